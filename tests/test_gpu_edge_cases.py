"""GPU parity on the method's edge cases and on heavy-tailed inputs, through the C ABI.

Same contract as tests/test_gpu_parity.py (tests/parity_utils.py).  What is added here:

  * Student-t(3) inputs and weights (paper Sec. 4.2 checks Gaussian and Student-t(3)
    inputs) on the small-expert, many-tiny-expert and wide layers at T = 1, 2, 4, 8;
  * an all-zero 128-group and an all-zero token row: the quantiser's zero-group branch
    (scale 0, codes 0) on the local input quantisation, on the exchanged one and in the
    multi-tile kernel; an all-zero token has equal logits for every expert, so its
    selection is an exact tie resolved by the lower-index rule and is compared as such;
  * a selected expert whose weights are all zero (its contribution is exactly zero and its
    requantised activation is the zero group), one with zero down-projection block scales
    and one with zero gate/up block scales;
  * exact logit ties forced by two identical router rows (and equal biases), so the k-th
    and (k+1)-th scores of a token are equal: the lower expert index must win, and the
    oracle's selection is injected for the rest of the comparison (the near-tie rule);
  * further seeds of the wide and coarse layers with every token compared.
"""
import numpy as np
import pytest
import torch

from paper_2609_04244_amd import monomoe as mm
from paper_2609_04244_amd import workloads as wl
from parity_utils import log, oracle_routing, run_case

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
_cache = {}


def layer(name, seed, Tmax, dist="gaussian", **over):
    key = (name, seed, Tmax, dist, tuple(sorted(over.items())))
    if key not in _cache:
        if len(_cache) >= 2:
            _cache.clear()
            torch.cuda.empty_cache()
        log("generating %s seed=%d Tmax=%d dist=%s %s" % (name, seed, Tmax, dist, over))
        _cache[key] = wl.generate(wl.config(name, **over), T=Tmax, seed=seed, device=DEV, dist=dist)
    return _cache[key]


def take(inp, T):
    d = dict(inp)
    d["x"] = inp["x"][:T].contiguous()
    d["T"] = T
    return d


def run(inp, kernel=mm.KERNEL_AUTO, tokens=None, **kw):
    plan = mm.Plan(inp["T"], inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"])
    if kernel != mm.KERNEL_AUTO:
        plan.set_schedule(kernel=kernel)
    info = plan.info()
    log("  kernel %s, grid %d" % ("multi-tile" if info["multi_tile"] else "single-tile", info["grid"]))
    rep = run_case(inp, tokens=tokens, plan=plan, **kw)
    plan.close()
    log("  -> %s" % rep)
    return info, rep


# ---------------------------------------------------------------- heavy-tailed inputs
@pytest.mark.parametrize("T", [1, 2, 4, 8])
@pytest.mark.parametrize("name", ["small_expert", "many_tiny_expert", "wide_fine"])
def test_student_t3_inputs(name, T):
    inp = take(layer(name, 11, 8, dist="student_t3"), T)
    log("case %s T=%d Student-t(3)" % (name, T))
    run(inp)


def test_student_t3_multi_tile():
    inp = take(layer("small_expert", 12, 24, dist="student_t3"), 24)
    log("case small_expert T=24 Student-t(3), multi-tile")
    info, _ = run(inp, tokens=[0, 7, 16, 23])
    assert info["multi_tile"] == 1


# ---------------------------------------------------------------- zero groups and tokens
def with_zero_rows(inp, T):
    """Token 0 gets an all-zero second 128-group; the last token is all zero."""
    d = take(inp, T)
    x = d["x"].clone()
    x[0, 128:256] = 0
    x[T - 1, :] = 0
    d["x"] = x
    return d


@pytest.mark.parametrize("name,T,kernel,path", [
    ("small_expert", 4, mm.KERNEL_AUTO, "local input quantisation"),
    ("many_tiny_expert", 8, mm.KERNEL_AUTO, "local input quantisation, biased logits"),
    ("wide_fine", 16, mm.KERNEL_AUTO, "exchanged input quantisation"),
    ("small_expert", 24, mm.KERNEL_AUTO, "multi-tile kernel"),
    ("tiny", 5, mm.KERNEL_MULTI, "multi-tile kernel within one tile"),
])
def test_zero_group_and_zero_token(name, T, kernel, path):
    inp = with_zero_rows(layer(name, 21, max(T, 8)), T)
    log("case %s T=%d zero group + zero token (%s)" % (name, T, path))
    info, rep = run(inp, kernel=kernel, exact_ties=True)
    assert info["multi_tile"] == (1 if "multi-tile" in path else 0)
    if inp["bias"] is None:   # an all-zero token ties every expert exactly
        assert rep["exact_tie_tokens"] >= 1


# ---------------------------------------------------------------- zero experts
def with_zero_experts(inp, T):
    """Token 0's first selected expert has all-zero weights, its second one zero down
    scales, token 1's first expert (when different) zero gate/up scales."""
    d = take(inp, T)
    _, oids, _ = oracle_routing(d)
    e0, e1 = int(oids[0][0]), int(oids[0][1])
    e2 = int(oids[1][0]) if T > 1 else e1
    w13, w2 = d["w13"].clone(), d["w2"].clone()
    w13s, w2s = d["w13_scale"].clone(), d["w2_scale"].clone()
    w13[e0] = 0
    w2[e0] = 0
    w2s[e1] = 0
    if e2 not in (e0, e1):
        w13s[e2] = 0
    d.update(w13=w13, w2=w2, w13_scale=w13s, w2_scale=w2s)
    return d, (e0, e1, e2)


@pytest.mark.parametrize("name,T", [("small_expert", 4), ("many_tiny_expert", 2), ("small_expert", 20),
                                    ("coarse", 8)])
def test_selected_zero_experts(name, T):
    inp, ex = with_zero_experts(layer(name, 31, max(T, 8)), T)
    log("case %s T=%d zero experts %s" % (name, T, ex))
    run(inp)


# ---------------------------------------------------------------- exact ties
def with_tied_rows(inp, T):
    """Router rows copied so that token 0's k-th selected expert ties exactly with an
    unselected expert of lower index (when one exists), and token 1's with one of higher
    index; biases are copied with the rows."""
    d = take(inp, T)
    _, oids, _ = oracle_routing(d)
    E, k = d["E"], d["k"]
    rw = d["router_w"].clone()
    bias = None if d["bias"] is None else d["bias"].clone()
    sel = None if d["sel_bias"] is None else d["sel_bias"].clone()
    used = set()
    pairs = []
    for t, lower in ((0, True), (1, False)):
        if t >= T:
            break
        a = int(oids[t][k - 1])
        chosen = set(int(e) for e in oids[t])
        cand = [b for b in range(E) if b not in chosen and b not in used and a not in used and
                ((b < a) if lower else (b > a))]
        if not cand:
            cand = [b for b in range(E) if b not in chosen and b not in used and a not in used]
        if not cand:
            continue
        b = cand[0] if lower else cand[-1]
        rw[b] = rw[a]
        if bias is not None:
            bias[b] = bias[a]
        if sel is not None:
            sel[b] = sel[a]
        used.update((a, b))
        pairs.append((t, a, b))
    d.update(router_w=rw, bias=bias, sel_bias=sel)
    return d, pairs


@pytest.mark.parametrize("name,T,kernel", [
    ("small_expert", 8, mm.KERNEL_AUTO), ("many_tiny_expert", 4, mm.KERNEL_AUTO),
    ("sigmoid_h7168_tp8", 4, mm.KERNEL_AUTO), ("small_expert", 20, mm.KERNEL_AUTO),
    ("tiny", 6, mm.KERNEL_MULTI),
])
def test_forced_exact_logit_ties(name, T, kernel):
    over = dict(E=64, k=4) if name == "tiny" else {}
    inp, pairs = with_tied_rows(layer(name, 41, max(T, 8), **over), T)
    log("case %s T=%d tied router rows (token, k-th expert, copy) %s" % (name, T, pairs))
    assert pairs
    _, rep = run(inp, kernel=kernel, exact_ties=True, min_near_ties=1)
    assert rep["exact_tie_tokens"] >= 1


# ---------------------------------------------------------------- more seeds, all tokens
@pytest.mark.parametrize("seed", [1, 2, 3])
@pytest.mark.parametrize("T", [1, 2, 4, 8])
def test_wide_fine_seeds(T, seed):
    inp = take(layer("wide_fine", seed, 8), T)
    log("case wide_fine T=%d seed=%d, every token" % (T, seed))
    run(inp)


@pytest.mark.parametrize("seed", [1, 2, 3])
@pytest.mark.parametrize("T", [1, 8])
def test_coarse_seeds(T, seed):
    inp = take(layer("coarse", seed, 8), T)
    log("case coarse T=%d seed=%d, every token" % (T, seed))
    run(inp)
