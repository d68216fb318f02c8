"""GPU tests of the operator's runtime behaviour through the C ABI: the token count as a
runtime argument (monomoe_forward_tokens), capture into a HIP graph and replay on new
inputs, and plans of one kernel created in any order.

Outputs are checked against the fp64 oracle under the output contract (tests/parity_utils.py)
and, where the same kernel and configuration run, bit for bit against a plan built for that
token count (whose debug forward is parity-tested in full).
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2609_04244_amd import monomoe as mm
from paper_2609_04244_amd import workloads as wl
from parity_utils import (MAX_ERR_REL_RMS, MEAN_REL_ERR, host_experts, log, near_tie_tokens, oracle_routing,
                          output_errors, run_case)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def args_of(inp, x=None):
    return (inp["x"] if x is None else x, inp["router_w"], inp["w13"], inp["w13_scale"], inp["w2"], inp["w2_scale"])


def check_output(inp, x, out):
    """The bf16 output of x (its T rows) against the oracle, tokens without a near tie."""
    d = dict(inp)
    d["x"] = x
    d["T"] = x.shape[0]
    logits, oids, ow = oracle_routing(d)
    keep = [t for t in range(d["T"]) if not near_tie_tokens(logits, d["k"])[t]]
    w13, w13s, w2, w2s = host_experts(d, oids[keep].reshape(-1))
    ref = oracle.forward(wl.bf16_bits(x)[keep], wl.bf16_bits(d["router_w"]), w13, w13s, w2, w2s, d["k"],
                         d["renorm"], ids_in=oids[keep], w_in=ow[keep])
    got = out.float().cpu().numpy().astype(np.float64)[keep]
    mx, rms, mre = output_errors(got, ref)
    log("  output: %d tokens compared, max err %.3g (bound %.3g), mean rel err %.3g" %
        (len(keep), mx, MAX_ERR_REL_RMS * rms, mre))
    assert mx <= MAX_ERR_REL_RMS * rms and mre <= MEAN_REL_ERR
    return len(keep)


def make_plan(inp, T):
    plan = mm.Plan(T, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"])
    if inp["bias"] is not None:
        plan.set_router_bias(inp["bias"])
    return plan


@pytest.mark.parametrize("name,Tplan,Ts", [
    ("small_expert", 8, [8, 5, 1, 3, 0, 8]),
    ("small_expert", 24, [24, 16, 9, 1, 20]),   # the multi-tile kernel's plan; at most one tile: single-tile
    ("many_tiny_expert", 8, [2, 7, 4]),
    ("coarse", 8, [1, 6, 8]),                   # sliced down projection: the multi-tile kernel from T = 2
])
def test_runtime_token_count(name, Tplan, Ts):
    inp = wl.generate(wl.config(name), T=Tplan, seed=51, device=DEV)
    plan = make_plan(inp, Tplan)
    info = plan.info()
    log("case %s plan T=%d (%s), calls with T=%s" % (name, Tplan, "multi-tile" if info["multi_tile"] else
                                                     "single-tile", Ts))
    outs = []
    for T in Ts:
        x = inp["x"][:T].contiguous()
        outs.append((T, x, plan.forward_tokens(T, *args_of(inp, x))))
    torch.cuda.synchronize()
    assert plan.status() == mm.MONOMOE_OK
    for T, x, out in outs:
        if T == 0:
            continue
        check_output(inp, x, out)
        # the single-tile kernel runs this call when the plan's kernel is single-tile, when
        # the call fits one tile and the down projection is not sliced, or when it has one
        # token; a plan built for T that also runs it computes the same bytes
        single = info["multi_tile"] == 0 or (T <= 16 and info["down_slices"] == 1) or T == 1
        ref_plan = make_plan(inp, T)
        if single and ref_plan.info()["multi_tile"] == 0:
            ref = ref_plan.forward(*args_of(inp, x))
            torch.cuda.synchronize()
            assert torch.equal(ref.view(torch.int16), out.view(torch.int16)), "T=%d" % T
        ref_plan.close()
    # the C entry point rejects a token count above the plan's bound, enqueueing nothing
    rc = mm.lib().monomoe_forward_tokens(plan._h, Tplan + 1, *[mm._ptr(t) for t in args_of(inp)],
                                         mm._ptr(outs[0][2]), mm._stream(None))
    assert rc == mm.MONOMOE_ERR_INVALID
    rc = mm.lib().monomoe_forward_tokens(plan._h, -1, *[mm._ptr(t) for t in args_of(inp)],
                                         mm._ptr(outs[0][2]), mm._stream(None))
    assert rc == mm.MONOMOE_ERR_INVALID
    plan.close()


def test_runtime_token_count_full_parity_after_small_calls():
    # calls with fewer tokens leave the workspace's tagged words of an earlier, smaller
    # layout behind; the full-size debug forward that follows must not be confused by them
    inp = wl.generate(wl.config("small_expert"), T=16, seed=52, device=DEV)
    plan = make_plan(inp, 16)
    for T in (3, 1, 11):
        x = inp["x"][:T].contiguous()
        plan.forward_tokens(T, *args_of(inp, x))
    torch.cuda.synchronize()
    run_case(inp, plan=plan)
    plan.close()


@pytest.mark.parametrize("name,T", [("small_expert", 8), ("tiny", 20), ("wide_fine", 4)])
def test_graph_capture_and_replay(name, T):
    inp = wl.generate(wl.config(name), T=T, seed=61, device=DEV)
    plan = make_plan(inp, T)
    xbuf = inp["x"].clone()
    out = torch.empty((T, inp["H"]), dtype=torch.bfloat16, device=DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up launch outside the capture
        plan.forward(*args_of(inp, xbuf), out=out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan.forward(*args_of(inp, xbuf), out=out)
    torch.cuda.synchronize()
    gen = torch.Generator(device=DEV)
    gen.manual_seed(7)
    for r in range(4):
        xr = torch.randn((T, inp["H"]), generator=gen, device=DEV).to(torch.bfloat16)
        xbuf.copy_(xr)
        g.replay()
        torch.cuda.synchronize()
        got = out.clone()
        eager = plan.forward(*args_of(inp, xr))   # eager work between replays, same plan
        torch.cuda.synchronize()
        assert plan.status() == mm.MONOMOE_OK
        log("case %s T=%d replay %d" % (name, T, r))
        assert torch.equal(got.view(torch.int16), eager.view(torch.int16)), "replay %d" % r
        check_output(inp, xr, got)
    del g
    plan.close()


def test_plans_created_in_descending_footprint():
    # the dynamic-LDS limit of a kernel symbol is shared by every plan: a later plan with a
    # smaller footprint must not break the launches of an earlier, larger one
    inp = wl.generate(wl.config("small_expert"), T=16, seed=71, device=DEV)
    Ts = (1, 2, 4, 8, 16)
    lds = {}
    for T in Ts:
        q = make_plan(inp, T)
        lds[T] = q.info()["lds_bytes"]
        q.close()
    Tb, Tsm = max(Ts, key=lambda T: lds[T]), min(Ts, key=lambda T: lds[T])
    log("LDS per workgroup by T: %s; larger plan T=%d, smaller T=%d" % (lds, Tb, Tsm))
    assert lds[Tb] > lds[Tsm]
    big = make_plan(inp, Tb)
    small = make_plan(inp, Tsm)

    def case(T):
        d = dict(inp)
        d["x"] = inp["x"][:T].contiguous()
        d["T"] = T
        return d
    run_case(case(Tb), plan=big)
    run_case(case(Tsm), plan=small)
    run_case(case(Tb), plan=big)
    small.close()
    big.close()
