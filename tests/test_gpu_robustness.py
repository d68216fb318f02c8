"""Race perturbation: the readiness protocol of both kernels under pseudo-random pauses at
every hand-off point (the race-perturbation build of the library, libmonomoe_perturb.so,
through the jitter_seed test hook of monomoe_forward_debug: partial sums
handed to the helper wavefront, activation and contribution stores, activation polls,
output reduction, kernel entry).  Every consumer must still see final data only, and the
output reduction has a fixed order, so each perturbed launch must reproduce the
unperturbed launch bit for bit: selections, routing weights, quantised input, SiLU
activations, requantised codes and scales, fp32 result and bf16 output.  One perturbed
launch per case is also checked against the oracle."""
import numpy as np
import pytest
import torch

from paper_2609_04244_amd import monomoe as mm
from paper_2609_04244_amd import workloads as wl
from parity_utils import log, run_case

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SEEDS = range(1, 9)
FIELDS = ("ids", "w", "xq", "xs", "act", "aq", "as", "out_f32")


ST_ENTRY, ST_EXIT = 0, 8   # phase-stamp columns: kernel entry and exit (s_memrealtime, 10 ns)


def launch(plan, inp, seed):
    out, d = plan.forward_debug(inp["x"], inp["router_w"], inp["w13"], inp["w13_scale"], inp["w2"],
                                inp["w2_scale"], jitter_seed=seed)
    torch.cuda.synchronize()
    st = d["stamps"].cpu().numpy()
    used = st[:, ST_EXIT] > 0   # workgroups of the (last) launch
    # the kernel's own duration, first entry to last exit, from its phase stamps
    d["us"] = float(st[used, ST_EXIT].max() - st[used, ST_ENTRY].min()) / 100.0
    assert plan.status() == mm.MONOMOE_OK, (seed, mm.status_string(plan.status()))
    d["out"] = out.view(torch.int16)
    return d


# (layer, T, oracle tokens, path exercised, schedule fields (None: the default schedule))
CASES = [
    ("small_expert", 1, None, "one-token kernel", None),
    ("small_expert", 8, None, "general kernel, input quantised locally", None),
    ("many_tiny_expert", 4, None, "general kernel, biased routing, 256 experts", None),
    ("wide_fine", 8, [0, 7], "general kernel, input quantised once and exchanged", None),
    ("coarse", 32, [0, 31], "multi-tile kernel", None),
    ("small_expert", 64, [0, 63], "multi-tile kernel", None),
    ("many_tiny_expert", 48, [0, 47], "multi-tile kernel", None),
    ("sigmoid_h7168_tp8", 4, [0, 3], "general kernel, sigmoid routing with selection bias", None),
    ("small_expert", 8, [0, 7], "general kernel, gate/up units dealt two at a time, down on 192 workgroups",
     dict(up_block=2, down_grid=192)),
    ("many_tiny_expert", 1, None, "one-token kernel, gate/up units dealt four at a time, down on 160 workgroups",
     dict(up_block=4, down_grid=160)),
]


@pytest.mark.parametrize("name,T,tokens,path,sched", CASES)
def test_perturbed_launches_are_bit_identical(name, T, tokens, path, sched):
    inp = wl.generate(wl.config(name), T=T, seed=0, device=DEV)
    plan = mm.Plan(T, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"], perturb=True)
    if inp["bias"] is not None:
        plan.set_router_bias(inp["bias"])
    if inp.get("policy", "softmax") == "sigmoid_bias":
        plan.set_routing(mm.ROUTING_SIGMOID_BIAS, inp["sel_bias"], inp["route_scale"])
    if sched is not None:
        plan.set_schedule(**sched)
    info = plan.info()
    log("case %s T=%d (%s): grid %d, multi_tile %d" % (name, T, path, info["grid"], info["multi_tile"]))
    assert bool(info["multi_tile"]) == path.startswith("multi-tile")
    ref = launch(plan, inp, 0)
    plain = [launch(plan, inp, 0)["us"] for _ in range(3)]
    perturbed = []
    for seed in SEEDS:
        got = launch(plan, inp, seed)
        perturbed.append(got["us"])
        for f in FIELDS + ("out",):
            assert torch.equal(got[f], ref[f]), "seed %d: %s differs from the unperturbed launch" % (seed, f)
    log("  %d perturbed launches bit-identical; kernel %.1f us unperturbed (median), %.1f .. %.1f us perturbed"
        % (len(SEEDS), float(np.median(plain)), min(perturbed), max(perturbed)))
    # the pauses were taken: the perturbed launches last longer (kernel time from the stamps,
    # first entry to last exit)
    assert float(np.mean(perturbed)) > float(np.median(plain))
    rep = run_case(inp, tokens=tokens, plan=plan, jitter_seed=SEEDS[-1])
    log("  oracle: %s" % rep)
    plan.close()


def test_jitter_seed_is_checked_and_only_the_perturbation_build_takes_it():
    inp = wl.generate(wl.config("tiny"), T=2, seed=0, device=DEV)
    args = (inp["x"], inp["router_w"], inp["w13"], inp["w13_scale"], inp["w2"], inp["w2_scale"])
    for perturb, code in ((True, mm.MONOMOE_ERR_INVALID), (False, mm.MONOMOE_ERR_INVALID)):
        plan = mm.Plan(2, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"], perturb=perturb)
        with pytest.raises(mm.MonoMoEError) as e:
            plan.forward_debug(*args, jitter_seed=65536)
        assert e.value.code == code
        plan.close()
    # the product library has no pauses compiled in and refuses a seed
    plan = mm.Plan(2, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"])
    with pytest.raises(mm.MonoMoEError) as e:
        plan.forward_debug(*args, jitter_seed=1)
    assert e.value.code == mm.MONOMOE_ERR_UNSUPPORTED
    plan.close()
