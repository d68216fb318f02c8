"""GPU parity of every tuned schedule (paper Sec. 3.4: serving uses a fixed, offline-tuned
schedule per shape; the tuner gates candidates against the default schedule's output, and
this test runs each schedule it recorded in paper_2609_04244_amd/tuned_schedules.json
against the fp64 oracle, through the C ABI, under the operator contract of
tests/parity_utils.py)."""
import pytest
import torch

from paper_2609_04244_amd import monomoe as mm
from paper_2609_04244_amd import tune
from paper_2609_04244_amd import workloads as wl
from parity_utils import log, run_case

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
CASES = [(w, int(T)) for w, ents in sorted(tune.load_table().items()) for T in sorted(ents, key=int)]
_layer = {}


def layer(name, Tmax):
    if _layer.get("key") != (name, Tmax):
        _layer.clear()
        torch.cuda.empty_cache()
        _layer["key"] = (name, Tmax)
        _layer["inp"] = wl.generate(wl.config(name), T=Tmax, seed=21, device=DEV)
    return _layer["inp"]


def test_table_is_present():
    assert CASES, "no tuned schedules recorded"


@pytest.mark.parametrize("name,T", CASES)
def test_tuned_schedule_matches_the_oracle(name, T):
    Tmax = max(t for w, t in CASES if w == name)
    inp = dict(layer(name, Tmax))
    inp["x"] = inp["x"][:T].contiguous()
    inp["T"] = T
    plan = mm.Plan(T, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"])
    assert tune.apply_tuned(plan, name, T)
    sch = tune.tuned_schedule(name, T)
    log("case %s T=%d tuned schedule %s" % (name, T, sch))
    if not plan.info()["multi_tile"]:   # the tuner's host gate, on the plan as configured
        assert tune.model_verdict(plan, wl.config(name), T, sch["general_only"]) is None
    rep = run_case(inp, plan=plan, tokens=sorted({0, T - 1}))
    log("  -> %s" % rep)
    plan.close()
