"""GPU test of monomoe_forward_noalloc, the allocation-free variant of monomoe_forward
(workspace in the library's static device array instead of a plan's buffer), through the C
ABI: its outputs must equal monomoe_forward's on the same inputs, on consecutive calls with
decreasing token counts (the second call reuses the array the first one left behind)."""
import ctypes

import pytest
import torch

from paper_2609_04244_amd import monomoe as mm
from paper_2609_04244_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def log(msg):
    print(msg, flush=True)


def plan_forward(inp, x):
    plan = mm.Plan(x.shape[0], inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"])
    if inp["bias"] is not None:
        plan.set_router_bias(inp["bias"])
    out = plan.forward(x, inp["router_w"], inp["w13"], inp["w13_scale"], inp["w2"], inp["w2_scale"])
    torch.cuda.synchronize()
    assert plan.status() == mm.MONOMOE_OK
    plan.close()
    return out


@pytest.mark.parametrize("name,Ts", [("small_expert", (8, 3)), ("many_tiny_expert", (4, 1)), ("tiny", (24, 20)),
                                     ("wide_fine", (16, 2))])
def test_noalloc_matches_forward(name, Ts):
    inp = wl.generate(wl.config(name), T=max(Ts), seed=81, device=DEV)
    status = torch.full((1,), 12345, dtype=torch.int32, device=DEV)
    for T in Ts:
        x = inp["x"][:T].contiguous()
        out = torch.empty((T, inp["H"]), dtype=torch.bfloat16, device=DEV)
        log("case %s T=%d: monomoe_forward_noalloc" % (name, T))
        mm.forward_noalloc(T, inp["H"], inp["E"], inp["I"], inp["k"], inp["renorm"], x, inp["router_w"], inp["w13"],
                           inp["w13_scale"], inp["w2"], inp["w2_scale"], out, bias=inp["bias"], status=status)
        torch.cuda.synchronize()
        assert int(status.item()) == mm.MONOMOE_OK
        ref = plan_forward(inp, x)
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), "%s T=%d" % (name, T)


def test_noalloc_rejects_what_it_cannot_serve():
    cfg = wl.config("coarse")
    L = mm.lib()
    dummy = torch.zeros(64, dtype=torch.uint8, device=DEV)
    p = ctypes.c_void_p(dummy.data_ptr())
    # 64 tokens of the 4096 x 14336 layer need more workspace than the static array holds
    rc = L.monomoe_forward_noalloc(ctypes.byref(mm.Shape(64, cfg["H"], cfg["E"], cfg["I"])), cfg["k"], 0, None,
                                   p, p, p, p, p, p, p, None, mm._stream(None))
    assert rc == mm.MONOMOE_ERR_UNSUPPORTED
    # a misaligned bias and a bad top-k are argument errors
    mis = ctypes.c_void_p(dummy.data_ptr() + 4)
    rc = L.monomoe_forward_noalloc(ctypes.byref(mm.Shape(1, 256, 8, 256)), 2, 1, mis, p, p, p, p, p, p, p, None,
                                   mm._stream(None))
    assert rc == mm.MONOMOE_ERR_INVALID
    rc = L.monomoe_forward_noalloc(ctypes.byref(mm.Shape(1, 256, 8, 256)), 9, 1, None, p, p, p, p, p, p, p, None,
                                   mm._stream(None))
    assert rc == mm.MONOMOE_ERR_INVALID
    torch.cuda.synchronize()
