"""Pins of the oracle's whole operator (gate/up projection with block scales, SwiGLU,
requantisation, down projection, top-k weighted reduction; Sec. 3 and Eq. 9).

Independent references: numpy float64 matmuls on dequantised operands (exact on the
integer/dyadic special case), torch's silu, torch's E4M3 cast, and invariants of the
definition (dense mean at k = E, zero experts, power-of-two scale equivariance, token
independence), plus the paper's accuracy criterion (cosine >= 0.998 against an
FP32 FFN with routing held fixed, Sec. 4.2).
"""
import numpy as np
import pytest
import torch

from paper_2609_04244_amd import workloads as wl


def decode_table():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    return codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()


DEC = decode_table()


def e4m3_codes_in(rng, shape, lo_exp_field, hi_exp_field, allow_zero=True):
    """Random E4M3 codes with exponent field in [lo, hi] (and sometimes zero)."""
    e = rng.integers(lo_exp_field, hi_exp_field + 1, size=shape)
    m = rng.integers(0, 8, size=shape)
    s = rng.integers(0, 2, size=shape)
    c = (s << 7) | (e << 3) | m
    if allow_zero:
        c = np.where(rng.random(shape) < 0.05, 0, c)
    return c.astype(np.uint8)


def bf16_of_values(v):
    return torch.as_tensor(v, dtype=torch.float64).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def torch_quantize_f32(v):
    t = torch.as_tensor(np.asarray(v, dtype=np.float32))
    amax = t.abs().max()
    s = amax / torch.tensor(448.0)
    if float(amax) == 0.0 or float(s) == 0.0:
        return np.zeros(t.shape[0], np.uint8), np.float32(0)
    return (t / s).clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy(), np.float32(s)


def dyadic_case(T=2, H=256, I=256, E=4, k=2, seed=0):
    """Inputs whose quantisation is known exactly: every input group holds E4M3 values and
    one element equal to 448, so the group scale is exactly 1 and the codes are the
    values' own codes; weight block scales are powers of two."""
    rng = np.random.default_rng(seed)
    xc = e4m3_codes_in(rng, (T, H), 5, 10)
    xc[:, ::128] = 0x7E
    x_vals = DEC[xc]
    x = bf16_of_values(x_vals)
    w13 = e4m3_codes_in(rng, (E, 2 * I, H), 4, 10)
    w2 = e4m3_codes_in(rng, (E, H, I), 4, 10)
    w13s = np.exp2(rng.integers(-3, 4, (E, 2 * I // 128, H // 128))).astype(np.float32)
    w2s = np.exp2(rng.integers(-3, 4, (E, H // 128, I // 128))).astype(np.float32)
    rw = bf16_of_values(rng.standard_normal((E, H)) * 0.05)
    return dict(x=x, xc=xc, rw=rw, w13=w13, w13s=w13s, w2=w2, w2s=w2s, T=T, H=H, I=I, E=E, k=k)


def dequant(codes, scales):
    R, C = codes.shape
    return DEC[codes] * np.kron(scales.astype(np.float64), np.ones((128, 128)))[:R, :C]


def test_input_quantisation_exact_on_dyadic_case(orc):
    c = dyadic_case()
    _, d = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], c["k"], True, debug=True)
    assert np.array_equal(d["xq"], c["xc"])
    assert np.all(d["xs"] == 1.0)


def test_gate_up_exact_against_integer_matmul(orc):
    c = dyadic_case()
    _, d = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], c["k"], True, debug=True)
    xv = DEC[c["xc"]]
    for t in range(c["T"]):
        for j in range(c["k"]):
            e = d["ids"][t, j]
            h_ref = dequant(c["w13"][e], c["w13s"][e]) @ xv[t]
            assert np.array_equal(d["h"][t * c["k"] + j], h_ref)   # exact: dyadic operands, < 53 bits


def test_swiglu_requant_down_reduce_against_libraries(orc):
    c = dyadic_case(seed=1)
    I, H, k = c["I"], c["H"], c["k"]
    ref, d = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], k, True, debug=True)
    h = torch.from_numpy(d["h"])
    act_ref = (torch.nn.functional.silu(h[:, :I]) * h[:, I:]).numpy()   # rows [0,I) gate, [I,2I) up
    np.testing.assert_allclose(d["act"], act_ref, rtol=1e-14, atol=1e-300)
    out = np.zeros((c["T"], H))
    for p in range(c["T"] * k):
        t, j = divmod(p, k)
        e = d["ids"][t, j]
        for g in range(I // 128):
            q, s = torch_quantize_f32(d["act"][p, g * 128:(g + 1) * 128].astype(np.float32))
            assert np.array_equal(d["aq"][p, g * 128:(g + 1) * 128], q)
            assert d["as"][p, g] == s
        a_deq = DEC[d["aq"][p]] * np.repeat(d["as"][p].astype(np.float64), 128)
        y_ref = dequant(c["w2"][e], c["w2s"][e]) @ a_deq
        np.testing.assert_allclose(d["y"][p], y_ref, rtol=1e-12, atol=1e-12 * np.abs(y_ref).max())
        out[t] += d["w"][t, j] * d["y"][p]
    np.testing.assert_allclose(ref, out, rtol=1e-14, atol=1e-14 * np.abs(out).max())


def tiny_inputs(T, seed=0, name="tiny", **over):
    inp = wl.generate(wl.config(name, **over), T=T, seed=seed)
    return dict(x=wl.bf16_bits(inp["x"]), rw=wl.bf16_bits(inp["router_w"]),
                bias=None if inp["bias"] is None else inp["bias"].numpy(),
                w13=inp["w13"].numpy(), w13s=inp["w13_scale"].numpy(),
                w2=inp["w2"].numpy(), w2s=inp["w2_scale"].numpy(), inp=inp)


def test_all_experts_with_uniform_logits_is_dense_mean(orc):
    c = tiny_inputs(T=2)
    E = c["w13"].shape[0]
    rw0 = np.zeros_like(c["rw"])
    full = orc.forward(c["x"], rw0, c["w13"], c["w13s"], c["w2"], c["w2s"], E, True)
    dense = []
    for e in range(E):   # each expert alone, through the selection-injection path
        ids = np.full((2, 1), e, np.int32)
        dense.append(orc.forward(c["x"], rw0, c["w13"], c["w13s"], c["w2"], c["w2s"], 1, True,
                                 ids_in=ids, w_in=np.ones((2, 1))))
    np.testing.assert_allclose(full, np.mean(dense, axis=0), rtol=1e-12, atol=1e-13)


def test_zero_expert_contributes_nothing(orc):
    c = tiny_inputs(T=1, seed=2)
    w13 = c["w13"].copy()
    w13[3] = 0
    w2s = c["w2s"].copy()
    w2s[5] = 0
    for z in (3, 5):
        ids = np.array([[1, z]], np.int32)
        w = np.array([[0.7, 0.3]])
        both = orc.forward(c["x"], c["rw"], w13, c["w13s"], c["w2"], w2s, 2, True, ids_in=ids, w_in=w)
        alone = orc.forward(c["x"], c["rw"], w13, c["w13s"], c["w2"], w2s, 1, True,
                            ids_in=np.array([[1]], np.int32), w_in=np.array([[0.7]]))
        np.testing.assert_array_equal(both, alone)


def test_down_scale_power_of_two_scales_that_expert_exactly(orc):
    c = tiny_inputs(T=2, seed=3)
    _, d0 = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True, debug=True)
    e = int(d0["ids"][0, 0])
    w2s = c["w2s"].copy()
    w2s[e] *= 8.0
    _, d1 = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], w2s, 2, True, debug=True)
    for p in range(4):
        t, j = divmod(p, 2)
        f = 8.0 if d0["ids"][t, j] == e else 1.0
        np.testing.assert_array_equal(d1["y"][p], d0["y"][p] * f)


def test_tokens_are_independent(orc):
    c = tiny_inputs(T=4, seed=4)
    full = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True)
    for t in range(4):
        one = orc.forward(c["x"][t:t + 1], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True)
        np.testing.assert_array_equal(one[0], full[t])


def test_bias_changes_selection_and_weights(orc):
    c = tiny_inputs(T=3, seed=5)
    E = c["w13"].shape[0]
    bias = np.zeros(E, np.float32)
    bias[6] = 50.0   # expert 6 must be selected first by every token, with weight ~1 after softmax
    _, d = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True, bias=bias, debug=True)
    assert np.all(d["ids"][:, 0] == 6)
    assert np.all(d["w"][:, 0] > 0.999)


def test_empty_token_tile_and_bad_shapes(orc):
    c = tiny_inputs(T=1)
    ref = orc.forward(c["x"][:0], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True)
    assert ref.shape == (0, 256)
    with pytest.raises(ValueError):
        orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 9, True)   # k > E
    with pytest.raises(ValueError):   # injected expert without weights
        orc.forward(c["x"], c["rw"], {0: c["w13"][0]}, {0: c["w13s"][0]}, {0: c["w2"][0]}, {0: c["w2s"][0]}, 1,
                    True, ids_in=np.array([[1]], np.int32), w_in=np.ones((1, 1)))


def float_reference(inp, ids, w):
    """The operator without its dynamic activation quantisation: bf16 input, the stored
    block-FP8 weights dequantised, every product and sum in fp64, routing fixed.  This is
    the reading of the paper's FP32 reference used throughout (the production BF16/FP8
    conversions applied to inputs and weights, no in-operator E4M3 activations)."""
    x = inp["x"].to(torch.float64)
    I = inp["I"]
    out = torch.zeros_like(x)
    for t in range(x.shape[0]):
        for j in range(ids.shape[1]):
            e = int(ids[t, j])
            w13 = torch.from_numpy(dequant(inp["w13"][e].numpy(), inp["w13_scale"][e].numpy()))
            w2 = torch.from_numpy(dequant(inp["w2"][e].numpy(), inp["w2_scale"][e].numpy()))
            h = w13 @ x[t]
            a = torch.nn.functional.silu(h[:I]) * h[I:]
            out[t] += float(w[t, j]) * (w2 @ a)
    return out.numpy()


@pytest.mark.parametrize("dist", ["gaussian", "student_t3"])
@pytest.mark.parametrize("name,T", [("tiny", 1), ("tiny", 2), ("tiny", 4), ("tiny", 8), ("mid", 2)])
def test_cosine_against_float_reference(orc, dist, name, T):
    cfg = wl.config("tiny") if name == "tiny" else wl.config("tiny", H=2048, I=768, E=8, k=2)
    inp = wl.generate(cfg, T=T, seed=21, dist=dist)
    ref, d = orc.forward(wl.bf16_bits(inp["x"]), wl.bf16_bits(inp["router_w"]), inp["w13"].numpy(),
                         inp["w13_scale"].numpy(), inp["w2"].numpy(), inp["w2_scale"].numpy(),
                         cfg["k"], cfg["renorm"], debug=True)
    unq = float_reference(inp, d["ids"], d["w"])
    cos = float(np.sum(ref * unq) / np.sqrt(np.sum(ref ** 2) * np.sum(unq ** 2)))
    assert cos >= 0.998, cos


def test_sigmoid_policy_equals_injected_sigmoid_selection(orc):
    # the sigmoid-routed operator is the operator with the sigmoid selection injected: the
    # selection is computed from the same fp64 logits, and the expert path is shared
    c = tiny_inputs(T=3, seed=7)
    E = c["w13"].shape[0]
    sel_bias = (np.random.default_rng(7).standard_normal(E) * 0.2).astype(np.float32)
    ref, d = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True, debug=True,
                         policy=orc.SIGMOID_BIAS, sel_bias=sel_bias, scale=2.5)
    ids, w = orc.select_sigmoid(orc.router_logits(c["x"], c["rw"]), 2, sel_bias, 2.5)
    assert np.array_equal(d["ids"], ids)
    np.testing.assert_array_equal(d["w"], w)
    inj = orc.forward(c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True, ids_in=ids, w_in=w)
    np.testing.assert_array_equal(ref, inj)
    np.testing.assert_allclose(d["w"].sum(axis=1), 2.5, rtol=1e-13)


def test_policy_arguments_are_checked(orc):
    c = tiny_inputs(T=1)
    args = (c["x"], c["rw"], c["w13"], c["w13s"], c["w2"], c["w2s"], 2, True)
    with pytest.raises(ValueError):   # softmax takes no selection bias
        orc.forward(*args, policy=orc.SOFTMAX, sel_bias=np.zeros(c["w13"].shape[0], np.float32))
    with pytest.raises(ValueError):   # nor a scaling factor
        orc.forward(*args, policy=orc.SOFTMAX, scale=2.5)
    with pytest.raises(ValueError):
        orc.forward(*args, policy=orc.SIGMOID_BIAS, scale=0.0)
    with pytest.raises(ValueError):
        orc.forward(*args, policy=7)
