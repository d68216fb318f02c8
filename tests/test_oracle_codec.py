"""Pins of the oracle's E4M3FN codec and group quantiser (format of Sec. 4.1: E4M3 FP8
weights and activations, activations quantised per 128-element group).

Independent references: the OCP FP8 table (tests/golden), torch's float8_e4m3fn casts
(an independent round-to-nearest-even implementation) and closed-form properties.
"""
import math
import os

import numpy as np
import pytest
import torch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_ocp_special_values.txt")


def torch_decode_all():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    return codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()


def torch_encode(v):
    """torch's RNE cast of float32 values already within [-448, 448]."""
    t = torch.as_tensor(np.asarray(v, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_ocp_table(orc):
    with open(GOLDEN) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 10
    for code, val in rows:
        got = orc.e4m3_decode(int(code, 16))
        if val == "nan":
            assert math.isnan(got), code
        else:
            assert got == float(val), code
            assert math.copysign(1.0, got) == math.copysign(1.0, float(val)), code


def test_decode_all_codes_match_torch(orc):
    ref = torch_decode_all()
    for c in range(256):
        got = orc.e4m3_decode(c)
        if math.isnan(ref[c]):
            assert math.isnan(got) and (c & 0x7F) == 0x7F
        else:
            assert got == ref[c], hex(c)
            assert math.copysign(1.0, got) == math.copysign(1.0, ref[c])


def test_encode_roundtrips_every_finite_code(orc):
    for c in range(256):
        v = orc.e4m3_decode(c)
        if math.isnan(v):
            continue
        assert orc.e4m3_encode(v) == c, hex(c)


def _sweep_values():
    vals = []
    finite = sorted({orc_v for orc_v in torch_decode_all().tolist() if not math.isnan(orc_v) and orc_v >= 0})
    for a, b in zip(finite[:-1], finite[1:]):
        mid = np.float32((a + b) / 2)
        for m in (mid, np.nextafter(mid, np.float32(0)), np.nextafter(mid, np.float32(1e9)),
                  np.float32(a * 0.75 + b * 0.25), np.float32(a * 0.25 + b * 0.75)):
            vals.append(m)
            vals.append(-m)
    rng = np.random.default_rng(7)
    vals.extend(rng.uniform(-448, 448, 20000).astype(np.float32))
    vals.extend((rng.standard_normal(20000) * np.exp2(rng.integers(-12, 6, 20000))).astype(np.float32))
    v = np.asarray(vals, dtype=np.float32)
    return v[np.abs(v) <= 448]


def test_encode_matches_torch_rne_in_range(orc):
    v = _sweep_values()
    ref = torch_encode(v)
    got = np.array([orc.e4m3_encode(x) for x in v], dtype=np.uint8)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(float(v[i]), hex(got[i]), hex(ref[i])) for i in bad[:10]]


@pytest.mark.parametrize("v,code", [
    (2.0 ** -10, 0x00),          # halfway 0 .. 2^-9: even is 0
    (3 * 2.0 ** -10, 0x02),      # halfway 0x01 .. 0x02: even is 0x02
    (1.0625, 0x38),              # halfway 1.0 (0x38) .. 1.125 (0x39)
    (1.1875, 0x3A),              # halfway 1.125 (0x39) .. 1.25 (0x3A)
    (-0.0, 0x80),                # sign of zero kept
    (448.0, 0x7E), (464.0, 0x7E), (1.0e6, 0x7E), (-1.0e6, 0xFE),   # saturation
    (float("inf"), 0x7E), (float("-inf"), 0xFE),
    (2.0 ** -6 * 15 / 16, 0x08),  # rounds up from the subnormal range into the smallest normal
])
def test_encode_ties_and_saturation(orc, v, code):
    assert orc.e4m3_encode(v) == code


def torch_quantize(v):
    """The group quantiser's definition evaluated with torch ops (fp32 division, torch RNE
    cast): an independent evaluation path for the oracle's C implementation."""
    t = torch.as_tensor(np.asarray(v, dtype=np.float32))
    amax = t.abs().max()
    s = amax / torch.tensor(448.0, dtype=torch.float32)
    if float(amax) == 0.0 or float(s) == 0.0:
        return np.zeros(t.shape[0], np.uint8), np.float32(0.0)
    q = (t / s).clamp(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return q, np.float32(s)


def _groups():
    rng = np.random.default_rng(11)
    out = []
    for j in range(200):
        g = rng.standard_normal(128).astype(np.float32) * np.float32(2.0 ** rng.integers(-20, 20))
        out.append(g)
    t3 = rng.standard_t(3, size=(50, 128)).astype(np.float32)
    out.extend(list(t3))
    g = rng.standard_normal(128).astype(np.float32)
    g[5] = -0.0
    g[6] = 0.0
    out.append(g)
    out.append(np.full(128, 3.0, np.float32))
    tiny = (rng.standard_normal(128) * 1e-38).astype(np.float32)
    out.append(tiny)
    return out


def test_quantizer_matches_torch_definition(orc):
    for g in _groups():
        q, s = orc.quantize_group(g)
        rq, rs = torch_quantize(g)
        assert np.float32(s) == rs
        assert np.array_equal(q, rq)


def test_quantizer_half_ulp_bound_and_max_code(orc):
    dec = torch_decode_all()
    for g in _groups():
        q, s = orc.quantize_group(g)
        assert s > 0
        r = g.astype(np.float64) / np.float64(s)
        d = dec[q]
        # half an E4M3 ulp of v/s (ulp of a normal value 2^(e-3), subnormal 2^-9), plus the
        # fp32 rounding of v/s itself
        e = np.floor(np.log2(np.maximum(np.abs(r), 2.0 ** -6)))
        half_ulp = 0.5 * np.exp2(e - 3)
        assert np.all(np.abs(d - r) <= half_ulp * (1 + 1e-6) + np.abs(r) * 2.0 ** -23)
        # the largest magnitude lands on +-448
        i = int(np.argmax(np.abs(g)))
        assert (q[i] & 0x7F) == 0x7E


def test_quantizer_power_of_two_equivariance(orc):
    rng = np.random.default_rng(3)
    for _ in range(50):
        g = rng.standard_normal(128).astype(np.float32)
        q0, s0 = orc.quantize_group(g)
        for j in (-7, -1, 1, 5, 12):
            q1, s1 = orc.quantize_group(g * np.float32(2.0 ** j))
            assert np.array_equal(q0, q1)
            assert np.float32(s1) == np.float32(s0 * np.float32(2.0 ** j))


def test_quantizer_zero_group(orc):
    for g in (np.zeros(128, np.float32), -np.zeros(128, np.float32)):
        q, s = orc.quantize_group(g)
        assert s == 0.0
        assert not q.any()


def test_bf16_decode_matches_torch(orc):
    rng = np.random.default_rng(5)
    bits = rng.integers(0, 1 << 16, 5000, dtype=np.uint32).astype(np.uint16)
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]   # finite only
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([orc.bf16_decode(b) for b in bits])
    assert np.array_equal(got, ref)
