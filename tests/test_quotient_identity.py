"""The kernel's quantisers take the fp32 quotient v / s as the fp64 product of v with an
fp64 reciprocal of s (within 2^-51 relative), rounded once to fp32, and the scale
amax / 448 the same way with the constant fp64 reciprocal of 448 (exact for every amax,
checked exhaustively below the normal range).  The claim: wherever v / s is an fp32 normal this
equals IEEE fp32 division, because fp32 rounding boundaries M (odd 25-bit integer times a
power of two) are never hit by v / s and are more than 2^-49 M away from it; below the
normal range the two may differ by a subnormal step, which no E4M3 code can see (every
|v / s| < 2^-10 encodes as a signed zero).  These checks exercise the claim on random
operands, on random bit patterns, and on quotients constructed to sit as close to a
rounding boundary as fp32 operands allow, with reciprocals perturbed by up to 2^-51;
numpy's float32 division is the IEEE reference.  The Newton refinement of the reciprocal
is checked with exact rational arithmetic."""
from fractions import Fraction

import numpy as np

TINY = np.float32(2.0 ** -126)


def reciprocal(s, rng):
    r = 1.0 / s.astype(np.float64)
    if rng is not None:   # any reciprocal within 2^-51 relative
        r = r * (1.0 + rng.uniform(-1, 1, r.size) * 2.0 ** -51)
    return r


def via_reciprocal(v, s, rng=None):
    return (v.astype(np.float64) * reciprocal(s, rng)).astype(np.float32)


def check(v, s, rng=None):
    v = v.astype(np.float32)
    s = s.astype(np.float32)
    with np.errstate(all="ignore"):
        ref = v / s
        got = via_reciprocal(v, s, rng)
    same = (ref.view(np.uint32) == got.view(np.uint32)) | (np.isnan(ref) & np.isnan(got))
    # below the normal range only the E4M3 code matters: both must encode as the same zero
    sub = (np.abs(ref) < TINY) & ~same
    same |= sub & (np.abs(got) < 2.0 ** -10) & (np.signbit(ref) == np.signbit(got))
    bad = np.flatnonzero(~same)
    assert bad.size == 0, [(float(v[i]), float(s[i]), float(ref[i]), float(got[i])) for i in bad[:5]]


def test_random_quantiser_operands():
    rng = np.random.default_rng(1)
    n = 1 << 21
    amax = np.abs(rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32) + np.float32(1e-30)
    s = amax / np.float32(448.0)
    v = (rng.uniform(-1, 1, n) * amax).astype(np.float32)
    check(v, s, rng)
    # bf16-valued inputs (the input quantiser's case)
    vb = (v.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)
    check(vb, s, rng)


def test_random_bit_patterns():
    rng = np.random.default_rng(2)
    n = 1 << 21
    v = rng.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32).view(np.float32)
    s = rng.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32).view(np.float32)
    keep = np.isfinite(v) & np.isfinite(s) & (s != 0)
    check(v[keep], s[keep], rng)


def test_quotients_next_to_rounding_boundaries():
    rng = np.random.default_rng(3)
    n = 1 << 19
    s = (np.abs(rng.standard_normal(n)) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    s = s[s > 0]
    q = rng.uniform(2.0 ** -9, 448.0, s.size).astype(np.float32)
    ulp = np.spacing(q).astype(np.float64)
    mid = q.astype(np.float64) + ulp / 2                      # an fp32 rounding boundary
    base = (mid * s.astype(np.float64)).astype(np.float32)   # v with v / s closest to it
    for d in (-2, -1, 0, 1, 2):
        v = (base.view(np.uint32).astype(np.int64) + d).astype(np.uint32).view(np.float32)
        check(v, s, rng)
        check(-v, s, rng)


def test_subnormal_scales_and_values():
    rng = np.random.default_rng(4)
    n = 1 << 18
    s = rng.integers(1, 1 << 23, n, dtype=np.uint32).view(np.float32)    # subnormal scales
    v = (s.astype(np.float64) * rng.uniform(-448, 448, n)).astype(np.float32)
    check(v, s, rng)
    vs = rng.integers(1, 1 << 23, n, dtype=np.uint32).view(np.float32)   # subnormal values
    check(vs, rng.uniform(1e-3, 1e3, n).astype(np.float32), rng)


def e4m3_scale(amax):
    """The kernel's scale: the fp64 product with RN64(1/448), rounded once to fp32."""
    return (amax.astype(np.float32).astype(np.float64) * (1.0 / 448.0)).astype(np.float32)


def test_scale_equals_ieee_division_everywhere():
    rng = np.random.default_rng(5)
    bits = rng.integers(0, 0x7F800000, 1 << 21, dtype=np.uint64).astype(np.uint32)   # finite positives
    amax = bits.view(np.float32)
    assert np.array_equal((amax / np.float32(448.0)).view(np.uint32), e4m3_scale(amax).view(np.uint32))
    # exhaustively, every amax whose scale is below the fp32 normal range (ties included)
    top = 0x04E00000   # bits of 448 * 2^-126
    for lo in range(0, top, 1 << 23):
        a = np.arange(lo, min(lo + (1 << 23), top), dtype=np.uint32).view(np.float32)
        assert np.array_equal((a / np.float32(448.0)).view(np.uint32), e4m3_scale(a).view(np.uint32)), lo


def _fma(a, b, c):
    return float(Fraction(a) * Fraction(b) + Fraction(c))


def test_newton_reciprocal_reaches_the_bound():
    rng = np.random.default_rng(6)
    for s in np.concatenate([rng.uniform(0.5, 1.0, 300), np.exp2(rng.uniform(-149, 127, 300))]).astype(np.float32):
        d = float(s)
        y = float(Fraction(1) / Fraction(d)) * (1.0 + rng.uniform(-1, 1) * 2.0 ** -7)   # crude estimate
        for _ in range(3):
            y = _fma(y, _fma(-d, y, 1.0), y)
        assert abs(Fraction(y) * Fraction(d) - 1) <= Fraction(1, 1 << 51), d
