"""CPU checks of two arithmetic facts the quantizing kernels rely on to match
the fp64 quantizer of the oracle bit for bit (Sec. 3.3, the group-wise
uniform quantizer with fp16 scale and minimum).  Both are emulated here with
IEEE fp32 (numpy float32) and exact extended-precision sums (the x86 long
double's 64-bit significand holds every product and sum below exactly, so a
single rounding to fp32 emulates an fma).

1. The scale's fp32 quotient range / (2^b - 1), b = 1..8, equals
   q0 + rq * (range - q0 * qmax) rounded once, with q0 = range * rq and rq
   the fp32 reciprocal of qmax (the kernels' three-instruction form of the
   division).
2. The code rint((c - m16) / s16), clamped to [0, 2^b - 1], is the same from
   the fp32 quotient (c - m16) * rcp(s16), for any reciprocal within 1 ulp,
   as from the fp64 quotient whenever the fp32 quotient lies farther than
   2^(b-21) from every half-integer (the kernels' fallback trigger).
"""
import numpy as np
import pytest

LD = np.longdouble


def fma32(a, b, c):
    """fp32 fma: the exact a * b + c rounded once to fp32."""
    return (a.astype(LD) * b.astype(LD) + c.astype(LD)).astype(np.float32)


def div_qmax(x, qmax, rq):
    q0 = (x * rq).astype(np.float32)
    return fma32(fma32(-q0, qmax, x), rq, q0)


def _binade(exp_bits, count=None, seed=0):
    if count is None:
        m = np.arange(1 << 23, dtype=np.uint32)
    else:
        m = np.random.default_rng(seed).integers(0, 1 << 23, size=count, dtype=np.uint32)
    return ((np.uint32(exp_bits) << np.uint32(23)) | m).view(np.float32)


def test_extended_precision_is_wide_enough():
    assert np.finfo(LD).nmant >= 63


@pytest.mark.parametrize("b", range(1, 9))
def test_division_by_qmax_whole_binade(b):
    """Every fp32 significand in [1, 2) (scaling carries the result to every
    binade whose quotient and residual stay normal)."""
    qmax = np.float32((1 << b) - 1)
    rq = np.float32(1) / qmax
    x = _binade(127)
    assert np.array_equal(div_qmax(x, qmax, rq), x / qmax)


@pytest.mark.parametrize("b", range(1, 9))
def test_division_by_qmax_extreme_binades(b):
    """Subnormal and smallest normal inputs (subnormal quotients and
    residuals), and the largest binade, sampled."""
    qmax = np.float32((1 << b) - 1)
    rq = np.float32(1) / qmax
    for e in (0, 1, 2, 9, 24, 254):
        x = _binade(e, count=1 << 18, seed=e + b)
        x = x[x > 0]
        with np.errstate(under="ignore", over="ignore"):
            assert np.array_equal(div_qmax(x, qmax, rq), x / qmax), (b, e)


def _codes_fp64(c, mf, sf, qmax):
    t = (c.astype(np.float64) - mf.astype(np.float64)) / sf.astype(np.float64)
    return np.clip(np.rint(t), 0, qmax)


@pytest.mark.parametrize("b", range(1, 9))
def test_fp32_code_rule_outside_the_margin(b):
    """Adversarial quotients near every half-integer of the code range (and
    near the clamp edges), with the reciprocal rounded down, to nearest and
    up: outside the margin the fp32 rule gives the fp64 code."""
    rng = np.random.default_rng(100 + b)
    qmax = (1 << b) - 1
    n = 400_000
    sf = (rng.uniform(0.5, 2.0, n) * 2.0 ** rng.integers(-20, 10, n)).astype(np.float16)
    sf = sf[(sf > 0) & np.isfinite(sf)].astype(np.float32)
    n = sf.size
    mf = (rng.standard_normal(n) * sf * rng.uniform(0, 8, n)).astype(np.float16).astype(np.float32)
    k = rng.integers(-1, qmax + 1, n).astype(np.float64)
    # quotients at k + 1/2 offset by a few multiples of the margin, both sides
    off = rng.choice([-1, 1], n) * rng.uniform(0, 4, n) * 2.0 ** (b - 21)
    c = (mf.astype(np.float64) + (k + 0.5 + off) * sf.astype(np.float64)).astype(np.float32)
    ref = _codes_fp64(c, mf, sf, qmax)
    near_at = np.float32(0.5) - np.float32(2.0 ** (b - 21))
    inv0 = np.float32(1) / sf
    checked = 0
    for inv in (np.nextafter(inv0, np.float32(0)), inv0, np.nextafter(inv0, np.float32(np.inf))):
        t = ((c - mf).astype(np.float32) * inv).astype(np.float32)
        r = np.rint(t)
        far = np.abs(t - r) <= near_at
        q = np.clip(r, 0, qmax)
        assert np.array_equal(q[far], ref[far]), b
        checked += int(far.sum())
    assert checked > n  # the margin leaves most samples to the fp32 rule


def test_fp32_code_rule_needs_a_margin():
    """Planting the mistake (no margin at b = 8): the same adversarial
    quotients then give codes that differ from fp64, so the test above can
    fail."""
    rng = np.random.default_rng(7)
    b, qmax, n = 8, 255, 400_000
    sf = (rng.uniform(0.5, 2.0, n) * 2.0 ** rng.integers(-20, 10, n)).astype(np.float16)
    sf = sf[(sf > 0) & np.isfinite(sf)].astype(np.float32)
    n = sf.size
    mf = (rng.standard_normal(n) * sf * rng.uniform(0, 8, n)).astype(np.float16).astype(np.float32)
    k = rng.integers(0, qmax, n).astype(np.float64)
    off = rng.choice([-1, 1], n) * rng.uniform(0, 4, n) * 2.0 ** (b - 21)
    c = (mf.astype(np.float64) + (k + 0.5 + off) * sf.astype(np.float64)).astype(np.float32)
    ref = _codes_fp64(c, mf, sf, qmax)
    inv = np.nextafter(np.float32(1) / sf, np.float32(np.inf))
    t = ((c - mf).astype(np.float32) * inv).astype(np.float32)
    q = np.clip(np.rint(t), 0, qmax)
    assert np.any(q != ref)
