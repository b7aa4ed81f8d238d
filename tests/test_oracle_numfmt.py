"""Pins of the oracle's half-precision rounding against library conversions.

The oracle rounds from the IEEE definition (quantum, ties to even, overflow
threshold).  Here it is checked against two independent library routines —
numpy's float32->float16 and float64->float16 conversions and torch's CPU
float32->bfloat16 conversion — over structured bit-pattern sets that include
every exponent, every rounding tie position, subnormals, overflow and NaN.
"""
import numpy as np
import pytest
import torch

from oracle.numfmt import MAX_FINITE, round_to


def _same(a, b):
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    na, nb = np.isnan(a), np.isnan(b)
    assert np.array_equal(na, nb)
    # compare bit patterns so that the sign of zero is checked too
    assert np.array_equal(a[~na].view(np.uint32), b[~nb].view(np.uint32))


def _f16_patterns():
    rng = np.random.default_rng(7)
    hi = np.arange(1 << 19, dtype=np.uint32) << 13           # sign, exponent, 10 mantissa bits
    lows = np.array([0, 1, 0x0FFF, 0x1000, 0x1001, 0x1FFF], np.uint32)
    pats = [(hi[:, None] | lows[None, :]).reshape(-1),
            hi | rng.integers(0, 1 << 13, size=hi.size, dtype=np.uint32)]
    return np.concatenate(pats).view(np.float32)


def _ties(p, emin, lo, hi_e):
    """Exact halfway points between neighbours of a format with p bits, +-1 f32 ulp."""
    out = []
    rng = np.random.default_rng(3)
    for e in range(lo, hi_e):
        q = np.ldexp(1.0, max(e, emin) - (p - 1))
        k = rng.integers(0, 1 << p, size=64) | 1              # odd multiples of q/2
        base = np.ldexp(1.0, e) + k * (q / 2)
        t = base.astype(np.float32)
        out += [t, np.nextafter(t, np.float32(np.inf)), np.nextafter(t, np.float32(0))]
    v = np.concatenate(out)
    return np.concatenate([v, -v])


def test_f16_matches_numpy_structured():
    x = _f16_patterns()
    with np.errstate(over="ignore", invalid="ignore"):
        ref = x.astype(np.float16).astype(np.float32)
    _same(round_to(x, "f16"), ref)


def test_f16_ties_and_subnormals_match_numpy():
    x = _ties(11, -14, -27, 16)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).astype(np.float32)
    _same(round_to(x, "f16"), ref)


def test_f16_from_float64_matches_numpy_direct():
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.normal(0, 1, 200_000), rng.normal(0, 3e4, 50_000),
                        rng.normal(0, 1e-6, 50_000)])
    # values that double rounding through float32 would get wrong
    x = np.concatenate([x, 1.0 + 2.0 ** -11 + 2.0 ** np.arange(-40, -25, dtype=np.float64)])
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).astype(np.float32)
    _same(round_to(x, "f16"), ref)


def test_bf16_matches_torch_structured():
    rng = np.random.default_rng(5)
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)
    pats = np.concatenate([(hi[:, None] | lows[None, :]).reshape(-1),
                           hi | rng.integers(0, 1 << 16, size=hi.size, dtype=np.uint32)])
    x = pats.view(np.float32)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    _same(round_to(x, "bf16"), ref)


def test_bf16_ties_match_torch():
    x = _ties(8, -126, -133, 128).astype(np.float32)
    x = x[np.isfinite(x)]
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    _same(round_to(x, "bf16"), ref)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_special_values(fmt):
    m = MAX_FINITE[fmt]
    x = np.array([np.inf, -np.inf, np.nan, 0.0, -0.0, m, -m], np.float64)
    r = round_to(x, fmt)
    assert np.isposinf(r[0]) and np.isneginf(r[1]) and np.isnan(r[2])
    assert r[3] == 0 and not np.signbit(r[3]) and r[4] == 0 and np.signbit(r[4])
    assert r[5] == m and r[6] == -m


def test_f16_overflow_threshold_and_subnormals():
    # 65520 is the midpoint between 65504 and 2**16: it rounds to even -> inf
    r = round_to(np.array([65519.99, 65520.0, -65520.0], np.float64), "f16")
    assert r[0] == 65504 and np.isposinf(r[1]) and np.isneginf(r[2])
    s = 2.0 ** -24                                      # smallest f16 subnormal
    r = round_to(np.array([s, 0.5 * s, 0.75 * s, 1.5 * s, 2.5 * s]), "f16")
    assert list(r) == [s, 0.0, s, 2 * s, 2 * s]


def test_bf16_overflow_threshold():
    top = np.ldexp(2.0 - 2.0 ** -7, 127)
    half_ulp = np.ldexp(1.0, 127 - 8)
    r = round_to(np.array([top + half_ulp * 0.99, top + half_ulp]), "bf16")
    assert r[0] == np.float32(top) and np.isposinf(r[1])
