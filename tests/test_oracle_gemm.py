"""Pins of the oracle's GEMM and linear layer.

The oracle accumulates half x half products in float32 (a library float32
matmul).  Each product is exact in float32, so the result differs from the
exact sum only by float32 accumulation error, bounded by K * 2^-24 * (|A||B|).
It is checked against a float64 matmul with that bound, and against a
brute-force element-by-element sum on a tiny case (which would catch a
transposed operand or a dropped bias).
"""
import numpy as np
import pytest

from oracle import ops
from oracle.numfmt import round_to
from oracle.policy import Policy


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
@pytest.mark.parametrize("mnk", [(64, 96, 512), (33, 17, 1537), (1, 5, 4096)])
def test_fp32_accumulation_within_bound(fmt, mnk):
    m, n, k = mnk
    rng = np.random.default_rng(m + n + k)
    a = round_to(rng.normal(0, 1, (m, k)), fmt)
    b = round_to(rng.normal(0, 1, (k, n)), fmt)
    pol = Policy(fmt)
    c32 = pol.mm(a, b)
    assert c32.dtype == np.float32
    c64 = a.astype(np.float64) @ b.astype(np.float64)
    bound = k * 2.0 ** -24 * (np.abs(a).astype(np.float64) @ np.abs(b).astype(np.float64))
    assert np.all(np.abs(c32 - c64) <= bound)
    # after the single rounding: within one half ulp of the correctly rounded sum
    r32 = pol.R(c32).astype(np.float64)
    p, emin = {"f16": (11, -14), "bf16": (8, -126)}[fmt]
    _, e = np.frexp(c64)
    ulp = np.ldexp(1.0, np.maximum(e - 1, emin) - (p - 1))
    # |R(c32) - exact| <= |R(c32) - c32| + |c32 - exact| <= ulp/2 + bound (+ ulp slack
    # for c32 rounding across a binade boundary)
    assert np.all(np.abs(r32 - c64) <= ulp + bound)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_linear_brute_force(fmt):
    rng = np.random.default_rng(1)
    M, N, K = 5, 3, 7
    x = round_to(rng.normal(0, 1, (M, K)), fmt)
    w = round_to(rng.normal(0, 1, (N, K)), fmt)
    b = round_to(rng.normal(0, 1, N), fmt)
    y = ops.linear_fwd(Policy(fmt), x, w, b)
    for i in range(M):
        for j in range(N):
            s = sum(float(x[i, kk]) * float(w[j, kk]) for kk in range(K)) + float(b[j])
            assert abs(float(y[i, j]) - s) <= abs(s) * 2.0 ** -7 + 1e-6
    dy = round_to(rng.normal(0, 1, (M, N)), fmt)
    dx, dw, db = ops.linear_bwd(Policy(fmt), x, w, dy)
    for i in range(M):
        for kk in range(K):
            s = sum(float(dy[i, j]) * float(w[j, kk]) for j in range(N))
            assert abs(float(dx[i, kk]) - s) <= abs(s) * 2.0 ** -7 + 1e-6
    for j in range(N):
        for kk in range(K):
            s = sum(float(dy[i, j]) * float(x[i, kk]) for i in range(M))
            assert abs(float(dw[j, kk]) - s) <= abs(s) * 2.0 ** -7 + 1e-6
        s = sum(float(dy[i, j]) for i in range(M))
        assert abs(float(db[j]) - s) <= abs(s) * 2.0 ** -7 + 1e-6


def test_gemm_output_is_representable_and_overflows_to_inf():
    pol = Policy("f16")
    a = np.full((2, 4), 256.0, np.float32)
    b = np.full((4, 2), 256.0, np.float32)          # sums of 4 * 65536 -> inf in f16
    c = pol.gemm(a, b)
    assert np.all(np.isposinf(c))
