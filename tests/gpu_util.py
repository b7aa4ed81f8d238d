"""Helpers for the GPU parity tests (test infrastructure only)."""
from __future__ import annotations

import numpy as np
import pytest

try:
    import torch
    HAVE_GPU = torch.cuda.is_available()
except Exception:  # pragma: no cover
    torch = None
    HAVE_GPU = False

needs_gpu = pytest.mark.skipif(not HAVE_GPU, reason="no GPU")

TORCH_HALF = {"f16": None, "bf16": None}
if torch is not None:
    TORCH_HALF = {"f16": torch.float16, "bf16": torch.bfloat16}
FMT_BITS = {"f16": (11, -14), "bf16": (8, -126), "f32": (24, -126)}


def to_dev_half(a: np.ndarray, fmt: str):
    """Upload half-representable float32 values as a half tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH_HALF[fmt]).cuda()


def to_host(t) -> np.ndarray:
    """Device tensor -> float32 numpy (exact widening of half values)."""
    return t.detach().float().cpu().numpy()


def ulp(x: np.ndarray, fmt: str) -> np.ndarray:
    """Spacing of the format (half, or float32) at |x| (subnormal spacing below
    the normal range)."""
    p, emin = FMT_BITS[fmt]
    x = np.abs(np.asarray(x, np.float64))
    _, e = np.frexp(np.where(np.isfinite(x), x, 1.0))
    return np.ldexp(1.0, np.maximum(e - 1, emin) - (p - 1))


def assert_same_values(gpu: np.ndarray, ref: np.ndarray, what: str = ""):
    """Bitwise equality of float32 arrays; NaN compared as a class."""
    gpu = np.asarray(gpu, np.float32)
    ref = np.asarray(ref, np.float32)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    ng, nr = np.isnan(gpu), np.isnan(ref)
    assert np.array_equal(ng, nr), f"{what}: NaN positions differ"
    bad = np.flatnonzero(gpu[~ng].view(np.uint32) != ref[~nr].view(np.uint32))
    assert bad.size == 0, f"{what}: {bad.size} values differ, first gpu={gpu[~ng][bad[0]]} ref={ref[~nr][bad[0]]}"


def gemm_bound(a: np.ndarray, b: np.ndarray, ref: np.ndarray, fmt: str, k: int, ulps: float = 1.0):
    """Per-element bound |gpu - ref| <= ulps*ulp(ref) + 2 K 2^-24 (|A||B|)."""
    absprod = np.abs(a.astype(np.float64)) @ np.abs(b.astype(np.float64))
    return ulps * ulp(ref, fmt) + 2.0 * k * 2.0 ** -24 * absprod


def assert_within(gpu, ref, bound, what=""):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(gpu), fin), f"{what}: finiteness differs"
    err = np.abs(gpu[fin] - ref[fin])
    bnd = np.broadcast_to(bound, ref.shape)[fin]
    bad = np.flatnonzero(err > bnd)
    assert bad.size == 0, (f"{what}: {bad.size}/{err.size} beyond bound; worst err "
                           f"{err[bad].max():.3g} vs bound {bnd[bad][np.argmax(err[bad])]:.3g}")


def rel_norm_err(gpu, ref) -> float:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(gpu - ref) / (den if den > 0 else 1.0))
