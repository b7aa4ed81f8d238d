"""Per-op precision policy and the GEMM definition (oracle).

MPX §3 relies on type promotion: an op runs in the precision its inputs were
cast to, so after the inputs are cast to half precision (§3.4) every layer
computes in half precision, while overflow-prone reductions (sums, means,
softmax) are forced to full precision (§3.2, ``force_full_precision``).  Half
products are accumulated in float32, as half-precision tensor units do.

The reading taken here (one rounding per layer-level op):

* GEMM: C = R(sum_k f32(A[m,k]) * f32(B[k,n]) [+ f32(bias[n])]), the sum in
  float32 (a library float32 matmul; every half x half product is exact in
  float32), the bias added in float32, then one rounding R to half.
* full-precision islands (GELU, LayerNorm, softmax, loss, bias sums of the
  backward) compute on the widened half inputs and round once at the output.
  The oracle computes these islands in float64, the closest it can get to the
  exact value; float32 arithmetic differs from it by far less than a half ulp.

``Policy("f64")`` switches every rounding off and computes GEMMs in float64:
the plain real-arithmetic model used for finite-difference checks.

``Policy("f32")`` is full-precision training (MPX's ``use_mixed_precision``
switched off, §3.4: nothing is cast to half): every op's output is rounded to
float32, GEMMs accumulate in float32 (a library float32 matmul) and the
full-precision islands are computed in float64 and rounded once to float32.
"""
from __future__ import annotations

import numpy as np

from .numfmt import round_to


class Policy:
    def __init__(self, fmt: str):
        if fmt not in ("f16", "bf16", "f32", "f64"):
            raise ValueError(fmt)
        self.fmt = fmt
        self.exact = fmt == "f64"

    def R(self, x) -> np.ndarray:
        """Round to the compute format (float32 carrier) or keep float64."""
        if self.exact:
            return np.asarray(x, dtype=np.float64)
        return round_to(x, self.fmt)

    def acc(self, x) -> np.ndarray:
        """Widen a half value to the accumulation type (exact)."""
        return np.asarray(x, dtype=np.float64 if self.exact else np.float32)

    def mm(self, a, b) -> np.ndarray:
        """Unrounded product a @ b: float32 accumulation (float64 when exact).

        Works on stacks of matrices (leading batch axes) like ``np.matmul``.
        """
        a = self.acc(a)
        b = self.acc(b)
        return np.matmul(a, b)

    def gemm(self, a, b, bias=None) -> np.ndarray:
        """C = R(a @ b [+ bias]) with a single rounding."""
        c = self.mm(a, b)
        if bias is not None:
            c = c + self.acc(bias)
        return self.R(c)

    def colsum(self, x) -> np.ndarray:
        """R(sum over rows) of a 2-D half array: the bias-gradient reduction."""
        return self.R(np.sum(np.asarray(x, dtype=np.float64), axis=0))
