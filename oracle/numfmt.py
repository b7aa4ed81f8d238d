"""IEEE-754 half formats used by mixed-precision training (oracle).

MPX §3.1 casts float leaves to ``float16`` or ``bfloat16``; §2 runs the
forward and backward passes in those 16-bit formats.  This module rounds any
real value (given as float32 or float64) to the nearest value of a target
format, ties to even, following the IEEE-754 definition of rounding:

* a finite x with leading-bit exponent e = floor(log2 |x|) has quantum
  q = 2**(max(e, emin) - (p - 1)) in a format with p significand bits and
  minimum normal exponent emin (below emin the quantum stays fixed: that is the
  subnormal range, which is kept, not flushed);
* the result is the multiple of q nearest to x, ties to the even multiple;
* a rounded magnitude of 2**(emax + 1) or more overflows to +-inf;
* +-inf and NaN pass through; the sign of zero is kept.

Half-precision values are carried as float32 arrays holding exactly
representable values (both 16-bit formats are subsets of float32).
"""
from __future__ import annotations

import numpy as np

# name -> (significand bits incl. the hidden bit, emin, emax)
FORMATS = {
    "f16": (11, -14, 15),
    "bf16": (8, -126, 127),
    "f32": (24, -126, 127),
}

MAX_FINITE = {
    "f16": 65504.0,
    "bf16": float(np.ldexp(2.0 - 2.0 ** -7, 127)),
}


def _round_block(x, p: int, emin: int, emax: int) -> np.ndarray:
    x64 = np.asarray(x, dtype=np.float64)
    _, E = np.frexp(x64)                     # x = m * 2**E, 0.5 <= |m| < 1
    e = np.maximum(E - 1, emin)              # leading-bit exponent, floored at emin
    q = np.ldexp(1.0, e - (p - 1))           # quantum of the target format
    r = np.rint(x64 / q) * q                 # np.rint: ties to even
    # overflow to +-inf; +-inf and NaN come through the division unchanged
    r = np.where(np.abs(r) >= np.ldexp(1.0, emax + 1), np.copysign(np.inf, x64), r)
    return r.astype(np.float32)


CHUNK = 1 << 16


def round_to(x, fmt: str) -> np.ndarray:
    """Round ``x`` (float32 or float64 values) to format ``fmt``; float32 out.

    One rounding straight from the given value: a float64 input is not passed
    through float32 first.  Elementwise; large arrays are processed in slices
    only to keep temporaries small.
    """
    p, emin, emax = FORMATS[fmt]
    x = np.asarray(x)
    with np.errstate(invalid="ignore"):      # signalling NaN inputs stay NaN
        if x.size <= CHUNK:
            return _round_block(x, p, emin, emax)
        xf = x.reshape(-1)
        out = np.empty(xf.shape, np.float32)
        for i in range(0, xf.size, CHUNK):
            out[i:i + CHUNK] = _round_block(xf[i:i + CHUNK], p, emin, emax)
        return out.reshape(x.shape)
