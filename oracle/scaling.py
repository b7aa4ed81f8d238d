"""Dynamic loss scaling: unscale, finite check and scale update (oracle).

MPX §3.3 defines the loss-scaling state with three operations:

* ``scale(x)`` multiplies by the current factor (here the seed of the
  backward pass: the loss cotangent is the scale itself, §3.4);
* ``unscale(x)`` divides by the factor and casts to full precision.  The
  order of the two is not stated; the reading taken here is: widen to float32
  first, then divide (float16 cannot hold 2**16, so dividing in half precision
  is not meant);
* ``adjust(grads_finite)`` updates the factor following the dynamic scheme of
  §2.1: when the scaled gradients overflow, reduce the factor (and the step is
  skipped); when they stay finite for a long enough run, increase it.

The reading of "long enough" taken here: ``period`` consecutive finite steps.
The counter resets on overflow and on growth; growth takes effect from the
next step.  The factor halves and doubles (``factor`` = 2), clamped to
[min_scale, max_scale].

The finite check (§3.4: "check whether the gradients are finite") covers
every gradient leaf; +-inf and NaN both count as non-finite.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class ScaleState:
    scale: np.float32
    counter: int
    period: int
    factor: np.float32 = np.float32(2.0)
    min_scale: np.float32 = np.float32(1.0)
    max_scale: np.float32 = np.float32(2.0 ** 127)


def make_state(scale: float, period: int, factor: float = 2.0,
               min_scale: float = 1.0, max_scale: float = 2.0 ** 127) -> ScaleState:
    return ScaleState(np.float32(scale), 0, int(period), np.float32(factor),
                      np.float32(min_scale), np.float32(max_scale))


def count_nonfinite(grads) -> int:
    """Number of non-finite values over every leaf (0 means all finite)."""
    return int(sum(int(np.count_nonzero(~np.isfinite(np.asarray(g)))) for g in grads))


def unscale(g_half, scale) -> np.ndarray:
    """float32(g) / scale, computed in float32 (cast first, then divide)."""
    return np.asarray(g_half, dtype=np.float32) / np.float32(scale)


def adjust(state: ScaleState, finite: bool) -> ScaleState:
    """One update of the dynamic loss-scale state."""
    if finite:
        counter = state.counter + 1
        scale = state.scale
        if counter == state.period:
            scale = np.float32(min(np.float32(scale * state.factor), state.max_scale))
            counter = 0
        return replace(state, scale=np.float32(scale), counter=counter)
    scale = np.float32(max(np.float32(state.scale / state.factor), state.min_scale))
    return replace(state, scale=scale, counter=0)
