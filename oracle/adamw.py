"""Masked AdamW on float32 master weights (oracle).

MPX §3.5: ``optimizer_update`` applies the optimizer only when the gradients
are finite; otherwise the model is left as it is.  The reading taken here
also leaves the optimizer state (first and second moments and the step
count) untouched on a skipped step, since updating moments with non-finite
gradients would poison them; the step count therefore counts applied steps
and drives the bias correction.

The optimizer is AdamW (Loshchilov & Hutter, decoupled weight decay, in the
form Optax implements): with t the applied-step count after increment,

    m <- b1 m + (1 - b1) g
    v <- b2 v + (1 - b2) g^2
    mhat = m / (1 - b1^t),  vhat = v / (1 - b2^t)
    p <- p - lr (mhat / (sqrt(vhat) + eps) + wd p)

Every constant derived from the hyperparameters (b1, b2, 1 - b1, 1 - b2,
1 - b1^t, 1 - b2^t, lr, eps, wd) is computed in float64 from the given values
and rounded to float32 once; the per-element arithmetic is float32 in the
order written.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class AdamWHP:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 1e-4


def bias_corrections(t: int, hp: AdamWHP):
    """(1 - b1^t, 1 - b2^t) as float32, computed in float64."""
    return (np.float32(1.0 - float(hp.beta1) ** t), np.float32(1.0 - float(hp.beta2) ** t))


def constants(hp: AdamWHP):
    """(b1, 1 - b1, b2, 1 - b2, lr, eps, wd) as float32, computed in float64."""
    f = np.float32
    b1, b2 = float(hp.beta1), float(hp.beta2)
    return (f(b1), f(1.0 - b1), f(b2), f(1.0 - b2), f(hp.lr), f(hp.eps), f(hp.weight_decay))


def adamw_update(p, m, v, g, t_new: int, hp: AdamWHP):
    """One AdamW update of float32 arrays; returns new (p, m, v)."""
    b1, omb1, b2, omb2, lr, eps, wd = constants(hp)
    g = np.asarray(g, dtype=np.float32)
    m = b1 * m + omb1 * g
    v = b2 * v + omb2 * (g * g)
    bc1, bc2 = bias_corrections(t_new, hp)
    mhat = m / bc1
    vhat = v / bc2
    upd = mhat / (np.sqrt(vhat) + eps) + wd * p
    p = p - lr * upd
    return p.astype(np.float32), m.astype(np.float32), v.astype(np.float32)


def adamw_masked(params, moms1, moms2, grads32, t: int, hp: AdamWHP, finite: bool):
    """Apply AdamW to every leaf when ``finite``; otherwise change nothing.

    ``params``, ``moms1``, ``moms2``, ``grads32`` are lists of float32 arrays.
    Returns (params, moms1, moms2, t) as new lists (inputs are not modified).
    """
    if not finite:
        return [a.copy() for a in params], [a.copy() for a in moms1], \
            [a.copy() for a in moms2], t
    t_new = t + 1
    out_p, out_m, out_v = [], [], []
    for p, m, v, g in zip(params, moms1, moms2, grads32):
        p2, m2, v2 = adamw_update(p, m, v, g, t_new, hp)
        out_p.append(p2)
        out_m.append(m2)
        out_v.append(v2)
    return out_p, out_m, out_v, t_new
