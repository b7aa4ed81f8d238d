"""The mixed-precision training step, composed from its parts (oracle).

The order follows MPX §3.4 (the transformed gradient function) and §3.5
(the masked optimizer update), which together carry out the recipe of §2.1:

1. cast every float input and every master weight to half precision
   (integer labels are left alone, §3.1);
2. run the forward pass and the loss (the loss in full precision);
3. scale: the backward pass is seeded with the current loss scale;
4. backward pass in half precision: scaled half gradients;
5. unscale: widen to float32 and divide by the scale;
6. check that every gradient is finite;
7. adjust the loss scale from that flag;
8. apply AdamW to the float32 masters only if the gradients were finite.

``finish_step`` takes already-computed half gradients, so tests can feed it
the GPU's gradients (lockstep parity) as well as the oracle's own.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Dict, List, Optional

import numpy as np

import workloads

from . import models, scaling
from .adamw import AdamWHP, adamw_masked
from .policy import Policy


@dataclass
class TrainState:
    names: List[str]
    masters: List[np.ndarray]      # float32
    m: List[np.ndarray]            # float32
    v: List[np.ndarray]            # float32
    t: int
    scale: scaling.ScaleState


@dataclass
class StepResult:
    loss: float
    nonfinite: int
    finite: bool
    scale_used: float
    grads_half: List[np.ndarray]   # scaled half gradients (after injection)


def hp_of(cfg) -> AdamWHP:
    return AdamWHP(cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay)


def init_state(cfg, masters: Optional[Dict[str, np.ndarray]] = None) -> TrainState:
    if masters is None:
        masters = workloads.init_params(cfg)
    names = [n for n, _, _ in workloads.param_specs(cfg)]
    ms = [np.array(masters[n], dtype=np.float32, copy=True) for n in names]
    return TrainState(names, ms, [np.zeros_like(a) for a in ms],
                      [np.zeros_like(a) for a in ms], 0,
                      scaling.make_state(cfg.scale_init, cfg.period, cfg.factor,
                                         cfg.min_scale, cfg.max_scale))


def cast_batch(pol: Policy, batch: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """Cast float inputs and float targets to half; integer labels untouched."""
    out = {}
    for k, a in batch.items():
        a = np.asarray(a)
        out[k] = pol.R(a) if np.issubdtype(a.dtype, np.floating) else a
    return out


def apply_injections(cfg, step: int, grads: List[np.ndarray]) -> None:
    for inj in cfg.injections:
        if inj.step == step:
            flat = grads[inj.tensor].reshape(-1)
            flat[inj.element] = np.float32(inj.value)


def gradients(cfg, state: TrainState, batch: Dict[str, np.ndarray], pol: Policy):
    """Steps 1-4: half forward/backward of the scaled loss.

    Returns (loss, list of scaled half gradients in parameter order).
    """
    P = {n: pol.R(w) for n, w in zip(state.names, state.masters)}
    hb = cast_batch(pol, batch)
    loss, dout, cache = models.forward_loss(pol, cfg, P, hb, state.scale.scale)
    G = models.backward(pol, cfg, P, cache, dout)
    return loss, [np.array(G[n], dtype=np.float32) for n in state.names]


def finish_step(cfg, state: TrainState, grads_half: List[np.ndarray]):
    """Steps 5-8 on given half gradients; returns (new_state, nonfinite)."""
    nonfinite = scaling.count_nonfinite(grads_half)
    finite = nonfinite == 0
    g32 = [scaling.unscale(g, state.scale.scale) for g in grads_half]
    new_scale = scaling.adjust(state.scale, finite)
    p, m, v, t = adamw_masked(state.masters, state.m, state.v, g32, state.t,
                              hp_of(cfg), finite)
    return replace(state, masters=p, m=m, v=v, t=t, scale=new_scale), nonfinite


def train_step(cfg, state: TrainState, batch, step: int, pol: Optional[Policy] = None):
    pol = pol or Policy(cfg.half)
    scale_used = float(state.scale.scale)
    loss, grads = gradients(cfg, state, batch, pol)
    apply_injections(cfg, step, grads)
    new_state, nonfinite = finish_step(cfg, state, grads)
    return new_state, StepResult(loss, nonfinite, nonfinite == 0, scale_used, grads)


def full_precision_step(cfg, state: TrainState, batch) -> tuple:
    """One training step with mixed precision switched off (MPX's
    ``use_mixed_precision=False``, §3.4): inputs and weights stay float32, the
    loss is not scaled, every op rounds to float32 (``Policy("f32")``), and
    AdamW is applied unconditionally to the float32 gradients.  The loss
    scale state is left as it is.  Returns (new_state, loss, gradients)."""
    pol = Policy("f32")
    P = {n: pol.R(w) for n, w in zip(state.names, state.masters)}
    loss, dout, cache = models.forward_loss(pol, cfg, P, cast_batch(pol, batch), 1.0)
    G = models.backward(pol, cfg, P, cache, dout)
    grads = [np.array(G[n], dtype=np.float32) for n in state.names]
    p, m, v, t = adamw_masked(state.masters, state.m, state.v, grads, state.t, hp_of(cfg), True)
    return replace(state, masters=p, m=m, v=v, t=t), loss, grads


def run(cfg, steps: Optional[int] = None, state: Optional[TrainState] = None):
    """Free-running: ``steps`` training steps on the fixed synthetic batch."""
    state = state or init_state(cfg)
    batch = workloads.make_batch(cfg)
    results = []
    for s in range(cfg.steps if steps is None else steps):
        state, r = train_step(cfg, state, batch, s)
        results.append(r)
    return state, results


# ------------------------------------------------------------ sweep (c5) --

@dataclass
class SweepState:
    p: List[np.ndarray]
    m: List[np.ndarray]
    v: List[np.ndarray]
    t: int
    scale: scaling.ScaleState


def sweep_init(cfg, grads_f32: List[np.ndarray], params: List[np.ndarray]):
    """Half gradients (rounded here) and the initial optimizer state."""
    grads_half = [Policy(cfg.half).R(g) for g in grads_f32]
    st = SweepState([p.copy() for p in params], [np.zeros_like(p) for p in params],
                    [np.zeros_like(p) for p in params], 0,
                    scaling.make_state(cfg.scale_init, cfg.period, cfg.factor,
                                       cfg.min_scale, cfg.max_scale))
    return grads_half, st


def sweep_step(cfg, st: SweepState, grads_half: List[np.ndarray], step: int):
    """unscale + finite check + scale update + masked AdamW on fixed gradients.

    Injections are applied to a copy of the gradient list for this step only.
    Returns (new_state, nonfinite, scale_used).
    """
    g = grads_half
    if any(inj.step == step for inj in cfg.injections):
        g = [a.copy() for a in grads_half]
        apply_injections(cfg, step, g)
    nonfinite = scaling.count_nonfinite(g)
    finite = nonfinite == 0
    g32 = [scaling.unscale(a, st.scale.scale) for a in g]
    scale_used = float(st.scale.scale)
    new_scale = scaling.adjust(st.scale, finite)
    p, m, v, t = adamw_masked(st.p, st.m, st.v, g32, st.t, hp_of(cfg), finite)
    return SweepState(p, m, v, t, new_scale), nonfinite, scale_used
