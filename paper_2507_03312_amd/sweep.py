"""The standalone optimizer sweep: unscale + all-finite check, masked AdamW
and the loss-scale update over a list of separately allocated half gradient
tensors (MPX §3.3-§3.5), one multi-tensor launch per call.

The gradients stay fixed across steps; an injected non-finite value is
written before a step and the original value restored after it.
"""
from __future__ import annotations

from typing import List

import numpy as np
import torch

import workloads

from . import binding as mx
from .train import TORCH_HALF, _ptr, _stream, pack_scale_state, unpack_scale_state


class SweepStep:
    def __init__(self, cfg, sizes=None, device="cuda", half_copy=True):
        self.cfg = cfg
        self.device = torch.device(device)
        self.dt = mx.DTYPES[cfg.half]
        hdt = TORCH_HALF[cfg.half]
        self.sizes = workloads.sweep_sizes(cfg) if sizes is None else np.asarray(sizes)
        dev = self.device
        self.p = [torch.zeros(int(n), dtype=torch.float32, device=dev) for n in self.sizes]
        self.m = [torch.zeros_like(t) for t in self.p]
        self.v = [torch.zeros_like(t) for t in self.p]
        self.g32 = [torch.zeros_like(t) for t in self.p]      # staging for the half cast
        self.g = [torch.zeros(int(n), dtype=hdt, device=dev) for n in self.sizes]
        self.h = [torch.zeros(int(n), dtype=hdt, device=dev) for n in self.sizes] if half_copy else None
        self.L_p, self.L_m, self.L_v = mx.TensorList(self.p), mx.TensorList(self.m), mx.TensorList(self.v)
        self.L_g, self.L_g32 = mx.TensorList(self.g), mx.TensorList(self.g32)
        self.L_h = mx.TensorList(self.h) if half_copy else None
        self.d_state = torch.from_numpy(pack_scale_state(cfg.scale_init, 0, cfg.period, cfg.factor,
                                                         cfg.min_scale, cfg.max_scale)).to(dev)
        self.d_nonfinite = torch.zeros(1, dtype=torch.int32, device=dev)
        self.d_step = torch.zeros(1, dtype=torch.int32, device=dev)
        self.hp = mx.AdamWHP(cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay)
        self.numel = int(self.sizes.sum())

    def load(self, grads_f32: List[np.ndarray], params: List[np.ndarray]):
        """Copy fp32 draws in and round the gradients to half on the device."""
        for t, a in zip(self.p, params):
            t.copy_(torch.from_numpy(a))
        for t, a in zip(self.g32, grads_f32):
            t.copy_(torch.from_numpy(a))
        for t in self.m + self.v:
            t.zero_()
        mx.mpx_cast_to_half(self.L_g32, self.L_g, self.dt, _stream())

    def step(self, s=None):
        s = _stream() if s is None else s
        mx.mpx_unscale_check(self.L_g, self.dt, _ptr(self.d_state), _ptr(self.d_nonfinite), None, s)
        mx.mpx_adamw_masked(self.L_p, self.L_m, self.L_v, self.L_g, self.dt, self.hp,
                            _ptr(self.d_step), _ptr(self.d_state), _ptr(self.d_nonfinite),
                            self.L_h, self.dt, s)
        mx.mpx_scale_update(_ptr(self.d_state), _ptr(self.d_nonfinite), s)

    def adamw(self, s):
        mx.mpx_adamw_masked(self.L_p, self.L_m, self.L_v, self.L_g, self.dt, self.hp,
                            _ptr(self.d_step), _ptr(self.d_state), _ptr(self.d_nonfinite),
                            self.L_h, self.dt, s)

    def time_graph(self, body, launches: int = 10, reps: int = 3) -> float:
        """Mean ms per call of ``body(stream)`` from HIP events around a graph
        of ``launches`` back-to-back calls."""
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(launches):
                body(_stream())
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (reps * launches)

    def injections_at(self, step: int):
        return [inj for inj in self.cfg.injections if inj.step == step]

    def inject(self, inj):
        flat = self.g[inj.tensor]
        idx = inj.element % flat.numel()
        old = flat[idx].clone()
        flat[idx] = inj.value
        return (flat, idx, old)

    @staticmethod
    def restore(saved):
        flat, idx, old = saved
        flat[idx] = old

    def scale_state(self):
        return unpack_scale_state(self.d_state.cpu().numpy())
