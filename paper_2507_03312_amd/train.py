"""The mixed-precision training step on the GPU, composed from libmpx calls.

The order of calls follows MPX §3.4 (the transformed gradient function) and
§3.5 (the masked optimizer update):

  cast masters and inputs to half -> half forward + full-precision loss ->
  backward seeded with the loss scale -> scaled half gradients ->
  unscale + all-finite check -> masked AdamW (+ half copy of the new
  masters) -> loss-scale update.

Every arithmetic step runs in libmpx's HIP kernels.  PyTorch is used only to
allocate device memory and to name the current stream; this module only
marshals pointers and sizes.  No call synchronises the host.

Memory layout: all parameters live in one float32 arena (masters), with
AdamW's m and v in arenas of the same layout, and the half working copy and
the half gradients in two half arenas of the same element offsets.  Every
tensor starts at a multiple of 128 elements (256-byte aligned in the half
arenas).  The multi-tensor sweeps see each arena as a single tensor; the
padding between tensors stays zero (AdamW maps zero to zero).
"""
from __future__ import annotations

import math
import struct
from typing import Dict, List, Optional

import numpy as np
import torch

import workloads

from . import binding as mx

TORCH_HALF = {"f16": torch.float16, "bf16": torch.bfloat16}
ALIGN = 128


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _off(t: torch.Tensor, elems: int) -> int:
    """Device address of element ``elems`` of tensor ``t``."""
    return t.data_ptr() + elems * t.element_size()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def pack_scale_state(scale, counter, period, factor=2.0, min_scale=1.0, max_scale=2.0 ** 127):
    raw = struct.pack("<fiifff", scale, counter, period, factor, min_scale, max_scale)
    return np.frombuffer(raw, dtype=np.int32).copy()


def unpack_scale_state(words: np.ndarray):
    scale, counter, period, factor, mn, mxs = struct.unpack("<fiifff", np.asarray(words, np.int32).tobytes())
    return {"scale": scale, "counter": counter, "period": period, "factor": factor,
            "min_scale": mn, "max_scale": mxs}


class Arena:
    """Flat arenas for masters (f32), m, v (f32), half copy and half grads.
    With ``full=True`` (full-precision training) there is no half copy (the
    layers read the masters) and the gradients are float32."""

    def __init__(self, specs, half: str, device, full: bool = False):
        self.names = [n for n, _, _ in specs]
        self.shapes = {n: tuple(s) for n, s, _ in specs}
        self.offsets: Dict[str, int] = {}
        off = 0
        for n, s, _ in specs:
            self.offsets[n] = off
            off += -(-int(np.prod(s)) // ALIGN) * ALIGN
        self.total = off
        hdt = torch.float32 if full else TORCH_HALF[half]
        self.p32 = torch.zeros(off, dtype=torch.float32, device=device)
        self.m32 = torch.zeros_like(self.p32)
        self.v32 = torch.zeros_like(self.p32)
        self.h = self.p32 if full else torch.zeros(off, dtype=hdt, device=device)
        self.g = torch.zeros(off, dtype=hdt, device=device)
        self.L_p = mx.TensorList([self.p32])
        self.L_m = mx.TensorList([self.m32])
        self.L_v = mx.TensorList([self.v32])
        self.L_h = None if full else mx.TensorList([self.h])
        self.L_g = mx.TensorList([self.g])

    def view(self, arena: torch.Tensor, name: str) -> torch.Tensor:
        n = int(np.prod(self.shapes[name]))
        return arena.narrow(0, self.offsets[name], n).view(self.shapes[name])

    def w(self, name):        # half working copy
        return self.view(self.h, name)

    def gr(self, name):       # half gradient
        return self.view(self.g, name)

    def load_masters(self, masters: Dict[str, np.ndarray]):
        host = np.zeros(self.total, np.float32)
        for n in self.names:
            o = self.offsets[n]
            a = np.asarray(masters[n], np.float32).reshape(-1)
            host[o:o + a.size] = a
        self.p32.copy_(torch.from_numpy(host))
        self.m32.zero_()
        self.v32.zero_()

    def read(self, arena: torch.Tensor) -> List[np.ndarray]:
        """Host copies (float32) of every tensor of an arena, in spec order."""
        a = arena.detach().float().cpu().numpy()
        return [a[self.offsets[n]:self.offsets[n] + int(np.prod(self.shapes[n]))]
                .reshape(self.shapes[n]).copy() for n in self.names]


class TrainStep:
    """Device state and the call sequence common to both model families."""

    def __init__(self, cfg, device="cuda", full_precision: bool = False):
        self.cfg = cfg
        self.device = torch.device(device)
        # full precision: MPX's use_mixed_precision switched off (the
        # baseline of the paper's comparison): float32 layers, no loss
        # scaling, AdamW on every step
        self.full = full_precision
        self.half = cfg.half
        self.dt = mx.MPX_F32 if self.full else mx.DTYPES[cfg.half]
        self.hdt = torch.float32 if self.full else TORCH_HALF[cfg.half]
        self.arena = Arena(workloads.param_specs(cfg), cfg.half, self.device, self.full)
        scale0 = 1.0 if self.full else cfg.scale_init
        self.d_state = torch.from_numpy(
            pack_scale_state(scale0, 0, cfg.period, cfg.factor, cfg.min_scale,
                             cfg.max_scale)).to(self.device)
        self.d_nonfinite = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.d_step = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.d_loss = torch.zeros(1, dtype=torch.float32, device=self.device)
        self.hp = mx.AdamWHP(cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay)
        self.half_copy_fresh = self.full  # full precision reads the masters directly
        # MPX §3.4's finite check fused into the kernels that write the
        # parameter gradients (they add their non-finite count to d_nonfinite,
        # zeroed at the start of the step); False: a separate unscale/check
        # pass over the whole gradient list after the backward
        self.fused_check = not self.full
        self.arena.load_masters(workloads.init_params(cfg))

    # ---- state access (harness only; each of these synchronises) ----
    def scale_state(self):
        return unpack_scale_state(self.d_state.cpu().numpy())

    def nonfinite(self) -> int:
        return int(self.d_nonfinite.item())

    def loss(self) -> float:
        return float(self.d_loss.item())

    def grads(self) -> List[np.ndarray]:
        return self.arena.read(self.arena.g)

    def masters(self) -> List[np.ndarray]:
        return self.arena.read(self.arena.p32)

    # ---- the step ----
    def cast_params(self):
        """MPX §3.1: half working copy of every master (first step only; later
        steps get it from the AdamW kernel's fused half-copy write)."""
        mx.mpx_cast_to_half(self.arena.L_p, self.arena.L_h, self.dt, _stream())
        self.half_copy_fresh = True

    def forward_backward(self):
        if not self.half_copy_fresh:
            self.cast_params()
        self._forward_backward(_stream())

    def _nf(self):
        """Counter argument of the gradient-writing calls."""
        return _ptr(self.d_nonfinite) if self.fused_check and not self.full else None

    def finish(self):
        """Finite check (unless fused into the backward), masked AdamW (+ half
        copy), scale update."""
        s = _stream()
        a = self.arena
        if self.full:  # no scaling, no check: AdamW on the float32 gradients
            mx.mpx_adamw_masked(a.L_p, a.L_m, a.L_v, a.L_g, mx.MPX_F32, self.hp,
                                _ptr(self.d_step), _ptr(self.d_state), _ptr(self.d_nonfinite),
                                None, self.dt, s)
            return
        if not self.fused_check:
            mx.mpx_unscale_check(a.L_g, self.dt, _ptr(self.d_state), _ptr(self.d_nonfinite), None,
                                 s)
        mx.mpx_adamw_masked(a.L_p, a.L_m, a.L_v, a.L_g, self.dt, self.hp, _ptr(self.d_step),
                            _ptr(self.d_state), _ptr(self.d_nonfinite), a.L_h, self.dt, s)
        mx.mpx_scale_update(_ptr(self.d_state), _ptr(self.d_nonfinite), s)

    def step(self):
        self.forward_backward()
        self.finish()

    # ---- HIP graph of the whole step ----
    graph = None

    def capture(self):
        """Record one whole step (forward, backward, unscale/check, masked
        AdamW, scale update) into a HIP graph; ``replay`` then launches it with
        a single host call.  Every piece of state the step reads (scale, flag,
        step count, half copy) lives in device memory, so replays advance the
        training state exactly as eager steps do."""
        if not self.half_copy_fresh:
            self.cast_params()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self._forward_backward(_stream())
            self.finish()
        torch.cuda.synchronize()
        self.graph = g

    def replay(self):
        self.graph.replay()

    # ---- timing of the dominant kernel ----
    def time_dominant(self, launches: int = 20, reps: int = 5) -> float:
        """Mean duration (ms) of one launch of the dominant kernel, from HIP
        events around a graph of ``launches`` back-to-back launches of it with
        the step's own operands (so no host launch gap is measured)."""
        return self.time_call(self._dominant_call, launches, reps)

    def gemm_sites(self):
        """(site, M, N, K, call) for each distinct linear-layer GEMM call of the
        step, as the step issues it; each does 2 M N K flops."""
        return []

    def time_call(self, call, launches: int = 20, reps: int = 5, groups: int = 5) -> float:
        """Duration (ms) of one ``call(stream)``: HIP events around ``reps``
        replays of a graph of ``launches`` back-to-back calls give one mean per
        group; the median over ``groups`` such groups is returned (one group
        alone moved by up to a third from box to box)."""
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(launches):
                call(_stream())
        g.replay()
        torch.cuda.synchronize()
        means = []
        for _ in range(groups):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                g.replay()
            e1.record()
            torch.cuda.synchronize()
            means.append(e0.elapsed_time(e1) / (reps * launches))
        return sorted(means)[groups // 2]

    def inject(self, tensor: int, element: int, value: float):
        """Harness fault injection: overwrite one gradient element (after the
        backward pass, before the finite check).  With the fused check the
        element is written after the kernels that count, so the count is
        adjusted here as they would have: +1 when a finite element becomes
        inf / NaN, -1 the other way round."""
        name = self.arena.names[tensor]
        flat = self.arena.gr(name).reshape(-1)
        i = element % flat.numel()
        was = bool(torch.isfinite(flat[i]).item())
        flat[i] = value
        now = bool(torch.isfinite(flat[i]).item())
        if self.fused_check and was != now:
            self.d_nonfinite += 1 if was else -1


def _linear_gelu_bytes(M: int, N: int, K: int) -> int:
    """Algorithmic HBM bytes of one linear_fwd + GELU launch in half precision:
    read X [M,K], W [N,K], b [N]; write the output and the pre-activation [M,N]."""
    return 2 * (M * K + N * K + N + 2 * M * N)


class MLPStep(TrainStep):
    """2-layer MLP with GELU and an MSE loss (mixed or full precision)."""

    def __init__(self, cfg, device="cuda", full_precision: bool = False):
        super().__init__(cfg, device, full_precision)
        B, D, Dh = cfg.batch, cfg.d_in, cfg.d_hidden
        dev, h = self.device, self.hdt
        self.x32 = torch.zeros(B, D, dtype=torch.float32, device=dev)
        self.t32 = torch.zeros(B, D, dtype=torch.float32, device=dev)
        if self.full:  # the float32 inputs are used as they are
            self.x16, self.t16 = self.x32, self.t32
        else:
            self.x16 = torch.zeros(B, D, dtype=h, device=dev)
            self.t16 = torch.zeros(B, D, dtype=h, device=dev)
            self.L_in = mx.TensorList([self.x32, self.t32])
            self.L_in16 = mx.TensorList([self.x16, self.t16])
        self.h_pre = torch.zeros(B, Dh, dtype=h, device=dev)
        self.hid = torch.zeros(B, Dh, dtype=h, device=dev)
        self.y = torch.zeros(B, D, dtype=h, device=dev)
        self.dy = torch.zeros(B, D, dtype=h, device=dev)
        self.dh_pre = torch.zeros(B, Dh, dtype=h, device=dev)
        ws = max(mx.mpx_linear_bwd_workspace(B, D, Dh), mx.mpx_linear_bwd_workspace(B, Dh, D),
                 mx.mpx_loss_workspace(B * D))
        self.ws = torch.zeros(ws, dtype=torch.uint8, device=dev)

    def _dominant_call(self, s):
        c, a = self.cfg, self.arena
        mx.mpx_linear_fwd(_ptr(self.x16), _ptr(a.w("fc1.w")), _ptr(a.w("fc1.b")), None,
                          _ptr(self.hid), _ptr(self.h_pre), c.batch, c.d_hidden, c.d_in, self.dt,
                          mx.MPX_ACT_GELU_TANH, s)

    def dominant_site(self):
        c = self.cfg
        M, N, K = c.batch, c.d_hidden, c.d_in
        width = 2 if self.full else 1  # float32 operands: twice the bytes
        return {"name": "fc1.fwd", "flops": 2.0 * M * N * K,
                "bytes": width * _linear_gelu_bytes(M, N, K),
                "desc": f"linear_fwd+GELU M={M} N={N} K={K} ({'f32' if self.full else c.half})"}

    def describe(self):
        c = self.cfg
        prec = "f32 (full precision)" if self.full else c.half
        return f"MLP {c.d_in}->{c.d_hidden}->{c.d_in} GELU, MSE, batch {c.batch}, {prec}"

    def set_batch(self, batch):
        self.x32.copy_(torch.from_numpy(batch["x"]))
        self.t32.copy_(torch.from_numpy(batch["target"]))

    def _forward_backward(self, s):
        c, a, dt = self.cfg, self.arena, self.dt
        B, D, Dh = c.batch, c.d_in, c.d_hidden
        nf = self._nf()
        if nf:
            mx.mpx_zero(nf, 4, s)
        if not self.full:
            mx.mpx_cast_to_half(self.L_in, self.L_in16, dt, s)
        self._dominant_call(s)
        mx.mpx_linear_fwd(_ptr(self.hid), _ptr(a.w("fc2.w")), _ptr(a.w("fc2.b")), None,
                          _ptr(self.y), None, B, D, Dh, dt, mx.MPX_ACT_NONE, s)
        mx.mpx_mse(_ptr(self.y), _ptr(self.t16), B * D, _ptr(self.d_state), _ptr(self.d_loss),
                   _ptr(self.dy), dt, _ptr(self.ws), self.ws.numel(), s)
        wsb = self.ws.numel()
        mx.mpx_linear_bwd(_ptr(self.hid), _ptr(a.w("fc2.w")), _ptr(self.dy), _ptr(self.h_pre),
                          mx.MPX_ACT_GELU_TANH, _ptr(self.dh_pre), _ptr(a.gr("fc2.w")),
                          _ptr(a.gr("fc2.b")), B, D, Dh, dt, _ptr(self.ws), wsb, nf, s)
        mx.mpx_linear_bwd(_ptr(self.x16), _ptr(a.w("fc1.w")), _ptr(self.dh_pre), None,
                          mx.MPX_ACT_NONE, None, _ptr(a.gr("fc1.w")), _ptr(a.gr("fc1.b")),
                          B, Dh, D, dt, _ptr(self.ws), wsb, nf, s)


class ViTStep(TrainStep):
    """Pre-LayerNorm ViT (token or image input), CLS pooling, CE loss (mixed
    or full precision; full precision takes the unfused attention and head)."""

    def __init__(self, cfg, device="cuda", full_precision: bool = False):
        super().__init__(cfg, device, full_precision)
        B, T, d, H, F, Cn = cfg.batch, cfg.tokens, cfg.d_model, cfg.heads, cfg.d_mlp, cfg.classes
        self.ldT = -(-T // 8) * 8
        M = B * T
        dev, h = self.device, self.hdt
        z = lambda *shape: torch.zeros(*shape, dtype=h, device=dev)
        if cfg.image:
            G, Pd = cfg.n_patches, cfg.patch_dim
            self.img = torch.zeros(B, cfg.image, cfg.image, cfg.channels, dtype=torch.float32,
                                   device=dev)
            self.patches = z(B * G, Pd)
            self.E = z(B * G, d)
            self.dE = z(B * G, d)
        else:
            self.tok32 = torch.zeros(M, d, dtype=torch.float32, device=dev)
            self.L_tok32 = mx.TensorList([self.tok32])
        if self.full and not cfg.image:  # the float32 tokens are the input as they are
            self.x0 = self.tok32
        else:
            self.x0 = z(M, d)
            self.L_x0 = mx.TensorList([self.x0])
        self.blocks = []
        for _ in range(cfg.depth):
            self.blocks.append({
                "a": z(M, d), "qkv": z(M, 3 * d), "P": z(B * H * T, self.ldT), "O": z(M, d),
                "x1": z(M, d), "c": z(M, d), "u_pre": z(M, F), "u": z(M, F), "x2": z(M, d)})
        if not self._fused_attention():   # score buffers of the unfused path
            self.S = z(B * H * T, self.ldT)
            self.dP = z(B * H * T, self.ldT)
            self.dS = z(B * H * T, self.ldT)
        self.zf = z(B, d)
        self.logits = z(B, Cn)
        self.dlogits = z(B, Cn)
        self.dz = z(B, d)
        # cotangents read by the weight-gradient stream are double (triple for
        # the residual stream) buffered, so the critical path of block k-1
        # never overwrites what the side stream still reads for block k
        self.dx = [z(M, d) for _ in range(3)]
        # the last block's cotangent from the final LayerNorm: only its CLS
        # rows are ever written, so it is zeroed once here, not every step
        self.dxf = z(M, d)
        self.du_pre = [z(M, F) for _ in range(2)]
        self.dx1 = [z(M, d) for _ in range(2)]
        self.dqkv = [z(M, 3 * d) for _ in range(2)]
        self.dcs = [z(M, d) for _ in range(2)]
        self.dO = z(M, d)
        self.das = [z(M, d) for _ in range(2)]
        self.labels = torch.zeros(B, dtype=torch.int32, device=dev)
        shapes = [(M, 3 * d, d), (M, d, d), (M, F, d), (M, d, F), (B, Cn, d)]
        if cfg.image:
            shapes.append((B * cfg.n_patches, d, cfg.patch_dim))
        # workspaces: the main stream's (LayerNorm, loss, attention) and the
        # weight-gradient stream's (split-K partials, bias column sums)
        ws = max(mx.mpx_layernorm_bwd_workspace(M, d), mx.mpx_loss_workspace(B),
                 mx.mpx_attention_bwd_workspace(B, T, H, cfg.head_dim),
                 mx.mpx_classifier_head_workspace(B, d),
                 # the last QKV bias (tokens) or the patch embedding's gradients (images)
                 mx.mpx_linear_bwd_workspace(B * cfg.n_patches, d, cfg.patch_dim) if cfg.image
                 else mx.mpx_linear_bwd_workspace(M, 3 * d, d))
        self.ws = torch.zeros(ws, dtype=torch.uint8, device=dev)
        ws2 = max(max(mx.mpx_linear_bwd_workspace(*s) for s in shapes),
                  mx.mpx_layernorm_bwd_workspace(M, d))
        self.ws2 = torch.zeros(ws2, dtype=torch.uint8, device=dev)
        self.side = torch.cuda.Stream(device=dev)  # default priority
        self.side_ln = None  # None: LayerNorm gamma / beta on the second stream
        self.split_last_ln = True
        self.last_bias_on_main = True
        self.patch_wgrad_on_main = True

    def _dominant_call(self, s):
        c, a, blk = self.cfg, self.arena, self.blocks[0]
        mx.mpx_linear_fwd(_ptr(blk["c"]), _ptr(a.w("blk0.up.w")), _ptr(a.w("blk0.up.b")), None,
                          _ptr(blk["u"]), _ptr(blk["u_pre"]), c.batch * c.tokens, c.d_mlp,
                          c.d_model, self.dt, mx.MPX_ACT_GELU_TANH, s)

    def gemm_sites(self):
        """Block 0's four linear layers (forward with the step's epilogue, dX,
        and dW + db with split-K) and the patch embedding, with the step's own
        operands and calls."""
        c, a, dt = self.cfg, self.arena, self.dt
        B, T, d, F = c.batch, c.tokens, c.d_model, c.d_mlp
        M = B * T
        W, G, blk = a.w, a.gr, self.blocks[0]
        GELU, NONE = mx.MPX_ACT_GELU_TANH, mx.MPX_ACT_NONE
        ws2p, ws2b = _ptr(self.ws2), self.ws2.numel()
        sites = []

        def layer(name, X, R, Y, pre, act, dY, Xpre, x_act, dX, Mr, N, K):
            w, b, gw, gb = W(name + ".w"), W(name + ".b"), G(name + ".w"), G(name + ".b")
            sites.append((name + ".fwd", Mr, N, K, lambda s: mx.mpx_linear_fwd(
                _ptr(X), _ptr(w), _ptr(b), _ptr(R), _ptr(Y), _ptr(pre), Mr, N, K, dt, act, s)))
            if dX is not None:
                sites.append((name + ".dX", Mr, N, K, lambda s: mx.mpx_linear_bwd(
                    None, _ptr(w), _ptr(dY), _ptr(Xpre), x_act, _ptr(dX), None, None, Mr, N, K, dt,
                    None, 0, None, s)))
            sites.append((name + ".dW", Mr, N, K, lambda s: mx.mpx_linear_bwd(
                _ptr(X), None, _ptr(dY), None, NONE, None, _ptr(gw), _ptr(gb), Mr, N, K, dt,
                ws2p, ws2b, None, s)))

        dx, du_pre, dx1, dqkv = self.dx[0], self.du_pre[0], self.dx1[0], self.dqkv[0]
        if c.image:
            layer("patch", self.patches, None, self.E, None, NONE, self.dE, None, NONE, None,
                  B * c.n_patches, d, c.patch_dim)
        p = "blk0."
        layer(p + "qkv", blk["a"], None, blk["qkv"], None, NONE, dqkv, None, NONE, self.das[0],
              M, 3 * d, d)
        layer(p + "proj", blk["O"], self.x0, blk["x1"], None, NONE, dx1, None, NONE, self.dO,
              M, d, d)
        layer(p + "up", blk["c"], None, blk["u"], blk["u_pre"], GELU, du_pre, None, NONE, self.dcs[0],
              M, F, d)
        layer(p + "down", blk["u"], blk["x1"], blk["x2"], None, NONE, dx, blk["u_pre"], GELU,
              du_pre, M, d, F)
        return sites

    def dominant_site(self):
        c = self.cfg
        M = c.batch * c.tokens
        width = 2 if self.full else 1  # float32 operands: twice the bytes
        prec = "f32" if self.full else c.half
        return {"name": "blk0.up.fwd", "flops": 2.0 * M * c.d_mlp * c.d_model,
                "bytes": width * _linear_gelu_bytes(M, c.d_mlp, c.d_model),
                "desc": f"linear_fwd+GELU (MLP up-projection) M={M} N={c.d_mlp} K={c.d_model} ({prec})"}

    def describe(self):
        c = self.cfg
        inp = (f"{c.image}x{c.image}x{c.channels} images, patch {c.patch}" if c.image
               else f"{c.tokens}x{c.d_model} token inputs")
        return (f"ViT pre-LN, {c.depth} block(s), d={c.d_model}, {c.heads} heads, MLP {c.d_mlp}, "
                f"{c.tokens} tokens, {inp}, {c.classes} classes, batch {c.batch}, {c.half}, "
                f"fp32 masters + masked AdamW, dynamic loss scaling")

    def set_batch(self, batch):
        c = self.cfg
        if c.image:
            self.img.copy_(torch.from_numpy(batch["x"]))
        else:
            self.tok32.copy_(torch.from_numpy(batch["x"].reshape(c.batch * c.tokens, c.d_model)))
        self.labels.copy_(torch.from_numpy(batch["labels"].astype(np.int32)))

    # attention core of one block: S = Q K^T, P = softmax, O = P V.  Sequences
    # up to 256 tokens with head dim 64 run the fused kernels; others the
    # batched GEMMs around the row softmax.
    def _fused_attention(self):
        c = self.cfg
        return not self.full and c.tokens <= 256 and c.head_dim == 64

    def _attn_fwd(self, blk, s):
        c, dt = self.cfg, self.dt
        B, T, d, H, hd, ldT = c.batch, c.tokens, c.d_model, c.heads, c.head_dim, self.ldT
        qkv, P, O = blk["qkv"], blk["P"], blk["O"]
        if self._fused_attention():
            mx.mpx_attention_fwd(_ptr(qkv), _ptr(O), _ptr(P), B, T, H, hd, dt, s)
            return
        mx.mpx_gemm_batched(0, 1, T, T, hd, B, H,
                            _ptr(qkv), 3 * d, T * 3 * d, hd,
                            _off(qkv, d), 3 * d, T * 3 * d, hd,
                            _ptr(self.S), ldT, H * T * ldT, T * ldT, dt, s)
        mx.mpx_softmax_fwd(_ptr(self.S), _ptr(P), B * H * T, T, ldT, 1.0 / math.sqrt(hd), dt, s)
        mx.mpx_gemm_batched(0, 0, T, hd, T, B, H,
                            _ptr(P), ldT, H * T * ldT, T * ldT,
                            _off(qkv, 2 * d), 3 * d, T * 3 * d, hd,
                            _ptr(O), d, T * d, hd, dt, s)

    def _attn_bwd(self, blk, dqkv, s):
        c, dt = self.cfg, self.dt
        B, T, d, H, hd, ldT = c.batch, c.tokens, c.d_model, c.heads, c.head_dim, self.ldT
        qkv, P, dO = blk["qkv"], blk["P"], self.dO
        if self._fused_attention():
            mx.mpx_attention_bwd(_ptr(qkv), _ptr(P), _ptr(dO), _ptr(dqkv), B, T, H, hd, dt,
                                 _ptr(self.ws), self.ws.numel(), s)
            return
        # dP = dO V^T
        mx.mpx_gemm_batched(0, 1, T, T, hd, B, H, _ptr(dO), d, T * d, hd,
                            _off(qkv, 2 * d), 3 * d, T * 3 * d, hd,
                            _ptr(self.dP), ldT, H * T * ldT, T * ldT, dt, s)
        # dV = P^T dO
        mx.mpx_gemm_batched(1, 0, T, hd, T, B, H, _ptr(P), ldT, H * T * ldT, T * ldT,
                            _ptr(dO), d, T * d, hd,
                            _off(dqkv, 2 * d), 3 * d, T * 3 * d, hd, dt, s)
        mx.mpx_softmax_bwd(_ptr(P), _ptr(self.dP), _ptr(self.dS), B * H * T, T, ldT,
                           1.0 / math.sqrt(hd), dt, s)
        # dQ = dS K
        mx.mpx_gemm_batched(0, 0, T, hd, T, B, H, _ptr(self.dS), ldT, H * T * ldT, T * ldT,
                            _off(qkv, d), 3 * d, T * 3 * d, hd,
                            _ptr(dqkv), 3 * d, T * 3 * d, hd, dt, s)
        # dK = dS^T Q
        mx.mpx_gemm_batched(1, 0, T, hd, T, B, H, _ptr(self.dS), ldT, H * T * ldT, T * ldT,
                            _ptr(qkv), 3 * d, T * 3 * d, hd,
                            _off(dqkv, d), 3 * d, T * 3 * d, hd, dt, s)

    def _forward_backward(self, s):
        c, a, dt = self.cfg, self.arena, self.dt
        B, T, d, F, Cn = c.batch, c.tokens, c.d_model, c.d_mlp, c.classes
        M = B * T
        W, G = a.w, a.gr
        wsp, wsb = _ptr(self.ws), self.ws.numel()
        GELU, NONE = mx.MPX_ACT_GELU_TANH, mx.MPX_ACT_NONE
        main = torch.cuda.current_stream()
        side, sh = self.side, self.side.cuda_stream
        nf = self._nf()
        if nf:
            # zeroed first on the step's stream: every gradient-writing call
            # below is ordered after it (zeroed on the second stream beside
            # the forward instead, the one-block step measured 1% slower than
            # with the separate check pass: the cross-stream wait cost more
            # than this launch)
            mx.mpx_zero(nf, 4, s)
        # ---- inputs (MPX §3.4: cast inputs to half) and embedding ----
        if c.image:
            mx.mpx_patchify_cast(_ptr(self.img), _ptr(self.patches), B, c.image, c.image,
                                 c.channels, c.patch, dt, s)
            mx.mpx_linear_fwd(_ptr(self.patches), _ptr(W("patch.w")), _ptr(W("patch.b")), None,
                              _ptr(self.E), None, B * c.n_patches, d, c.patch_dim, dt, NONE, s)
            mx.mpx_embed_assemble(_ptr(self.E), _ptr(W("cls")), _ptr(W("pos")), _ptr(self.x0),
                                  B, T, d, dt, s)
        # token inputs in mixed precision: their cast to half is fused with
        # the first block's LayerNorm (one pass instead of two)
        cast_in_ln = not c.image and not self.full
        # ---- blocks ----
        x = self.x0
        for i, blk in enumerate(self.blocks):
            p = f"blk{i}."
            if i == 0 and cast_in_ln:
                mx.mpx_layernorm_fwd_cast(_ptr(self.tok32), d, _ptr(W(p + "ln1.g")),
                                          _ptr(W(p + "ln1.b")), _ptr(self.x0), _ptr(blk["a"]), None,
                                          M, d, dt, s)
            else:
                mx.mpx_layernorm_fwd(_ptr(x), d, _ptr(W(p + "ln1.g")), _ptr(W(p + "ln1.b")),
                                     _ptr(blk["a"]), None, M, d, dt, s)
            mx.mpx_linear_fwd(_ptr(blk["a"]), _ptr(W(p + "qkv.w")), _ptr(W(p + "qkv.b")), None,
                              _ptr(blk["qkv"]), None, M, 3 * d, d, dt, NONE, s)
            self._attn_fwd(blk, s)
            mx.mpx_linear_fwd(_ptr(blk["O"]), _ptr(W(p + "proj.w")), _ptr(W(p + "proj.b")),
                              _ptr(x), _ptr(blk["x1"]), None, M, d, d, dt, NONE, s)
            mx.mpx_layernorm_fwd(_ptr(blk["x1"]), d, _ptr(W(p + "ln2.g")), _ptr(W(p + "ln2.b")),
                                 _ptr(blk["c"]), None, M, d, dt, s)
            mx.mpx_linear_fwd(_ptr(blk["c"]), _ptr(W(p + "up.w")), _ptr(W(p + "up.b")), None,
                              _ptr(blk["u"]), _ptr(blk["u_pre"]), M, F, d, dt, GELU, s)
            mx.mpx_linear_fwd(_ptr(blk["u"]), _ptr(W(p + "down.w")), _ptr(W(p + "down.b")),
                              _ptr(blk["x1"]), _ptr(blk["x2"]), None, M, d, F, dt, NONE, s)
            x = blk["x2"]
        # ---- head: LN on the CLS rows, linear, cross-entropy seeded with the scale ----
        # Up to 32 classes (C d <= 16384, 2048 rows) the head's forward and its backward
        # down to the final LayerNorm's input are one pass per row, the same
        # bits as the separate calls (three launches instead of seven on the
        # critical path); its weight gradients follow below.
        fused_head = not self.full and Cn <= 32 and Cn * d <= 16384 and B <= 2048
        if fused_head:
            mx.mpx_classifier_head(_ptr(x), T * d, _ptr(W("lnf.g")), _ptr(W("lnf.b")),
                                   _ptr(W("head.w")), _ptr(W("head.b")), _ptr(self.labels), B, d, Cn,
                                   _ptr(self.d_state), _ptr(self.zf), _ptr(self.d_loss),
                                   _ptr(self.dlogits), _ptr(self.dxf), T * d, _ptr(G("lnf.g")),
                                   _ptr(G("lnf.b")), dt, wsp, wsb, nf, s)
        else:
            mx.mpx_layernorm_fwd(_ptr(x), T * d, _ptr(W("lnf.g")), _ptr(W("lnf.b")), _ptr(self.zf),
                                 None, B, d, dt, s)
            mx.mpx_linear_fwd(_ptr(self.zf), _ptr(W("head.w")), _ptr(W("head.b")), None,
                              _ptr(self.logits), None, B, Cn, d, dt, NONE, s)
            mx.mpx_cross_entropy(_ptr(self.logits), Cn, _ptr(self.labels), B, Cn,
                                 _ptr(self.d_state), _ptr(self.d_loss), _ptr(self.dlogits), dt, wsp,
                                 wsb, s)
        # ---- backward ----
        # The critical path (dX of every layer, LayerNorm and attention
        # backward) runs on the step's stream; the weight and bias gradients
        # of each linear layer, which nothing later in the backward reads, run
        # on a second stream forked at the point their cotangent is ready.
        ws2p, ws2b = _ptr(self.ws2), self.ws2.numel()

        def wgrad(X, dY, dW, db, Mr, N, K):
            side.wait_stream(main)
            mx.mpx_linear_bwd(_ptr(X), None, _ptr(dY), None, NONE, None, _ptr(dW), _ptr(db),
                              Mr, N, K, dt, ws2p, ws2b, nf, sh)

        # the step's last weight gradient (the first block's QKV projection,
        # token inputs) ends the second stream's queue; its bias column sum
        # runs on the step's stream instead, which is idle by then
        last_bias_main = self.last_bias_on_main and not c.image

        # LayerNorm backward: dX alone on the step's stream and gamma / beta
        # (re-reading X and dY) on the second stream, which takes their final
        # column reduction off the critical path (ViT-S +1.3%, ViT-B +1.7%;
        # the one-block model +6.2% since the dX-only call got its wider grid)
        side_ln = True if self.side_ln is None else self.side_ln

        def ln_bwd(X, ldx, g, dY, R, dX, ldo, gg, gb, rows, fused=False):
            if dX is None:  # only gamma / beta are needed
                mx.mpx_layernorm_bwd(_ptr(X), ldx, _ptr(g), _ptr(dY), None, None, d, _ptr(gg),
                                     _ptr(gb), rows, d, dt, wsp, wsb, nf, s)
                return
            if fused or not side_ln:
                mx.mpx_layernorm_bwd(_ptr(X), ldx, _ptr(g), _ptr(dY), _ptr(R), _ptr(dX), ldo,
                                     _ptr(gg), _ptr(gb), rows, d, dt, wsp, wsb, nf, s)
                return
            mx.mpx_layernorm_bwd(_ptr(X), ldx, _ptr(g), _ptr(dY), _ptr(R), _ptr(dX), ldo, None, None,
                                 rows, d, dt, None, 0, None, s)
            side.wait_stream(main)
            mx.mpx_layernorm_bwd(_ptr(X), ldx, _ptr(g), _ptr(dY), None, None, d, _ptr(gg), _ptr(gb),
                                 rows, d, dt, ws2p, ws2b, nf, sh)

        def dgrad(W_, dY, Xpre, act, dX, Mr, N, K):
            mx.mpx_linear_bwd(None, _ptr(W_), _ptr(dY), None if Xpre is None else _ptr(Xpre), act,
                              _ptr(dX), None, None, Mr, N, K, dt, None, 0, None, s)

        wgrad(self.zf, self.dlogits, G("head.w"), G("head.b"), B, Cn, d)
        if not fused_head:
            dgrad(W("head.w"), self.dlogits, None, NONE, self.dz, B, Cn, d)
            ln_bwd(x, T * d, W("lnf.g"), self.dz, None, self.dxf, T * d, G("lnf.g"), G("lnf.b"), B)
        dx = self.dxf
        done = []  # side-stream completion of each block's weight gradients
        for k, i in enumerate(reversed(range(c.depth))):
            blk = self.blocks[i]
            p = f"blk{i}."
            xin = self.x0 if i == 0 else self.blocks[i - 1]["x2"]
            if k >= 2:  # block k-2's side work read the buffers block k is about to reuse
                main.wait_event(done[k - 2])
            dx_out = self.dx[(k + 1) % 3]
            du_pre, dx1, dqkv = self.du_pre[k % 2], self.dx1[k % 2], self.dqkv[k % 2]
            dc, da = self.dcs[k % 2], self.das[k % 2]
            wgrad(blk["u"], dx, G(p + "down.w"), G(p + "down.b"), M, d, F)
            dgrad(W(p + "down.w"), dx, blk["u_pre"], GELU, du_pre, M, d, F)
            wgrad(blk["c"], du_pre, G(p + "up.w"), G(p + "up.b"), M, F, d)
            dgrad(W(p + "up.w"), du_pre, None, NONE, dc, M, F, d)
            ln_bwd(blk["x1"], d, W(p + "ln2.g"), dc, dx, dx1, d, G(p + "ln2.g"), G(p + "ln2.b"), M)
            wgrad(blk["O"], dx1, G(p + "proj.w"), G(p + "proj.b"), M, d, d)
            dgrad(W(p + "proj.w"), dx1, None, NONE, self.dO, M, d, d)
            self._attn_bwd(blk, dqkv, s)
            bias_main = last_bias_main and i == 0
            wgrad(blk["a"], dqkv, G(p + "qkv.w"), None if bias_main else G(p + "qkv.b"), M, 3 * d, d)
            dgrad(W(p + "qkv.w"), dqkv, None, NONE, da, M, 3 * d, d)
            # the backward's last LayerNorm: with token inputs nothing reads the
            # input cotangent, so only gamma / beta are computed; with images
            # it is split like the others (gamma / beta beside the embedding
            # backward), unless split_last_ln is switched off
            last_dx = None if (i == 0 and not c.image) else dx_out
            ln_bwd(xin, d, W(p + "ln1.g"), da, dx1, last_dx, d, G(p + "ln1.g"), G(p + "ln1.b"), M,
                   fused=(i == 0 and not self.split_last_ln))
            if bias_main:
                mx.mpx_linear_bwd(None, None, _ptr(dqkv), None, NONE, None, None, _ptr(G(p + "qkv.b")),
                                  M, 3 * d, d, dt, wsp, wsb, nf, s)
            ev = torch.cuda.Event()
            ev.record(side)
            done.append(ev)
            dx = dx_out
        if c.image:
            mx.mpx_embed_assemble_bwd(_ptr(dx), _ptr(self.dE), _ptr(G("cls")), _ptr(G("pos")),
                                      B, T, d, dt, nf, s)
            if self.patch_wgrad_on_main:
                # the step's last weight gradient: on the step's stream, idle
                # once the embedding backward is done, beside the second
                # stream's last LayerNorm gamma / beta instead of after it
                mx.mpx_linear_bwd(_ptr(self.patches), None, _ptr(self.dE), None, NONE, None,
                                  _ptr(G("patch.w")), _ptr(G("patch.b")), B * c.n_patches, d,
                                  c.patch_dim, dt, wsp, wsb, nf, s)
            else:
                wgrad(self.patches, self.dE, G("patch.w"), G("patch.b"), B * c.n_patches, d,
                      c.patch_dim)
        main.wait_stream(side)  # join: the optimizer reads every gradient


def make_step(cfg, device="cuda", full_precision: bool = False) -> TrainStep:
    cls = MLPStep if cfg.kind == "mlp" else ViTStep
    return cls(cfg, device, full_precision)
