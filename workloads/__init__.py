"""Seeded synthetic workloads for the mixed-precision training step.

This module is shared by the CPU oracle and the HIP path.  It holds only
shapes, hyperparameters and random draws: no rounding, no casts, no GEMMs and
none of the method's arithmetic.  Every array it returns is float32 (or int32
for labels and int64 for sizes); each side casts to half precision with its
own code.

The paper's workloads are vision transformers trained on CIFAR-100 and
ImageNet-1k (MPX §5, Evaluation).  Neither dataset is available, so seeded
synthetic tensors with the same shapes stand in for them (32x32x3 images with
100 classes, 224x224x3 images with 1000 classes).

Seeds: ``numpy.random.default_rng(0)`` draws parameters, ``default_rng(1)``
draws inputs and labels, ``default_rng(2)`` draws anything else.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED_PARAMS = 0
SEED_DATA = 1
SEED_OTHER = 2


@dataclass(frozen=True)
class Injection:
    """A non-finite value written into one gradient before the finite check.

    ``tensor`` indexes the gradient list in parameter order, ``element`` the
    flat element (negative counts from the end), ``value`` is +inf, -inf or nan.
    """
    step: int
    tensor: int
    element: int
    value: float


@dataclass(frozen=True)
class TrainConfig:
    """One synthetic training workload: an MLP or a pre-LN ViT."""
    name: str
    kind: str                     # "mlp" or "vit"
    half: str                     # "f16" or "bf16"
    batch: int
    steps: int
    scale_init: float
    period: int                   # consecutive finite steps before growth
    # MLP
    d_in: int = 0
    d_hidden: int = 0
    # ViT
    depth: int = 0
    d_model: int = 0
    heads: int = 0
    d_mlp: int = 0
    classes: int = 0
    tokens: int = 0               # sequence length including CLS
    image: int = 0                # image side (0: inputs are tokens)
    patch: int = 0
    channels: int = 3
    injections: Tuple[Injection, ...] = ()
    # AdamW (decoupled weight decay), constant learning rate
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 1e-4
    min_scale: float = 1.0
    max_scale: float = 2.0 ** 127
    factor: float = 2.0

    @property
    def head_dim(self) -> int:
        return self.d_model // self.heads if self.heads else 0

    @property
    def n_patches(self) -> int:
        return (self.image // self.patch) ** 2 if self.image else 0

    @property
    def patch_dim(self) -> int:
        return self.patch * self.patch * self.channels if self.image else 0


@dataclass(frozen=True)
class SweepConfig:
    """The standalone optimizer sweep over a list of half gradient tensors."""
    name: str
    half: str
    n_tensors: int
    total: int
    sigma: float                  # gradient std before scaling
    steps: int
    scale_init: float
    period: int
    injections: Tuple[Injection, ...] = ()
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 1e-4
    min_scale: float = 1.0
    max_scale: float = 2.0 ** 127
    factor: float = 2.0


def _sweep_injections(n_tensors: int, steps: int) -> Tuple[Injection, ...]:
    out = []
    for s in range(steps):
        if s % 100 == 37:
            t = (7919 * s) % n_tensors
            if s % 200 == 37:
                out.append(Injection(s, t, -1, float("inf")))
            else:
                out.append(Injection(s, t, 0, float("nan")))
    return tuple(out)


CONFIGS: Dict[str, object] = {
    # 2-layer MLP 512->1024->512 with GELU, MSE, fp16, +inf into dW1 at step 3
    "mlp": TrainConfig(
        name="mlp", kind="mlp", half="f16", batch=64, steps=10,
        scale_init=2.0 ** 15, period=4, d_in=512, d_hidden=1024,
        injections=(Injection(3, 0, 0, float("inf")),)),
    # one pre-LN ViT encoder block on 128x65x384 tokens, bf16, 10 classes
    "vit_block": TrainConfig(
        name="vit_block", kind="vit", half="bf16", batch=128, steps=10,
        scale_init=2.0 ** 15, period=2000, depth=1, d_model=384, heads=6,
        d_mlp=1536, classes=10, tokens=65),
    # ViT-Small-like, 32x32x3 images, patch 4, fp16, 100 classes
    "vit_s": TrainConfig(
        name="vit_s", kind="vit", half="f16", batch=256, steps=10,
        scale_init=2.0 ** 16, period=2000, depth=12, d_model=384, heads=6,
        d_mlp=1536, classes=100, tokens=65, image=32, patch=4),
    # ViT-Base-like, 224x224x3 images, patch 16, bf16, 1000 classes
    "vit_b": TrainConfig(
        name="vit_b", kind="vit", half="bf16", batch=64, steps=10,
        scale_init=2.0 ** 15, period=2000, depth=12, d_model=768, heads=12,
        d_mlp=3072, classes=1000, tokens=197, image=224, patch=16),
    # standalone sweep: 200 fp16 tensors, 1e8 elements, 1% of steps injected
    "sweep": SweepConfig(
        name="sweep", half="f16", n_tensors=200, total=100_000_000,
        sigma=1e-3, steps=200, scale_init=2.0 ** 16, period=2000,
        injections=_sweep_injections(200, 200)),
}

# Ordered as the five workloads of the build: tiny MLP, one ViT block,
# ViT-S, ViT-B, optimizer sweep.
CONFIG_ORDER = ["mlp", "vit_block", "vit_s", "vit_b", "sweep"]


def get(name: str):
    return CONFIGS[name]


def scaled_down(cfg: TrainConfig, **kw) -> TrainConfig:
    """A copy of ``cfg`` with some fields replaced (for small parity cases)."""
    d = dict(cfg.__dict__)
    d.update(kw)
    return TrainConfig(**d)


# --------------------------------------------------------------------------
# Parameters
# --------------------------------------------------------------------------

def param_specs(cfg: TrainConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Parameter names, shapes and init kinds, in the fixed arena order.

    Weights are stored [out, in] so a linear layer computes X @ W^T.
    Init kinds: "normal" (N(0, 0.02)), "zeros", "ones".
    """
    specs: List[Tuple[str, Tuple[int, ...], str]] = []
    if cfg.kind == "mlp":
        specs += [("fc1.w", (cfg.d_hidden, cfg.d_in), "normal"),
                  ("fc1.b", (cfg.d_hidden,), "zeros"),
                  ("fc2.w", (cfg.d_in, cfg.d_hidden), "normal"),
                  ("fc2.b", (cfg.d_in,), "zeros")]
        return specs
    d, f = cfg.d_model, cfg.d_mlp
    if cfg.image:
        specs += [("patch.w", (d, cfg.patch_dim), "normal"),
                  ("patch.b", (d,), "zeros"),
                  ("cls", (d,), "zeros"),
                  ("pos", (cfg.tokens, d), "normal")]
    for i in range(cfg.depth):
        p = f"blk{i}."
        specs += [(p + "ln1.g", (d,), "ones"), (p + "ln1.b", (d,), "zeros"),
                  (p + "qkv.w", (3 * d, d), "normal"), (p + "qkv.b", (3 * d,), "zeros"),
                  (p + "proj.w", (d, d), "normal"), (p + "proj.b", (d,), "zeros"),
                  (p + "ln2.g", (d,), "ones"), (p + "ln2.b", (d,), "zeros"),
                  (p + "up.w", (f, d), "normal"), (p + "up.b", (f,), "zeros"),
                  (p + "down.w", (d, f), "normal"), (p + "down.b", (d,), "zeros")]
    specs += [("lnf.g", (d,), "ones"), ("lnf.b", (d,), "zeros"),
              ("head.w", (cfg.classes, d), "normal"), ("head.b", (cfg.classes,), "zeros")]
    return specs


def param_count(cfg: TrainConfig) -> int:
    return int(sum(int(np.prod(s)) for _, s, _ in param_specs(cfg)))


def init_params(cfg: TrainConfig) -> Dict[str, np.ndarray]:
    """fp32 master parameters, drawn in spec order from one generator."""
    rng = np.random.default_rng(SEED_PARAMS)
    out: Dict[str, np.ndarray] = {}
    for name, shape, kind in param_specs(cfg):
        if kind == "normal":
            out[name] = rng.normal(0.0, 0.02, size=shape).astype(np.float32)
        elif kind == "zeros":
            out[name] = np.zeros(shape, np.float32)
        else:
            out[name] = np.ones(shape, np.float32)
    return out


# --------------------------------------------------------------------------
# Batches
# --------------------------------------------------------------------------

def make_batch(cfg: TrainConfig) -> Dict[str, np.ndarray]:
    """One fixed synthetic batch (the same batch is used at every step).

    mlp:        x ~ N(0,1) [B, d_in], target ~ N(0,1) [B, d_in]
    vit tokens: x ~ N(0,1) [B, T, d], labels ~ U{0..classes-1}
    vit images: x ~ U(0,1) [B, H, W, C] (NHWC), labels ~ U{0..classes-1}
    """
    rng = np.random.default_rng(SEED_DATA)
    if cfg.kind == "mlp":
        x = rng.normal(0.0, 1.0, size=(cfg.batch, cfg.d_in)).astype(np.float32)
        t = rng.normal(0.0, 1.0, size=(cfg.batch, cfg.d_in)).astype(np.float32)
        return {"x": x, "target": t}
    if cfg.image:
        x = rng.uniform(0.0, 1.0, size=(cfg.batch, cfg.image, cfg.image,
                                        cfg.channels)).astype(np.float32)
    else:
        x = rng.normal(0.0, 1.0, size=(cfg.batch, cfg.tokens, cfg.d_model)).astype(np.float32)
    y = rng.integers(0, cfg.classes, size=(cfg.batch,)).astype(np.int32)
    return {"x": x, "labels": y}


# --------------------------------------------------------------------------
# Optimizer sweep
# --------------------------------------------------------------------------

def sweep_sizes(cfg: SweepConfig) -> np.ndarray:
    """Lognormal tensor sizes summing exactly to ``cfg.total`` (each >= 1)."""
    rng = np.random.default_rng(SEED_PARAMS)
    e = np.exp(rng.normal(0.0, 1.5, size=cfg.n_tensors))
    sizes = np.floor(cfg.total * e / e.sum()).astype(np.int64)
    sizes = np.maximum(sizes, 1)
    sizes[int(np.argmax(sizes))] += cfg.total - int(sizes.sum())
    return sizes


def sweep_tensors(cfg: SweepConfig, sizes: Optional[np.ndarray] = None):
    """fp32 draws for the sweep: (grad_values, params), each a list of arrays.

    grad_values are N(0, sigma) times the initial loss scale (a power of two);
    each side rounds them to half precision itself.  Moments start at zero.
    """
    if sizes is None:
        sizes = sweep_sizes(cfg)
    rng_p = np.random.default_rng(SEED_PARAMS + 100)
    rng_g = np.random.default_rng(SEED_DATA)
    params = [rng_p.normal(0.0, 0.02, size=int(n)).astype(np.float32) for n in sizes]
    grads = [(rng_g.normal(0.0, cfg.sigma, size=int(n)) * cfg.scale_init).astype(np.float32)
             for n in sizes]
    return grads, params


def small_sweep(n_tensors: int = 13, total: int = 50_000, steps: int = 12,
                period: int = 3, half: str = "f16") -> SweepConfig:
    """A sweep small enough for the oracle to run in well under a second."""
    inj = (Injection(4, 5, -1, float("inf")), Injection(9, 2, 0, float("nan")))
    return SweepConfig(name="sweep_small", half=half, n_tensors=n_tensors,
                       total=total, sigma=1e-3, steps=steps,
                       scale_init=2.0 ** 16, period=period, injections=inj)
