"""Layer forward and backward passes under a precision policy (oracle).

Each forward takes half-valued inputs and returns half-valued outputs plus
what its backward needs; each backward takes the half cotangent of the
output and returns half cotangents, at the same precision as the forward
(MPX §3: every op runs in the precision of its inputs; §2.1: the gradients of
the scaled loss are computed in half precision).  ``pol`` is a
``policy.Policy``.

Layouts: activations are row-major [rows, features]; a weight is [out, in], so
a linear layer computes X @ W^T; tokens are [batch * seq, d] with the
sequence index fastest over rows; the fused QKV projection's output columns
are (q heads, k heads, v heads), head h of each taking columns h*hd..h*hd+hd-1.
"""
from __future__ import annotations

import math

import numpy as np

GELU_C = math.sqrt(2.0 / math.pi)
GELU_A = 0.044715
LN_EPS = 1e-5


def f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


# ----------------------------------------------------------------- linear --

def linear_fwd(pol, x, w, b):
    """Y = R(X W^T + b): one GEMM, bias added before the single rounding."""
    return pol.gemm(x, np.asarray(w).T, b)


def linear_bwd(pol, x, w, dy, need_dx=True):
    """Gradients of Y = X W^T + b for a half cotangent dY.

    dX = R(dY W), dW = R(dY^T X), db = R(sum_rows dY).
    """
    dx = pol.gemm(dy, w) if need_dx else None
    dw = pol.gemm(np.asarray(dy).T, x)
    db = pol.colsum(dy)
    return dx, dw, db


# ------------------------------------------------------------------- GELU --

def _elementwise(fn, *arrays, chunk=1 << 16):
    """fn applied to flat slices of same-shape arrays (keeps temporaries small)."""
    flat = [np.asarray(a).reshape(-1) for a in arrays]
    out = np.empty(flat[0].shape, np.float64)
    for i in range(0, out.size, chunk):
        out[i:i + chunk] = fn(*[f[i:i + chunk] for f in flat])
    return out.reshape(np.shape(arrays[0]))


def _sigmoid_2u(z):
    """1 / (1 + exp(-2u)) with u = c (z + a z^3), i.e. (1 + tanh(u)) / 2."""
    u = GELU_C * (z + GELU_A * z ** 3)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-2.0 * u))


def _gelu64(x):
    """0.5 x (1 + tanh(u)), evaluated as x / (1 + exp(-2u)) (the same function;
    this form has no cancellation for negative x)."""
    z = f64(x)
    return z * _sigmoid_2u(z)


def gelu_grad(x):
    """d/dx of the tanh-form GELU, in float64:
    sigma + 2 x sigma (1 - sigma) c (1 + 3 a x^2), with sigma = (1 + tanh(u)) / 2."""
    z = f64(x)
    sg = _sigmoid_2u(z)
    return sg + 2.0 * z * sg * (1.0 - sg) * GELU_C * (1.0 + 3.0 * GELU_A * z * z)


def gelu_fwd(pol, x):
    """GELU, tanh form: 0.5 x (1 + tanh(c (x + a x^3))), full precision inside."""
    return pol.R(_elementwise(_gelu64, x))


def gelu_bwd(pol, x_pre, dy):
    """dX_pre = R(dY * gelu'(X_pre))."""
    return pol.R(_elementwise(lambda a, b: f64(b) * gelu_grad(a), x_pre, dy))


# ---------------------------------------------------------------- residual --

def add(pol, a, b):
    """R(a + b)."""
    return pol.R(f64(a) + f64(b))


# -------------------------------------------------------------- LayerNorm --

def layernorm_fwd(pol, x, g, b):
    """Row LayerNorm in full precision: two-pass mean and variance, eps 1e-5."""
    z = f64(x)
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + LN_EPS)
    xhat = (z - mu) * rstd
    return pol.R(xhat * f64(g) + f64(b))


def layernorm_bwd(pol, x, g, dy):
    """Cotangents of LayerNorm: (dX, dgamma, dbeta), each rounded once."""
    z = f64(x)
    d = z.shape[-1]
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + LN_EPS)
    xhat = (z - mu) * rstd
    dyv = f64(dy)
    dxhat = dyv * f64(g)
    dx = rstd * (dxhat - dxhat.sum(axis=-1, keepdims=True) / d
                 - xhat * (dxhat * xhat).sum(axis=-1, keepdims=True) / d)
    rows = dyv.reshape(-1, d)
    dg = (rows * xhat.reshape(-1, d)).sum(axis=0)
    db = rows.sum(axis=0)
    return pol.R(dx), pol.R(dg), pol.R(db)


# -------------------------------------------------------------- attention --

def split_heads(qkv, batch, seq, heads, hd):
    """[B*T, 3*d] -> three arrays [B, H, T, hd] (views, no arithmetic)."""
    a = np.asarray(qkv).reshape(batch, seq, 3, heads, hd)
    return (a[:, :, 0].transpose(0, 2, 1, 3), a[:, :, 1].transpose(0, 2, 1, 3),
            a[:, :, 2].transpose(0, 2, 1, 3))


def merge_heads(o):
    """[B, H, T, hd] -> [B*T, H*hd]."""
    b, h, t, hd = o.shape
    return np.ascontiguousarray(o.transpose(0, 2, 1, 3)).reshape(b * t, h * hd)


def softmax_fwd(pol, s, scale):
    """P = R(softmax(scale * S)) over the last axis, in full precision."""
    z = f64(s) * scale
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return pol.R(e / e.sum(axis=-1, keepdims=True))


def softmax_bwd(pol, p, dp, scale):
    """dS = R(scale * P * (dP - sum_j dP_j P_j)) for P = softmax(scale * S)."""
    pv = f64(p)
    dpv = f64(dp)
    return pol.R(scale * pv * (dpv - (dpv * pv).sum(axis=-1, keepdims=True)))


def attention_fwd(pol, qkv, batch, seq, heads, hd):
    """Multi-head self-attention core on a fused QKV activation.

    S = R(Q K^T), P = R(softmax(S / sqrt(hd))) in full precision, O = R(P V).
    Returns O as [B*T, d] and the cache for the backward pass.
    """
    q, k, v = split_heads(qkv, batch, seq, heads, hd)
    scale = 1.0 / math.sqrt(hd)
    s = pol.R(pol.mm(q, np.swapaxes(k, -1, -2)))
    p = softmax_fwd(pol, s, scale)
    o = pol.R(pol.mm(p, v))
    return merge_heads(o), (q, k, v, p, scale)


def attention_bwd(pol, cache, do_flat, batch, seq, heads, hd):
    """Cotangent of the fused QKV activation, [B*T, 3d].

    dP = R(dO V^T), dV = R(P^T dO), dS = softmax backward, dQ = R(dS K),
    dK = R(dS^T Q).
    """
    q, k, v, p, scale = cache
    do = np.asarray(do_flat).reshape(batch, seq, heads, hd).transpose(0, 2, 1, 3)
    dp = pol.R(pol.mm(do, np.swapaxes(v, -1, -2)))
    dv = pol.R(pol.mm(np.swapaxes(p, -1, -2), do))
    ds = softmax_bwd(pol, p, dp, scale)
    dq = pol.R(pol.mm(ds, k))
    dk = pol.R(pol.mm(np.swapaxes(ds, -1, -2), q))
    out = np.stack([dq, dk, dv], axis=0)               # [3, B, H, T, hd]
    out = out.transpose(1, 3, 0, 2, 4)                 # [B, T, 3, H, hd]
    return np.ascontiguousarray(out).reshape(batch * seq, 3 * heads * hd)


# ------------------------------------------------------------------ losses --

def mse_fwd_bwd(pol, y, target, scale):
    """Mean squared error in full precision and its scaled half cotangent.

    loss = mean((y - t)^2) over all elements; dY = R(scale * 2 (y - t) / n).
    """
    diff = f64(y) - f64(target)
    n = diff.size
    loss = float(np.mean(diff * diff))
    return loss, pol.R(float(scale) * 2.0 * diff / n)


def ce_fwd_bwd(pol, logits, labels, scale):
    """Mean softmax cross-entropy in full precision and its scaled cotangent.

    loss = mean_b(logsumexp(z_b) - z_b[y_b]);
    dZ = R(scale * (softmax(z) - onehot(y)) / B).
    """
    z = f64(logits)
    bsz = z.shape[0]
    zm = z - z.max(axis=1, keepdims=True)
    e = np.exp(zm)
    se = e.sum(axis=1, keepdims=True)
    lse = np.log(se)[:, 0]
    rows = np.arange(bsz)
    loss = float(np.mean(lse - zm[rows, labels]))
    g = e / se
    g[rows, labels] -= 1.0
    return loss, pol.R(float(scale) * g / bsz)


# ---------------------------------------------------------------- patches --

def patchify(images, patch):
    """[B, H, W, C] -> [B * n_patches, patch*patch*C] (a relabelling, no math).

    Patches are taken row-major over the patch grid; a patch vector lists its
    pixels row-major, channels fastest: index (i * patch + j) * C + c.
    """
    b, h, w, c = images.shape
    gh, gw = h // patch, w // patch
    a = np.asarray(images).reshape(b, gh, patch, gw, patch, c)
    a = a.transpose(0, 1, 3, 2, 4, 5)
    return np.ascontiguousarray(a).reshape(b * gh * gw, patch * patch * c)
