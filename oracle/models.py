"""The two model families of the workloads, forward and backward (oracle).

MLP: Y = fc2(GELU(fc1(X))), loss = MSE(Y, target).

ViT (pre-LayerNorm encoder, MPX §5 trains vision transformers):
    tokens: either the input itself [B, T, d], or
            x[b, 0] = R(cls + pos[0]),  x[b, 1 + g] = R(R(patch_g W_p^T + b_p) + pos[1 + g])
    block:  a = LN1(x); qkv = a W_qkv^T + b; o = attention(qkv) W_proj^T + b;
            x1 = R(x + o); c = LN2(x1); u = GELU(c W_up^T + b); dn = u W_down^T + b;
            x2 = R(x1 + dn)
    head:   z = LN_f(x[:, 0]) (the CLS token), logits = z W_h^T + b_h,
            loss = mean cross-entropy.

``params`` maps names (``workloads.param_specs``) to half-valued arrays (the
cast working copies).  The backward takes the scaled half cotangent of the
loss output and returns scaled half gradients for every parameter.
"""
from __future__ import annotations

import numpy as np

from . import ops


# --------------------------------------------------------------------- MLP --

def mlp_forward(pol, P, x):
    h_pre = ops.linear_fwd(pol, x, P["fc1.w"], P["fc1.b"])
    h = ops.gelu_fwd(pol, h_pre)
    y = ops.linear_fwd(pol, h, P["fc2.w"], P["fc2.b"])
    return y, (x, h_pre, h)


def mlp_backward(pol, P, cache, dy):
    x, h_pre, h = cache
    G = {}
    dh, G["fc2.w"], G["fc2.b"] = ops.linear_bwd(pol, h, P["fc2.w"], dy)
    dh_pre = ops.gelu_bwd(pol, h_pre, dh)
    _, G["fc1.w"], G["fc1.b"] = ops.linear_bwd(pol, x, P["fc1.w"], dh_pre, need_dx=False)
    return G


# --------------------------------------------------------------------- ViT --

def embed_forward(pol, cfg, P, x_in):
    """Token matrix [B*T, d] from images (patch embedding) or given tokens."""
    B, T, d = cfg.batch, cfg.tokens, cfg.d_model
    if not cfg.image:
        return np.asarray(x_in).reshape(B * T, d), None
    patches = ops.patchify(x_in, cfg.patch)
    pe = ops.linear_fwd(pol, patches, P["patch.w"], P["patch.b"])      # [B*G, d]
    pos = np.asarray(P["pos"])
    x = np.empty((B, T, d), dtype=pe.dtype)
    x[:, 0, :] = ops.add(pol, P["cls"], pos[0])[None, :]
    x[:, 1:, :] = ops.add(pol, pe.reshape(B, T - 1, d), pos[None, 1:, :])
    return x.reshape(B * T, d), patches


def block_forward(pol, cfg, P, i, x):
    p = f"blk{i}."
    B, T, H, hd = cfg.batch, cfg.tokens, cfg.heads, cfg.head_dim
    a = ops.layernorm_fwd(pol, x, P[p + "ln1.g"], P[p + "ln1.b"])
    qkv = ops.linear_fwd(pol, a, P[p + "qkv.w"], P[p + "qkv.b"])
    o, acache = ops.attention_fwd(pol, qkv, B, T, H, hd)
    proj = ops.linear_fwd(pol, o, P[p + "proj.w"], P[p + "proj.b"])
    x1 = ops.add(pol, x, proj)
    c = ops.layernorm_fwd(pol, x1, P[p + "ln2.g"], P[p + "ln2.b"])
    u_pre = ops.linear_fwd(pol, c, P[p + "up.w"], P[p + "up.b"])
    u = ops.gelu_fwd(pol, u_pre)
    dn = ops.linear_fwd(pol, u, P[p + "down.w"], P[p + "down.b"])
    x2 = ops.add(pol, x1, dn)
    return x2, (x, a, qkv, acache, o, x1, c, u_pre, u)


def block_backward(pol, cfg, P, i, cache, dx2):
    p = f"blk{i}."
    B, T, H, hd = cfg.batch, cfg.tokens, cfg.heads, cfg.head_dim
    x, a, qkv, acache, o, x1, c, u_pre, u = cache
    G = {}
    du, G[p + "down.w"], G[p + "down.b"] = ops.linear_bwd(pol, u, P[p + "down.w"], dx2)
    du_pre = ops.gelu_bwd(pol, u_pre, du)
    dc, G[p + "up.w"], G[p + "up.b"] = ops.linear_bwd(pol, c, P[p + "up.w"], du_pre)
    dx1_ln, G[p + "ln2.g"], G[p + "ln2.b"] = ops.layernorm_bwd(pol, x1, P[p + "ln2.g"], dc)
    dx1 = ops.add(pol, dx2, dx1_ln)
    do, G[p + "proj.w"], G[p + "proj.b"] = ops.linear_bwd(pol, o, P[p + "proj.w"], dx1)
    dqkv = ops.attention_bwd(pol, acache, do, B, T, H, hd)
    da, G[p + "qkv.w"], G[p + "qkv.b"] = ops.linear_bwd(pol, a, P[p + "qkv.w"], dqkv)
    dx_ln, G[p + "ln1.g"], G[p + "ln1.b"] = ops.layernorm_bwd(pol, x, P[p + "ln1.g"], da)
    dx = ops.add(pol, dx1, dx_ln)
    return dx, G


def vit_forward(pol, cfg, P, x_in):
    B, T, d = cfg.batch, cfg.tokens, cfg.d_model
    x, patches = embed_forward(pol, cfg, P, x_in)
    caches = []
    for i in range(cfg.depth):
        x, bc = block_forward(pol, cfg, P, i, x)
        caches.append(bc)
    xc = x.reshape(B, T, d)[:, 0, :]
    z = ops.layernorm_fwd(pol, xc, P["lnf.g"], P["lnf.b"])
    logits = ops.linear_fwd(pol, z, P["head.w"], P["head.b"])
    return logits, (patches, caches, xc, z)


def vit_backward(pol, cfg, P, cache, dlogits):
    B, T, d = cfg.batch, cfg.tokens, cfg.d_model
    patches, caches, xc, z = cache
    G = {}
    dz, G["head.w"], G["head.b"] = ops.linear_bwd(pol, z, P["head.w"], dlogits)
    dxc, G["lnf.g"], G["lnf.b"] = ops.layernorm_bwd(pol, xc, P["lnf.g"], dz)
    dx = np.zeros((B, T, d), dtype=dxc.dtype)
    dx[:, 0, :] = dxc
    dx = dx.reshape(B * T, d)
    for i in reversed(range(cfg.depth)):
        dx, Gi = block_backward(pol, cfg, P, i, caches[i], dx)
        G.update(Gi)
    if cfg.image:
        dx3 = dx.reshape(B, T, d)
        G["cls"] = pol.colsum(dx3[:, 0, :])
        G["pos"] = pol.R(np.sum(np.asarray(dx3, dtype=np.float64), axis=0))
        dpe = dx3[:, 1:, :].reshape(B * (T - 1), d)
        _, G["patch.w"], G["patch.b"] = ops.linear_bwd(pol, patches, P["patch.w"], dpe,
                                                       need_dx=False)
    return G


# ----------------------------------------------------------------- dispatch --

def forward_loss(pol, cfg, P, batch, scale):
    """Forward pass and loss; returns (loss, scaled half cotangent, cache)."""
    if cfg.kind == "mlp":
        y, cache = mlp_forward(pol, P, batch["x"])
        loss, dy = ops.mse_fwd_bwd(pol, y, batch["target"], scale)
        return loss, dy, cache
    logits, cache = vit_forward(pol, cfg, P, batch["x"])
    loss, dl = ops.ce_fwd_bwd(pol, logits, batch["labels"], scale)
    return loss, dl, cache


def backward(pol, cfg, P, cache, dout):
    if cfg.kind == "mlp":
        return mlp_backward(pol, P, cache, dout)
    return vit_backward(pol, cfg, P, cache, dout)
