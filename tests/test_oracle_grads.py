"""Pins of the oracle's hand-written backward passes.

* Finite differences: in the float64 policy (no rounding) every parameter
  gradient of a tiny MLP and of tiny ViTs (with and without patch embedding)
  must match central differences of the loss.
* Mixed precision: the unscaled half-precision gradients must match the
  float64 gradients normwise within 2e-2 (float16) / 5e-2 (bfloat16).
* Scale equivariance: with power-of-two scales, every backward op is linear in
  the cotangent and rounding commutes with power-of-two scaling in the normal
  range, so unscaled gradients at two scales are bit-identical.
"""
import numpy as np
import pytest

import workloads
from oracle import models, ops, scaling
from oracle.numfmt import round_to
from oracle.policy import Policy
from oracle.step import cast_batch


def tiny_cfgs():
    mlp = workloads.TrainConfig(name="tiny_mlp", kind="mlp", half="f16", batch=2, steps=1,
                                scale_init=1.0, period=10, d_in=3, d_hidden=4)
    vit_tok = workloads.TrainConfig(name="tiny_vit_tok", kind="vit", half="bf16", batch=2,
                                    steps=1, scale_init=1.0, period=10, depth=2, d_model=8,
                                    heads=2, d_mlp=16, classes=3, tokens=3)
    vit_img = workloads.TrainConfig(name="tiny_vit_img", kind="vit", half="f16", batch=2,
                                    steps=1, scale_init=1.0, period=10, depth=1, d_model=8,
                                    heads=2, d_mlp=16, classes=3, tokens=5, image=4, patch=2)
    return [mlp, vit_tok, vit_img]


def _params(cfg, std=0.3):
    """Larger-than-default init so that tiny networks have O(1) signals."""
    rng = np.random.default_rng(42)
    P = {}
    for name, shape, kind in workloads.param_specs(cfg):
        if kind == "ones":
            P[name] = (1.0 + 0.1 * rng.normal(size=shape))
        else:
            P[name] = rng.normal(0, std, size=shape)
    return P


def _loss(cfg, P, batch):
    pol = Policy("f64")
    loss, _, _ = models.forward_loss(pol, cfg, P, batch, 1.0)
    return loss


@pytest.mark.parametrize("cfg", tiny_cfgs(), ids=lambda c: c.name)
def test_float64_gradients_match_finite_differences(cfg):
    pol = Policy("f64")
    P = _params(cfg)
    batch = {k: (v.astype(np.float64) if v.dtype.kind == "f" else v)
             for k, v in workloads.make_batch(cfg).items()}
    _, dout, cache = models.forward_loss(pol, cfg, P, batch, 1.0)
    G = models.backward(pol, cfg, P, cache, dout)
    assert set(G) == set(P)
    for name, w in P.items():
        g = G[name]
        assert g.shape == w.shape, name
        flat = w.reshape(-1)
        fd = np.empty(flat.size)
        for i in range(flat.size):
            h = 1e-6 * max(1.0, abs(flat[i]))
            old = flat[i]
            flat[i] = old + h
            lp = _loss(cfg, P, batch)
            flat[i] = old - h
            lm = _loss(cfg, P, batch)
            flat[i] = old
            fd[i] = (lp - lm) / (2 * h)
        err = np.max(np.abs(fd - g.reshape(-1)))
        assert err <= 1e-6 * max(1.0, np.max(np.abs(fd))), (name, err)


def _half_grads(cfg, fmt, scale, P64, batch):
    pol = Policy(fmt)
    P = {k: pol.R(v) for k, v in P64.items()}
    hb = cast_batch(pol, batch)
    _, dout, cache = models.forward_loss(pol, cfg, P, hb, scale)
    G = models.backward(pol, cfg, P, cache, dout)
    return {k: scaling.unscale(v, np.float32(scale)) for k, v in G.items()}


@pytest.mark.parametrize("cfg", tiny_cfgs(), ids=lambda c: c.name)
@pytest.mark.parametrize("fmt,tol", [("f16", 2e-2), ("bf16", 5e-2)])
def test_half_gradients_close_to_float64(cfg, fmt, tol):
    P64 = _params(cfg)
    batch = workloads.make_batch(cfg)
    pol64 = Policy("f64")
    # float64 gradients at the half-rounded weights and inputs, so that only the
    # arithmetic differs
    Pr = {k: round_to(v, fmt).astype(np.float64) for k, v in P64.items()}
    br = {k: (round_to(v, fmt).astype(np.float64) if v.dtype.kind == "f" else v)
          for k, v in batch.items()}
    _, dout, cache = models.forward_loss(pol64, cfg, Pr, br, 1.0)
    G64 = models.backward(pol64, cfg, Pr, cache, dout)
    Gh = _half_grads(cfg, fmt, 2.0 ** 10, P64, batch)
    num = np.sqrt(sum(np.sum((Gh[k] - G64[k]) ** 2) for k in G64))
    den = np.sqrt(sum(np.sum(G64[k] ** 2) for k in G64))
    assert num <= tol * den, num / den


@pytest.mark.parametrize("cfg", tiny_cfgs(), ids=lambda c: c.name)
def test_scale_equivariance_bf16(cfg):
    P64 = _params(cfg)
    batch = workloads.make_batch(cfg)
    a = _half_grads(cfg, "bf16", 2.0 ** 3, P64, batch)
    b = _half_grads(cfg, "bf16", 2.0 ** 17, P64, batch)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_scale_equivariance_f16_normal_range():
    cfg = tiny_cfgs()[0]
    P64 = _params(cfg)
    batch = workloads.make_batch(cfg)
    a = _half_grads(cfg, "f16", 2.0 ** 10, P64, batch)
    b = _half_grads(cfg, "f16", 2.0 ** 12, P64, batch)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_cross_entropy_uniform_logits_is_log_classes():
    pol = Policy("f16")
    z = np.zeros((4, 10), np.float32)
    loss, dz = ops.ce_fwd_bwd(pol, z, np.array([0, 3, 9, 9]), 2.0 ** 15)
    assert abs(loss - np.log(10.0)) < 1e-12
    # cotangent: scale * (1/C - onehot) / B
    assert np.allclose(dz[0, 1], round_to(2.0 ** 15 * 0.1 / 4, "f16"))
    assert np.allclose(dz[0, 0], round_to(2.0 ** 15 * (0.1 - 1) / 4, "f16"))


def test_mse_closed_form():
    pol = Policy("f16")
    y = np.array([[1.0, 2.0]], np.float32)
    t = np.array([[0.0, 0.0]], np.float32)
    loss, dy = ops.mse_fwd_bwd(pol, y, t, 4.0)
    assert loss == 2.5
    assert list(dy[0]) == [4.0, 8.0]


def test_layernorm_and_softmax_invariants():
    pol = Policy("f64")
    x = np.random.default_rng(0).normal(3, 2, size=(16, 24))
    y = ops.layernorm_fwd(pol, x, np.ones(24), np.zeros(24))
    assert np.allclose(y.mean(axis=1), 0, atol=1e-12)
    assert np.allclose(y.var(axis=1), 1 / (1 + 1e-5 / x.var(axis=1)), rtol=1e-10)
    p = ops.softmax_fwd(pol, x, 0.125)
    assert np.allclose(p.sum(axis=1), 1.0)
    assert np.allclose(p[0], np.exp(x[0] / 8) / np.exp(x[0] / 8).sum())


def test_attention_layout_brute_force():
    """Heads, q/k/v column blocks and token order, element by element."""
    pol = Policy("f64")
    B, T, H, hd = 2, 3, 2, 4
    d = H * hd
    qkv = np.random.default_rng(1).normal(size=(B * T, 3 * d))
    o, _ = ops.attention_fwd(pol, qkv, B, T, H, hd)
    for b in range(B):
        for h in range(H):
            q = np.array([[qkv[b * T + i, h * hd + c] for c in range(hd)] for i in range(T)])
            k = np.array([[qkv[b * T + i, d + h * hd + c] for c in range(hd)] for i in range(T)])
            v = np.array([[qkv[b * T + i, 2 * d + h * hd + c] for c in range(hd)] for i in range(T)])
            for i in range(T):
                s = [sum(q[i, c] * k[j, c] for c in range(hd)) / np.sqrt(hd) for j in range(T)]
                e = np.exp(np.array(s) - max(s))
                pr = e / e.sum()
                for c in range(hd):
                    ref = sum(pr[j] * v[j, c] for j in range(T))
                    assert abs(o[b * T + i, h * hd + c] - ref) < 1e-12


def test_patchify_brute_force():
    img = np.arange(2 * 4 * 6 * 3).reshape(2, 4, 6, 3).astype(np.float32)
    pt = ops.patchify(img, 2)
    assert pt.shape == (2 * 2 * 3, 12)
    for b in range(2):
        for gy in range(2):
            for gx in range(3):
                row = (b * 2 + gy) * 3 + gx
                for i in range(2):
                    for j in range(2):
                        for c in range(3):
                            assert pt[row, (i * 2 + j) * 3 + c] == img[b, gy * 2 + i, gx * 2 + j, c]


def test_gelu_against_high_precision():
    """The oracle's GELU (and derivative) against 50-digit evaluations of the
    tanh form 0.5 x (1 + tanh(c (x + a x^3))), including the far negative tail
    where 1 + tanh cancels in float64."""
    import mpmath
    mpmath.mp.dps = 1000   # 1 + tanh(u) cancels down to ~1e-860 at x = -30
    xs = np.concatenate([np.linspace(-12, 6, 181), [-30.0, -9.5, -0.75, 0.0, 1e-3]])
    c = mpmath.sqrt(2 / mpmath.pi)
    for x in xs:
        X = mpmath.mpf(float(x))
        u = c * (X + mpmath.mpf("0.044715") * X ** 3)
        ref = 0.5 * X * (1 + mpmath.tanh(u))
        got = ops._gelu64(np.array([x]))[0]
        assert abs(got - float(ref)) <= 1e-13 * abs(float(ref)) + 1e-300, x
        dref = mpmath.diff(lambda t: 0.5 * t * (1 + mpmath.tanh(c * (t + mpmath.mpf("0.044715") * t ** 3))), X)
        dgot = ops.gelu_grad(np.array([x]))[0]
        assert abs(dgot - float(dref)) <= 1e-12 * abs(float(dref)) + 1e-300, x
    # the bf16 GELU of a far-negative input is a tiny negative number, not zero
    assert ops.gelu_fwd(Policy("bf16"), np.array([-8.0]))[0] < 0
