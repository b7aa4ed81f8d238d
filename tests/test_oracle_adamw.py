"""Pins of the oracle's masked AdamW.

* first step closed form: with m = v = 0, the bias-corrected ratio is g/|g|;
* agreement with torch.optim.AdamW (a library implementation, float64, CPU)
  over several applied steps, decoupled weight decay included;
* a skipped step changes nothing, and the step count only advances on
  applied steps, so bias correction follows the applied-step count.
"""
import numpy as np
import torch

from oracle.adamw import AdamWHP, adamw_masked

HP = AdamWHP(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-4)


def _rand(n, seed, s=1.0):
    return np.random.default_rng(seed).normal(0, s, size=n).astype(np.float32)


def test_first_step_closed_form():
    p0 = _rand(10_000, 0, 0.02)
    g = _rand(10_000, 1, 1e-3)
    z = np.zeros_like(p0)
    (p1,), _, _, t = adamw_masked([p0], [z], [z], [g], 0, HP, True)
    ref = p0.astype(np.float64) - HP.lr * (np.sign(g) * np.abs(g) / (np.abs(g) + HP.eps)
                                           + HP.weight_decay * p0)
    assert t == 1
    # float32 arithmetic: a few ulps of p plus a tiny fraction of the step size
    assert np.all(np.abs(p1 - ref) <= 2.0 ** -21 * np.abs(ref) + 1e-6 * HP.lr)


def _torch_run(p0, grads, hp):
    p = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay)
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


def test_matches_torch_adamw_with_skips():
    n = 20_000
    p = [_rand(n, 0, 0.02)]
    m = [np.zeros(n, np.float32)]
    v = [np.zeros(n, np.float32)]
    applied = []
    t = 0
    for s in range(8):
        g = _rand(n, 10 + s, 1e-2)
        finite = s not in (2, 5)
        if not finite:
            g = g.copy()
            g[17] = np.inf
        before = (p[0].copy(), m[0].copy(), v[0].copy(), t)
        p, m, v, t = adamw_masked(p, m, v, [g], t, HP, finite)
        if finite:
            applied.append(g)
        else:
            # a skipped step leaves every state bit-identical
            assert np.array_equal(p[0], before[0]) and np.array_equal(m[0], before[1])
            assert np.array_equal(v[0], before[2]) and t == before[3]
    assert t == len(applied) == 6
    pr, mr, vr = _torch_run(_rand(n, 0, 0.02), applied, HP)
    assert np.max(np.abs(p[0] - pr)) <= 1e-6 * max(np.max(np.abs(pr)), HP.lr)
    assert np.max(np.abs(m[0] - mr)) <= 1e-6 * np.max(np.abs(mr))
    assert np.max(np.abs(v[0] - vr)) <= 1e-6 * np.max(np.abs(vr))


def test_no_weight_decay_matches_torch_adam_direction():
    hp = AdamWHP(lr=1e-2, weight_decay=0.0)
    n = 1000
    p0 = _rand(n, 3, 0.5)
    gs = [_rand(n, 30 + s, 1.0) for s in range(3)]
    p, m, v, t = [p0], [np.zeros(n, np.float32)], [np.zeros(n, np.float32)], 0
    for g in gs:
        p, m, v, t = adamw_masked(p, m, v, [g], t, hp, True)
    pr, _, _ = _torch_run(p0, gs, hp)
    assert np.max(np.abs(p[0] - pr)) <= 1e-6
