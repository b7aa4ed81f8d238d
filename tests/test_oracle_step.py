"""Step-level pins of the oracle on the MLP workload (fp16, scale 2^15, growth
interval 4, +inf written into dW1 at step 3).

The loss-scale trajectory and the skip decision are closed forms worked out by
hand from the dynamic scaling rule; a skipped step must leave the masters, the
moments and the step count bit-identical.
"""
import numpy as np

import workloads
from oracle import step


def test_mlp_workload_trajectory_and_skip():
    cfg = workloads.get("mlp")
    st = step.init_state(cfg)
    batch = workloads.make_batch(cfg)
    used, flags = [], []
    for s in range(cfg.steps):
        before = st
        st, r = step.train_step(cfg, st, batch, s)
        used.append(r.scale_used)
        flags.append(r.nonfinite)
        if s == 3:
            for a, b in zip(before.masters, st.masters):
                assert np.array_equal(a, b)
            for a, b in zip(before.m, st.m):
                assert np.array_equal(a, b)
            assert st.t == before.t
        else:
            assert r.nonfinite == 0 and st.t == before.t + 1
    assert flags[3] == 1
    assert used == [2.0 ** 15] * 4 + [2.0 ** 14] * 4 + [2.0 ** 15] * 2
    assert st.t == 9 and float(st.scale.scale) == 2.0 ** 15 and st.scale.counter == 2


def test_mlp_gradients_are_half_and_scaled():
    cfg = workloads.get("mlp")
    st = step.init_state(cfg)
    batch = workloads.make_batch(cfg)
    _, grads = step.gradients(cfg, st, batch, step.Policy("f16"))
    for g in grads:
        assert np.array_equal(g.astype(np.float16).astype(np.float32), g)
    # scaled by 2^15: the gradients are far from the f16 subnormal range
    assert max(float(np.max(np.abs(g))) for g in grads) > 1.0


def test_full_precision_step_matches_float64_gradients():
    """Full precision (mixed precision switched off): with every op rounded
    to float32 the MLP workload's gradients agree with the float64 policy's
    (the exact-arithmetic model pinned by finite differences) to float32
    accuracy, the loss is unscaled, the scale state is untouched, and the
    step applies AdamW (step count advances)."""
    cfg = workloads.get("mlp")
    st = step.init_state(cfg)
    batch = workloads.make_batch(cfg)
    new, loss, grads = step.full_precision_step(cfg, st, batch)
    pol = step.Policy("f64")
    P = {n: np.asarray(w, np.float64) for n, w in zip(st.names, st.masters)}
    fb = {k: np.asarray(v, np.float64) for k, v in batch.items()}
    loss64, dout, cache = step.models.forward_loss(pol, cfg, P, fb, 1.0)
    G = step.models.backward(pol, cfg, P, cache, dout)
    assert abs(loss - loss64) <= 1e-6 * abs(loss64)
    for n, g in zip(st.names, grads):
        assert g.dtype == np.float32
        ref = np.asarray(G[n], np.float64)
        err = np.linalg.norm(g - ref) / np.linalg.norm(ref)
        assert err <= 1e-5, (n, err)
        # a float32 result, not a half one: some values are not half-representable
        assert not np.array_equal(g.astype(np.float16).astype(np.float32), g)
    assert new.t == st.t + 1 and new.scale == st.scale
    assert any(not np.array_equal(a, b) for a, b in zip(new.masters, st.masters))
