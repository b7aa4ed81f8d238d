"""Pins of the oracle's dynamic loss scaling (unscale, finite check, adjust).

The scale trajectories below were worked out by hand from the rule (halve and
reset on a non-finite step; double after ``period`` consecutive finite steps)
and are closed forms independent of the code.
"""
import numpy as np
import pytest

import workloads
from oracle import scaling, step
from oracle.numfmt import round_to


def _trajectory(scale0, period, bad_steps, n):
    st = scaling.make_state(scale0, period)
    used, skips = [], []
    for s in range(n):
        used.append(float(st.scale))
        finite = s not in bad_steps
        if not finite:
            skips.append(s)
        st = scaling.adjust(st, finite)
    return used, skips, st


def test_mlp_workload_trajectory_closed_form():
    used, skips, st = _trajectory(2.0 ** 15, 4, {3}, 10)
    assert used == [2.0 ** 15] * 4 + [2.0 ** 14] * 4 + [2.0 ** 15] * 2
    assert skips == [3]
    assert float(st.scale) == 2.0 ** 15 and st.counter == 2


def test_sweep_trajectory_period_2000():
    used, skips, st = _trajectory(2.0 ** 16, 2000, {37, 137}, 200)
    assert skips == [37, 137]
    assert used[:38] == [2.0 ** 16] * 38
    assert used[38:138] == [2.0 ** 15] * 100
    assert used[138:] == [2.0 ** 14] * 62
    assert float(st.scale) == 2.0 ** 14 and st.counter == 62


def test_sweep_trajectory_period_25():
    used, _, st = _trajectory(2.0 ** 16, 25, {37, 137}, 200)
    changes = [(s, used[s]) for s in range(1, 200) if used[s] != used[s - 1]]
    assert changes == [(25, 2.0 ** 17), (38, 2.0 ** 16), (63, 2.0 ** 17), (88, 2.0 ** 18),
                       (113, 2.0 ** 19), (138, 2.0 ** 18), (163, 2.0 ** 19), (188, 2.0 ** 20)]
    assert float(st.scale) == 2.0 ** 20 and st.counter == 12


def test_floor_and_cap():
    st = scaling.make_state(2.0, 1, min_scale=1.0, max_scale=4.0)
    st = scaling.adjust(st, False)
    assert float(st.scale) == 1.0
    st = scaling.adjust(st, False)
    assert float(st.scale) == 1.0 and st.counter == 0
    for expect in (2.0, 4.0, 4.0):
        st = scaling.adjust(st, True)
        assert float(st.scale) == expect and st.counter == 0


def test_counter_resets_on_overflow():
    st = scaling.make_state(8.0, 3)
    st = scaling.adjust(st, True)
    st = scaling.adjust(st, True)
    assert st.counter == 2
    st = scaling.adjust(st, False)
    assert st.counter == 0 and float(st.scale) == 4.0
    st = scaling.adjust(st, True)
    st = scaling.adjust(st, True)
    assert float(st.scale) == 4.0
    st = scaling.adjust(st, True)
    assert float(st.scale) == 8.0 and st.counter == 0


@pytest.mark.parametrize("bad", [np.inf, -np.inf, np.nan])
@pytest.mark.parametrize("where", [0, -1, 12345])
def test_nonfinite_anywhere_is_counted(bad, where):
    rng = np.random.default_rng(0)
    grads = [round_to(rng.normal(size=n), "f16") for n in (7, 1, 20000, 33)]
    assert scaling.count_nonfinite(grads) == 0
    for t in range(len(grads)):
        g = [a.copy() for a in grads]
        flat = g[t].reshape(-1)
        flat[where % flat.size] = bad
        assert scaling.count_nonfinite(g) == 1


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_finite_extremes_not_counted(fmt):
    mx = {"f16": 65504.0, "bf16": float(np.ldexp(2.0 - 2.0 ** -7, 127))}[fmt]
    sub = {"f16": 2.0 ** -24, "bf16": 2.0 ** -133}[fmt]
    g = round_to(np.array([0.0, -0.0, sub, -sub, mx, -mx]), fmt)
    assert scaling.count_nonfinite([g]) == 0


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
@pytest.mark.parametrize("k", [0, 1, 10, 15, 16, 24])
def test_unscale_power_of_two_is_exact(fmt, k):
    rng = np.random.default_rng(k)
    x = round_to(rng.normal(0, 1e-2, size=50_000), fmt)
    scaled = round_to(x.astype(np.float64) * 2.0 ** k, fmt)
    ok = np.isfinite(scaled) & (np.abs(scaled) >= (2.0 ** -14 if fmt == "f16" else 2.0 ** -126))
    un = scaling.unscale(scaled, np.float32(2.0 ** k))
    assert un.dtype == np.float32
    # division by 2^k equals an exponent shift (a library ldexp) ...
    assert np.array_equal(un[ok], np.ldexp(scaled[ok], -k))
    # ... and scale-then-unscale returns the value whenever the scaled value is normal
    assert np.array_equal(un[ok], x[ok])


def test_small_sweep_trajectory():
    cfg = workloads.small_sweep()
    sizes = workloads.sweep_sizes(cfg)
    gf, params = workloads.sweep_tensors(cfg, sizes)
    gh, st = step.sweep_init(cfg, gf, params)
    used, flags = [], []
    for s in range(cfg.steps):
        st, nf, sc = step.sweep_step(cfg, st, gh, s)
        used.append(sc)
        flags.append(nf)
    # period 3, injections at steps 4 and 9
    assert [f > 0 for f in flags] == [s in (4, 9) for s in range(cfg.steps)]
    s16 = 2.0 ** 16
    assert used == [s16, s16, s16, 2 * s16, 2 * s16, s16, s16, s16, 2 * s16, 2 * s16, s16, s16]
    assert st.t == cfg.steps - 2
