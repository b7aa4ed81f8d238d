"""GPU parity of the multi-tensor sweeps against the oracle, through the C ABI:
cast to half (MPX §3.1), unscale + finite check (§3.3/§3.4), loss-scale update
(§3.3 adjust) and masked AdamW (§3.5).

Bars: the cast, the non-finite count, the unscaled float32 values and the
scale state are bit-exact; the AdamW update is within 1e-5 relative (it is
expected to be bit-exact: both sides evaluate the same float32 expression in
the same order with correctly rounded division and square root).
"""
import numpy as np
import pytest

import workloads
from oracle import adamw as oadamw
from oracle import scaling as oscale
from oracle import step as ostep
from oracle.numfmt import round_to
from tests.gpu_util import HAVE_GPU, assert_same_values, to_dev_half, to_host

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="no GPU")]

if HAVE_GPU:
    import torch
    from paper_2507_03312_amd import binding as mx
    from paper_2507_03312_amd.train import pack_scale_state, unpack_scale_state


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _bit_patterns(n_random=1 << 20):
    rng = np.random.default_rng(0)
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x0FFF, 0x1000, 0x1001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)
    pats = [(hi[:, None] | lows[None, :]).reshape(-1),
            rng.integers(0, 1 << 32, size=n_random, dtype=np.uint64).astype(np.uint32)]
    return np.concatenate(pats).view(np.float32)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_cast_to_half_bit_exact(fmt):
    x = _bit_patterns()
    # three tensors: a large aligned one, a small one, and one misaligned by a
    # single element (scalar path), with ragged sizes
    sizes = [x.size - 1000 - 37, 1000, 37]
    src_all = torch.from_numpy(np.concatenate([x, np.zeros(1, np.float32)])).cuda()
    views = [src_all[0:sizes[0]], src_all[sizes[0]:sizes[0] + sizes[1]],
             src_all[sizes[0] + sizes[1] + 1:sizes[0] + sizes[1] + 1 + sizes[2]]]
    dst_all = torch.zeros(sum(sizes) + 1, dtype=torch.float16 if fmt == "f16" else torch.bfloat16,
                          device="cuda")
    dviews = [dst_all[0:sizes[0]], dst_all[sizes[0] + 1:sizes[0] + 1 + sizes[1]],
              dst_all[sizes[0] + 1 + sizes[1]:sizes[0] + 1 + sizes[1] + sizes[2]]]
    Ls, Ld = mx.TensorList(views), mx.TensorList(dviews)
    mx.mpx_cast_to_half(Ls, Ld, mx.DTYPES[fmt], _stream())
    torch.cuda.synchronize()
    for v, dv in zip(views, dviews):
        src = v.cpu().numpy()
        assert_same_values(to_host(dv), round_to(src, fmt), f"cast {fmt}")


def _grad_list(fmt, sizes, seed=0):
    rng = np.random.default_rng(seed)
    return [round_to(rng.normal(0, 1e-3, size=n) * 2.0 ** 16, fmt) for n in sizes]


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_unscale_check_count_and_values(fmt):
    sizes = [1, 7, 8, 16384, 16385, 100_003, 3]
    grads = _grad_list(fmt, sizes)
    dev = [to_dev_half(g, fmt) for g in grads]
    out = [torch.zeros(n, dtype=torch.float32, device="cuda") for n in sizes]
    Lg, Lo = mx.TensorList(dev), mx.TensorList(out)
    state = torch.from_numpy(pack_scale_state(2.0 ** 16, 0, 2000)).cuda()
    nf = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    dt = mx.DTYPES[fmt]
    mx.mpx_unscale_check(Lg, dt, state.data_ptr(), nf.data_ptr(), Lo, _stream())
    assert int(nf.item()) == oscale.count_nonfinite(grads) == 0
    for o, g in zip(out, grads):
        assert_same_values(o.cpu().numpy(), oscale.unscale(g, np.float32(2.0 ** 16)), "unscale")
    # injections at the first, last and tail elements of several tensors
    cases = [(0, 0, np.inf), (6, 2, -np.inf), (4, 16384, np.nan), (5, -1, np.inf), (3, 16383, np.nan)]
    for k in range(1, len(cases) + 1):
        gi = [g.copy() for g in grads]
        for t, e, val in cases[:k]:
            gi[t].reshape(-1)[e] = val
            dev[t].view(-1)[e] = float(val)
        mx.mpx_unscale_check(Lg, dt, state.data_ptr(), nf.data_ptr(), None, _stream())
        assert int(nf.item()) == oscale.count_nonfinite(gi) == k
    # finite extremes are not counted
    for t, e, _ in cases:
        dev[t].view(-1)[e] = 65504.0 if fmt == "f16" else 3.0e38
    dev[0].view(-1)[0] = 2.0 ** -24 if fmt == "f16" else 2.0 ** -133
    mx.mpx_unscale_check(Lg, dt, state.data_ptr(), nf.data_ptr(), None, _stream())
    assert int(nf.item()) == 0


def test_unscale_check_empty_list_writes_zero():
    Lg = mx.TensorList([])
    nf = torch.full((1,), 9, dtype=torch.int32, device="cuda")
    mx.mpx_unscale_check(Lg, mx.MPX_F16, 0, nf.data_ptr(), None, _stream())
    assert int(nf.item()) == 0


def test_scale_update_matches_oracle_state_machine():
    cases = [(2.0 ** 15, 4, {3}, 10), (2.0 ** 16, 25, {37, 137}, 200), (2.0, 1, {0, 1, 2}, 6)]
    for scale0, period, bad, n in cases:
        st = oscale.make_state(scale0, period, max_scale=2.0 ** 20 if period == 1 else 2.0 ** 127)
        dst = torch.from_numpy(pack_scale_state(scale0, 0, period, 2.0, 1.0, float(st.max_scale))).cuda()
        nf = torch.zeros(1, dtype=torch.int32, device="cuda")
        for s in range(n):
            nf.fill_(1 if s in bad else 0)
            mx.mpx_scale_update(dst.data_ptr(), nf.data_ptr(), _stream())
            st = oscale.adjust(st, s not in bad)
            got = unpack_scale_state(dst.cpu().numpy())
            assert got["scale"] == float(st.scale) and got["counter"] == st.counter, (s, got, st)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_adamw_masked_small_sweep_trajectory(fmt):
    from paper_2507_03312_amd.sweep import SweepStep
    cfg = workloads.small_sweep(half=fmt)
    sizes = workloads.sweep_sizes(cfg)
    gf, params = workloads.sweep_tensors(cfg, sizes)
    gpu = SweepStep(cfg, sizes)
    gpu.load(gf, params)
    gh, ost = ostep.sweep_init(cfg, gf, params)
    for g_dev, g_ref in zip(gpu.g, gh):
        assert_same_values(to_host(g_dev), g_ref, "initial half gradients")
    for s in range(cfg.steps):
        before = [to_host(t) for t in gpu.p]
        saved = [gpu.inject(inj) for inj in gpu.injections_at(s)]
        gpu.step()
        for sv in saved:
            gpu.restore(sv)
        ost, nf_ref, _ = ostep.sweep_step(cfg, ost, gh, s)
        assert int(gpu.d_nonfinite.item()) == nf_ref
        st = gpu.scale_state()
        assert st["scale"] == float(ost.scale.scale) and st["counter"] == ost.scale.counter
        assert int(gpu.d_step.item()) == ost.t
        for i in range(len(sizes)):
            p = to_host(gpu.p[i])
            if nf_ref:
                assert np.array_equal(p, before[i]), "skipped step must not write"
            tol = 1e-5 * np.maximum(np.abs(ost.p[i]), cfg.lr)
            assert np.all(np.abs(p - ost.p[i]) <= tol)
            for dv, ref in ((gpu.m[i], ost.m[i]), (gpu.v[i], ost.v[i])):
                r = to_host(dv)
                assert np.all(np.abs(r - ref) <= 1e-5 * np.max(np.abs(ref)) + 1e-30)
            # the half copy is the rounding of the GPU's own new masters
            assert_same_values(to_host(gpu.h[i]), round_to(p, fmt), "half copy")


def test_adamw_bit_exact_against_oracle_expression():
    """Same float32 expression, same order: expected bit-identical."""
    n = 300_001
    rng = np.random.default_rng(4)
    p = rng.normal(0, 0.02, n).astype(np.float32)
    m = rng.normal(0, 1e-3, n).astype(np.float32)
    v = np.abs(rng.normal(0, 1e-6, n)).astype(np.float32)
    g16 = round_to(rng.normal(0, 1e-3, n) * 2.0 ** 16, "f16")
    hp = oadamw.AdamWHP()
    t0 = 7
    tp, tm, tv = (torch.from_numpy(a.copy()).cuda() for a in (p, m, v))
    tg = to_dev_half(g16, "f16")
    L = [mx.TensorList([x]) for x in (tp, tm, tv, tg)]
    state = torch.from_numpy(pack_scale_state(2.0 ** 16, 0, 2000)).cuda()
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    step = torch.full((1,), t0, dtype=torch.int32, device="cuda")
    mx.mpx_adamw_masked(L[0], L[1], L[2], L[3], mx.MPX_F16, mx.AdamWHP(hp.lr, hp.beta1, hp.beta2,
                        hp.eps, hp.weight_decay), step.data_ptr(), state.data_ptr(), nf.data_ptr(),
                        None, mx.MPX_F16, _stream())
    g32 = oscale.unscale(g16, np.float32(2.0 ** 16))
    rp, rm, rv = oadamw.adamw_update(p, m, v, g32, t0 + 1, hp)
    assert int(step.item()) == t0 + 1
    for dev, ref, name in ((tp, rp, "p"), (tm, rm, "m"), (tv, rv, "v")):
        got = dev.cpu().numpy()
        assert np.all(np.abs(got - ref) <= 1e-5 * np.maximum(np.abs(ref), hp.lr)), name
        assert_same_values(got, ref, name)


@pytest.mark.slow
def test_full_sweep_workload_sampled():
    """1e8 elements in 200 tensors: scale/skip trajectory over the 200 steps
    bit-exact against the oracle's state machine driven by the oracle's own
    finite count; AdamW (p, m, v and the half copy) checked on up to 64
    sampled elements of EVERY tensor after the first three steps, on the two
    skipped steps (nothing written) and on the first applied step after each
    skip (bias corrections use the count of applied steps), and at the end.
    AdamW is elementwise, so the oracle follows the sampled elements alone."""
    from paper_2507_03312_amd.sweep import SweepStep
    cfg = workloads.get("sweep")
    sizes = workloads.sweep_sizes(cfg)
    gf, params = workloads.sweep_tensors(cfg, sizes)
    gpu = SweepStep(cfg, sizes)
    gpu.load(gf, params)
    rng = np.random.default_rng(9)
    samples = [np.unique(rng.integers(0, n, size=min(n, 64))) for n in sizes]
    idx = [torch.from_numpy(i).cuda() for i in samples]
    g_s = [round_to(g[i], "f16") for g, i in zip(gf, samples)]
    p_s = [p[i].copy() for p, i in zip(params, samples)]
    m_s = [np.zeros_like(x) for x in p_s]
    v_s = [np.zeros_like(x) for x in p_s]
    # N(0, 1e-3) * 2^16 stays far below the float16 maximum: only injections overflow
    assert max(float(np.max(np.abs(g))) for g in gf) < 65504 / 4
    skips = [inj.step for inj in cfg.injections]
    check_at = {0, 1, 2, cfg.steps - 1} | set(skips) | {s + 1 for s in skips}
    st = oscale.make_state(cfg.scale_init, cfg.period)
    hp = oadamw.AdamWHP(cfg.lr, cfg.beta1, cfg.beta2, cfg.eps, cfg.weight_decay)
    t = 0
    checked = 0
    for s in range(cfg.steps):
        injs = gpu.injections_at(s)
        saved = [gpu.inject(inj) for inj in injs]
        gpu.step()
        for sv in saved:
            gpu.restore(sv)
        finite = not injs
        assert int(gpu.d_nonfinite.item()) == len(injs)
        g32 = [oscale.unscale(g, st.scale) for g in g_s]
        p_s, m_s, v_s, t = oadamw.adamw_masked(p_s, m_s, v_s, g32, t, hp, finite)
        if s in check_at:
            for i in range(len(sizes)):
                for dev, ref, what in ((gpu.p, p_s, "p"), (gpu.m, m_s, "m"), (gpu.v, v_s, "v")):
                    got = dev[i][idx[i]].cpu().numpy()
                    tol = 1e-5 * (np.maximum(np.abs(ref[i]), cfg.lr) if what == "p"
                                  else max(float(np.max(np.abs(ref[i]))), 1e-30))
                    assert np.all(np.abs(got - ref[i]) <= tol), (s, i, what)
                got_p = gpu.p[i][idx[i]].cpu().numpy()
                assert_same_values(to_host(gpu.h[i][idx[i]]), round_to(got_p, "f16"), "half copy")
            checked += 1
        st = oscale.adjust(st, finite)
        got = gpu.scale_state()
        assert got["scale"] == float(st.scale) and got["counter"] == st.counter
        assert int(gpu.d_step.item()) == t
    assert int(gpu.d_step.item()) == cfg.steps - 2
    assert checked == len(check_at)
