"""GPU parity of the half GEMMs (float32 accumulation) against the oracle,
through the C ABI: linear forward with bias / GELU / residual epilogues,
linear backward (dX, dX through GELU', split-K dW, db) and the batched GEMM of
the attention core, in float16 and bfloat16.

Bar (per element): |gpu - oracle| <= ulp(oracle) + 2 K 2^-24 (|A||B|), the
difference allowed between two float32 summation orders followed by one
rounding to half.  Epilogues that round again (GELU, residual) are checked
against the oracle's op applied to the GPU's own pre-activation, within one
half ulp (float32 vs float64 math inside the op).
"""
import numpy as np
import pytest

from oracle import ops
from oracle.numfmt import round_to
from oracle.policy import Policy
from tests.gpu_util import (HAVE_GPU, assert_within, gemm_bound, to_dev_half, to_host, ulp)

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="no GPU")]

if HAVE_GPU:
    import torch
    from paper_2507_03312_amd import binding as mx

FMTS = ["f16", "bf16"]


def _s():
    return torch.cuda.current_stream().cuda_stream


def _rand(shape, fmt, seed, std=1.0):
    return round_to(np.random.default_rng(seed).normal(0, std, size=shape), fmt)


def _empty(shape, fmt):
    return torch.zeros(*shape, dtype=torch.float16 if fmt == "f16" else torch.bfloat16, device="cuda")


SHAPES = [
    (64, 1024, 512),     # MLP fc1
    (70, 100, 72),       # ragged in M and N, K a multiple of 8
    (33, 17, 50),        # every dim ragged, K not a multiple of 8 (scalar loads)
    (300, 200, 1000),
    (128, 10, 384),      # a 10-class head
    (1, 8, 8),
]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("mnk", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_linear_fwd(fmt, mnk):
    M, N, K = mnk
    pol = Policy(fmt)
    x = _rand((M, K), fmt, 1)
    w = _rand((N, K), fmt, 2, 0.05)
    b = _rand((N,), fmt, 3, 0.5)
    r = _rand((M, N), fmt, 4)
    dx, dw, db, dr = (to_dev_half(a, fmt) for a in (x, w, b, r))
    y, pre, y2 = _empty((M, N), fmt), _empty((M, N), fmt), _empty((M, N), fmt)
    dt = mx.DTYPES[fmt]
    # plain + bias
    mx.mpx_linear_fwd(dx.data_ptr(), dw.data_ptr(), db.data_ptr(), None, y.data_ptr(), None,
                      M, N, K, dt, mx.MPX_ACT_NONE, _s())
    ref = ops.linear_fwd(pol, x, w, b)
    bound = gemm_bound(x, w.T, ref, fmt, K)
    assert_within(to_host(y), ref, bound, "linear")
    # GELU epilogue: pre-activation within the GEMM bound, output = gelu(own pre)
    mx.mpx_linear_fwd(dx.data_ptr(), dw.data_ptr(), db.data_ptr(), None, y.data_ptr(),
                      pre.data_ptr(), M, N, K, dt, mx.MPX_ACT_GELU_TANH, _s())
    gpre = to_host(pre)
    assert_within(gpre, ref, bound, "pre-activation")
    g_ref = ops.gelu_fwd(pol, gpre)
    assert_within(to_host(y), g_ref, ulp(g_ref, fmt), "gelu epilogue")
    # residual epilogue, no bias
    mx.mpx_linear_fwd(dx.data_ptr(), dw.data_ptr(), None, dr.data_ptr(), y2.data_ptr(), None,
                      M, N, K, dt, mx.MPX_ACT_NONE, _s())
    mx.mpx_linear_fwd(dx.data_ptr(), dw.data_ptr(), None, None, y.data_ptr(), None,
                      M, N, K, dt, mx.MPX_ACT_NONE, _s())
    own = to_host(y)
    ref0 = ops.linear_fwd(pol, x, w, None)
    assert_within(own, ref0, gemm_bound(x, w.T, ref0, fmt, K), "linear no bias")
    assert_within(to_host(y2), ops.add(pol, own, r), 0.0, "residual epilogue")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("mnk", SHAPES + [(4096, 384, 384), (2500, 96, 40), (8192, 33, 50)],
                         ids=lambda s: "x".join(map(str, s)))
def test_linear_bwd(fmt, mnk):
    M, N, K = mnk
    pol = Policy(fmt)
    x = _rand((M, K), fmt, 11)
    w = _rand((N, K), fmt, 12, 0.05)
    dy = _rand((M, N), fmt, 13)
    xpre = _rand((M, K), fmt, 14)
    tx, tw, tdy, txp = (to_dev_half(a, fmt) for a in (x, w, dy, xpre))
    gdx, gdw, gdb = _empty((M, K), fmt), _empty((N, K), fmt), _empty((N,), fmt)
    ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    dt = mx.DTYPES[fmt]
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), None, mx.MPX_ACT_NONE,
                      gdx.data_ptr(), gdw.data_ptr(), gdb.data_ptr(), M, N, K, dt,
                      ws.data_ptr(), ws_n, None, _s())
    rdx, rdw, rdb = ops.linear_bwd(pol, x, w, dy)
    assert_within(to_host(gdx), rdx, gemm_bound(dy, w, rdx, fmt, N), "dX")
    assert_within(to_host(gdw), rdw, gemm_bound(dy.T, x, rdw, fmt, M), "dW")
    colb = ulp(rdb, fmt) + 2.0 * M * 2.0 ** -24 * np.abs(dy.astype(np.float64)).sum(axis=0)
    assert_within(to_host(gdb), rdb, colb, "db")
    # dX through GELU': half(half(dY W) * gelu'(Xpre))
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), txp.data_ptr(),
                      mx.MPX_ACT_GELU_TANH, gdx.data_ptr(), gdw.data_ptr(), None, M, N, K, dt,
                      ws.data_ptr(), ws_n, None, _s())
    got = to_host(gdx)
    ref = ops.gelu_bwd(pol, xpre, rdx)
    # GPU's own dX may differ from rdx by the GEMM bound, scaled by |gelu'| <= 1.13
    bound = 1.13 * gemm_bound(dy, w, rdx, fmt, N) + ulp(ref, fmt)
    assert_within(got, ref, bound, "dX through gelu'")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("mnk", [(4096, 384, 384), (256, 256, 256), (70, 100, 72), (128, 10, 384),
                                 (2500, 96, 40), (33, 17, 50)],
                         ids=lambda s: "x".join(map(str, s)))
def test_linear_bwd_counts_nonfinite(fmt, mnk):
    """MPX §3.4's finite check fused into the kernels that write dW and db
    (split-K reduction, both GEMM epilogues, the skinny-product kernel, the
    column sum): the count they add equals the separate check's count over
    [dW, db], dX is never counted, and a second call adds to the counter."""
    M, N, K = mnk
    x = _rand((M, K), fmt, 21)
    w = _rand((N, K), fmt, 22, 0.05)
    dy = _rand((M, N), fmt, 23)
    big = 60000.0 if fmt == "f16" else 3.0e38  # finite, but dW and db overflow in places
    dy[0, ::2] = big
    dy[min(1, M - 1), :] = big / 2
    dy = round_to(dy, fmt)
    tx, tw, tdy = (to_dev_half(a, fmt) for a in (x, w, dy))
    gdx, gdw, gdb = _empty((M, K), fmt), _empty((N, K), fmt), _empty((N,), fmt)
    ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    dt = mx.DTYPES[fmt]
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    ref = torch.zeros(1, dtype=torch.int32, device="cuda")
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), None, mx.MPX_ACT_NONE,
                      gdx.data_ptr(), gdw.data_ptr(), gdb.data_ptr(), M, N, K, dt,
                      ws.data_ptr(), ws_n, nf.data_ptr(), _s())
    mx.mpx_unscale_check(mx.TensorList([gdw, gdb]), dt, 0, ref.data_ptr(), None, _s())
    count, want = int(nf.item()), int(ref.item())
    assert count == want and 0 < want < N * K + N, (count, want)
    mx.mpx_linear_bwd(tx.data_ptr(), None, tdy.data_ptr(), None, mx.MPX_ACT_NONE, None,
                      gdw.data_ptr(), gdb.data_ptr(), M, N, K, dt, ws.data_ptr(), ws_n,
                      nf.data_ptr(), _s())
    assert int(nf.item()) == 2 * want


def test_linear_bwd_workspace_is_checked():
    M, N, K = 256, 256, 256
    t = _empty((M, K), "f16")
    with pytest.raises(mx.MPXError, match="workspace"):
        mx.mpx_linear_bwd(t.data_ptr(), t.data_ptr(), t.data_ptr(), None, 0, t.data_ptr(),
                          t.data_ptr(), None, M, N, K, mx.MPX_F16, None, 0, None, _s())


def test_invalid_arguments_raise_before_launch():
    t = _empty((8, 8), "f16")
    with pytest.raises(mx.MPXError):
        mx.mpx_linear_fwd(t.data_ptr(), None, None, None, t.data_ptr(), None, 8, 8, 8,
                          mx.MPX_F16, 0, _s())
    with pytest.raises(mx.MPXError):
        mx.mpx_linear_fwd(t.data_ptr(), t.data_ptr(), None, None, t.data_ptr(), None, 0, 8, 8,
                          mx.MPX_F16, 0, _s())
    with pytest.raises(mx.MPXError):
        mx.mpx_linear_fwd(t.data_ptr(), t.data_ptr(), None, None, t.data_ptr(), None, 8, 8, 8,
                          7, 0, _s())


ATTN = [(2, 3, 65, 64), (1, 2, 197, 64), (3, 1, 5, 16)]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("bhtd", ATTN, ids=lambda s: "x".join(map(str, s)))
def test_gemm_batched_attention_layouts(fmt, bhtd):
    """The four operand layouts the attention core uses, on the real strides."""
    B, H, T, hd = bhtd
    d = H * hd
    ldT = -(-T // 8) * 8
    pol = Policy(fmt)
    qkv = _rand((B * T, 3 * d), fmt, 21)
    Pm = np.zeros((B, H, T, ldT), np.float32)
    Pm[..., :T] = _rand((B, H, T, T), fmt, 22, 0.1)
    tq, tp = to_dev_half(qkv, fmt), to_dev_half(Pm.reshape(B * H * T, ldT), fmt)
    out_s = _empty((B * H * T, ldT), fmt)
    out_o = _empty((B * T, d), fmt)
    dt = mx.DTYPES[fmt]
    e = tq.element_size()
    q, k, v = ops.split_heads(qkv, B, T, H, hd)
    # S = Q K^T
    mx.mpx_gemm_batched(0, 1, T, T, hd, B, H, tq.data_ptr(), 3 * d, T * 3 * d, hd,
                        tq.data_ptr() + d * e, 3 * d, T * 3 * d, hd,
                        out_s.data_ptr(), ldT, H * T * ldT, T * ldT, dt, _s())
    got = to_host(out_s).reshape(B, H, T, ldT)[..., :T]
    k_t = np.swapaxes(k, -1, -2)
    ref = pol.R(pol.mm(q, k_t))
    bnd = ulp(ref, fmt) + 2 * hd * 2.0 ** -24 * (np.abs(q.astype(np.float64)) @ np.abs(k_t.astype(np.float64)))
    assert_within(got, ref, bnd, "QK^T")
    # O = P V  (k-major P with padded rows, V as a K x N slice)
    mx.mpx_gemm_batched(0, 0, T, hd, T, B, H, tp.data_ptr(), ldT, H * T * ldT, T * ldT,
                        tq.data_ptr() + 2 * d * e, 3 * d, T * 3 * d, hd,
                        out_o.data_ptr(), d, T * d, hd, dt, _s())
    Pv = Pm[..., :T]
    ref = pol.R(pol.mm(Pv, v))
    bnd = ulp(ref, fmt) + 2 * T * 2.0 ** -24 * (np.abs(Pv.astype(np.float64)) @ np.abs(v.astype(np.float64)))
    got = to_host(out_o).reshape(B, T, H, hd).transpose(0, 2, 1, 3)
    assert_within(got, ref, bnd, "PV")
    # dV-like: P^T X (trans_a = 1) and dK-like with trans_a = 1, trans_b = 0
    mx.mpx_gemm_batched(1, 0, T, hd, T, B, H, tp.data_ptr(), ldT, H * T * ldT, T * ldT,
                        tq.data_ptr(), 3 * d, T * 3 * d, hd,
                        out_o.data_ptr(), d, T * d, hd, dt, _s())
    Pt = np.swapaxes(Pv, -1, -2)
    ref = pol.R(pol.mm(Pt, q))
    bnd = ulp(ref, fmt) + 2 * T * 2.0 ** -24 * (np.abs(Pt.astype(np.float64)) @ np.abs(q.astype(np.float64)))
    got = to_host(out_o).reshape(B, T, H, hd).transpose(0, 2, 1, 3)
    assert_within(got, ref, bnd, "P^T Q")


@pytest.mark.parametrize("fmt,mnk", [("bf16", (12608, 2304, 768)), ("bf16", (12608, 768, 3072)),
                                     ("f16", (16640, 1536, 384)), ("f16", (16384, 384, 48))],
                         ids=lambda s: str(s))
def test_full_size_linear_sampled(fmt, mnk):
    """Full ViT-B / ViT-S layer shapes, forward and backward, in the launch
    configuration the training step uses; sampled outputs against the oracle."""
    M, N, K = mnk
    pol = Policy(fmt)
    rng = np.random.default_rng(5)
    x = _rand((M, K), fmt, 31)
    w = _rand((N, K), fmt, 32, 0.02)
    dy = _rand((M, N), fmt, 33, 1e-2)
    tx, tw, tdy = (to_dev_half(a, fmt) for a in (x, w, dy))
    y, gdx, gdw, gdb = _empty((M, N), fmt), _empty((M, K), fmt), _empty((N, K), fmt), _empty((N,), fmt)
    dt = mx.DTYPES[fmt]
    mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), None, None, y.data_ptr(), None, M, N, K, dt, 0, _s())
    ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), None, 0, gdx.data_ptr(),
                      gdw.data_ptr(), gdb.data_ptr(), M, N, K, dt, ws.data_ptr(), ws_n, None, _s())
    rows = np.unique(rng.integers(0, M, 48))
    cols = np.unique(rng.integers(0, N, 48))
    ref = pol.gemm(x[rows], w[cols].T)
    assert_within(to_host(y)[np.ix_(rows, cols)], ref, gemm_bound(x[rows], w[cols].T, ref, fmt, K), "Y")
    kc = np.unique(rng.integers(0, K, 48))
    ref = pol.gemm(dy[rows], w[:, kc])
    assert_within(to_host(gdx)[np.ix_(rows, kc)], ref, gemm_bound(dy[rows], w[:, kc], ref, fmt, N), "dX")
    ref = pol.gemm(dy[:, cols].T, x[:, kc])
    assert_within(to_host(gdw)[np.ix_(cols, kc)], ref, gemm_bound(dy[:, cols].T, x[:, kc], ref, fmt, M), "dW")


CONFIGS = [1, 2, 3, 4, 5, 6, 7, 9, 10, 11]


@pytest.fixture
def gemm_config(request):
    mx.mpx_gemm_set_config(request.param)
    yield request.param
    mx.mpx_gemm_set_config(0)


@pytest.mark.parametrize("gemm_config", CONFIGS, indirect=True)
@pytest.mark.parametrize("fmt", FMTS)
def test_every_tile_config(gemm_config, fmt):
    """Each tile configuration forced in turn (the direct-to-LDS ones need k a
    multiple of 64): forward with bias + GELU on a ragged output, backward
    with dX through GELU' and split-K dW, all three operand layouts."""
    pol = Policy(fmt)
    dt = mx.DTYPES[fmt]
    # forward, ragged M and N
    M, N, K = 300, 200, 320
    x, w, b = _rand((M, K), fmt, 41), _rand((N, K), fmt, 42, 0.05), _rand((N,), fmt, 43, 0.5)
    tx, tw, tb = (to_dev_half(a, fmt) for a in (x, w, b))
    y, pre = _empty((M, N), fmt), _empty((M, N), fmt)
    mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), tb.data_ptr(), None, y.data_ptr(),
                      pre.data_ptr(), M, N, K, dt, mx.MPX_ACT_GELU_TANH, _s())
    ref = ops.linear_fwd(pol, x, w, b)
    gpre = to_host(pre)
    assert_within(gpre, ref, gemm_bound(x, w.T, ref, fmt, K), "pre-activation")
    g_ref = ops.gelu_fwd(pol, gpre)
    assert_within(to_host(y), g_ref, ulp(g_ref, fmt), "gelu epilogue")
    # backward: every reduction a multiple of 64, outputs ragged w.r.t. the tiles
    M, N, K = 2112, 448, 320
    x, w = _rand((M, K), fmt, 44), _rand((N, K), fmt, 45, 0.05)
    dy, xpre = _rand((M, N), fmt, 46), _rand((M, K), fmt, 47)
    tx, tw, tdy, txp = (to_dev_half(a, fmt) for a in (x, w, dy, xpre))
    gdx, gdw = _empty((M, K), fmt), _empty((N, K), fmt)
    ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), txp.data_ptr(),
                      mx.MPX_ACT_GELU_TANH, gdx.data_ptr(), gdw.data_ptr(), None, M, N, K, dt,
                      ws.data_ptr(), ws_n, None, _s())
    rdx, rdw, _ = ops.linear_bwd(pol, x, w, dy)
    assert_within(to_host(gdw), rdw, gemm_bound(dy.T, x, rdw, fmt, M), "dW")
    ref = ops.gelu_bwd(pol, xpre, rdx)
    assert_within(to_host(gdx), ref, 1.13 * gemm_bound(dy, w, rdx, fmt, N) + ulp(ref, fmt),
                  "dX through gelu'")
    # batched, both transposed layouts, head dim 64 and 128 tokens
    B, H, T, hd = 2, 2, 128, 64
    d = H * hd
    qkv = _rand((B * T, 3 * d), fmt, 48)
    tq = to_dev_half(qkv, fmt)
    e = tq.element_size()
    q, k, v = ops.split_heads(qkv, B, T, H, hd)
    out_s, out_o = _empty((B * H * T, T), fmt), _empty((B * T, d), fmt)
    mx.mpx_gemm_batched(0, 1, T, T, hd, B, H, tq.data_ptr(), 3 * d, T * 3 * d, hd,
                        tq.data_ptr() + d * e, 3 * d, T * 3 * d, hd,
                        out_s.data_ptr(), T, H * T * T, T * T, dt, _s())
    k_t = np.swapaxes(k, -1, -2)
    ref = pol.R(pol.mm(q, k_t))
    bnd = ulp(ref, fmt) + 2 * hd * 2.0 ** -24 * (np.abs(q.astype(np.float64)) @ np.abs(k_t.astype(np.float64)))
    assert_within(to_host(out_s).reshape(B, H, T, T), ref, bnd, "QK^T")
    # K^T V-like product: both operands mn-major (trans_a = 1, trans_b = 0)
    mx.mpx_gemm_batched(1, 0, hd, hd, T, B, H, tq.data_ptr() + d * e, 3 * d, T * 3 * d, hd,
                        tq.data_ptr() + 2 * d * e, 3 * d, T * 3 * d, hd,
                        out_o.data_ptr(), d, T * d, hd, dt, _s())
    kt_v = pol.R(pol.mm(k_t, v))
    bnd = ulp(kt_v, fmt) + 2 * T * 2.0 ** -24 * (np.abs(k_t.astype(np.float64)) @ np.abs(v.astype(np.float64)))
    got = to_host(out_o).reshape(B, T, H, hd)[:, :hd].transpose(0, 2, 1, 3)
    assert_within(got, kt_v, bnd, "K^T V")


@pytest.mark.parametrize("persistent,plain", [(10, 7), (11, 9)])
@pytest.mark.parametrize("fmt", FMTS)
def test_persistent_configs_walk_many_tiles(fmt, persistent, plain):
    """The persistent configurations on outputs with more tiles than the grid
    has workgroups (each walks 2 or 3 tiles, ragged edges included): bit-equal
    to the same tile shape launched one workgroup per tile, and sampled
    outputs within the GEMM bar of the oracle.  Forward with bias + GELU and
    dX through GELU', the two epilogues with an LDS-staged variant."""
    pol = Policy(fmt)
    dt = mx.DTYPES[fmt]
    M, N, K = 4200, 2100, 192
    x, w, b = _rand((M, K), fmt, 61), _rand((N, K), fmt, 62, 0.05), _rand((N,), fmt, 63, 0.5)
    dy, xpre = _rand((M, N), fmt, 64), _rand((M, K), fmt, 65)
    tx, tw, tb, tdy, txp = (to_dev_half(a, fmt) for a in (x, w, b, dy, xpre))
    out = {}
    try:
        for cfg in (plain, persistent):
            mx.mpx_gemm_set_config(cfg)
            y, pre, gdx = _empty((M, N), fmt), _empty((M, N), fmt), _empty((M, K), fmt)
            mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), tb.data_ptr(), None, y.data_ptr(),
                              pre.data_ptr(), M, N, K, dt, mx.MPX_ACT_GELU_TANH, _s())
            mx.mpx_linear_bwd(None, tw.data_ptr(), tdy.data_ptr(), txp.data_ptr(),
                              mx.MPX_ACT_GELU_TANH, gdx.data_ptr(), None, None, M, N, K, dt,
                              None, 0, None, _s())
            torch.cuda.synchronize()
            out[cfg] = (y, pre, gdx)
    finally:
        mx.mpx_gemm_set_config(0)
    for a, c, what in zip(out[plain], out[persistent], ("Y", "pre-activation", "dX")):
        assert torch.equal(a, c), what
    rng = np.random.default_rng(7)
    rows, cols = np.unique(rng.integers(0, M, 40)), np.unique(rng.integers(0, N, 40))
    ref = ops.linear_fwd(pol, x[rows], w[cols], b[cols])
    assert_within(to_host(out[persistent][1])[np.ix_(rows, cols)], ref,
                  gemm_bound(x[rows], w[cols].T, ref, fmt, K), "pre-activation")
    kc = np.unique(rng.integers(0, K, 40))
    rdx = pol.gemm(dy[rows], w[:, kc])
    ref = ops.gelu_bwd(pol, xpre[np.ix_(rows, kc)], rdx)
    assert_within(to_host(out[persistent][2])[np.ix_(rows, kc)], ref,
                  1.13 * gemm_bound(dy[rows], w[:, kc], rdx, fmt, N) + ulp(ref, fmt), "dX")


@pytest.mark.parametrize("fmt", FMTS)
def test_skinny_path_forced(fmt):
    """The one-wave / one-lane-per-output path (configuration 8) on shapes that
    are not skinny, both reduction branches and all operand layouts."""
    pol = Policy(fmt)
    dt = mx.DTYPES[fmt]
    mx.mpx_gemm_set_config(8)
    try:
        for (M, N, K) in [(70, 100, 72), (300, 50, 16), (64, 96, 40)]:
            x, w = _rand((M, K), fmt, 51), _rand((N, K), fmt, 52, 0.05)
            b, dy = _rand((N,), fmt, 53, 0.5), _rand((M, N), fmt, 54)
            tx, tw, tb, tdy = (to_dev_half(a, fmt) for a in (x, w, b, dy))
            y, gdx, gdw = _empty((M, N), fmt), _empty((M, K), fmt), _empty((N, K), fmt)
            mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), tb.data_ptr(), None, y.data_ptr(), None,
                              M, N, K, dt, mx.MPX_ACT_NONE, _s())
            ref = ops.linear_fwd(pol, x, w, b)
            assert_within(to_host(y), ref, gemm_bound(x, w.T, ref, fmt, K), f"Y {M}x{N}x{K}")
            ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
            ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
            mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), None, mx.MPX_ACT_NONE,
                              gdx.data_ptr(), gdw.data_ptr(), None, M, N, K, dt, ws.data_ptr(), ws_n, None,
                              _s())
            rdx, rdw, _ = ops.linear_bwd(pol, x, w, dy)
            assert_within(to_host(gdx), rdx, gemm_bound(dy, w, rdx, fmt, N), f"dX {M}x{N}x{K}")
            assert_within(to_host(gdw), rdw, gemm_bound(dy.T, x, rdw, fmt, M), f"dW {M}x{N}x{K}")
    finally:
        mx.mpx_gemm_set_config(0)


@pytest.mark.parametrize("fmt", FMTS)
def test_linear_bwd_subsets_match_full_call(fmt):
    """dX alone (no workspace) and dW + db alone, as the two-stream backward
    issues them, give the bits of the full call; an empty request is rejected."""
    M, N, K = 2112, 448, 320
    dt = mx.DTYPES[fmt]
    x, w = _rand((M, K), fmt, 61), _rand((N, K), fmt, 62, 0.05)
    dy, xp = _rand((M, N), fmt, 63), _rand((M, K), fmt, 64)
    tx, tw, tdy, txp = (to_dev_half(a, fmt) for a in (x, w, dy, xp))
    full = [_empty((M, K), fmt), _empty((N, K), fmt), _empty((N,), fmt)]
    part = [_empty((M, K), fmt), _empty((N, K), fmt), _empty((N,), fmt)]
    ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), txp.data_ptr(),
                      mx.MPX_ACT_GELU_TANH, *(t.data_ptr() for t in full), M, N, K, dt,
                      ws.data_ptr(), ws_n, None, _s())
    mx.mpx_linear_bwd(None, tw.data_ptr(), tdy.data_ptr(), txp.data_ptr(), mx.MPX_ACT_GELU_TANH,
                      part[0].data_ptr(), None, None, M, N, K, dt, None, 0, None, _s())
    mx.mpx_linear_bwd(tx.data_ptr(), None, tdy.data_ptr(), None, mx.MPX_ACT_NONE, None,
                      part[1].data_ptr(), part[2].data_ptr(), M, N, K, dt, ws.data_ptr(), ws_n, None, _s())
    for f, q, what in zip(full, part, ("dX", "dW", "db")):
        assert torch.equal(f, q), what
    with pytest.raises(mx.MPXError, match="nothing to compute"):
        mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), None, 0, None, None, None,
                          M, N, K, dt, ws.data_ptr(), ws_n, None, _s())
    with pytest.raises(mx.MPXError, match="workspace"):
        mx.mpx_linear_bwd(tx.data_ptr(), None, tdy.data_ptr(), None, 0, None, part[1].data_ptr(),
                          None, M, N, K, dt, None, 0, None, _s())


# ------------------------------------------- full precision (MPX_F32) --

def _dev32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _rand32(shape, seed, std=1.0):
    return np.random.default_rng(seed).normal(0, std, size=shape).astype(np.float32)


def _zeros32(*shape):
    return torch.zeros(*shape, dtype=torch.float32, device="cuda")


# hardware exp2 / reciprocal inside GELU and GELU': a few float32 ulps
GELU_F32_REL = 4e-6


@pytest.mark.parametrize("mnk", [(64, 1024, 512), (70, 100, 72), (33, 17, 50), (300, 200, 1000),
                                 (4096, 384, 384), (129, 130, 131), (1, 8, 8)],
                         ids=lambda s: "x".join(map(str, s)))
def test_linear_f32_matches_full_precision_oracle(mnk):
    """Full-precision training (mixed precision switched off): the float32
    products, their epilogues and the bias sums against the oracle's float32
    policy, within the bound of two float32 summation orders."""
    M, N, K = mnk
    pol = Policy("f32")
    F32 = mx.MPX_F32
    x, w, b, r = _rand32((M, K), 1), _rand32((N, K), 2, 0.05), _rand32((N,), 3, 0.5), _rand32((M, N), 4)
    tx, tw, tb, tr = (_dev32(a) for a in (x, w, b, r))
    y, pre = _zeros32(M, N), _zeros32(M, N)
    ref = ops.linear_fwd(pol, x, w, b)
    bnd = gemm_bound(x, w.T, ref, "f32", K) + ulp(ref, "f32")
    mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), tb.data_ptr(), None, y.data_ptr(), None, M, N, K,
                      F32, mx.MPX_ACT_NONE, _s())
    assert_within(to_host(y), ref, bnd, "Y")
    mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), tb.data_ptr(), None, y.data_ptr(), pre.data_ptr(),
                      M, N, K, F32, mx.MPX_ACT_GELU_TANH, _s())
    gpre = to_host(pre)
    assert_within(gpre, ref, bnd, "pre-activation")
    gref = ops.gelu_fwd(pol, gpre)
    assert_within(to_host(y), gref, GELU_F32_REL * np.abs(gref) + ulp(gref, "f32"), "GELU")
    mx.mpx_linear_fwd(tx.data_ptr(), tw.data_ptr(), tb.data_ptr(), tr.data_ptr(), y.data_ptr(), None,
                      M, N, K, F32, mx.MPX_ACT_NONE, _s())
    rref = ops.add(pol, ref, r)
    assert_within(to_host(y), rref, bnd + ulp(rref, "f32"), "Y + R")
    # backward
    dy, xp = _rand32((M, N), 13), _rand32((M, K), 14)
    tdy, txp = _dev32(dy), _dev32(xp)
    gdx, gdw, gdb = _zeros32(M, K), _zeros32(N, K), _zeros32(N)
    ws_n = mx.mpx_linear_bwd_workspace(M, N, K)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), None, mx.MPX_ACT_NONE,
                      gdx.data_ptr(), gdw.data_ptr(), gdb.data_ptr(), M, N, K, F32, ws.data_ptr(), ws_n,
                      None, _s())
    rdx, rdw, rdb = ops.linear_bwd(pol, x, w, dy)
    assert_within(to_host(gdx), rdx, gemm_bound(dy, w, rdx, "f32", N), "dX")
    assert_within(to_host(gdw), rdw, gemm_bound(dy.T, x, rdw, "f32", M), "dW")
    colb = ulp(rdb, "f32") + 2.0 * M * 2.0 ** -24 * np.abs(dy.astype(np.float64)).sum(axis=0)
    assert_within(to_host(gdb), rdb, colb, "db")
    mx.mpx_linear_bwd(tx.data_ptr(), tw.data_ptr(), tdy.data_ptr(), txp.data_ptr(),
                      mx.MPX_ACT_GELU_TANH, gdx.data_ptr(), None, None, M, N, K, F32, ws.data_ptr(),
                      ws_n, None, _s())
    gref = ops.gelu_bwd(pol, xp, rdx)
    bound = 1.13 * gemm_bound(dy, w, rdx, "f32", N) + GELU_F32_REL * np.abs(gref) + ulp(gref, "f32")
    assert_within(to_host(gdx), gref, bound, "dX through gelu'")
    with pytest.raises(mx.MPXError, match="half gradients only"):
        nf = torch.zeros(1, dtype=torch.int32, device="cuda")
        mx.mpx_linear_bwd(tx.data_ptr(), None, tdy.data_ptr(), None, 0, None, gdw.data_ptr(), None,
                          M, N, K, F32, ws.data_ptr(), ws_n, nf.data_ptr(), _s())


@pytest.mark.parametrize("tr", [(0, 1), (0, 0), (1, 0)])
def test_gemm_batched_f32(tr):
    """The attention products of full-precision training (per-head strided
    operands of a fused QKV activation), against float64 products."""
    ta, tb = tr
    B, H, T, hd = 3, 2, 65, 64
    M, N, K = (T, T, hd) if (ta, tb) == (0, 1) else (T, hd, T)
    rng = np.random.default_rng(sum(tr))
    A = rng.normal(size=(B, H, M, K) if not ta else (B, H, K, M)).astype(np.float32)
    Bm = rng.normal(size=(B, H, N, K) if tb else (B, H, K, N)).astype(np.float32)
    a, b = A.reshape(B * H, *A.shape[2:]), Bm.reshape(B * H, *Bm.shape[2:])
    opa = a.transpose(0, 2, 1) if ta else a
    opb = b.transpose(0, 2, 1) if tb else b
    ref = np.matmul(opa.astype(np.float64), opb.astype(np.float64))
    tA, tB = _dev32(A), _dev32(Bm)
    C = _zeros32(B, H, M, N)
    lda, ldb = A.shape[-1], Bm.shape[-1]
    mx.mpx_gemm_batched(ta, tb, M, N, K, B, H, tA.data_ptr(), lda, H * A.shape[2] * lda, A.shape[2] * lda,
                        tB.data_ptr(), ldb, H * Bm.shape[2] * ldb, Bm.shape[2] * ldb,
                        C.data_ptr(), N, H * M * N, M * N, mx.MPX_F32, _s())
    got = to_host(C).reshape(B * H, M, N)
    bound = ulp(ref, "f32") + 2.0 * K * 2.0 ** -24 * np.matmul(np.abs(opa).astype(np.float64),
                                                               np.abs(opb).astype(np.float64))
    assert_within(got, ref, bound, "batched f32")
