"""GPU parity of the support ops (full-precision islands and embedding data
movement) against the oracle, through the C ABI.

The GPU computes these ops in float32, the oracle in float64; both round once
to half, so outputs agree within one half ulp (exactly, for data movement).
Column sums (LayerNorm dgamma/dbeta, embedding dpos/dcls) also carry a float32
summation-order term.
"""
import math

import numpy as np
import pytest

from oracle import ops
from oracle.numfmt import round_to
from oracle.policy import Policy
from tests.gpu_util import (HAVE_GPU, assert_same_values, assert_within, gemm_bound, to_dev_half,
                            to_host, ulp)

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="no GPU")]

if HAVE_GPU:
    import torch
    from paper_2507_03312_amd import binding as mx

FMTS = ["f16", "bf16"]


def _s():
    return torch.cuda.current_stream().cuda_stream


def _rand(shape, fmt, seed, std=1.0, mean=0.0):
    return round_to(np.random.default_rng(seed).normal(mean, std, size=shape), fmt)


def _empty(shape, fmt):
    return torch.zeros(*shape, dtype=torch.float16 if fmt == "f16" else torch.bfloat16, device="cuda")


def _sum_bound(x, fmt, ref):
    return 2 * ulp(ref, fmt) + 2.0 * x.shape[0] * 2.0 ** -24 * np.abs(x.astype(np.float64)).sum(axis=0)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("rows,d", [(130, 384), (7, 768), (33, 100), (5, 2048), (8321, 384), (3001, 768)])
def test_layernorm_fwd_bwd(fmt, rows, d):
    pol = Policy(fmt)
    x = _rand((rows, d), fmt, 1, 2.0, 0.5)
    g = _rand((d,), fmt, 2, 0.2, 1.0)
    b = _rand((d,), fmt, 3, 0.2)
    dy = _rand((rows, d), fmt, 4)
    rg = _rand((rows, d), fmt, 5)
    tx, tg, tb, tdy, trg = (to_dev_half(a, fmt) for a in (x, g, b, dy, rg))
    y = _empty((rows, d), fmt)
    dt = mx.DTYPES[fmt]
    mx.mpx_layernorm_fwd(tx.data_ptr(), d, tg.data_ptr(), tb.data_ptr(), y.data_ptr(), None,
                         rows, d, dt, _s())
    ref = ops.layernorm_fwd(pol, x, g, b)
    # float32 evaluation of xhat*g + b: a few float32 ulps of |xhat*g| + |b| (matters
    # where the two cancel to a tiny result) plus one half ulp of the result
    xh = ops.layernorm_fwd(Policy("f64"), x, np.ones(d), np.zeros(d))
    f32_err = 2.0 ** -21 * (np.abs(xh * g.astype(np.float64)) + np.abs(b.astype(np.float64)))
    assert_within(to_host(y), ref, ulp(ref, fmt) + f32_err, "LN fwd")
    dx, dg, db = _empty((rows, d), fmt), _empty((d,), fmt), _empty((d,), fmt)
    wsn = mx.mpx_layernorm_bwd_workspace(rows, d)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), trg.data_ptr(),
                         dx.data_ptr(), d, dg.data_ptr(), db.data_ptr(), rows, d, dt,
                         ws.data_ptr(), wsn, None, _s())
    rdx, rdg, rdb = ops.layernorm_bwd(pol, x, g, dy)
    rtot = ops.add(pol, rg, rdx)
    assert_within(to_host(dx), rtot, 2 * ulp(rtot, fmt) + ulp(rdx, fmt) + 1e-4 * np.abs(rdx), "LN dX")
    xhat_abs = np.abs(ops.layernorm_fwd(Policy("f64"), x, np.ones(d), np.zeros(d)))
    assert_within(to_host(dg), rdg, _sum_bound(dy * xhat_abs, fmt, rdg) + 1e-4 * np.abs(rdg), "LN dgamma")
    assert_within(to_host(db), rdb, _sum_bound(dy, fmt, rdb), "LN dbeta")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("B,T,d", [(64, 197, 768), (5, 3, 12)])
def test_embed_assemble_bwd_vector_form_matches_scalar_form(fmt, B, T, d):
    """The token-assembly backward on 8-byte aligned operands (4 outputs per
    lane from 65536 outputs T d on) and on a cotangent one element off that
    alignment (one output per lane) sum in the same order: dpos, dcls, dE and
    the non-finite count agree bit for bit, with overflowing columns
    included (the small shape takes the one-output form both times)."""
    dX = _rand((B * T, d), fmt, 41, 100.0)
    big = 60000.0 if fmt == "f16" else 3e38
    dX[:, 0] = big  # column 0 (a CLS and a patch position) overflows when summed
    flat = np.concatenate([np.zeros(1, np.float32), dX.reshape(-1)])
    tflat = to_dev_half(flat, fmt)
    t_al = tflat[1:].clone()              # 8-byte aligned copy
    outs = []
    for src in (t_al, tflat[1:]):         # the view is 2 bytes off
        dE, dcls, dpos = _empty((B * (T - 1), d), fmt), _empty((d,), fmt), _empty((T, d), fmt)
        nf = torch.zeros(1, dtype=torch.int32, device="cuda")
        mx.mpx_embed_assemble_bwd(src.data_ptr(), dE.data_ptr(), dcls.data_ptr(), dpos.data_ptr(), B, T, d,
                                  mx.DTYPES[fmt], nf.data_ptr(), _s())
        torch.cuda.synchronize()
        outs.append((dE, dcls, dpos, int(nf.item())))
    (e1, c1, p1, n1), (e2, c2, p2, n2) = outs
    for a, b_, what in ((e1, e2, "dE"), (c1, c2, "dcls"), (p1, p2, "dpos")):
        assert torch.equal(a.view(torch.int16), b_.view(torch.int16)), what
    assert n1 == n2 and n1 >= T + 1


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("rows,d", [(12608, 768), (16640, 384), (37, 768), (9, 384), (1, 768), (3, 384)])
def test_layernorm_row_groups_match_one_wave_rows(fmt, rows, d):
    """At d = 384 and 768 with 16-byte aligned rows, the forward and the
    dX-only backward give each row 16 or 32 lanes; the same values with rows
    4 halves apart (ldx = d + 4) take the one-wave-per-row kernels.  The two
    sum in the same order, so every output bit agrees: normal rows, a
    constant row (zero variance), an all-zero row, an all -0 row, and row
    counts that leave the last wave partly empty."""
    x = _rand((rows, d), fmt, 31, 2.0, 0.5)
    x[0] = 0.0
    if rows > 1:
        x[1] = 3.0
    if rows > 2:
        x[2] = -0.0
    g, b = _rand((d,), fmt, 32, 0.2, 1.0), _rand((d,), fmt, 33, 0.2)
    dy, rg = _rand((rows, d), fmt, 34), _rand((rows, d), fmt, 35)
    tx, tg, tb, tdy, trg = (to_dev_half(a, fmt) for a in (x, g, b, dy, rg))
    wide = _empty((rows, d + 4), fmt)
    wide[:, :d] = tx
    dt = mx.DTYPES[fmt]
    y1, y2 = _empty((rows, d), fmt), _empty((rows, d), fmt)
    mr1 = torch.zeros(2 * rows, dtype=torch.float32, device="cuda")
    mr2 = torch.zeros_like(mr1)
    mx.mpx_layernorm_fwd(tx.data_ptr(), d, tg.data_ptr(), tb.data_ptr(), y1.data_ptr(), mr1.data_ptr(),
                         rows, d, dt, _s())
    mx.mpx_layernorm_fwd(wide.data_ptr(), d + 4, tg.data_ptr(), tb.data_ptr(), y2.data_ptr(),
                         mr2.data_ptr(), rows, d, dt, _s())
    for res in (None, trg):
        dx1, dx2 = _empty((rows, d), fmt), _empty((rows, d), fmt)
        rp = None if res is None else res.data_ptr()
        mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), rp, dx1.data_ptr(), d,
                             None, None, rows, d, dt, None, 0, None, _s())
        mx.mpx_layernorm_bwd(wide.data_ptr(), d + 4, tg.data_ptr(), tdy.data_ptr(), rp, dx2.data_ptr(), d,
                             None, None, rows, d, dt, None, 0, None, _s())
        torch.cuda.synchronize()
        assert torch.equal(dx1.view(torch.int16), dx2.view(torch.int16)), ("dX", res is None)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16)), "Y"
    assert torch.equal(mr1.view(torch.int32), mr2.view(torch.int32)), "mean / rstd"


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("rows,d", [(8321, 384), (12608, 768), (37, 768), (1000, 256)])
def test_layernorm_bwd_subsets_match_full_call(fmt, rows, d):
    """dX alone (no workspace) and dgamma / dbeta alone, as the two-stream
    backward issues them, give the bits of the full call (row groups at
    d = 384 and 768, one wave per row at d = 256)."""
    x = _rand((rows, d), fmt, 11, 2.0, 0.5)
    g = _rand((d,), fmt, 12, 0.2, 1.0)
    dy, rg = _rand((rows, d), fmt, 13), _rand((rows, d), fmt, 14)
    tx, tg, tdy, trg = (to_dev_half(a, fmt) for a in (x, g, dy, rg))
    dt = mx.DTYPES[fmt]
    full = [_empty((rows, d), fmt), _empty((d,), fmt), _empty((d,), fmt)]
    part = [_empty((rows, d), fmt), _empty((d,), fmt), _empty((d,), fmt)]
    wsn = mx.mpx_layernorm_bwd_workspace(rows, d)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), trg.data_ptr(),
                         full[0].data_ptr(), d, full[1].data_ptr(), full[2].data_ptr(), rows, d, dt,
                         ws.data_ptr(), wsn, None, _s())
    mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), trg.data_ptr(),
                         part[0].data_ptr(), d, None, None, rows, d, dt, None, 0, None, _s())
    mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), None, None, d,
                         part[1].data_ptr(), part[2].data_ptr(), rows, d, dt, ws.data_ptr(), wsn, None, _s())
    for f, q, what in zip(full, part, ("dX", "dgamma", "dbeta")):
        assert torch.equal(f, q), what
    with pytest.raises(mx.MPXError, match="nothing to compute"):
        mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), None, None, d, None,
                             None, rows, d, dt, None, 0, None, _s())
    with pytest.raises(mx.MPXError, match="together"):
        mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), None, None, d,
                             part[1].data_ptr(), None, rows, d, dt, ws.data_ptr(), wsn, None, _s())


def test_layernorm_strided_rows_cls_pooling():
    """Final LayerNorm on the CLS rows of a [B, T, d] token matrix."""
    fmt, B, T, d = "bf16", 6, 5, 384
    pol = Policy(fmt)
    x = _rand((B, T, d), fmt, 7)
    g, b = _rand((d,), fmt, 8, 0.1, 1.0), _rand((d,), fmt, 9, 0.1)
    tx, tg, tb = (to_dev_half(a, fmt) for a in (x, g, b))
    z = _empty((B, d), fmt)
    mx.mpx_layernorm_fwd(tx.data_ptr(), T * d, tg.data_ptr(), tb.data_ptr(), z.data_ptr(), None,
                         B, d, mx.MPX_BF16, _s())
    ref = ops.layernorm_fwd(pol, x[:, 0, :], g, b)
    assert_within(to_host(z), ref, ulp(ref, fmt), "LN CLS rows")
    dz = _rand((B, d), fmt, 10)
    tdz = to_dev_half(dz, fmt)
    dx = _empty((B * T, d), fmt)
    dx.fill_(7.0)
    dg, db = _empty((d,), fmt), _empty((d,), fmt)
    wsn = mx.mpx_layernorm_bwd_workspace(B, d)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_layernorm_bwd(tx.data_ptr(), T * d, tg.data_ptr(), tdz.data_ptr(), None, dx.data_ptr(),
                         T * d, dg.data_ptr(), db.data_ptr(), B, d, mx.MPX_BF16, ws.data_ptr(), wsn, None, _s())
    got = to_host(dx).reshape(B, T, d)
    rdx, _, _ = ops.layernorm_bwd(pol, x[:, 0, :], g, dz)
    assert_within(got[:, 0, :], rdx, ulp(rdx, fmt) + 1e-4 * np.abs(rdx), "LN dX CLS rows")
    assert np.all(got[:, 1:, :] == 7.0), "rows outside the CLS rows must not be written"


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("T", [65, 197, 5])
def test_softmax_fwd_bwd(fmt, T):
    pol = Policy(fmt)
    rows = 37
    ld = -(-T // 8) * 8
    s = np.zeros((rows, ld), np.float32)
    s[:, :T] = _rand((rows, T), fmt, 1, 3.0)
    dp = np.zeros((rows, ld), np.float32)
    dp[:, :T] = _rand((rows, T), fmt, 2)
    ts, tdp = to_dev_half(s, fmt), to_dev_half(dp, fmt)
    p = _empty((rows, ld), fmt)
    p.fill_(3.0)
    scale = 1.0 / math.sqrt(64)
    mx.mpx_softmax_fwd(ts.data_ptr(), p.data_ptr(), rows, T, ld, scale, mx.DTYPES[fmt], _s())
    gp = to_host(p)
    ref = ops.softmax_fwd(pol, s[:, :T], scale)
    assert_within(gp[:, :T], ref, ulp(ref, fmt), "softmax")
    assert np.all(gp[:, T:] == 0)
    ds = _empty((rows, ld), fmt)
    tp = to_dev_half(gp, fmt)
    mx.mpx_softmax_bwd(tp.data_ptr(), tdp.data_ptr(), ds.data_ptr(), rows, T, ld, scale,
                       mx.DTYPES[fmt], _s())
    ref = ops.softmax_bwd(pol, gp[:, :T], dp[:, :T], scale)
    got = to_host(ds)
    dot = np.abs((dp[:, :T].astype(np.float64) * gp[:, :T]).sum(axis=1, keepdims=True))
    bnd = ulp(ref, fmt) + 1e-5 * scale * np.abs(gp[:, :T]) * (np.abs(dp[:, :T]) + dot)
    assert_within(got[:, :T], ref, bnd, "softmax bwd")
    assert np.all(got[:, T:] == 0)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("B,C", [(64, 1000), (256, 100), (3, 10)])
def test_cross_entropy(fmt, B, C):
    from paper_2507_03312_amd.train import pack_scale_state
    pol = Policy(fmt)
    z = _rand((B, C), fmt, 3, 2.0)
    y = np.random.default_rng(4).integers(0, C, B).astype(np.int32)
    scale = 2.0 ** 15
    tz = to_dev_half(z, fmt)
    ty = torch.from_numpy(y).cuda()
    st = torch.from_numpy(pack_scale_state(scale, 0, 10)).cuda()
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dz = _empty((B, C), fmt)
    wsn = mx.mpx_loss_workspace(B)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_cross_entropy(tz.data_ptr(), C, ty.data_ptr(), B, C, st.data_ptr(), loss.data_ptr(),
                         dz.data_ptr(), mx.DTYPES[fmt], ws.data_ptr(), wsn, _s())
    rl, rdz = ops.ce_fwd_bwd(pol, z, y, scale)
    assert abs(float(loss.item()) - rl) <= 1e-5 * abs(rl)
    assert_within(to_host(dz), rdz, ulp(rdz, fmt) + 1e-5 * np.abs(rdz), "CE cotangent")


@pytest.mark.parametrize("fmt", FMTS)
def test_mse(fmt):
    from paper_2507_03312_amd.train import pack_scale_state
    pol = Policy(fmt)
    yv, tv = _rand((64, 512), fmt, 5), _rand((64, 512), fmt, 6)
    st = torch.from_numpy(pack_scale_state(2.0 ** 15, 0, 4)).cuda()
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dy = _empty((64, 512), fmt)
    ty, tt = to_dev_half(yv, fmt), to_dev_half(tv, fmt)
    wsn = mx.mpx_loss_workspace(yv.size)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_mse(ty.data_ptr(), tt.data_ptr(), yv.size, st.data_ptr(), loss.data_ptr(), dy.data_ptr(),
               mx.DTYPES[fmt], ws.data_ptr(), wsn, _s())
    rl, rdy = ops.mse_fwd_bwd(pol, yv, tv, 2.0 ** 15)
    assert abs(float(loss.item()) - rl) <= 1e-5 * rl
    assert_within(to_host(dy), rdy, ulp(rdy, fmt), "MSE cotangent")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("B,Hh,C,p,d", [(3, 8, 3, 4, 16), (9, 32, 3, 4, 384), (2, 48, 3, 16, 100),
                                         (2, 64, 3, 16, 768), (3, 8, 3, 4, 50)],
                         ids=lambda v: str(v))
def test_patchify_embed_assemble_and_backward(fmt, B, Hh, C, p, d):
    pol = Policy(fmt)
    G = (Hh // p) ** 2
    T = G + 1
    img = np.random.default_rng(1).uniform(0, 1, (B, Hh, Hh, C)).astype(np.float32)
    timg = torch.from_numpy(img).cuda()
    pt = _empty((B * G, p * p * C), fmt)
    mx.mpx_patchify_cast(timg.data_ptr(), pt.data_ptr(), B, Hh, Hh, C, p, mx.DTYPES[fmt], _s())
    assert_same_values(to_host(pt), pol.R(ops.patchify(img, p)), "patchify")
    E = _rand((B * G, d), fmt, 2)
    cls = _rand((d,), fmt, 3)
    pos = _rand((T, d), fmt, 4)
    tE, tc, tpos = (to_dev_half(a, fmt) for a in (E, cls, pos))
    X = _empty((B * T, d), fmt)
    mx.mpx_embed_assemble(tE.data_ptr(), tc.data_ptr(), tpos.data_ptr(), X.data_ptr(), B, T, d,
                          mx.DTYPES[fmt], _s())
    ref = np.empty((B, T, d), np.float32)
    ref[:, 0] = ops.add(pol, cls, pos[0])
    ref[:, 1:] = ops.add(pol, E.reshape(B, G, d), pos[None, 1:])
    assert_same_values(to_host(X).reshape(B, T, d), ref, "embed assemble")
    dX = _rand((B * T, d), fmt, 5)
    tdX = to_dev_half(dX, fmt)
    dE, dcls, dpos = _empty((B * G, d), fmt), _empty((d,), fmt), _empty((T, d), fmt)
    mx.mpx_embed_assemble_bwd(tdX.data_ptr(), dE.data_ptr(), dcls.data_ptr(), dpos.data_ptr(), B,
                              T, d, mx.DTYPES[fmt], None, _s())
    d3 = dX.reshape(B, T, d)
    assert_same_values(to_host(dE), d3[:, 1:].reshape(B * G, d), "dE")
    rpos = pol.R(d3.astype(np.float64).sum(axis=0))
    assert_within(to_host(dpos), rpos, _sum_bound(d3.reshape(B, -1), fmt, rpos.reshape(-1)).reshape(T, d), "dpos")
    assert_same_values(to_host(dcls), to_host(dpos)[0], "dcls")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("B,T,d,C", [(128, 65, 384, 10), (5, 3, 100, 7), (33, 2, 512, 32),
                                     (2, 1, 2048, 8)], ids=lambda v: str(v))
def test_classifier_head_matches_separate_calls(fmt, B, T, d, C):
    """The fused classifier head (final LayerNorm on the CLS rows, linear,
    cross-entropy with the scaled seed, backward to the LayerNorm input and
    gamma / beta) gives the bits of the separate calls, each of which is
    checked against the oracle above; at the widths where the separate
    LayerNorm backward works in row groups its gamma / beta sums add the same
    terms in another grouping and agree within that reordering's bound."""
    from paper_2507_03312_amd.train import pack_scale_state
    dt = mx.DTYPES[fmt]
    x = _rand((B * T, d), fmt, 21, 2.0, 0.5)
    g, be = _rand((d,), fmt, 22, 0.2, 1.0), _rand((d,), fmt, 23, 0.2)
    w, bias = _rand((C, d), fmt, 24, 0.05), _rand((C,), fmt, 25, 0.5)
    y = np.random.default_rng(26).integers(0, C, B).astype(np.int32)
    tx, tg, tb, tw, tbias = (to_dev_half(a, fmt) for a in (x, g, be, w, bias))
    ty = torch.from_numpy(y).cuda()
    st = torch.from_numpy(pack_scale_state(2.0 ** 15, 0, 10)).cuda()
    ld = T * d

    def outs():
        return ([_empty((B, d), fmt), _empty((B, C), fmt), _empty((B * T, d), fmt), _empty((d,), fmt),
                 _empty((d,), fmt)], torch.zeros(1, dtype=torch.float32, device="cuda"))

    (z1, dl1, dx1, dg1, db1), loss1 = outs()
    wsn = mx.mpx_classifier_head_workspace(B, d)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_classifier_head(tx.data_ptr(), ld, tg.data_ptr(), tb.data_ptr(), tw.data_ptr(),
                           tbias.data_ptr(), ty.data_ptr(), B, d, C, st.data_ptr(), z1.data_ptr(),
                           loss1.data_ptr(), dl1.data_ptr(), dx1.data_ptr(), ld, dg1.data_ptr(),
                           db1.data_ptr(), dt, ws.data_ptr(), wsn, None, _s())

    (z2, dl2, dx2, dg2, db2), loss2 = outs()
    logits, dz = _empty((B, C), fmt), _empty((B, d), fmt)
    ws2n = max(mx.mpx_loss_workspace(B), mx.mpx_layernorm_bwd_workspace(B, d))
    ws2 = torch.zeros(ws2n, dtype=torch.uint8, device="cuda")
    mx.mpx_layernorm_fwd(tx.data_ptr(), ld, tg.data_ptr(), tb.data_ptr(), z2.data_ptr(), None, B, d,
                         dt, _s())
    mx.mpx_linear_fwd(z2.data_ptr(), tw.data_ptr(), tbias.data_ptr(), None, logits.data_ptr(), None,
                      B, C, d, dt, mx.MPX_ACT_NONE, _s())
    mx.mpx_cross_entropy(logits.data_ptr(), C, ty.data_ptr(), B, C, st.data_ptr(), loss2.data_ptr(),
                         dl2.data_ptr(), dt, ws2.data_ptr(), ws2n, _s())
    mx.mpx_linear_bwd(None, tw.data_ptr(), dl2.data_ptr(), None, mx.MPX_ACT_NONE, dz.data_ptr(),
                      None, None, B, C, d, dt, None, 0, None, _s())
    mx.mpx_layernorm_bwd(tx.data_ptr(), ld, tg.data_ptr(), dz.data_ptr(), None, dx2.data_ptr(), ld,
                         dg2.data_ptr(), db2.data_ptr(), B, d, dt, ws2.data_ptr(), ws2n, None, _s())
    torch.cuda.synchronize()
    same = [(z1, z2, "Z"), (dl1, dl2, "dlogits"), (dx1, dx2, "dX"), (loss1, loss2, "loss")]
    if d in (384, 768):
        # the separate LayerNorm backward sums gamma / beta over rows in row
        # groups of 16 or 32 lanes, the head one row per wave: the same float32
        # terms added in another grouping, so a float32 ulp of the magnitude per
        # addition apart before the one rounding to half
        xh = ops.layernorm_fwd(Policy("f64"), x[::T], np.ones(d), np.zeros(d))
        dzv = to_host(dz).astype(np.float64)
        for got, ref, terms, what in ((dg1, dg2, dzv * xh, "dgamma"), (db1, db2, dzv, "dbeta")):
            r = to_host(ref)
            bound = ulp(r, fmt) + B * 2.0 ** -23 * np.abs(terms).sum(axis=0)
            assert_within(to_host(got), r, bound, what)
    else:
        same += [(dg1, dg2, "dgamma"), (db1, db2, "dbeta")]
    for a, b_, what in same:
        assert torch.equal(a, b_), what


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("B,T,d,C", [(128, 65, 384, 10), (33, 2, 512, 32)], ids=lambda v: str(v))
def test_classifier_head_against_oracle(fmt, B, T, d, C):
    """The fused classifier head against the oracle's ops, per element, stage
    by stage: each stage the GPU exposes (Z, dlogits, dX, dgamma, dbeta) is
    compared with the oracle's op on the GPU's own exposed input, and the
    stages it keeps internal (the logits, dZ) enter through their propagated
    bounds:
      Z        = LN(x)                       one half ulp + float32 evaluation
      logits   = half(Z W^T + b)             within the GEMM bound delta of
                                             the oracle's logits from the GPU's Z
      dlogits  = CE cotangent of the logits: a logit error of at most Delta
                 per row moves every softmax probability by a factor within
                 exp(+-2 Delta), so |d dlogits| <= scale/B p (exp(2 Delta) - 1)
                 on top of one ulp and the float32 evaluation term;
      loss     = mean(logsumexp - logit_y):  within mean(2 Delta) + 1e-5 |loss|
      dZ       = half(dlogits W)             within the GEMM bound eps of the
                                             oracle's dZ from the GPU's dlogits
      dX, dgamma, dbeta = LN backward of dZ: the oracle's values plus the
                 linear propagation of eps through the LN backward."""
    from paper_2507_03312_amd.train import pack_scale_state
    pol = Policy(fmt)
    dt = mx.DTYPES[fmt]
    x = _rand((B * T, d), fmt, 31, 2.0, 0.5)
    g, be = _rand((d,), fmt, 32, 0.2, 1.0), _rand((d,), fmt, 33, 0.2)
    w, bias = _rand((C, d), fmt, 34, 0.05), _rand((C,), fmt, 35, 0.5)
    y = np.random.default_rng(36).integers(0, C, B).astype(np.int32)
    scale = 2.0 ** 15
    tx, tg, tb, tw, tbias = (to_dev_half(a, fmt) for a in (x, g, be, w, bias))
    ty = torch.from_numpy(y).cuda()
    st = torch.from_numpy(pack_scale_state(scale, 0, 10)).cuda()
    ld = T * d
    z, dl, dx = _empty((B, d), fmt), _empty((B, C), fmt), _empty((B * T, d), fmt)
    dg, db = _empty((d,), fmt), _empty((d,), fmt)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    wsn = mx.mpx_classifier_head_workspace(B, d)
    ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_classifier_head(tx.data_ptr(), ld, tg.data_ptr(), tb.data_ptr(), tw.data_ptr(),
                           tbias.data_ptr(), ty.data_ptr(), B, d, C, st.data_ptr(), z.data_ptr(),
                           loss.data_ptr(), dl.data_ptr(), dx.data_ptr(), ld, dg.data_ptr(),
                           db.data_ptr(), dt, ws.data_ptr(), wsn, None, _s())
    torch.cuda.synchronize()
    xc = x.reshape(B, T, d)[:, 0, :]
    # Z
    gz = to_host(z)
    rz = ops.layernorm_fwd(pol, xc, g, be)
    xhat = ops.layernorm_fwd(Policy("f64"), xc, np.ones(d), np.zeros(d))
    f32_err = 2.0 ** -21 * (np.abs(xhat * g.astype(np.float64)) + np.abs(be.astype(np.float64)))
    assert_within(gz, rz, ulp(rz, fmt) + f32_err, "head Z")
    # logits (internal) -> dlogits and the loss
    rl = ops.linear_fwd(pol, gz, w, bias)
    delta = np.max(gemm_bound(gz, w.T, rl, fmt, d), axis=1, keepdims=True)      # per row
    rloss, rdl = ops.ce_fwd_bwd(pol, rl, y, scale)
    l64 = rl.astype(np.float64)
    p = np.exp(l64 - l64.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    sens = scale / B * p * np.expm1(2.0 * delta)
    gdl = to_host(dl)
    assert_within(gdl, rdl, ulp(rdl, fmt) + 1e-5 * np.abs(rdl) + sens, "head dlogits")
    assert abs(float(loss.item()) - rloss) <= float(np.mean(2.0 * delta)) + 1e-5 * abs(rloss)
    # dZ (internal) -> dX, dgamma, dbeta
    rdz, _, _ = ops.linear_bwd(pol, gz, w, gdl)
    eps = gemm_bound(gdl, w, rdz, fmt, C)
    rdx, rdg, rdb = ops.layernorm_bwd(pol, xc, g, rdz)
    x64 = xc.astype(np.float64)
    rstd = 1.0 / np.sqrt(x64.var(axis=1, keepdims=True) + 1e-5)
    ge = np.abs(g.astype(np.float64)) * eps
    prop = rstd * (ge + ge.mean(axis=1, keepdims=True)
                   + np.abs(xhat) * (ge * np.abs(xhat)).mean(axis=1, keepdims=True))
    gx = to_host(dx).reshape(B, T, d)
    assert_within(gx[:, 0, :], rdx, 2 * ulp(rdx, fmt) + 1e-4 * np.abs(rdx) + prop, "head dX")
    assert_within(to_host(dg), rdg, _sum_bound(rdz * np.abs(xhat), fmt, rdg) + 1e-4 * np.abs(rdg)
                  + (eps * np.abs(xhat)).sum(axis=0), "head dgamma")
    assert_within(to_host(db), rdb, _sum_bound(rdz, fmt, rdb) + eps.sum(axis=0), "head dbeta")


def test_classifier_head_limits():
    t = _empty((64, 64), "bf16")
    p = t.data_ptr()
    with pytest.raises(mx.MPXError, match="C must be"):
        mx.mpx_classifier_head(p, 64, p, p, p, p, p, 4, 64, 33, p, p, p, p, p, 64, p, p, mx.MPX_BF16,
                               p, 1 << 20, None, _s())
    with pytest.raises(mx.MPXError, match="workspace"):
        mx.mpx_classifier_head(p, 64, p, p, p, p, p, 4, 64, 10, p, p, p, p, p, 64, p, p, mx.MPX_BF16,
                               p, 16, None, _s())


# ------------------------------------------- full precision (MPX_F32) --
# The float32 support ops against the oracle's float32 policy (float64
# inside, one rounding to float32): the GPU's float32 reductions differ from
# that by a few float32 ulps of the row's magnitude.

def _f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _close32(got, ref, scale, rel=2e-6, what=""):
    """|got - ref| <= rel * (|ref| + scale) elementwise (scale: the row's size)."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, what
    err = np.abs(got - ref)
    bnd = rel * (np.abs(ref) + scale)
    assert np.all(err <= bnd), f"{what}: worst {err.max():.3g} (bound {bnd[np.argmax(err - bnd)]:.3g})"


@pytest.mark.parametrize("rows,d", [(130, 384), (7, 768), (65, 100), (33, 1500), (9, 2048)])
def test_layernorm_f32(rows, d):
    pol = Policy("f32")
    rng = np.random.default_rng(rows + d)
    x = rng.normal(0.5, 2.0, size=(rows, d)).astype(np.float32)
    g = rng.normal(1.0, 0.1, size=d).astype(np.float32)
    b = rng.normal(0.0, 0.1, size=d).astype(np.float32)
    dy = rng.normal(0, 1, size=(rows, d)).astype(np.float32)
    r = rng.normal(0, 1, size=(rows, d)).astype(np.float32)
    tx, tg, tb, tdy, tr = (_f32(a) for a in (x, g, b, dy, r))
    y = torch.zeros(rows, d, device="cuda")
    F32 = mx.MPX_F32
    mx.mpx_layernorm_fwd(tx.data_ptr(), d, tg.data_ptr(), tb.data_ptr(), y.data_ptr(), None, rows, d,
                         F32, _s())
    _close32(to_host(y), ops.layernorm_fwd(pol, x, g, b), 4.0, 4e-6, "LN fwd")
    dx = torch.zeros(rows, d, device="cuda")
    dg, db = torch.zeros(d, device="cuda"), torch.zeros(d, device="cuda")
    ws_n = mx.mpx_layernorm_bwd_workspace(rows, d)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), tr.data_ptr(), dx.data_ptr(),
                         d, dg.data_ptr(), db.data_ptr(), rows, d, F32, ws.data_ptr(), ws_n, None, _s())
    rdx, rdg, rdb = ops.layernorm_bwd(pol, x, g, dy)
    _close32(to_host(dx), ops.add(pol, rdx, r), 4.0, 4e-6, "LN dX + R")
    _close32(to_host(dg), rdg, math.sqrt(rows) * 4.0, 4e-6, "dgamma")
    _close32(to_host(db), rdb, math.sqrt(rows) * 4.0, 4e-6, "dbeta")


@pytest.mark.parametrize("rows,n,ld", [(300, 65, 72), (20, 197, 200), (4, 1024, 1024)])
def test_softmax_f32(rows, n, ld):
    pol = Policy("f32")
    rng = np.random.default_rng(n)
    s = rng.normal(0, 3, size=(rows, ld)).astype(np.float32)
    dp = rng.normal(0, 1, size=(rows, ld)).astype(np.float32)
    ts, tdp = _f32(s), _f32(dp)
    p = torch.full((rows, ld), 7.0, device="cuda")
    ds = torch.full((rows, ld), 7.0, device="cuda")
    scale = 0.125
    mx.mpx_softmax_fwd(ts.data_ptr(), p.data_ptr(), rows, n, ld, scale, mx.MPX_F32, _s())
    gp = to_host(p)
    _close32(gp[:, :n], ops.softmax_fwd(pol, s[:, :n], scale), 0.0, 4e-6, "P")
    assert np.all(gp[:, n:] == 0)
    mx.mpx_softmax_bwd(p.data_ptr(), tdp.data_ptr(), ds.data_ptr(), rows, n, ld, scale, mx.MPX_F32, _s())
    gds = to_host(ds)
    ref = ops.softmax_bwd(pol, gp[:, :n], dp[:, :n], scale)
    _close32(gds[:, :n], ref, scale * np.abs(gp[:, :n]) * 4.0, 4e-6, "dS")
    assert np.all(gds[:, n:] == 0)


def test_cross_entropy_embed_patchify_f32():
    pol = Policy("f32")
    rng = np.random.default_rng(5)
    B, C = 37, 100
    z = rng.normal(0, 2, size=(B, C)).astype(np.float32)
    y = rng.integers(0, C, size=B).astype(np.int32)
    tz, ty = _f32(z), torch.from_numpy(y).cuda()
    state = torch.from_numpy(np.frombuffer(np.array([1.0], np.float32).tobytes() + np.zeros(5, np.int32).tobytes(),
                                           dtype=np.int32).copy()).cuda()
    loss = torch.zeros(1, device="cuda")
    dz = torch.zeros(B, C, device="cuda")
    ws_n = mx.mpx_loss_workspace(B)
    ws = torch.zeros(ws_n, dtype=torch.uint8, device="cuda")
    mx.mpx_cross_entropy(tz.data_ptr(), C, ty.data_ptr(), B, C, state.data_ptr(), loss.data_ptr(),
                         dz.data_ptr(), mx.MPX_F32, ws.data_ptr(), ws_n, _s())
    rl, rdz = ops.ce_fwd_bwd(pol, z, y, 1.0)
    assert abs(float(loss.item()) - rl) <= 2e-6 * abs(rl)
    _close32(to_host(dz), rdz, 1.0 / B, 4e-6, "dZ")
    # patches and token assembly (and its backward)
    Bi, H, W, Ch, p, d = 2, 8, 8, 3, 4, 16
    img = rng.uniform(0, 1, size=(Bi, H, W, Ch)).astype(np.float32)
    G, T = (H // p) * (W // p), (H // p) * (W // p) + 1
    pt = torch.zeros(Bi * G, p * p * Ch, device="cuda")
    timg = _f32(img)  # kept alive: a freed temporary's memory can be reused before the launch
    mx.mpx_patchify_cast(timg.data_ptr(), pt.data_ptr(), Bi, H, W, Ch, p, mx.MPX_F32, _s())
    assert np.array_equal(to_host(pt), ops.patchify(img, p))
    E = rng.normal(size=(Bi * G, d)).astype(np.float32)
    cls = rng.normal(size=d).astype(np.float32)
    pos = rng.normal(size=(T, d)).astype(np.float32)
    X = torch.zeros(Bi * T, d, device="cuda")
    tE, tcls, tpos = _f32(E), _f32(cls), _f32(pos)
    mx.mpx_embed_assemble(tE.data_ptr(), tcls.data_ptr(), tpos.data_ptr(), X.data_ptr(),
                          Bi, T, d, mx.MPX_F32, _s())
    ref = np.empty((Bi, T, d), np.float32)
    ref[:, 0] = cls + pos[0]
    ref[:, 1:] = E.reshape(Bi, G, d) + pos[None, 1:]
    assert np.array_equal(to_host(X), ref.reshape(Bi * T, d))
    dX = rng.normal(size=(Bi * T, d)).astype(np.float32)
    dE, dcls, dpos = (torch.zeros(Bi * G, d, device="cuda"), torch.zeros(d, device="cuda"),
                      torch.zeros(T, d, device="cuda"))
    tdX = _f32(dX)
    mx.mpx_embed_assemble_bwd(tdX.data_ptr(), dE.data_ptr(), dcls.data_ptr(), dpos.data_ptr(), Bi, T,
                              d, mx.MPX_F32, None, _s())
    d3 = dX.reshape(Bi, T, d)
    assert np.array_equal(to_host(dE), d3[:, 1:].reshape(Bi * G, d))
    _close32(to_host(dpos), d3.astype(np.float64).sum(axis=0), 2.0, 4e-7, "dpos")
    _close32(to_host(dcls), d3[:, 0].astype(np.float64).sum(axis=0), 2.0, 4e-7, "dcls")


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_nonfinite_counts_of_layernorm_head_and_embedding(fmt):
    """MPX §3.4's finite check fused into the LayerNorm, classifier-head and
    token-assembly backward: the count each adds equals the separate check's
    count over the parameter gradients it writes (dgamma / dbeta; dcls /
    dpos), with cotangents large enough that some of those sums overflow."""
    from paper_2507_03312_amd.train import pack_scale_state
    dt = mx.DTYPES[fmt]
    big = 30000.0 if fmt == "f16" else 1.0e38
    rng = np.random.default_rng(3)
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    ref = torch.zeros(1, dtype=torch.int32, device="cuda")

    def check(grads, add_to):
        torch.cuda.synchronize()
        mx.mpx_unscale_check(mx.TensorList(grads), dt, 0, ref.data_ptr(), None, _s())
        got, want = int(nf.item()), int(ref.item())
        assert got == add_to + want and want > 0, (got, add_to, want)
        return got

    # LayerNorm: rows whose cotangent is large in every other column (one
    # wave per row at d = 256, row groups at d = 384)
    total = 0
    for rows, d in ((96, 256), (96, 384)):
        x = round_to(rng.normal(size=(rows, d)), fmt)
        g = round_to(1.0 + 0.1 * rng.normal(size=d), fmt)
        dy = rng.normal(size=(rows, d))
        dy[:, ::2] = big
        dy = round_to(dy, fmt)
        tx, tg, tdy = (to_dev_half(a, fmt) for a in (x, g, dy))
        dg, db = _empty((d,), fmt), _empty((d,), fmt)
        wsn = mx.mpx_layernorm_bwd_workspace(rows, d)
        ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
        mx.mpx_layernorm_bwd(tx.data_ptr(), d, tg.data_ptr(), tdy.data_ptr(), None, None, d, dg.data_ptr(),
                             db.data_ptr(), rows, d, dt, ws.data_ptr(), wsn, nf.data_ptr(), _s())
        total = check([dg, db], total)
    # token assembly backward: large CLS-position cotangents in some columns
    B, T = 4, 5
    dX = rng.normal(size=(B * T, d))
    dX.reshape(B, T, d)[:, 0, :64] = big
    dX = round_to(dX, fmt)
    tdX = to_dev_half(dX, fmt)
    dE, dcls, dpos = _empty((B * (T - 1), d), fmt), _empty((d,), fmt), _empty((T, d), fmt)
    mx.mpx_embed_assemble_bwd(tdX.data_ptr(), dE.data_ptr(), dcls.data_ptr(), dpos.data_ptr(), B, T, d,
                              dt, nf.data_ptr(), _s())
    total = check([dcls, dpos], total)
    # classifier head: the loss scale (and for bfloat16 a huge W) pushes the
    # head's cotangents, and so dgamma / dbeta, past the format's range
    Bh, C = 64, 10
    xh = round_to(rng.normal(size=(Bh, d)), fmt)
    w = round_to((0.5 if fmt == "f16" else 1.0e30) * rng.normal(size=(C, d)), fmt)
    y = rng.integers(0, C, size=Bh).astype(np.int32)
    scale = 2.0 ** 24 if fmt == "f16" else 2.0 ** 100
    st = torch.from_numpy(pack_scale_state(scale, 0, 10)).cuda()
    txh, tw, tb0 = to_dev_half(xh, fmt), to_dev_half(w, fmt), _empty((C,), fmt)
    ty = torch.from_numpy(y).cuda()
    z, dl, dxh = _empty((Bh, d), fmt), _empty((Bh, C), fmt), _empty((Bh, d), fmt)
    dgh, dbh = _empty((d,), fmt), _empty((d,), fmt)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    wsn = mx.mpx_classifier_head_workspace(Bh, d)
    wsh = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
    mx.mpx_classifier_head(txh.data_ptr(), d, tg.data_ptr(), tb0.data_ptr(), tw.data_ptr(), tb0.data_ptr(),
                           ty.data_ptr(), Bh, d, C, st.data_ptr(), z.data_ptr(), loss.data_ptr(),
                           dl.data_ptr(), dxh.data_ptr(), d, dgh.data_ptr(), dbh.data_ptr(), dt,
                           wsh.data_ptr(), wsn, nf.data_ptr(), _s())
    check([dgh, dbh], total)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
@pytest.mark.parametrize("rows,d,ldx", [(8320, 384, 384), (65, 100, 104), (7, 768, 768), (33, 1500, 1501),
                                        (9, 384, 386), (12608, 768, 768)])
def test_layernorm_fwd_cast_matches_cast_then_layernorm(fmt, rows, d, ldx):
    """The input cast fused with the first LayerNorm gives the same bits as
    the cast followed by the LayerNorm (both outputs and the row stats)."""
    dt = mx.DTYPES[fmt]
    rng = np.random.default_rng(rows + d)
    x = rng.normal(0.3, 1.5, size=(rows, ldx)).astype(np.float32)
    g = to_dev_half(round_to(1.0 + 0.1 * rng.normal(size=d), fmt), fmt)
    b = to_dev_half(round_to(0.1 * rng.normal(size=d), fmt), fmt)
    tx = torch.from_numpy(x).cuda()
    xh1, y1 = _empty((rows, d), fmt), _empty((rows, d), fmt)
    mr1 = torch.zeros(rows, 2, device="cuda")
    mx.mpx_layernorm_fwd_cast(tx.data_ptr(), ldx, g.data_ptr(), b.data_ptr(), xh1.data_ptr(), y1.data_ptr(),
                              mr1.data_ptr(), rows, d, dt, _s())
    # reference: the cast (x as dense rows), then the LayerNorm
    tdense = torch.from_numpy(np.ascontiguousarray(x[:, :d])).cuda()
    xh2, y2 = _empty((rows, d), fmt), _empty((rows, d), fmt)
    mr2 = torch.zeros(rows, 2, device="cuda")
    src, dst = mx.TensorList([tdense]), mx.TensorList([xh2])
    mx.mpx_cast_to_half(src, dst, dt, _s())
    mx.mpx_layernorm_fwd(xh2.data_ptr(), d, g.data_ptr(), b.data_ptr(), y2.data_ptr(), mr2.data_ptr(), rows, d,
                         dt, _s())
    torch.cuda.synchronize()
    assert torch.equal(xh1, xh2) and torch.equal(y1, y2) and torch.equal(mr1, mr2)


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
@pytest.mark.parametrize("rows,d,ldx", [(8320, 384, 384), (33, 1500, 1501)])
def test_layernorm_fwd_cast_against_oracle(fmt, rows, d, ldx):
    """The fused input cast + LayerNorm against the oracle directly: the half
    copy is the oracle's rounding of the float32 inputs, bit for bit, and the
    normalised output is the oracle's LayerNorm of that copy within one half
    ulp plus the float32 evaluation term."""
    pol = Policy(fmt)
    dt = mx.DTYPES[fmt]
    rng = np.random.default_rng(rows + 7 * d)
    x = rng.normal(0.3, 1.5, size=(rows, ldx)).astype(np.float32)
    g = round_to(1.0 + 0.1 * rng.normal(size=d), fmt)
    b = round_to(0.1 * rng.normal(size=d), fmt)
    tg, tb = to_dev_half(g, fmt), to_dev_half(b, fmt)
    tx = torch.from_numpy(x).cuda()
    xh, yv = _empty((rows, d), fmt), _empty((rows, d), fmt)
    mx.mpx_layernorm_fwd_cast(tx.data_ptr(), ldx, tg.data_ptr(), tb.data_ptr(), xh.data_ptr(),
                              yv.data_ptr(), None, rows, d, dt, _s())
    torch.cuda.synchronize()
    rxh = pol.R(x[:, :d])
    assert_same_values(to_host(xh), rxh, "half copy")
    ref = ops.layernorm_fwd(pol, rxh, g, b)
    xhat = ops.layernorm_fwd(Policy("f64"), rxh, np.ones(d), np.zeros(d))
    f32_err = 2.0 ** -21 * (np.abs(xhat * g.astype(np.float64)) + np.abs(b.astype(np.float64)))
    assert_within(to_host(yv), ref, ulp(ref, fmt) + f32_err, "LN of the cast")
