"""mpx_linear_bwd_noalloc (the linear backward that allocates nothing: its
partials live in the library's static per-GPU scratch array) against
mpx_linear_bwd with a caller's workspace, through the C ABI.

Both run the same kernels, so every output (dX through GELU', dW with split-K,
db) and the non-finite count must be the same bits.  Two calls in a row on
the shared array, the second with a smaller product, show that nothing the
first call left behind leaks into the second; the second call also overflows
in part (the count is compared).  A product whose partials exceed the array
is rejected before anything is launched."""
import numpy as np
import pytest

from oracle.numfmt import round_to
from tests.gpu_util import HAVE_GPU

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="no GPU")]

if HAVE_GPU:
    import torch
    from paper_2507_03312_amd import binding as mx


def _s():
    return torch.cuda.current_stream().cuda_stream


def _half(a, fmt):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(
        torch.float16 if fmt == "f16" else torch.bfloat16).cuda()


def _run_both(M, N, K, fmt, seed, big=1.0):
    rng = np.random.default_rng(seed)
    X = _half(round_to(rng.normal(0, 1, (M, K)), fmt), fmt)
    Xpre = _half(round_to(rng.normal(0, 1, (M, K)), fmt), fmt)   # the layer below's pre-activation
    W = _half(round_to(rng.normal(0, 0.05, (N, K)), fmt), fmt)
    dY = _half(round_to(rng.normal(0, big, (M, N)), fmt), fmt)
    dt = mx.DTYPES[fmt]
    outs = []
    for noalloc in (False, True):
        dX = torch.zeros(M, K, dtype=X.dtype, device="cuda")
        dW = torch.zeros(N, K, dtype=X.dtype, device="cuda")
        db = torch.zeros(N, dtype=X.dtype, device="cuda")
        nf = torch.zeros(1, dtype=torch.int32, device="cuda")
        xp = Xpre
        if noalloc:
            mx.mpx_linear_bwd_noalloc(X.data_ptr(), W.data_ptr(), dY.data_ptr(), xp.data_ptr(),
                                      mx.MPX_ACT_GELU_TANH, dX.data_ptr(), dW.data_ptr(), db.data_ptr(),
                                      M, N, K, dt, nf.data_ptr(), _s())
        else:
            wsn = mx.mpx_linear_bwd_workspace(M, N, K)
            ws = torch.zeros(wsn, dtype=torch.uint8, device="cuda")
            mx.mpx_linear_bwd(X.data_ptr(), W.data_ptr(), dY.data_ptr(), xp.data_ptr(),
                              mx.MPX_ACT_GELU_TANH, dX.data_ptr(), dW.data_ptr(), db.data_ptr(),
                              M, N, K, dt, ws.data_ptr(), wsn, nf.data_ptr(), _s())
        torch.cuda.synchronize()
        outs.append((dX, dW, db, int(nf.item())))
    (a_dx, a_dw, a_db, a_nf), (b_dx, b_dw, b_db, b_nf) = outs
    for a, b, what in ((a_dx, b_dx, "dX"), (a_dw, b_dw, "dW"), (a_db, b_db, "db")):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), what
    assert a_nf == b_nf
    return a_nf


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_noalloc_matches_workspace_call_twice(fmt):
    # first: a ViT-B projection-sized product (split-K over 12608 rows, every
    # partial of the array in use); second: a smaller ragged product whose
    # fp16 gradients overflow in part
    M, N, K = 12608, 768, 768
    assert mx.mpx_linear_bwd_workspace(M, N, K) <= mx.MPX_LINEAR_BWD_NOALLOC_SCRATCH
    assert _run_both(M, N, K, fmt, 1) == 0
    nf = _run_both(1030, 200, 136, fmt, 2, big=2000.0 if fmt == "f16" else 1.0)
    if fmt == "f16":
        assert nf > 0


def test_noalloc_rejects_products_beyond_the_array():
    M, N, K = 64, 1 << 25, 8   # 2^25 bias columns: 128 MiB of column partials
    assert mx.mpx_linear_bwd_workspace(M, N, K) > mx.MPX_LINEAR_BWD_NOALLOC_SCRATCH
    p = 256   # never dereferenced: the size check fails before any launch
    with pytest.raises(mx.MPXError, match="static scratch"):
        mx.mpx_linear_bwd_noalloc(p, p, p, None, 0, None, p, p, M, N, K, mx.MPX_BF16, None, _s())
