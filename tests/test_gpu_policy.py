"""GPU parity of MPX's casting transformations through the C ABI: the widening
cast half -> float32 (§3.1 cast_to_float32), the PyTree casts of §3.1
(cast_tree and its named forms) and the function casts of §3.2
(cast_function, force_full_precision) built on mpx_cast_to_half and
mpx_cast_to_float.

Bars: every cast is bit-exact; the product computed inside a cast function
is within the GEMM bound of the other parity tests.  The expected widening is the value each
half bit pattern encodes by the format's definition (bfloat16: the pattern
as the upper half of a float32; binary16: numpy's IEEE decoder), not a
conversion of the library under test; the expected narrowing is the
oracle's round_to.
"""
import collections

import numpy as np
import pytest

from oracle import ops as oops
from oracle.numfmt import round_to
from oracle.policy import Policy
from tests.gpu_util import HAVE_GPU, assert_same_values, assert_within, gemm_bound, to_host

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not HAVE_GPU, reason="no GPU")]

if HAVE_GPU:
    import torch
    from paper_2507_03312_amd import binding as mx
    from paper_2507_03312_amd import policy

THALF = {"f16": "float16", "bf16": "bfloat16"}


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _decode(bits: np.ndarray, fmt: str) -> np.ndarray:
    """float32 values of 16-bit patterns, by the format's definition."""
    if fmt == "bf16":
        return (bits.astype(np.uint32) << 16).view(np.float32)
    return bits.view(np.float16).astype(np.float32)


def _half_from_bits(bits: np.ndarray, fmt: str):
    """Device half tensor holding exactly these bit patterns (no conversion)."""
    return torch.from_numpy(bits.view(np.int16).copy()).cuda().view(getattr(torch, THALF[fmt]))


@pytest.mark.parametrize("fmt", ["f16", "bf16"])
def test_cast_to_float_every_bit_pattern(fmt):
    every = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    rng = np.random.default_rng(1)
    # one tensor of all 65536 patterns (three times over, so the vector loop
    # runs), one ragged, and one misaligned by an element (scalar path)
    pats = [np.tile(every, 3), rng.integers(0, 1 << 16, 1237).astype(np.uint16),
            rng.integers(0, 1 << 16, 45).astype(np.uint16)]
    flat = np.concatenate([pats[0], pats[1], np.zeros(1, np.uint16), pats[2]])
    src_all = _half_from_bits(flat, fmt)
    n0, n1 = pats[0].size, pats[1].size
    views = [src_all[:n0], src_all[n0:n0 + n1], src_all[n0 + n1 + 1:]]
    dst_all = torch.full((flat.size + 1,), -7.0, dtype=torch.float32, device="cuda")
    dviews = [dst_all[:n0], dst_all[n0 + 1:n0 + 1 + n1], dst_all[n0 + 1 + n1:n0 + 1 + n1 + pats[2].size]]
    mx.mpx_cast_to_float(mx.TensorList(views), mx.TensorList(dviews), mx.DTYPES[fmt], _stream())
    torch.cuda.synchronize()
    for p, dv in zip(pats, dviews):
        ref = _decode(p, fmt)
        assert_same_values(dv.cpu().numpy(), ref, f"widen {fmt}")
        # the widened values are the half values: rounding them back is the identity
        assert_same_values(round_to(ref, fmt), ref, f"{fmt} values")
    assert float(dst_all[n0].item()) == -7.0          # the gap between views is untouched


def test_cast_to_float_rejects_bad_lists():
    a = torch.zeros(10, dtype=torch.float16, device="cuda")
    b = torch.zeros(11, dtype=torch.float32, device="cuda")
    with pytest.raises(mx.MPXError, match="differ"):
        mx.mpx_cast_to_float(mx.TensorList([a]), mx.TensorList([b]), mx.MPX_F16, _stream())
    with pytest.raises(mx.MPXError, match="MPX_F16 or MPX_BF16"):
        mx.mpx_cast_to_float(mx.TensorList([a]), mx.TensorList([b[:10]]), mx.MPX_F32, _stream())
    # an empty list is a no-op
    mx.mpx_cast_to_float(mx.TensorList([]), mx.TensorList([]), mx.MPX_BF16, _stream())


Pair = collections.namedtuple("Pair", "w b")


def _tree(seed=0):
    rng = np.random.default_rng(seed)
    f32 = rng.normal(0, 3e3, size=70_001).astype(np.float32)        # overflows in f16 at the tails
    f32[:4] = [np.inf, -np.inf, np.nan, 6e-8]
    h16 = round_to(rng.normal(0, 1, 513), "f16")
    b16 = round_to(rng.normal(0, 1e5, 257), "bf16")
    ints = rng.integers(0, 1000, 99, dtype=np.int64)
    dev = {
        "w": torch.from_numpy(f32).cuda(),
        "layers": [Pair(torch.from_numpy(h16).half().cuda(), torch.from_numpy(b16).bfloat16().cuda()),
                   (torch.from_numpy(ints).cuda(), 3.5, None)],
        "empty": torch.zeros(0, dtype=torch.float32, device="cuda"),
    }
    host = {"w": f32, "h16": h16, "b16": b16, "ints": ints}
    return dev, host


@pytest.mark.parametrize("fmt", ["f16", "bf16", "f32"])
def test_cast_tree_values_structure_and_passthrough(fmt):
    dev, host = _tree()
    out = policy.cast_tree(dev, fmt)
    torch.cuda.synchronize()
    want = getattr(torch, {"f16": "float16", "bf16": "bfloat16", "f32": "float32"}[fmt])
    assert isinstance(out, dict) and set(out) == set(dev)
    assert isinstance(out["layers"], list) and isinstance(out["layers"][0], Pair)
    assert isinstance(out["layers"][1], tuple)
    for t in (out["w"], out["layers"][0].w, out["layers"][0].b, out["empty"]):
        assert t.dtype == want
    assert out["empty"].shape == (0,)
    # integer leaves and non-tensor leaves come back as the same objects (§3.1)
    assert out["layers"][1][0] is dev["layers"][1][0]
    assert out["layers"][1][1] == 3.5 and out["layers"][1][2] is None
    assert np.array_equal(out["layers"][1][0].cpu().numpy(), host["ints"])
    # a leaf already in the target type is returned as it is
    for src, dst in ((dev["w"], out["w"]), (dev["layers"][0].w, out["layers"][0].w),
                     (dev["layers"][0].b, out["layers"][0].b)):
        assert (dst is src) == (src.dtype == want)
    # values: one rounding from the source value (exact when widening)
    if fmt == "f32":
        exp = {"w": host["w"], "h16": host["h16"], "b16": host["b16"]}
    else:
        exp = {k: round_to(host[k], fmt) for k in ("w", "h16", "b16")}
    assert_same_values(to_host(out["w"]), exp["w"], "w")
    assert_same_values(to_host(out["layers"][0].w), exp["h16"], "f16 leaf")
    assert_same_values(to_host(out["layers"][0].b), exp["b16"], "bf16 leaf")


def test_named_casts_are_cast_tree():
    dev, host = _tree(3)
    for fn, fmt in ((policy.cast_to_float16, "f16"), (policy.cast_to_bfloat16, "bf16")):
        assert_same_values(to_host(fn(dev)["w"]), round_to(host["w"], fmt), fmt)
    assert_same_values(to_host(policy.cast_to_half_precision(dev, "bf16")["w"]),
                       round_to(host["w"], "bf16"), "half bf16")
    assert_same_values(to_host(policy.cast_to_float32(policy.cast_to_float16(dev))["w"]),
                       round_to(host["w"], "f16"), "f16 then f32")


def _linear(x, w):
    """A function computing in the precision of its inputs: Y = X W^T through
    mpx_linear_fwd, dtype taken from the buffers."""
    m, k = x.shape
    n = w.shape[0]
    assert w.dtype == x.dtype
    y = torch.empty(m, n, dtype=x.dtype, device=x.device)
    dt = {torch.float32: mx.MPX_F32, torch.float16: mx.MPX_F16, torch.bfloat16: mx.MPX_BF16}[x.dtype]
    mx.mpx_linear_fwd(x.data_ptr(), w.data_ptr(), None, None, y.data_ptr(), None, m, n, k, dt,
                      mx.MPX_ACT_NONE, _stream())
    return y


def test_cast_function_and_force_full_precision():
    # a product whose exact value (200 * 512 = 102400) is beyond float16's range
    m, n, k = 64, 48, 512
    x = torch.full((m, k), 200.0, device="cuda")
    w = torch.ones(n, k, device="cuda")
    half_fn = policy.cast_function(_linear, "f16")
    y16 = half_fn(x, w=w)
    assert y16.dtype == torch.float16
    assert torch.isinf(y16).all()                  # overflow in half precision (§3.2)
    full_fn = policy.force_full_precision(half_fn, "f16")
    assert full_fn.__name__ == "_linear"
    y = policy.force_full_precision(_linear, "bf16")(x.half(), w.bfloat16())
    torch.cuda.synchronize()
    assert y.dtype == torch.bfloat16
    assert_same_values(to_host(y), np.full((m, n), round_to(np.float64(102400.0), "bf16"), np.float32),
                       "full precision product")
    # cast_function with a return type: outputs in float32, computed in bf16
    xs = np.random.default_rng(5).normal(0, 1, (m, k)).astype(np.float32)
    ws = np.random.default_rng(6).normal(0, 1, (n, k)).astype(np.float32)
    yb = policy.cast_function(_linear, "bf16", return_dtype="f32")(
        torch.from_numpy(xs).cuda(), torch.from_numpy(ws).cuda())
    torch.cuda.synchronize()
    assert yb.dtype == torch.float32
    xr, wr = round_to(xs, "bf16"), round_to(ws, "bf16")
    ref = oops.linear_fwd(Policy("bf16"), xr, wr, None)
    assert_within(to_host(yb), ref, gemm_bound(xr, wr.T, ref, "bf16", k), "bf16 linear through cast_function")
