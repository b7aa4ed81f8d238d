"""ctypes binding of libmpx (include/mpx.h): the same names, argument
marshalling only.

Every function takes device pointers as Python ints (``tensor.data_ptr()``),
tensor lists as ``TensorList`` handles and the stream as an int
(``torch.cuda.current_stream().cuda_stream``).  A non-zero return code raises
``MPXError`` with the library's message.  The library must have been built
(``python -m paper_2507_03312_amd.build``); importing this module without it
raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmpx.so")

MPX_F32, MPX_F16, MPX_BF16 = 0, 1, 2
MPX_ACT_NONE, MPX_ACT_GELU_TANH = 0, 1
DTYPES = {"f32": MPX_F32, "f16": MPX_F16, "bf16": MPX_BF16}


class MPXError(RuntimeError):
    pass


class ScaleState(C.Structure):
    _fields_ = [("scale", C.c_float), ("counter", C.c_int32), ("period", C.c_int32),
                ("factor", C.c_float), ("min_scale", C.c_float), ("max_scale", C.c_float)]


class AdamWHP(C.Structure):
    _fields_ = [("lr", C.c_double), ("beta1", C.c_double), ("beta2", C.c_double),
                ("eps", C.c_double), ("weight_decay", C.c_double)]


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_2507_03312_amd.build` (no fallback exists)")
    return C.CDLL(_LIB_PATH)


lib = _load()

P = C.c_void_p
I64 = C.c_int64
I32 = C.c_int32
F = C.c_float
SZ = C.c_size_t

_SIGS = {
    "mpx_tlist_create": (C.c_int, [C.POINTER(P), C.POINTER(I64), I32, C.POINTER(P)]),
    "mpx_tlist_destroy": (C.c_int, [P]),
    "mpx_tlist_numel": (I64, [P]),
    "mpx_cast_to_half": (C.c_int, [P, P, I32, P]),
    "mpx_cast_to_float": (C.c_int, [P, P, I32, P]),
    "mpx_unscale_check": (C.c_int, [P, I32, P, P, P, P]),
    "mpx_scale_update": (C.c_int, [P, P, P]),
    "mpx_adamw_masked": (C.c_int, [P, P, P, P, I32, C.POINTER(AdamWHP), P, P, P, P, I32, P]),
    "mpx_linear_fwd": (C.c_int, [P, P, P, P, P, P, I64, I64, I64, I32, I32, P]),
    "mpx_linear_bwd": (C.c_int, [P, P, P, P, I32, P, P, P, I64, I64, I64, I32, P, SZ, P, P]),
    "mpx_linear_bwd_workspace": (SZ, [I64, I64, I64]),
    "mpx_linear_bwd_noalloc": (C.c_int, [P, P, P, P, I32, P, P, P, I64, I64, I64, I32, P, P]),
    "mpx_gemm_batched": (C.c_int, [I32, I32, I64, I64, I64, I64, I64, P, I64, I64, I64, P, I64,
                                   I64, I64, P, I64, I64, I64, I32, P]),
    "mpx_gemm_set_config": (C.c_int, [I32]),
    "mpx_attention_fwd": (C.c_int, [P, P, P, I64, I64, I64, I64, I32, P]),
    "mpx_attention_bwd": (C.c_int, [P, P, P, P, I64, I64, I64, I64, I32, P, SZ, P]),
    "mpx_attention_bwd_workspace": (SZ, [I64, I64, I64, I64]),
    "mpx_layernorm_fwd": (C.c_int, [P, I64, P, P, P, P, I64, I64, I32, P]),
    "mpx_layernorm_fwd_cast": (C.c_int, [P, I64, P, P, P, P, P, I64, I64, I32, P]),
    "mpx_layernorm_bwd": (C.c_int, [P, I64, P, P, P, P, I64, P, P, I64, I64, I32, P, SZ, P, P]),
    "mpx_layernorm_bwd_workspace": (SZ, [I64, I64]),
    "mpx_softmax_fwd": (C.c_int, [P, P, I64, I64, I64, F, I32, P]),
    "mpx_softmax_bwd": (C.c_int, [P, P, P, I64, I64, I64, F, I32, P]),
    "mpx_loss_workspace": (SZ, [I64]),
    "mpx_cross_entropy": (C.c_int, [P, I64, P, I64, I64, P, P, P, I32, P, SZ, P]),
    "mpx_mse": (C.c_int, [P, P, I64, P, P, P, I32, P, SZ, P]),
    "mpx_classifier_head_workspace": (SZ, [I64, I64]),
    "mpx_classifier_head": (C.c_int, [P, I64, P, P, P, P, P, I64, I64, I64, P, P, P, P, P, I64, P, P,
                                      I32, P, SZ, P, P]),
    "mpx_patchify_cast": (C.c_int, [P, P, I64, I64, I64, I64, I64, I32, P]),
    "mpx_embed_assemble": (C.c_int, [P, P, P, P, I64, I64, I64, I32, P]),
    "mpx_embed_assemble_bwd": (C.c_int, [P, P, P, P, I64, I64, I64, I32, P, P]),
    "mpx_gather_rows": (C.c_int, [P, I64, P, I64, I64, I32, P]),
    "mpx_zero": (C.c_int, [P, SZ, P]),
    "mpx_last_error": (C.c_char_p, []),
}

for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = sorted(_SIGS)


def _check(rc: int, name: str) -> None:
    if rc != 0:
        raise MPXError(f"{name} failed ({rc}): {lib.mpx_last_error().decode()}")


def _call(name):
    fn = getattr(lib, name)

    def wrapper(*args):
        _check(fn(*args), name)
    wrapper.__name__ = name
    wrapper.__doc__ = f"{name} (include/mpx.h); raises MPXError on failure."
    return wrapper


class TensorList:
    """Owner of an ``mpx_tlist`` over device tensors (kept alive here)."""

    def __init__(self, tensors):
        self.tensors = list(tensors)
        n = len(self.tensors)
        ptrs = (P * max(n, 1))(*[t.data_ptr() for t in self.tensors])
        numels = (I64 * max(n, 1))(*[t.numel() for t in self.tensors])
        h = P()
        _check(lib.mpx_tlist_create(ptrs, numels, n, C.byref(h)), "mpx_tlist_create")
        self.handle = h

    @property
    def numel(self) -> int:
        return int(lib.mpx_tlist_numel(self.handle))

    def close(self):
        if getattr(self, "handle", None):
            lib.mpx_tlist_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _h(t):
    return None if t is None else t.handle


def mpx_cast_to_half(src: TensorList, dst: TensorList, half: int, stream: int):
    _check(lib.mpx_cast_to_half(src.handle, dst.handle, half, stream), "mpx_cast_to_half")


def mpx_cast_to_float(src: TensorList, dst: TensorList, half: int, stream: int):
    _check(lib.mpx_cast_to_float(src.handle, dst.handle, half, stream), "mpx_cast_to_float")


def mpx_unscale_check(grads: TensorList, gdt: int, d_state: int, d_nonfinite: int,
                      out_f32, stream: int):
    _check(lib.mpx_unscale_check(grads.handle, gdt, d_state, d_nonfinite, _h(out_f32), stream),
           "mpx_unscale_check")


def mpx_scale_update(d_state: int, d_nonfinite: int, stream: int):
    _check(lib.mpx_scale_update(d_state, d_nonfinite, stream), "mpx_scale_update")


def mpx_adamw_masked(p32: TensorList, m32: TensorList, v32: TensorList, grads: TensorList,
                     gdt: int, hp: AdamWHP, d_step: int, d_state: int, d_nonfinite: int,
                     half_copy, half: int, stream: int):
    _check(lib.mpx_adamw_masked(p32.handle, m32.handle, v32.handle, grads.handle, gdt,
                                C.byref(hp), d_step, d_state, d_nonfinite, _h(half_copy), half,
                                stream), "mpx_adamw_masked")


mpx_linear_fwd = _call("mpx_linear_fwd")
mpx_linear_bwd = _call("mpx_linear_bwd")
mpx_linear_bwd_noalloc = _call("mpx_linear_bwd_noalloc")
MPX_LINEAR_BWD_NOALLOC_SCRATCH = 64 << 20   # bytes (include/mpx.h)
mpx_gemm_batched = _call("mpx_gemm_batched")
mpx_gemm_set_config = _call("mpx_gemm_set_config")
mpx_attention_fwd = _call("mpx_attention_fwd")
mpx_attention_bwd = _call("mpx_attention_bwd")
mpx_layernorm_fwd = _call("mpx_layernorm_fwd")
mpx_layernorm_fwd_cast = _call("mpx_layernorm_fwd_cast")
mpx_layernorm_bwd = _call("mpx_layernorm_bwd")
mpx_softmax_fwd = _call("mpx_softmax_fwd")
mpx_softmax_bwd = _call("mpx_softmax_bwd")
mpx_cross_entropy = _call("mpx_cross_entropy")
mpx_mse = _call("mpx_mse")
mpx_classifier_head = _call("mpx_classifier_head")
mpx_patchify_cast = _call("mpx_patchify_cast")
mpx_embed_assemble = _call("mpx_embed_assemble")
mpx_embed_assemble_bwd = _call("mpx_embed_assemble_bwd")
mpx_gather_rows = _call("mpx_gather_rows")
mpx_zero = _call("mpx_zero")


def mpx_linear_bwd_workspace(M: int, N: int, K: int) -> int:
    return int(lib.mpx_linear_bwd_workspace(M, N, K))


def mpx_attention_bwd_workspace(B: int, T: int, H: int, hd: int) -> int:
    return int(lib.mpx_attention_bwd_workspace(B, T, H, hd))


def mpx_loss_workspace(n: int) -> int:
    return int(lib.mpx_loss_workspace(n))


def mpx_layernorm_bwd_workspace(rows: int, d: int) -> int:
    return int(lib.mpx_layernorm_bwd_workspace(rows, d))


def mpx_classifier_head_workspace(B: int, d: int) -> int:
    return int(lib.mpx_classifier_head_workspace(B, d))


def mpx_last_error() -> str:
    return lib.mpx_last_error().decode()
