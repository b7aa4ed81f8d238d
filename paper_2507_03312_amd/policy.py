"""MPX's casting transformations over device tensors: the PyTree casts of
§3.1 (cast_tree, cast_to_half_precision, cast_to_float16, cast_to_bfloat16,
cast_to_float32) and the function casts of §3.2 (cast_function,
force_full_precision).  The conversions run in libmpx's multi-tensor cast
kernels (mpx_cast_to_half: float32 -> half, rounding to nearest even;
mpx_cast_to_float: half -> float32, exact); this module only walks the
trees and marshals pointers.

A tree is any nesting of dicts, lists and tuples whose leaves are torch
tensors on the GPU (the device buffers the libmpx calls take), Python
scalars or None.  A cast visits the floating-point tensor leaves only:
integer tensors (random keys, labels, indices) are never touched (§3.1).
Leaves already in the target type are returned as they are; every other
floating leaf gets a new dense buffer of the target type.  The casts of one
call go out as at most two multi-tensor launches per half type on the
current stream (half -> other half is widened to float32 first, then
rounded once: the same value as one rounding, since the widening is exact).
Each call uploads its small pointer tables synchronously, so these casts
belong around a step, not inside a captured one.
"""
from __future__ import annotations

import collections
import copy
import functools
from typing import Any, Callable, List, Optional, Tuple

import torch

from . import binding as mx

_DTYPES = {"f32": torch.float32, "float32": torch.float32,
           "f16": torch.float16, "float16": torch.float16,
           "bf16": torch.bfloat16, "bfloat16": torch.bfloat16}
_HALF_CODE = {torch.float16: mx.MPX_F16, torch.bfloat16: mx.MPX_BF16}

# descriptor tables of launched casts, released once their launch has run
_in_flight: "collections.deque" = collections.deque()


def _target(dtype) -> torch.dtype:
    if isinstance(dtype, torch.dtype):
        if dtype not in (torch.float32, torch.float16, torch.bfloat16):
            raise ValueError(f"unsupported floating-point type {dtype}")
        return dtype
    try:
        return _DTYPES[str(dtype)]
    except KeyError:
        raise ValueError(f"unsupported floating-point type {dtype!r}") from None


def _flatten(tree) -> Tuple[List[Any], Callable[[List[Any]], Any]]:
    """Leaves of a tree in a fixed order, and the function that rebuilds the
    tree's structure around a list of new leaves."""
    if isinstance(tree, dict):
        keys = list(tree.keys())
        parts = [_flatten(tree[k]) for k in keys]
    elif isinstance(tree, (list, tuple)):
        keys = None
        parts = [_flatten(x) for x in tree]
    else:
        return [tree], lambda leaves: leaves[0]
    sizes = [len(p[0]) for p in parts]
    leaves = [leaf for p in parts for leaf in p[0]]

    def rebuild(new):
        out, i = [], 0
        for (_, rb), n in zip(parts, sizes):
            out.append(rb(new[i:i + n]))
            i += n
        if keys is not None:
            if type(tree) is dict:
                return dict(zip(keys, out))
            new = copy.copy(tree)  # dict subclasses keep their type and state (a default factory)
            new.clear()
            new.update(zip(keys, out))
            return new
        if isinstance(tree, tuple) and hasattr(tree, "_fields"):  # named tuple
            return type(tree)(*out)
        return type(tree)(out)
    return leaves, rebuild


def _release_finished():
    while _in_flight and _in_flight[0][0].query():
        _in_flight.popleft()


def _launch(fn, pairs, code):
    src = mx.TensorList([s for s, _ in pairs])
    dst = mx.TensorList([d for _, d in pairs])
    fn(src, dst, code, torch.cuda.current_stream().cuda_stream)
    done = torch.cuda.Event()
    done.record()
    _in_flight.append((done, src, dst))


def cast_tree(tree, dtype):
    """§3.1 cast_tree: every floating-point tensor leaf of `tree` in `dtype`
    ("f32", "f16", "bf16" or the torch type); everything else unchanged."""
    target = _target(dtype)
    _release_finished()
    leaves, rebuild = _flatten(tree)
    out = list(leaves)
    widen = {torch.float16: [], torch.bfloat16: []}   # half -> float32
    narrow = {torch.float16: [], torch.bfloat16: []}  # float32 -> half
    for i, t in enumerate(leaves):
        if not isinstance(t, torch.Tensor) or not t.is_floating_point() or t.dtype == target:
            continue
        if t.dtype not in (torch.float32, torch.float16, torch.bfloat16):
            raise ValueError(f"leaf {i}: unsupported floating-point type {t.dtype}")
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"leaf {i}: casts take dense device tensors")
        dst = torch.empty(t.shape, dtype=target, device=t.device)
        if target == torch.float32:
            widen[t.dtype].append((t, dst))
        elif t.dtype == torch.float32:
            narrow[target].append((t, dst))
        else:  # half -> the other half, through float32
            mid = torch.empty(t.shape, dtype=torch.float32, device=t.device)
            widen[t.dtype].append((t, mid))
            narrow[target].append((mid, dst))
        out[i] = dst
    for h, pairs in widen.items():
        if pairs:
            _launch(mx.mpx_cast_to_float, pairs, _HALF_CODE[h])
    for h, pairs in narrow.items():
        if pairs:
            _launch(mx.mpx_cast_to_half, pairs, _HALF_CODE[h])
    return rebuild(out)


def cast_to_half_precision(tree, half: str = "f16"):
    """§3.1 cast_to_half_precision (half: "f16" or "bf16")."""
    if _target(half) == torch.float32:
        raise ValueError("half must be f16 or bf16")
    return cast_tree(tree, half)


def cast_to_float16(tree):
    return cast_tree(tree, "f16")


def cast_to_bfloat16(tree):
    return cast_tree(tree, "bf16")


def cast_to_float32(tree):
    return cast_tree(tree, "f32")


def cast_function(func: Callable, dtype, return_dtype: Optional[object] = None) -> Callable:
    """§3.2 cast_function: a function that casts every input tree to `dtype`,
    calls `func`, and casts its outputs to `return_dtype` when given.  The
    precision `func` computes in follows from its inputs: the libmpx calls
    it makes take their dtype from the buffers it passes."""
    target = _target(dtype)
    ret = None if return_dtype is None else _target(return_dtype)

    @functools.wraps(func)
    def cast_func(*args, **kwargs):
        args, kwargs = cast_tree((list(args), kwargs), target)
        out = func(*args, **kwargs)
        return out if ret is None else cast_tree(out, ret)
    return cast_func


def force_full_precision(func: Callable, return_dtype) -> Callable:
    """§3.2 force_full_precision: `func` on float32 inputs (for operations
    that overflow in float16: sums, means, large products), outputs cast to
    `return_dtype`."""
    return cast_function(func, torch.float32, return_dtype)
