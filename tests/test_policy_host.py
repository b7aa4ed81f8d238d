"""Host logic of the casting transformations (§3.1, §3.2) that needs no GPU:
tree walking, leaf selection and the errors raised before any launch."""
import collections

import pytest
import torch

from paper_2507_03312_amd import policy


def test_trees_without_floating_leaves_pass_through_unchanged():
    ints = torch.arange(5)
    keys = torch.zeros(2, dtype=torch.uint32)
    T = collections.namedtuple("T", "a b")
    tree = {"x": [ints, (keys, 1.5)], "y": T(None, "label"), "z": []}
    for fmt in ("f16", "bf16", "f32", torch.float16):
        out = policy.cast_tree(tree, fmt)
        assert out == {"x": [ints, (keys, 1.5)], "y": T(None, "label"), "z": []}
        assert out["x"][0] is ints and out["x"][1][0] is keys
        assert type(out["y"]) is T and type(out["x"][1]) is tuple


def test_dict_subclasses_keep_their_type_and_state():
    dd = collections.defaultdict(list, {"a": torch.arange(2)})
    od = collections.OrderedDict([("z", 1), ("y", torch.arange(3))])
    out = policy.cast_tree({"dd": dd, "od": od}, "f16")
    assert type(out["dd"]) is collections.defaultdict and out["dd"].default_factory is list
    assert type(out["od"]) is collections.OrderedDict and list(out["od"]) == ["z", "y"]
    assert out["dd"]["a"] is dd["a"] and out["od"]["y"] is od["y"]


def test_leaves_already_in_the_target_type_are_not_copied():
    # host tensors are fine as long as nothing has to be cast
    a = torch.ones(3, dtype=torch.bfloat16)
    out = policy.cast_to_bfloat16({"a": a, "n": torch.arange(3)})
    assert out["a"] is a


@pytest.mark.parametrize("bad", ["f64", "int8", torch.float64, torch.int32, None])
def test_unknown_target_types_raise(bad):
    with pytest.raises(ValueError, match="unsupported"):
        policy.cast_tree([torch.arange(2)], bad)


def test_leaves_that_cannot_be_cast_raise_before_any_launch():
    with pytest.raises(ValueError, match="dense device tensors"):
        policy.cast_to_float16([torch.ones(4)])                   # host float32
    with pytest.raises(ValueError, match="unsupported floating-point type"):
        policy.cast_to_float32({"d": torch.ones(2, dtype=torch.float64)})
    with pytest.raises(ValueError, match="f16 or bf16"):
        policy.cast_to_half_precision([], "f32")


def test_cast_function_wraps_and_passes_non_float_arguments():
    seen = {}

    def f(n, *, labels, scale=2.0):
        """doc"""
        seen.update(n=n, labels=labels, scale=scale)
        return n + 1

    labels = torch.arange(4)
    g = policy.cast_function(f, "bf16")
    assert g.__name__ == "f" and g.__doc__ == "doc"
    assert g(3, labels=labels) == 4
    assert seen["labels"] is labels and seen["n"] == 3 and seen["scale"] == 2.0
    h = policy.force_full_precision(f, "f16")
    assert h(1, labels=labels, scale=0.5) == 2 and seen["scale"] == 0.5
