"""Host arithmetic of the benchmark's whole-step roofline: the per-call
algorithmic flops of every workload against closed forms written out per
model, and the bound's assembly."""
import numpy as np
import pytest

import bench
import workloads


def _n_params(cfg):
    return sum(int(np.prod(s)) for _, s, _ in workloads.param_specs(cfg))


def _gemm_flops_closed_form(cfg):
    """Linear-layer flops of one training step: forward, dX and dW of every
    layer (2 M N K each), except the dX of the first layer that reads the
    inputs (the MLP's fc1, the patch embedding)."""
    B = cfg.batch
    if cfg.kind == "mlp":
        one = 2.0 * B * cfg.d_in * cfg.d_hidden
        return 3 * one + 2 * one          # fc2: fwd, dX, dW; fc1: fwd, dW
    M, d, F = B * cfg.tokens, cfg.d_model, cfg.d_mlp
    block = 2.0 * M * d * (3 * d + d + F + F)
    total = 3 * cfg.depth * block + 3 * 2.0 * B * cfg.classes * d
    if cfg.image:
        total += 2 * 2.0 * B * cfg.n_patches * d * cfg.patch_dim
    return total


@pytest.mark.parametrize("name", ["mlp", "vit_block", "vit_s", "vit_b"])
def test_step_gemm_flops_match_closed_form(name):
    cfg = workloads.get(name)
    calls = bench.step_calls(cfg, _n_params(cfg))
    g = sum(f for kind, _, f, _ in calls if kind == "gemm")
    assert g == pytest.approx(_gemm_flops_closed_form(cfg), rel=1e-12)
    # attention: 4 T^2 hd per (batch, head) forward, 10 T^2 hd backward
    if cfg.kind == "vit":
        a = sum(f for kind, _, f, _ in calls if kind == "attention")
        per = cfg.batch * cfg.heads * cfg.tokens ** 2 * cfg.head_dim
        assert a == pytest.approx(cfg.depth * 14.0 * per, rel=1e-12)
    # the optimizer moves 28 B per parameter
    opt = [b for kind, _, _, b in calls if kind == "optimizer"]
    assert opt == [28 * _n_params(cfg)]


def test_vit_b_step_flops_near_the_stated_total():
    # linear layers plus attention of the ViT-B step: about 6.7e12 flops
    cfg = workloads.get("vit_b")
    calls = bench.step_calls(cfg, _n_params(cfg))
    total = sum(f for kind, _, f, _ in calls if kind in ("gemm", "attention"))
    assert 6.6e12 < total < 6.8e12


def test_step_roofline_sums_the_per_call_bounds():
    cfg = workloads.get("vit_s")
    n = _n_params(cfg)
    r = bench.step_roofline(cfg, n, 2500.0, 10.0)
    want = sum(max(f / 2.5e15, b / 8e12) for _, _, f, b in bench.step_calls(cfg, n)) * 1e3
    assert r["ms"] == pytest.approx(want, abs=1e-4)
    assert r["frac"] == pytest.approx(r["ms"] / 10.0, abs=1e-4)
    assert sum(r["parts_ms"].values()) == pytest.approx(r["ms"], abs=1e-3)
    assert set(r["parts_ms"]) == {"gemm", "attention", "support", "optimizer"}
