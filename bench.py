"""Benchmark of the mixed-precision training step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--config NAME]
                [--no-cpu-baseline] [--no-sweep] [--step-only]

A step is one pass of the whole hot path over one synthetic batch: cast the
inputs, half forward, loss with the scale seed, half backward, unscale +
finite check, masked AdamW with the fused half copy, loss-scale update.
Inputs and parameters are resident in HBM before the timed region starts;
the step runs as one captured HIP graph.  The default workload is the
ViT-Base-like model (12 blocks, d 768, 197 tokens, batch 64, bf16), the
largest of the workloads.

Prints ONE JSON line.  `value` is train steps/s for the model workloads (or
unscale+AdamW GB/s for the optimizer sweep).  `roofline` covers the dominant
kernel: its launch duration comes from HIP events around a graph of
back-to-back launches with the step's own operands, on the stream they run
on (the median of five groups of replays); `bound` is whichever of the MFMA and HBM ceilings is the binding one for
its algorithmic flops and bytes (`frac` against that one; the other fraction
is given too).  `traffic` is the HBM bytes per launch from the FETCH_SIZE /
WRITE_SIZE counters, scaled by a plain copy's reading, or null when the
kernel sources changed since the counters were taken.  `gemm` times every
linear-layer GEMM call of one block against the dense MFMA peak.  `sweep`
(model workloads, unless --no-sweep) is the standalone optimizer sweep over
1e8 fp16 gradient elements in 200 tensors: unscale + check + masked AdamW +
scale update GB/s on applied steps (28 B per element), and the time of a
skipped step (a non-finite gradient: check, no AdamW write, scale halved)
separately.  `step_roofline` is the whole step's lower bound: every call of
the step at the larger of its MFMA time and its HBM time at peak for its
algorithmic flops and bytes, summed, and its ratio to the measured step
time.  `cpu_baseline` times the CPU oracle on a bounded sample.

--step-only runs the warmup and the timed steps and nothing else (no
per-kernel timing graphs, no sweep, no oracle), so that a kernel trace of
the run holds exactly the step's launches; it prints how many steps ran.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

import workloads

PEAK_MFMA_TFLOPS = {"f16": 2500.0, "bf16": 2500.0}   # dense, MI355X
PEAK_HBM_GBS = 8000.0
PEAK_F32_TFLOPS = 157.3                               # dense float32 MFMA, MI355X
DEFAULT_CONFIG = "vit_b"

# HBM bytes per launch of the dominant kernels from two rocprofv3 --pmc runs
# (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch), each scaled by what the
# same counter reads for a plain 256 MiB device copy in the same run (fetch
# about 131087 KiB -> factor 2.0000, write 262144.0 KiB -> factor 1.0000).  Each
# entry records the SHA-256 of the sources its kernel was built from; when
# they no longer match, the figure is stale and reported as null.
TRAFFIC = {
    "vit_block/blk0.up.fwd": {
        "fetch_kib": 13947.7, "write_kib": 49920.0,
        "fetch_factor": 262144.0 / 131088.8, "write_factor": 262144.0 / 262144.0,
        "sources": {
            "paper_2507_03312_amd/csrc/gemm_kernels.h": "8e0c308ac1b5d6809b80c6ae9e9dc05a12e6987d72d8b54d85ccd4a643a873ca",
            "paper_2507_03312_amd/csrc/mfma.h": "46e04f5162db64f2c8dc7bd5c5aae35c9ba491888000bfd3597337920e363231",
            "paper_2507_03312_amd/csrc/common.h": "2084a1c1294723c666ae58a2f812b765b2e5ea388fca5027c911b15626f0d620",
        },
    },
    "vit_s/blk0.up.fwd": {
        "fetch_kib": 23660.5, "write_kib": 99840.0,
        "fetch_factor": 262144.0 / 131088.3, "write_factor": 262144.0 / 262144.0,
        "sources": {
            "paper_2507_03312_amd/csrc/gemm_kernels.h": "8e0c308ac1b5d6809b80c6ae9e9dc05a12e6987d72d8b54d85ccd4a643a873ca",
            "paper_2507_03312_amd/csrc/mfma.h": "46e04f5162db64f2c8dc7bd5c5aae35c9ba491888000bfd3597337920e363231",
            "paper_2507_03312_amd/csrc/common.h": "2084a1c1294723c666ae58a2f812b765b2e5ea388fca5027c911b15626f0d620",
        },
    },
    "vit_b/blk0.up.fwd": {
        "fetch_kib": 70788.5, "write_kib": 151342.8,
        "fetch_factor": 262144.0 / 131093.6, "write_factor": 262144.0 / 262144.0,
        "sources": {
            "paper_2507_03312_amd/csrc/gemm_kernels.h": "8e0c308ac1b5d6809b80c6ae9e9dc05a12e6987d72d8b54d85ccd4a643a873ca",
            "paper_2507_03312_amd/csrc/mfma.h": "46e04f5162db64f2c8dc7bd5c5aae35c9ba491888000bfd3597337920e363231",
            "paper_2507_03312_amd/csrc/common.h": "2084a1c1294723c666ae58a2f812b765b2e5ea388fca5027c911b15626f0d620",
        },
    },
    "sweep/adamw": {
        "fetch_kib": 686821.7, "write_kib": 1367203.9,
        "fetch_factor": 262144.0 / 131088.6, "write_factor": 262144.0 / 262144.0,
        "sources": {
            "paper_2507_03312_amd/csrc/sweep.hip": "f6f3065d68b04a498769c3ad2b517512429bc5c108dc6a722f6d23eff5d6b987",
            "paper_2507_03312_amd/csrc/common.h": "2084a1c1294723c666ae58a2f812b765b2e5ea388fca5027c911b15626f0d620",
        },
    },
}


def traffic_bytes(name):
    """HBM bytes of one launch of a workload's dominant kernel ("workload/site"),
    from the stored counter readings, or None when none were taken for that
    workload or a source they depend on has changed since."""
    import hashlib
    t = TRAFFIC.get(name)
    if not t:
        return None
    root = os.path.dirname(os.path.abspath(__file__))
    for rel, digest in t["sources"].items():
        with open(os.path.join(root, rel), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    return int(round((t["fetch_kib"] * t["fetch_factor"] + t["write_kib"] * t["write_factor"]) * 1024))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--config", default=None, choices=workloads.CONFIG_ORDER,
                    help=f"workload (default {DEFAULT_CONFIG}; mlp for --compare-precision)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="model workloads: leave out the optimizer-sweep sub-object")
    ap.add_argument("--step-only", action="store_true",
                    help="warmup and timed steps only (for kernel traces of the step)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--compare-precision", action="store_true",
                    help="step time and peak device memory of full precision (mixed precision "
                         "switched off) against mixed precision over batch sizes, for the "
                         "workload of --config (mlp when the default is left)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB "
                         "(reference dispatch for hardware byte counters)")
    return ap.parse_args()


def cpu_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        return int(max(n)) if n else 1
    except Exception:
        return 1


def cpu_baseline_train(cfg, budget_s):
    """Oracle training steps on the host, as many as fit the time budget (>= 1).

    When one step of the full model would take far longer than the budget
    (ViT-S, ViT-B), the sample is the oracle's gradient computation and
    update at depths 1 and 2 of the same workload (full batch, width and
    token count); the per-block cost t2 - t1 and the rest (embedding, head,
    optimizer) t1 - (t2 - t1) give the full step by a linear model in the
    depth, which is how the oracle's work grows (blocks are identical)."""
    from oracle import step as ostep
    if cfg.kind == "vit" and cfg.depth > 2 and cfg.batch * cfg.tokens * cfg.d_model * cfg.depth > 1e8:
        times = []
        for depth in (1, 2):
            c = workloads.scaled_down(cfg, depth=depth)
            st = ostep.init_state(c)
            batch = workloads.make_batch(c)
            t0 = time.perf_counter()
            ostep.train_step(c, st, batch, 0)
            times.append(time.perf_counter() - t0)
        per_block = max(times[1] - times[0], 1e-9)
        est = times[0] - per_block + cfg.depth * per_block
        return {"value": 1.0 / est, "unit": "steps/s", "cores": cpu_threads(), "kind": "oracle",
                "sample": f"one oracle training step of the '{cfg.name}' workload at depth 1 "
                          f"({times[0]:.1f} s) and at depth 2 ({times[1]:.1f} s), full batch and "
                          f"width; the {cfg.depth}-block step is extrapolated linearly in the "
                          f"depth: {est:.1f} s"}
    st = ostep.init_state(cfg)
    batch = workloads.make_batch(cfg)
    t0 = time.perf_counter()
    n = 0
    while True:
        st, _ = ostep.train_step(cfg, st, batch, n)
        n += 1
        if time.perf_counter() - t0 >= budget_s or n >= cfg.steps:
            break
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "steps/s", "cores": cpu_threads(), "kind": "oracle",
            "sample": f"{n} full oracle training step(s) of the '{cfg.name}' workload, "
                      f"{dt:.1f} s"}


def cpu_baseline_sweep(cfg, budget_s):
    """Oracle unscale + check + adjust + AdamW over a prefix of the tensor list."""
    from oracle import step as ostep
    sizes = workloads.sweep_sizes(cfg)
    take, tot = [], 0
    for i, n in enumerate(sizes):               # about 1e7 elements
        take.append(int(n))
        tot += int(n)
        if tot >= 10_000_000:
            break
    cfg_s = workloads.SweepConfig(**{**cfg.__dict__, "n_tensors": len(take), "total": tot,
                                     "injections": ()})
    gf, params = workloads.sweep_tensors(cfg_s, np.array(take, np.int64))
    gh, st = ostep.sweep_init(cfg_s, gf, params)
    t0 = time.perf_counter()
    n = 0
    while True:
        st, _, _ = ostep.sweep_step(cfg_s, st, gh, n)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    gbs = n * tot * 28 / dt / 1e9
    return {"value": gbs, "unit": "GB/s", "cores": cpu_threads(), "kind": "oracle",
            "sample": f"{n} applied sweep step(s) over the first {len(take)} tensors "
                      f"({tot} elements) of the sweep workload, {dt:.1f} s"}


def calibration_copy(args, dev):
    """One plain device copy of --copy-calibration-mib MiB after the timed
    region: the reference dispatch that scales the hardware byte counters."""
    if not args.copy_calibration_mib:
        return
    import torch
    n = args.copy_calibration_mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()


def step_calls(cfg, n_params: int):
    """(kind, name, flops, bytes) of every call of one mixed-precision step:
    the algorithmic work, each operand read once and each result written once
    (half values 2 B, float32 4 B; split-K partials, re-reads and workspaces
    are not algorithmic).  kind is "gemm", "attention", "support" or
    "optimizer"."""
    h = 2
    out = []

    def gemm(name, M, N, K, extra_in=0, outs=1, bias=True, kind="gemm"):
        # C[M, N] = A[M, K] B[N, K]^T (+ bias, + extra operands of M x N)
        b = h * (M * K + N * K + (N if bias else 0) + (extra_in + outs) * M * N)
        out.append((kind, name, 2.0 * M * N * K, b))

    def support(name, b):
        out.append(("support", name, 0.0, b))

    B = cfg.batch
    if cfg.kind == "mlp":
        D, Hd = cfg.d_in, cfg.d_hidden
        support("cast inputs, targets", 2 * B * D * (4 + h))
        gemm("fc1.fwd+gelu", B, Hd, D, outs=2)
        gemm("fc2.fwd", B, D, Hd)
        support("mse", 2 * B * D * h + B * D * h)
        gemm("fc2.dW", D, Hd, B, bias=False)                       # dW = dY^T H (+ db)
        gemm("fc2.dX+gelu'", B, Hd, D, extra_in=1, bias=False)
        gemm("fc1.dW", Hd, D, B, bias=False)
    else:
        T, d, F, H, hd, L, C = cfg.tokens, cfg.d_model, cfg.d_mlp, cfg.heads, cfg.head_dim, cfg.depth, cfg.classes
        M, ldP = B * T, -(-T // 8) * 8
        att_f = B * H * (4.0 * T * T * hd)
        att_fb = h * B * H * (4 * T * hd + T * ldP)               # Q, K, V read; O, P written
        att_bf = B * H * (10.0 * T * T * hd)
        att_bb = h * B * H * (7 * T * hd + T * ldP)               # Q, K, V, dO, P read; dQKV written
        if cfg.image:
            G, Pd = cfg.n_patches, cfg.patch_dim
            support("patchify+cast", B * cfg.image * cfg.image * cfg.channels * 4 + B * G * Pd * h)
            gemm("patch.fwd", B * G, d, Pd)
            support("embed assemble", h * (B * G * d + T * d + M * d))
        for i in range(L):
            p = f"blk{i}."
            if i == 0 and not cfg.image:
                support(p + "ln1.fwd+cast", M * d * (4 + 2 * h))
            else:
                support(p + "ln1.fwd", 2 * h * M * d)
            gemm(p + "qkv.fwd", M, 3 * d, d)
            out.append(("attention", p + "attn.fwd", att_f, att_fb))
            gemm(p + "proj.fwd+res", M, d, d, extra_in=1)
            support(p + "ln2.fwd", 2 * h * M * d)
            gemm(p + "up.fwd+gelu", M, F, d, outs=2)
            gemm(p + "down.fwd+res", M, d, F, extra_in=1)
        # fused head: final LN on the CLS rows, logits, CE with the scale seed,
        # backward to the LN input; its weight gradient
        gemm("head.fwd", B, C, d)
        gemm("head.dX", B, d, C, bias=False)
        gemm("head.dW", C, d, B, bias=False)
        for i in reversed(range(L)):
            p = f"blk{i}."
            gemm(p + "down.dW", d, F, M, bias=False)
            gemm(p + "down.dX+gelu'", M, F, d, extra_in=1, bias=False)
            gemm(p + "up.dW", F, d, M, bias=False)
            gemm(p + "up.dX", M, d, F, bias=False)
            support(p + "ln2.bwd", 4 * h * M * d)                   # x1, dc, residual read; dx1 written
            gemm(p + "proj.dW", d, d, M, bias=False)
            gemm(p + "proj.dX", M, d, d, bias=False)
            out.append(("attention", p + "attn.bwd", att_bf, att_bb))
            gemm(p + "qkv.dW", 3 * d, d, M, bias=False)
            gemm(p + "qkv.dX", M, d, 3 * d, bias=False)
            last_tokens = i == 0 and not cfg.image                 # gamma / beta only
            support(p + "ln1.bwd", (2 if last_tokens else 4) * h * M * d)
        if cfg.image:
            support("embed assemble.bwd", h * (M * d + B * G * d))
            gemm("patch.dW", d, Pd, B * G, bias=False)
    out.append(("optimizer", "masked AdamW + half copy", 0.0, 28 * n_params))
    return out


def step_roofline(cfg, n_params: int, peak_tflops: float, ms_per_step: float):
    """The step's lower bound: each call at the larger of its MFMA time and
    its HBM time at peak, summed (calls that run side by side could overlap
    one's compute with another's traffic, so this is the serial bound)."""
    parts = {}
    flops = byts = 0.0
    for kind, _, f, b in step_calls(cfg, n_params):
        t = max(f / (peak_tflops * 1e12), b / (PEAK_HBM_GBS * 1e9)) * 1e3
        parts[kind] = parts.get(kind, 0.0) + t
        flops += f
        byts += b
    ms = sum(parts.values())
    return {"ms": round(ms, 4), "frac": round(ms / ms_per_step, 4),
            "parts_ms": {k: round(v, 4) for k, v in parts.items()},
            "flops": flops, "bytes": int(byts),
            "rule": "sum over the step's calls of max(flops / MFMA peak, algorithmic bytes / HBM peak)"}


def gemm_table(st, peak):
    """TFLOP/s of each distinct linear-layer GEMM call of the step (forward,
    dX, dW + db), each timed like the dominant kernel, and the FLOP-weighted
    aggregate over one block's calls, against the dense MFMA peak."""
    sites = st.gemm_sites()
    if not sites:
        return None
    out, fl, tm = {}, 0.0, 0.0
    for name, M, N, K, call in sites:
        ms = st.time_call(call)
        f = 2.0 * M * N * K
        out[name] = {"M": M, "N": N, "K": K, "us": round(ms * 1e3, 2),
                     "tflops": round(f / (ms * 1e-3) / 1e12, 1)}
        if name.startswith("blk0."):
            fl += f
            tm += ms
    agg = fl / (tm * 1e-3) / 1e12
    return {"sites": out, "block_aggregate_tflops": round(agg, 1), "peak": peak,
            "block_aggregate_frac": round(agg / peak, 4)}


def compare_precision(args, dev):
    """Full precision vs mixed precision over batch sizes: graph-replayed step
    time and the peak device memory the step allocates (parameters, optimizer
    state, inputs, activations, workspaces), the shape of the paper's
    comparison (§4).  MLP workload: batches 64 .. 131072; a ViT workload: half
    to four times its batch (ViT-S: 128 .. 1024, the paper's range)."""
    import torch
    from paper_2507_03312_amd.train import make_step
    name = args.config or "mlp"
    if name == "sweep":
        raise SystemExit("--compare-precision needs a training workload")
    base_cfg = workloads.get(name)
    rows = []
    gemm = {}
    if name == "mlp":
        batches = [64, 1024, 8192, 32768, 131072]
    else:
        batches = [base_cfg.batch // 2, base_cfg.batch, 2 * base_cfg.batch, 4 * base_cfg.batch]
    for B in batches:
        cfg = workloads.scaled_down(base_cfg, batch=B)
        batch = workloads.make_batch(cfg)
        row = {"batch": B}
        for full in (True, False):
            key = "full" if full else "mixed"
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            torch.cuda.reset_peak_memory_stats(dev)
            base = torch.cuda.memory_allocated(dev)
            st = make_step(cfg, dev, full_precision=full)
            st.set_batch(batch)
            st.step()
            st.capture()
            for _ in range(2):
                st.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            st.replay()
            e1.record()
            torch.cuda.synchronize()
            # about half a second of replays per point
            steps = int(max(3, min(2000, 500.0 / max(e0.elapsed_time(e1), 1e-3))))
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            t0.record()
            for _ in range(steps):
                st.replay()
            t1.record()
            torch.cuda.synchronize()
            row[key + "_ms"] = round(t0.elapsed_time(t1) / steps, 4)
            row[key + "_mib"] = round((torch.cuda.max_memory_allocated(dev) - base) / 2 ** 20, 1)
            if B == batches[-1]:
                site = st.dominant_site()
                k_ms = st.time_dominant()
                tf = site["flops"] / (k_ms * 1e-3) / 1e12
                peak = PEAK_F32_TFLOPS if full else PEAK_MFMA_TFLOPS[cfg.half]
                gemm[key] = {"kernel": site["desc"], "us": round(k_ms * 1e3, 2),
                             "tflops": round(tf, 1), "peak": peak, "frac": round(tf / peak, 4)}
            del st
        row["speedup"] = round(row["full_ms"] / row["mixed_ms"], 3)
        row["memory_ratio"] = round(row["full_mib"] / row["mixed_mib"], 3)
        rows.append(row)
        print(json.dumps(row), file=sys.stderr, flush=True)
    last = rows[-1]
    st = make_step(workloads.scaled_down(base_cfg, batch=1), dev)
    desc = st.describe().split(", batch")[0]
    del st
    line = {"metric": "full-precision / mixed-precision step time", "value": last["speedup"],
            "unit": "x", "n_gpus": 1, "steps": None, "warmup": 3,
            "ms_per_step": last["mixed_ms"], "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "f32 vs " + base_cfg.half, "data": "synthetic",
            "config": {"workload": desc + "; full precision (f32 layers, no loss scaling) vs "
                                          "mixed precision (" + base_cfg.half + " layers, dynamic "
                                          "loss scaling), batch sizes " + ",".join(map(str, batches)),
                       "parallelism": "none"},
            "comparison": rows, "gemm_at_largest_batch": gemm}
    print(json.dumps(line))


def measure_sweep(dev, steps, warm, step_only=False):
    """The optimizer-sweep workload (1e8 fp16 gradient elements in 200
    tensors): GB/s of whole applied steps (unscale + check, masked AdamW with
    the half copy, scale update; 28 B per element algorithmic), the time of a
    skipped step (one +inf in the gradients: the check, AdamW writing
    nothing, the scale halved), and the AdamW kernel alone (the dominant
    kernel).  Each step runs as one captured HIP graph."""
    import torch
    from paper_2507_03312_amd.sweep import SweepStep
    cfg = workloads.get("sweep")
    sw = SweepStep(cfg, device=dev)
    gf, params = workloads.sweep_tensors(cfg, sw.sizes)
    sw.load(gf, params)
    del gf, params
    torch.cuda.synchronize()
    for _ in range(warm):
        sw.step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sw.step()
    torch.cuda.synchronize()

    def timed(n):
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(n):
            g.replay()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n

    applied_ms = timed(steps)
    if step_only:
        print(f"step-only: {warm} eager sweep steps, then {steps + 2} graph replays of the step",
              file=sys.stderr)
        return {"value": round(sw.numel * 28 / (applied_ms * 1e-3) / 1e9, 1),
                "ms_per_applied_step": round(applied_ms, 4)}
    k_ms = sw.time_graph(sw.adamw)   # AdamW alone (applied)
    saved = sw.inject(workloads.Injection(0, 0, 0, float("inf")))
    applied_before = int(sw.d_step.item())
    skipped_ms = timed(max(steps // 2, 5))
    assert int(sw.d_step.item()) == applied_before, "a skipped step applied AdamW"
    sw.restore(saved)
    bytes_per = sw.numel * 28
    gbs = bytes_per / (applied_ms * 1e-3) / 1e9
    k_gbs = bytes_per / (k_ms * 1e-3) / 1e9
    out = {"metric": "unscale+AdamW GB/s", "value": round(gbs, 1), "unit": "GB/s",
           "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "ms_per_applied_step": round(applied_ms, 4),
           "skipped_step_ms": round(skipped_ms, 4), "elements": sw.numel, "bytes_per_element": 28,
           "steps": steps, "workload": "200 fp16 gradient tensors, lognormal sizes summing to 1e8 "
                                       "elements, fp32 masters/m/v, scale 2^16; a step = unscale + "
                                       "check, masked AdamW + half copy, scale update",
           "adamw_kernel": {"bound": "hbm", "achieved": round(k_gbs, 1), "peak": PEAK_HBM_GBS,
                            "unit": "GB/s", "frac": round(k_gbs / PEAK_HBM_GBS, 4),
                            "traffic": traffic_bytes("sweep/adamw"),
                            "kernel": "masked AdamW + half copy, 28 B/element",
                            "avg_launch_ms": round(k_ms, 4)}}
    del sw, g
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(data-parallel sharding is not implemented)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2507_03312_amd.train import make_step

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    if args.compare_precision:
        compare_precision(args, dev)
        return
    name = args.config or DEFAULT_CONFIG
    cfg = workloads.get(name)

    if name == "sweep":
        steps = args.steps or 50
        warm = args.warmup if args.warmup is not None else 5
        sw = measure_sweep(dev, steps, warm, args.step_only)
        if args.step_only:
            print(json.dumps({"metric": "unscale+AdamW GB/s", "value": sw["value"], "unit": "GB/s",
                              "ms_per_step": sw["ms_per_applied_step"], "steps": steps,
                              "warmup": warm, "step_only": True}))
            return
        calibration_copy(args, dev)
        line = {"metric": "unscale+AdamW GB/s", "value": sw["value"], "unit": "GB/s",
                "n_gpus": 1, "steps": steps, "warmup": warm, "ms_per_step": sw["ms_per_applied_step"],
                "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                "dtype": "f32 (f16 gradients)", "data": "synthetic",
                "config": {"workload": "sweep: " + sw["workload"], "elements": sw["elements"],
                           "parallelism": "none"},
                "roofline": sw["adamw_kernel"], "skipped_step_ms": sw["skipped_step_ms"]}
        if not args.no_cpu_baseline:
            line["cpu_baseline"] = cpu_baseline_sweep(cfg, args.cpu_seconds)
        print(json.dumps(line))
        return

    steps = args.steps or {"mlp": 500, "vit_block": 300, "vit_s": 50, "vit_b": 30}[name]
    warm = args.warmup if args.warmup is not None else 5
    st = make_step(cfg, dev)
    st.set_batch(workloads.make_batch(cfg))
    site = st.dominant_site()
    torch.cuda.synchronize()
    for _ in range(warm):                 # eager steps (also the first cast)
        st.step()
    st.capture()                          # the whole step as one HIP graph
    for _ in range(warm):
        st.replay()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        st.replay()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    if args.step_only:
        calibration_copy(args, dev)
        print(f"step-only: {warm} eager steps, then {warm + steps} graph replays of the step "
              f"({2 * warm + steps} steps in all; the first eager step also casts the masters)",
              file=sys.stderr)
        print(json.dumps({"metric": "train steps/s", "value": round(1000.0 / ms, 3), "unit": "steps/s",
                          "n_gpus": 1, "steps": steps, "warmup": warm, "ms_per_step": round(ms, 4),
                          "config": {"workload": st.describe()}, "step_only": True}))
        return
    k_ms = st.time_dominant()
    calibration_copy(args, dev)
    peak = PEAK_MFMA_TFLOPS[cfg.half]
    tflops = site["flops"] / (k_ms * 1e-3) / 1e12
    gbs = site["bytes"] / (k_ms * 1e-3) / 1e9
    # the binding ceiling: the larger of the MFMA time and the HBM time at peak
    hbm_bound = site["bytes"] / PEAK_HBM_GBS > site["flops"] / (peak * 1e3)
    if hbm_bound:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "mfma_frac": round(tflops / peak, 4)}
    else:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(tflops / peak, 4), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
    roof.update({"traffic": traffic_bytes(name + "/" + site["name"]), "algorithmic_bytes": site["bytes"],
                 "flops": site["flops"], "kernel": site["desc"], "avg_launch_ms": round(k_ms, 5)})
    gemm = gemm_table(st, peak)
    line = {"metric": "train steps/s", "value": round(1000.0 / ms, 3), "unit": "steps/s",
            "n_gpus": 1, "steps": steps, "warmup": warm, "ms_per_step": round(ms, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": cfg.half, "data": "synthetic",
            "config": {"workload": st.describe(), "global_batch": cfg.batch,
                       "seq_len": cfg.tokens or None, "parallelism": "none"},
            "roofline": roof}
    if gemm:
        line["gemm"] = gemm
    n_params = sum(int(np.prod(shape)) for _, shape, _ in workloads.param_specs(cfg))
    line["step_roofline"] = step_roofline(cfg, n_params, peak, ms)
    del st
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_sweep:
        line["sweep"] = measure_sweep(dev, 50, 5)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_train(cfg, args.cpu_seconds)
        if not args.no_sweep:
            line["sweep"]["cpu_baseline"] = cpu_baseline_sweep(workloads.get("sweep"),
                                                               min(args.cpu_seconds, 8.0))
    print(json.dumps(line))


if __name__ == "__main__":
    main()
