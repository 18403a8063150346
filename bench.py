"""Benchmark of the ReLU-sparse FFN forward on one MI355X.

Workload: one non-gated bf16 FFN layer, T=8192 tokens, d=4096, f=16384, 99% of the
hidden units inactive (uniformly random active units per token), ELL width K=256,
TwELL tiles T_n=256 with S=32 slots. Inputs are seeded synthetic data resident in HBM.

A step is one sfl_ffn_forward call: up projection with the fused ReLU -> TwELL
epilogue, hybrid classification, sparse down projection and the dense-backup rows.
The library's dense FFN (sfl_dense_ffn_baseline) is timed the same way for the
speedup. Per-stage times come from HIP events the library records on its stream.

Prints one JSON line (see the keys below). `--gpus` above 1 is refused: this build
runs on one GPU.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--sparsity", type=float, default=0.99)
    p.add_argument("--tokens", type=int, default=8192)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--skip-dense", action="store_true")
    return p.parse_args()


def file_hash(*paths):
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel_key, src_hash):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken
    on the current kernel source; None otherwise."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(kernel_key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != src_hash:
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(w, seconds):
    """The oracle's hybrid forward (fp64) on a bounded, seeded sample of the same rows."""
    import oracle.ffn as off
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    rng = np.random.default_rng(123)
    X = w.as_f64(w.X)
    Wu = w.as_f64(w.W_up)
    Wd = w.as_f64(w.W_down)
    n = 64
    done_rows, spent = 0, 0.0
    while spent < seconds and done_rows < w.T:
        rows = rng.choice(w.T, size=min(n, w.T), replace=False)
        t0 = time.perf_counter()
        off.ffn_hybrid_forward(X[rows], Wu, Wd, w.bias_f, w.shift_t[rows], tile_cols=w.cfg["tile_cols"],
                               tile_slots=w.cfg["tile_slots"], ell_width=w.cfg["ell_width"], val_dtype="bf16")
        dt = time.perf_counter() - t0
        spent += dt
        done_rows += len(rows)
        if dt < seconds / 8:
            n = min(w.T, n * 2)
    return {"value": done_rows / spent, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{done_rows} seeded random rows of the same workload (fp64 oracle: pre-activation, "
                      f"TwELL extraction, hybrid classification, ELL gather / dense rows), {spent:.1f} s"}


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)
    import torch

    import workloads as wl
    from paper_2603_23198_amd import binding as b

    torch.cuda.set_device(0)
    w = wl.c4_sweep(a.sparsity, T=a.tokens)
    T, d, f = w.T, w.d, w.f
    bf = lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).cuda().view(torch.bfloat16)
    X, Wu, Wd = bf(w.X), bf(w.W_up), bf(w.W_down)
    shift = torch.from_numpy(w.shift_t).cuda()
    cfg = b.make_cfg(**w.cfg)
    bufs = b.alloc_twell(T, f, "bf16", cfg)
    Y = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    stats = b.alloc_stats()
    # inference weights are laid out once, before any step: W_down also in the slice-major
    # copy the sparse down projection reads (sfl_pack_down_weights)
    WdP = torch.empty_like(Wd)
    b.sfl_pack_down_weights(Wd, WdP)
    args = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, W_down_packed=WdP, shift_t=shift, stats=stats)
    ws = torch.empty(max(1, b.sfl_workspace_size(args)), dtype=torch.uint8, device="cuda")
    args = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, W_down_packed=WdP, shift_t=shift, stats=stats, workspace=ws)
    stream = torch.cuda.current_stream()

    def fwd(ar):
        b.sfl_ffn_forward(ar, stream)

    for _ in range(a.warmup):
        fwd(args)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(a.steps):
        fwd(args)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / a.steps
    st = b.read_stats(stats)

    # per-stage times from events recorded by the library on the same stream
    n_ev = 5
    stage_ms = np.zeros(n_ev - 1)
    for _ in range(a.steps):
        ev = b.create_events(n_ev)
        sa = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, W_down_packed=WdP, shift_t=shift, stats=stats,
                        workspace=ws, events=ev)
        fwd(sa)
        torch.cuda.synchronize()
        stage_ms += np.array([b.event_ms(ev, i, i + 1) for i in range(n_ev - 1)])
    stage_ms /= a.steps
    stages = dict(zip(["up_gemm_twell", "classify", "gather_down", "dense_backup"], stage_ms.round(4).tolist()))

    # the same step when W_down is re-laid out inside every call (no pre-packed copy)
    uargs = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, shift_t=shift, stats=stats)
    uws = torch.empty(max(1, b.sfl_workspace_size(uargs)), dtype=torch.uint8, device="cuda")
    uargs = b.ffn_args(X, Wu, Wd, cfg, Y=Y, bufs=bufs, shift_t=shift, stats=stats, workspace=uws)
    for _ in range(a.warmup):
        fwd(uargs)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(a.steps):
        fwd(uargs)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_unpacked = e0.elapsed_time(e1) / a.steps
    del uws

    dense_ms = None
    if not a.skip_dense:
        dws = torch.empty(b.sfl_workspace_size(args, 2), dtype=torch.uint8, device="cuda")
        Yd = torch.empty_like(Y)
        dargs = b.ffn_args(X, Wu, Wd, cfg, Y=Yd, shift_t=shift, workspace=dws)
        for _ in range(a.warmup):
            b.sfl_dense_ffn_baseline(dargs, stream)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(a.steps):
            b.sfl_dense_ffn_baseline(dargs, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        dense_ms = e0.elapsed_time(e1) / a.steps
        del dws, Yd

    # roofline of the dominant kernel (the up-projection GEMM with the TwELL epilogue)
    up_flops = 2.0 * T * d * f
    up_s = stages["up_gemm_twell"] * 1e-3
    achieved = up_flops / up_s / 1e12
    csrc = os.path.join(ROOT, "paper_2603_23198_amd", "csrc")
    gemm_hash = file_hash(os.path.join(csrc, "gemm.hip"), os.path.join(csrc, "common.h"))
    gather_hash = file_hash(os.path.join(csrc, "gather.hip"), os.path.join(csrc, "common.h"))
    traffic = measured_traffic("up_gemm_twell", gemm_hash)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_MFMA_PEAK_TFLOPS, 4), "traffic": traffic,
                "kernel": "k_gemm_bf16<KC,RC,TWELL>", "work": "2*T*d*f flops per launch"}
    # the sparse down projection: algorithmic bytes = sum_t nnz_t*(2d + 4) + 2d + 5
    nnz = int(st["total_nnz"])
    n_sparse = T - int(st["n_ovf_rows"])
    gbytes = nnz * (2 * d + 4) + n_sparse * (2 * d + 5)
    g_s = stages["gather_down"] * 1e-3
    gather = {"bound": "hbm", "achieved": round(gbytes / g_s / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
              "frac": round(gbytes / g_s / 1e9 / HBM_PEAK_GBS, 4), "algorithmic_bytes": gbytes,
              "traffic": measured_traffic("gather_down", gather_hash),
              "note": "effective rate: W_down rows are re-read per token and served mostly from L2/MALL"}

    out = {
        "metric": "sparse FFN tokens/sec at 99% sparsity; HBM GB/s % peak; speedup vs dense FFN",
        "value": round(T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian X and weights; per-row shift gives uniformly random active units)",
        "config": {"workload": f"non-gated ReLU FFN forward, bf16, T={T}, d={d}, f={f}, sparsity={a.sparsity}",
                   "tokens": T, "d": d, "f": f, "sparsity_target": a.sparsity,
                   "realised_sparsity": round(1 - nnz / (T * f), 5), "ell_width": cfg.ell_width,
                   "tile_cols": cfg.tile_cols, "tile_slots": cfg.tile_slots, "parallelism": "single GPU"},
        "dense_ms_per_step": None if dense_ms is None else round(dense_ms, 4),
        "speedup_vs_dense": None if dense_ms is None else round(dense_ms / ms, 4),
        "stages_ms": stages,
        "ms_per_step_w_down_packed_per_call": round(ms_unpacked, 4),
        "n_ovf_rows": int(st["n_ovf_rows"]),
        "roofline": roofline,
        "gather_roofline": gather,
    }
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
