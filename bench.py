"""Benchmark of the ReLU-sparse FFN layer on one MI355X.

Headline workload: one non-gated bf16 FFN layer, T=8192 tokens, d=4096, f=16384, 99% of
the hidden units inactive (uniformly random active units per token), ELL width K=256,
TwELL tiles T_n=256 with S=32 slots. Inputs are seeded synthetic data resident in HBM;
the weights are laid out once before timing (W_down also in the slice-major copy the
sparse down projection reads).

A step is one sfl_ffn_forward call: up projection with the fused ReLU -> TwELL
epilogue, hybrid classification, sparse down projection and the dense-backup rows.
The library's dense FFN (sfl_dense_ffn_baseline) is timed the same way for the
speedup. Per-stage times come from HIP events the library records on its stream.

The same JSON line also reports the other workloads of the hot path (sparsity sweep,
lognormal row counts with dense-backup rows, gated forward at prefill and decode sizes,
the training step: forward + backward with the L1 term, and one GPU's share of the
headline layer split eight ways over hidden units or over tokens). `--quick` skips them.
`--gpus` above 1 is refused: the benchmark runs on one GPU.
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
    p.add_argument("--quick", action="store_true", help="headline workload only")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="first run one plain 256 MiB device copy (reference for HBM byte counters)")
    p.add_argument("--only", choices=["lognormal", "gated", "decode", "train", "gated_train", "tp8", "dp8", "fp32",
                                       "splitd"],
                   help="run one secondary workload and print its record (for profiling); no headline line")
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
    rec = profile_record(kernel_key, src_hash)
    return None if rec is None else rec.get("hbm_bytes_per_launch")


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def profile_record(kernel_key, src_hash):
    """The committed rocprofv3 figures (kernel-trace average duration, counter readings) of
    one kernel, if they were taken on the current kernel source; None otherwise."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(kernel_key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != src_hash:
        return None
    return rec


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
    while spent < seconds:
        rows = rng.choice(w.T, size=min(n, w.T), replace=False)
        t0 = time.perf_counter()
        off.ffn_hybrid_forward(X[rows], Wu, Wd, w.bias_f, w.shift_t[rows], tile_cols=w.cfg["tile_cols"],
                               tile_slots=w.cfg["tile_slots"], ell_width=w.cfg["ell_width"], val_dtype="bf16")
        dt = time.perf_counter() - t0
        spent += dt
        done_rows += len(rows)
        if dt < seconds / 8:
            n = min(w.T, n * 2)
    return {"value": round(done_rows / spent, 1), "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{done_rows} seeded random rows of the same workload (fp64 oracle: pre-activation, "
                      f"TwELL extraction, hybrid classification, ELL gather / dense rows), {spent:.1f} s"}


def dense_fallback_taken(b, s, w):
    """Whether sfl_ffn_forward took its dense fallback for this workload (the library's rule:
    a candidate by ELL width, then the sparse rows' entries against T f / 64)."""
    if w.gated or w.dtype != "bf16" or w.T <= 256 or w.cfg["ell_width"] * 32 < w.f:
        return False
    nnz = s["bufs"]["row_nnz"][:w.T].cpu().numpy()
    ovf = s["bufs"]["row_ovf"][:w.T].cpu().numpy()
    return bool(int(nnz[ovf == 0].sum()) * 64 > w.T * w.f)


class Bench:
    def __init__(self, b, torch, steps, warmup):
        self.b, self.torch, self.steps, self.warmup = b, torch, steps, warmup
        self.stream = torch.cuda.current_stream()

    def dev(self, a):
        t = self.torch
        if a is None:
            return None
        if a.dtype == np.uint16:
            return t.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(t.bfloat16)
        return t.from_numpy(np.ascontiguousarray(a)).cuda()

    def time(self, fn, steps=None, warmup=None):
        """Mean ms per call over `steps` back-to-back calls, after `warmup` calls."""
        t = self.torch
        steps = steps or self.steps
        for _ in range(self.warmup if warmup is None else warmup):
            fn()
        t.cuda.synchronize()
        e0, e1 = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for _ in range(steps):
            fn()
        e1.record(self.stream)
        t.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    def per_call(self, fn, n=50, flush=None):
        """Per-call ms of n calls, each timed alone (events around it); with `flush`, that
        callable runs before each call, outside the timed span (cold caches)."""
        t = self.torch
        out = []
        for _ in range(n):
            if flush is not None:
                flush()
            e0, e1 = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
            e0.record(self.stream)
            fn()
            e1.record(self.stream)
            t.cuda.synchronize()
            out.append(e0.elapsed_time(e1))
        return np.array(out)

    def ceilings(self):
        """Bandwidth ceilings of this GPU (sfl_bandwidth_probe): HBM copy (1 GiB buffers),
        HBM read (4 GiB, one pass), L2 read (16 MiB, i.e. 2 MiB per XCD, re-read 400 times)."""
        b, t = self.b, self.torch
        sink = t.zeros(1, dtype=t.int32, device="cuda")
        out = {}

        def rate(fn):
            moved = fn()
            t.cuda.synchronize()
            e0, e1 = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
            e0.record(self.stream)
            moved = fn()
            e1.record(self.stream)
            t.cuda.synchronize()
            return round(moved / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)

        src = t.empty(1 << 30, dtype=t.uint8, device="cuda")
        dst = t.empty_like(src)
        out["hbm_copy_GBs"] = rate(lambda: b.sfl_bandwidth_probe(src, dst, reps=3, stream=self.stream))
        del dst
        big = t.empty(4 << 30, dtype=t.uint8, device="cuda")
        out["hbm_read_GBs"] = rate(lambda: b.sfl_bandwidth_probe(big, None, reps=1, sink=sink, stream=self.stream))
        del big
        small = src[:16 << 20]
        out["l2_read_GBs"] = rate(lambda: b.sfl_bandwidth_probe(small, None, reps=400, sink=sink,
                                                                stream=self.stream))
        del src, small
        out["how"] = ("sfl_bandwidth_probe: copy of 1 GiB (bytes read + written), one read pass over 4 GiB, "
                      "400 read passes over 16 MiB split so that each XCD re-reads its own 2 MiB")
        return out

    def stage_times(self, make_args, call, n_ev, steps=None):
        b = self.b
        steps = steps or self.steps
        acc = np.zeros(n_ev - 1)
        for _ in range(steps):
            ev = b.create_events(n_ev)
            call(make_args(ev), self.stream)
            self.torch.cuda.synchronize()
            acc += [b.event_ms(ev, i, i + 1) for i in range(n_ev - 1)]
        return (acc / steps).round(4).tolist()

    def setup_forward(self, w, packed=True):
        b, t = self.b, self.torch
        X, Wu, Wd = self.dev(w.X), self.dev(w.W_up), self.dev(w.W_down)
        Wg = self.dev(w.W_gate) if w.gated else None
        cfg = b.make_cfg(**w.cfg)
        act = t.bfloat16 if w.dtype == "bf16" else t.float32
        bufs = b.alloc_twell(w.T, w.f, "bf16" if w.dtype == "bf16" else "f32", cfg)
        Y = t.empty((w.T, w.d), dtype=act, device="cuda")
        stats = b.alloc_stats()
        WdP = WuP = WupT = WgT = WdT = None
        if packed and w.dtype == "bf16" and w.d % 512 == 0:
            WdP = t.empty_like(Wd)
            b.sfl_pack_down_weights(Wd, WdP)

        def transposed(W):
            out = t.empty((W.shape[1], W.shape[0]), dtype=W.dtype, device="cuda")
            b.sfl_transpose(W, out)
            return out

        if w.dtype == "bf16":
            # Transposed weight copies are kept beside the weights, like W_down's slice-major
            # copy: one-time layouts that let every dense GEMM (the up / gate projection, the
            # dense-backup rows, the dense baseline) read both operands K-contiguously.
            WupT, WdT = transposed(Wu), transposed(Wd)
            if w.gated:
                WgT = transposed(Wg)
            if packed and w.d % 512 == 0:
                # slice-major W_up^T: the gated forward's up-dots and the backward's dX read it
                WuP = t.empty_like(Wu)
                b.sfl_pack_down_weights(WupT, WuP)
        kw = dict(Y=Y, bufs=bufs, W_gate=Wg, W_upT=WupT, W_gateT=WgT, W_downT=WdT, W_down_packed=WdP,
                  W_up_packed=WuP if w.gated else None,
                  bias_f=self.dev(w.bias_f), shift_t=self.dev(w.shift_t), stats=stats)
        a0 = b.ffn_args(X, Wu, Wd, cfg, **kw)
        ws = t.empty(max(1, b.sfl_workspace_size(a0)), dtype=t.uint8, device="cuda")
        dws = t.empty(max(1, b.sfl_workspace_size(a0, 2)), dtype=t.uint8, device="cuda")
        s = dict(X=X, Wu=Wu, Wd=Wd, WupT=WupT, WdP=WdP, WuP=WuP, cfg=cfg, bufs=bufs, stats=stats, kw=kw, ws=ws,
                 dws=dws, Y=Y)
        s["args"] = b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws)
        dkw = dict(kw)
        dkw["Y"] = t.empty_like(Y)
        s["dargs"] = b.ffn_args(X, Wu, Wd, cfg, **dkw, workspace=dws)
        s["dkw"] = dkw
        s["mk"] = lambda ev: b.ffn_args(X, Wu, Wd, cfg, **kw, workspace=ws, events=ev)
        return s

    def forward_record(self, w, dense=True, stages=True, order_ab=False, fallback_ab=False):
        b = self.b
        s = self.setup_forward(w)
        ms = self.time(lambda: b.sfl_ffn_forward(s["args"], self.stream))
        if fallback_ab:
            # the same call with the dense fallback disabled (ELL gather for every sparse row)
            os.environ["SFL_DENSE_FALLBACK"] = "off"
            ms_off = self.time(lambda: b.sfl_ffn_forward(s["args"], self.stream))
            os.environ.pop("SFL_DENSE_FALLBACK", None)
        if order_ab:
            # the sparse down projection's token order: descending row count / token order
            # (the default picks one of them by batch size and ELL width)
            ab = {}
            for order in ("nnz", "token", "nnz", "token"):
                os.environ["SFL_TOKEN_ORDER"] = order
                ab.setdefault(order, []).append((self.time(lambda: b.sfl_ffn_forward(s["args"], self.stream)),
                                                 self.stage_times(s["mk"], b.sfl_ffn_forward, 5)[2]))
            os.environ.pop("SFL_TOKEN_ORDER", None)
        st = b.read_stats(s["stats"])
        rec = {"workload": w.name, "dtype": w.dtype, "tokens": w.T, "ms": round(ms, 4),
               "tokens_per_s": round(w.T / ms * 1e3, 1),
               "dense_fallback_taken": dense_fallback_taken(b, s, w),
               "realised_sparsity": round(1 - st["total_nnz"] / (w.T * w.f), 5), "n_ovf_rows": st["n_ovf_rows"]}
        if stages:
            rec["stages_ms"] = dict(zip(["up_gemm_twell", "classify", "sparse_down", "dense_backup"],
                                        self.stage_times(s["mk"], b.sfl_ffn_forward, 5)))
        if fallback_ab:
            rec["ms_dense_fallback_off"] = round(ms_off, 4)
        if order_ab:
            rec["token_order_ab"] = {
                o: {"ms": round(float(np.mean([x[0] for x in v])), 4),
                    "sparse_down_ms": round(float(np.mean([x[1] for x in v])), 4)} for o, v in ab.items()}
            rec["token_order_ab"]["note"] = ("SFL_TOKEN_ORDER=nnz (descending row count) / token; the order kernel "
                                             "runs inside the sparse down projection stage")
        if w.T <= 256:
            # launch-bound shapes: the same call captured once in a HIP graph and replayed
            t = self.torch
            g = t.cuda.CUDAGraph()
            side = t.cuda.Stream()
            side.wait_stream(self.stream)
            with t.cuda.stream(side):
                b.sfl_ffn_forward(s["args"], side)  # warm the code paths outside the capture
            self.stream.wait_stream(side)
            t.cuda.synchronize()
            with t.cuda.graph(g):
                b.sfl_ffn_forward(s["args"], t.cuda.current_stream())
            rec["graph_ms"] = round(self.time(g.replay), 4)
        if dense:
            dms = self.time(lambda: b.sfl_dense_ffn_baseline(s["dargs"], self.stream))
            rec["dense_ms"] = round(dms, 4)
            rec["speedup_vs_dense"] = round(dms / ms, 4)
            if w.T <= 256:
                t = self.torch
                g = t.cuda.CUDAGraph()
                with t.cuda.graph(g):
                    b.sfl_dense_ffn_baseline(s["dargs"], t.cuda.current_stream())
                rec["dense_graph_ms"] = round(self.time(g.replay), 4)
                rec["graph_speedup_vs_dense"] = round(rec["dense_graph_ms"] / rec["graph_ms"], 4)
            rec["dense_stages_ms"] = dict(zip(["up_gemm_relu", "down_gemm"],
                                              self.stage_times(lambda ev: b.ffn_args(
                                                  s["X"], s["Wu"], s["Wd"], s["cfg"], **s["dkw"],
                                                  workspace=s["dws"], events=ev),
                                                  b.sfl_dense_ffn_baseline, 3)))
            if not w.gated and w.dtype == "bf16":
                # the same dense FFN through torch (hipBLASLt GEMMs), for context
                t = self.torch
                X, Wd, WupT = s["X"], s["Wd"], s["WupT"]
                bias = None if w.bias_f is None else self.dev(w.bias_f).to(t.bfloat16)
                sh = None if w.shift_t is None else self.dev(w.shift_t).to(t.bfloat16)[:, None]

                def torch_dense():
                    Z = X @ WupT.t()
                    if bias is not None:
                        Z += bias
                    if sh is not None:
                        Z += sh
                    return t.relu_(Z) @ Wd

                tms = self.time(torch_dense)
                rec["dense_torch_ms"] = round(tms, 4)
                rec["speedup_vs_dense_torch"] = round(tms / ms, 4)
        return rec, s, st

    def splitd_record(self, w, splits=(1, 2, 4, 8)):
        """The forward's sparse down projection (slice-major walk, stage events) against the
        paper-shaped row-wise kernel (sfl_down_projection_rowwise) on the same ELL rows, for
        each split of d."""
        b = self.b
        s = self.setup_forward(w)
        b.sfl_ffn_forward(s["args"], self.stream)
        stages = dict(zip(["up_gemm_twell", "classify", "sparse_down", "dense_backup"],
                          self.stage_times(s["mk"], b.sfl_ffn_forward, 5)))
        Y2 = self.torch.empty_like(s["Y"])
        a2 = b.ffn_args(s["X"], s["Wu"], s["Wd"], s["cfg"], Y=Y2, bufs=s["bufs"])
        rw = {str(sp): round(self.time(lambda: b.sfl_down_projection_rowwise(a2, sp, self.stream)), 4)
              for sp in splits}
        best = min(rw, key=rw.get)
        return {"workload": w.name, "ell_width": w.cfg["ell_width"], "slice_walk_ms": stages["sparse_down"],
                "rowwise_ms_by_split": rw, "rowwise_best_split": int(best),
                "slice_walk_speedup_vs_best_rowwise": round(rw[best] / stages["sparse_down"], 3)}

    def training_record(self, w, lam):
        """Forward + backward (sfl_ffn_backward) of the layer, gated or not; the same dense
        layer through torch matmuls (hipBLASLt) for context."""
        b, t = self.b, self.torch
        s = self.setup_forward(w)
        dY = self.dev(w.dY)
        dX = t.empty((w.T, w.d), dtype=t.bfloat16, device="cuda")
        dWu = t.empty((w.d, w.f), dtype=t.float32, device="cuda")
        dWd = t.empty((w.f, w.d), dtype=t.float32, device="cuda")
        extra = dict(W_upT=s["WupT"], W_down_packed=s["WdP"], W_up_packed=s["WuP"])
        if w.gated:
            dWg = t.empty((w.d, w.f), dtype=t.float32, device="cuda")
            WgT = s["kw"]["W_gateT"]
            WgP = t.empty_like(WgT)
            b.sfl_pack_down_weights(WgT, WgP)
            extra.update(W_gate=s["kw"]["W_gate"], W_gateT=WgT, W_gate_packed=WgP, dW_gate=dWg,
                         bias_f=s["kw"]["bias_f"], shift_t=s["kw"]["shift_t"])
        bws = t.empty(max(1, b.sfl_workspace_size(
            b.bwd_args(s["X"], s["Wu"], s["Wd"], dY, s["cfg"], s["bufs"], lam, dX, dWu, dWd, **extra), 1)),
            dtype=t.uint8, device="cuda")
        mkb = lambda ev=None: b.bwd_args(s["X"], s["Wu"], s["Wd"], dY, s["cfg"], s["bufs"], lam, dX, dWu, dWd,
                                         workspace=bws, events=ev, **extra)
        bargs = mkb()

        def step():
            b.sfl_ffn_forward(s["args"], self.stream)
            b.sfl_ffn_backward(bargs, self.stream)

        steps = max(3, self.steps // 4)
        ms = self.time(step, steps=steps, warmup=2)
        bwd = self.stage_times(lambda ev: mkb(ev), b.sfl_ffn_backward, 6, steps=steps)
        rec = {"workload": w.name, "tokens": w.T, "ms_fwd_bwd": round(ms, 4),
               "tokens_per_s": round(w.T / ms * 1e3, 1), "lambda_l1": lam,
               "backward_stages_ms": dict(zip(["dh_at_pattern", "dx_gather", "pattern_transpose", "dw_gathers",
                                               "dense_backup_rows"], bwd))}
        if not w.gated:
            # dead-unit record of this batch, and the targeted re-initialisation of the
            # pattern-deciding projection (on a copy): with this batch's dead units, and
            # with every unit dead (the bound: every weight read, blended, written)
            last = t.zeros((w.f,), dtype=t.int64, device="cuda")
            rec["track_active_units_ms"] = round(self.time(lambda: b.sfl_track_active_units(
                s["bufs"], w.T, w.f, "bf16", s["cfg"], 1, last, self.stream), steps=steps, warmup=1), 4)
            Wc = s["Wu"].clone()
            noise = t.randn((w.d, w.f), dtype=t.float32, device="cuda")
            rec["reinit_dead_units_ms"] = round(self.time(lambda: b.sfl_reinit_dead_units(
                Wc, last, 1, 0.1, 0.02, noise, stream=self.stream), steps=steps, warmup=1), 4)
            t.cuda.synchronize()
            rec["dead_units_in_batch"] = int((last < 1).sum().item())
            rec["reinit_all_dead_ms"] = round(self.time(lambda: b.sfl_reinit_dead_units(
                Wc, last, 2, 0.1, 0.02, noise, stream=self.stream), steps=steps, warmup=1), 4)
            del Wc, noise
        # dense reference (torch / hipBLASLt)
        X, Wu, Wd = s["X"], s["Wu"], s["Wd"]
        WuT, WdT, XT = Wu.t().contiguous(), Wd.t().contiguous(), X.t().contiguous()
        if w.gated:
            Wg = s["kw"]["W_gate"]
            WgTc = Wg.t().contiguous()

            def dense_step():
                G = X @ Wg
                U = X @ Wu
                H = t.relu(G) * U
                _ = H @ Wd
                dH = dY @ WdT
                dU = dH * t.relu(G)
                dG = dH * U * (G > 0)
                _ = dU @ WuT + dG @ WgTc
                _ = XT @ dU
                _ = XT @ dG
                _ = H.t().contiguous() @ dY
        else:
            def dense_step():
                H = t.relu(X @ Wu)
                _ = H @ Wd
                dZ = (dY @ WdT) * (H > 0)
                _ = dZ @ WuT
                _ = XT @ dZ
                _ = H.t().contiguous() @ dY

        dms = self.time(dense_step, steps=steps, warmup=2)
        rec["dense_torch_ms_fwd_bwd"] = round(dms, 4)
        rec["speedup_vs_dense_torch"] = round(dms / ms, 4)
        del bws
        return rec


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU; --gpus must be 1"}))
        sys.exit(2)
    import torch

    import workloads as wl
    from paper_2603_23198_amd import binding as b

    torch.cuda.set_device(0)
    if a.calibrate_copy:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    B = Bench(b, torch, a.steps, a.warmup)
    if a.only:
        if a.only == "splitd":
            recs = [B.splitd_record(wl.c4_sweep(sp, ell_width=k)) for sp, k in
                    ((0.99, 256), (0.995, 192), (0.998, 128), (0.999, 64))]
            print(json.dumps({"only": a.only, "records": recs}), flush=True)
            return
        if a.only in ("train", "gated_train"):
            wt = wl.c5_training() if a.only == "train" else wl.gated_training()
            rec = B.training_record(wt, 2e-5)
        else:
            wo = {"lognormal": wl.c2_lognormal, "gated": lambda: wl.c3_gated(T=8192),
                  "decode": lambda: wl.c3_gated(T=32), "tp8": lambda: wl.c4_shard("tp8"),
                  "dp8": lambda: wl.c4_shard("dp8"), "fp32": wl.c1_small_fp32}[a.only]()
            rec = B.forward_record(wo)[0]
        print(json.dumps({"only": a.only, "record": rec}), flush=True)
        return
    w = wl.c4_sweep(a.sparsity, T=a.tokens)
    T, d, f = w.T, w.d, w.f
    head, s, st = B.forward_record(w, order_ab=True)
    ms = head["ms"]
    stages = head["stages_ms"]

    # the persistent GEMMs' tile order: a Hilbert curve over 32 x 32 blocks of tiles (default)
    # against the XCD-grouped order, for the up projection of the sparse forward and for the
    # dense FFN's two GEMMs (interleaved runs)
    order_ab = {}
    dmk = lambda ev: b.ffn_args(s["X"], s["Wu"], s["Wd"], s["cfg"], **s["dkw"], workspace=s["dws"], events=ev)
    for order in ("grouped", "hilbert", "grouped", "hilbert", "grouped", "hilbert"):
        os.environ["SFL_GEMM_TILE_ORDER"] = order
        order_ab.setdefault(order + "_ms", []).append(
            B.stage_times(s["mk"], b.sfl_ffn_forward, 5)[0])
        order_ab.setdefault("dense_" + order + "_ms", []).append(
            float(sum(B.stage_times(dmk, b.sfl_dense_ffn_baseline, 3))))
    os.environ.pop("SFL_GEMM_TILE_ORDER", None)
    order_ab = {k: round(float(np.mean(v)), 4) for k, v in order_ab.items()}

    # the same step when W_down is re-laid out inside every call (no pre-packed copy)
    kw = dict(s["kw"])
    kw["W_down_packed"] = None
    ua = b.ffn_args(s["X"], s["Wu"], s["Wd"], s["cfg"], **kw)
    uws = torch.empty(max(1, b.sfl_workspace_size(ua)), dtype=torch.uint8, device="cuda")
    ua = b.ffn_args(s["X"], s["Wu"], s["Wd"], s["cfg"], **kw, workspace=uws)
    ms_unpacked = B.time(lambda: b.sfl_ffn_forward(ua, B.stream))
    del uws

    # roofline of the dominant kernel (the up-projection GEMM with the TwELL epilogue).
    # `achieved` divides the algorithmic flops by this run's HIP-event time of the up
    # projection stage (one kernel launch on the library's stream); the committed rocprofv3
    # kernel-trace average of the same kernel, and the MFMA busy share read from its counters,
    # are reported beside it (when they were taken on the current kernel source).
    up_flops = 2.0 * T * d * f
    achieved = up_flops / (stages["up_gemm_twell"] * 1e-3) / 1e12
    csrc = os.path.join(ROOT, "paper_2603_23198_amd", "csrc")
    gemm_hash = file_hash(os.path.join(csrc, "gemm.hip"), os.path.join(csrc, "common.h"))
    gather_hash = file_hash(os.path.join(csrc, "gather.hip"), os.path.join(csrc, "common.h"))
    gprof = profile_record("up_gemm_twell", gemm_hash) or {}
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_MFMA_PEAK_TFLOPS, 4),
                "traffic": gprof.get("hbm_bytes_per_launch"),
                "kernel": "k_gemm_kc<EPI_TWELL, 256, LAY_KC>", "work": "2*T*d*f flops per launch",
                "timing": "HIP events around the up-projection stage, this run"}
    if gprof.get("avg_duration_us"):
        pa = up_flops / (gprof["avg_duration_us"] * 1e-6) / 1e12
        roofline["profile"] = {"avg_us": gprof["avg_duration_us"], "achieved": round(pa, 2),
                               "frac": round(pa / BF16_MFMA_PEAK_TFLOPS, 4),
                               "mfma_busy_frac": gprof.get("mfma_busy_frac"),
                               "source": "profiles/traffic.json (rocprofv3 kernel trace and counters)"}
    # the sparse down projection: algorithmic bytes = sum_t nnz_t*(2d + 4) + (2d + 5) per sparse
    # row. Each token re-reads its W_down rows, which the XCDs' L2 caches serve (W_down is read
    # slice by slice), so the effective rate is compared with the measured L2 read ceiling;
    # the DRAM side is the counter bytes that came from beyond L2 over the kernel's duration.
    nnz = int(st["total_nnz"])
    n_sparse = T - int(st["n_ovf_rows"])
    gbytes = nnz * (2 * d + 4) + n_sparse * (2 * d + 5)
    g_rate = gbytes / (stages["sparse_down"] * 1e-3) / 1e9
    ceil = B.ceilings()
    dprof = profile_record("gather_down", gather_hash) or {}
    gather = {"bound": "l2", "achieved": round(g_rate, 1), "peak": ceil["l2_read_GBs"], "unit": "GB/s",
              "frac": round(g_rate / ceil["l2_read_GBs"], 4), "algorithmic_bytes": gbytes,
              "effective_frac_of_hbm_spec": round(g_rate / HBM_PEAK_GBS, 4),
              "traffic": dprof.get("hbm_bytes_per_launch"),
              "kernel": "k_gather_down_b16",
              "timing": "HIP events around the sparse down projection stage, this run",
              "peak_source": "measured L2 read ceiling (ceilings.l2_read_GBs)"}
    if dprof.get("hbm_bytes_per_launch") and dprof.get("avg_duration_us"):
        dram = dprof["hbm_bytes_per_launch"] / (dprof["avg_duration_us"] * 1e-6) / 1e9
        gather["dram_side"] = {"GBs": round(dram, 1), "frac_of_hbm_spec": round(dram / HBM_PEAK_GBS, 4),
                               "frac_of_measured_hbm_read": round(dram / ceil["hbm_read_GBs"], 4),
                               "avg_us": dprof["avg_duration_us"],
                               "source": "profiles/traffic.json (FETCH_SIZE + WRITE_SIZE, kernel trace)"}

    # distribution of single calls, warm and cold: before each cold call a 1 GiB buffer is
    # written, which evicts W_up, W_down and X from L2 and the 256 MiB infinity cache
    scratch = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    flush = lambda: scratch.fill_(1)
    warm = B.per_call(lambda: b.sfl_ffn_forward(s["args"], B.stream))
    cold = B.per_call(lambda: b.sfl_ffn_forward(s["args"], B.stream), flush=flush)
    cold_dense = B.per_call(lambda: b.sfl_dense_ffn_baseline(s["dargs"], B.stream), flush=flush)
    del scratch
    pct = lambda v: {"median": round(float(np.median(v)), 4), "p10": round(float(np.percentile(v, 10)), 4),
                     "p90": round(float(np.percentile(v, 90)), 4)}
    timing = {"calls": len(warm), "warm_ms": pct(warm), "cold_ms": pct(cold), "cold_dense_ms": pct(cold_dense),
              "cold_tokens_per_s": round(T / float(np.median(cold)) * 1e3, 1),
              "cold_speedup_vs_dense": round(float(np.median(cold_dense)) / float(np.median(cold)), 4)}

    out = {
        "metric": "sparse FFN tokens/sec at 99% sparsity; HBM GB/s % peak; speedup vs dense FFN",
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian X and weights; per-row shift gives uniformly random active units)",
        "config": {"workload": f"non-gated ReLU FFN forward, bf16, T={T}, d={d}, f={f}, sparsity={a.sparsity}",
                   "tokens": T, "d": d, "f": f, "sparsity_target": a.sparsity,
                   "realised_sparsity": head["realised_sparsity"], "ell_width": s["cfg"].ell_width,
                   "tile_cols": s["cfg"].tile_cols, "tile_slots": s["cfg"].tile_slots,
                   "parallelism": "single GPU"},
        "dense_ms_per_step": head["dense_ms"],
        "speedup_vs_dense": head["speedup_vs_dense"],
        "dense_stages_ms": head["dense_stages_ms"],
        "dense_torch_ms_per_step": head.get("dense_torch_ms"),
        "speedup_vs_dense_torch": head.get("speedup_vs_dense_torch"),
        "stages_ms": stages,
        "token_order_ab": head.get("token_order_ab"),
        "single_call_timing": timing,
        "ms_per_step_w_down_packed_per_call": round(ms_unpacked, 4),
        "up_gemm_tile_order_ab": order_ab,
        "n_ovf_rows": head["n_ovf_rows"],
        "roofline": roofline,
        "gather_roofline": gather,
        "ceilings": ceil,
        # the fused ReLU -> TwELL epilogue measured as the difference to the same GEMM with a
        # plain ReLU + bf16 store epilogue (the dense FFN's first GEMM)
        "twell_epilogue_delta_ms": round(stages["up_gemm_twell"] - head["dense_stages_ms"]["up_gemm_relu"], 4),
        # dense-equivalent work per second: the dense FFN's 4 T d f flops over the sparse time
        "tflops_equivalent": round(4.0 * T * d * f / (ms * 1e-3) / 1e12, 1),
    }
    del s
    if not a.quick:
        others = []
        for sp_ in (0.9, 0.95, 0.999):
            r, s2, _ = B.forward_record(wl.c4_sweep(sp_, T=a.tokens), stages=True, fallback_ab=sp_ < 0.99)
            others.append(r)
            del s2
        r, s2, _ = B.forward_record(wl.c2_lognormal(), order_ab=True)
        others.append(r)
        del s2
        r, s2, _ = B.forward_record(wl.c1_small_fp32())
        others.append(r)
        del s2
        for tt in (8192, 32):
            r, s2, _ = B.forward_record(wl.c3_gated(T=tt), order_ab=True)
            others.append(r)
            del s2
        out["other_workloads"] = others
        # TwELL storage: the packed 32-bit words (Appendix A's inference format) against the
        # planes with the same 31 slots, at the headline workload
        lay = {}
        for name, layout in (("planes_s31", 0), ("packed32", 1)):
            wp = wl.c4_sweep(0.99, T=a.tokens, tile_slots=31)
            wp.cfg["layout"] = layout
            r, s2, _ = B.forward_record(wp, dense=False)
            lay[name] = {"ms": r["ms"], "stages_ms": r["stages_ms"]}
            del s2
        out["twell_layout_ab"] = lay
        # the paper's row-wise down kernel against the slice walk at the headline workload
        out["down_projection_ab"] = B.splitd_record(wl.c4_sweep(0.99, T=a.tokens))
        # one GPU's share of the headline layer run on eight GPUs: hidden units split eight
        # ways (tensor parallel, f = 2048) or tokens split eight ways (data parallel, T = 1024);
        # the collectives around them are not part of this record
        shards = []
        for kind in ("tp8", "dp8"):
            r, s2, _ = B.forward_record(wl.c4_shard(kind, T=a.tokens))
            r["shard"] = kind
            shards.append(r)
            del s2
        out["shard_shapes"] = shards
        torch.cuda.empty_cache()
        w5 = wl.c5_training()
        out["training_step"] = B.training_record(w5, 2e-5)
        del w5
        torch.cuda.empty_cache()
        out["gated_training_step"] = B.training_record(wl.gated_training(), 2e-5)
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, a.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
