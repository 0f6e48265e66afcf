#!/usr/bin/env python3
"""Throughput of the l1-phase CSR training step on one MI355X.

A step is one pass of the hot path over one batch of the large fully
connected layer 9216 -> 4096 (W: 4096 x 9216 CSR, 9% density with Zipf(1.1)
row lengths, batch 1024, fp32):

    Y  = W.X                          csr_spmm_fwd
    bitmap index of W, CSC(W)         csr_bitmap_build, csc_build
    dX = W^T.dY                       csr_spmm_bwd_t
    Z  = S_t(W - eta*dY.X^T)          dense_wgrad_prox (fp32 matrix cores, prox in the epilogue)
    W' = CSR(Z)                       csr_recompress_counted

The timed step is L1.l1_step: these calls with the dependencies of a
training loop on two streams (bitmap index and CSC beside the forward
product, the backward product beside the weight update).  The serial
schedule is timed beside it and gives the per-call split; each call is also
timed cold (a 1 GiB write between repetitions evicts L2 and the MALL).  Every
step reads the same resident inputs and writes W' to its own buffers, so all
timed steps do identical work.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--no-cpu-baseline]
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

METRIC = "sparse train-step GFLOP/s (nnz-effective) and achieved HBM GB/s vs peak"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_MFMA_F32_TFLOPS = 157.3   # MI355X dense fp32 matrix
PEAK_MFMA_BF16_TFLOPS = 2500.0  # MI355X dense bf16 matrix
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum host time spent timing the oracle")
    ap.add_argument("--workload", default="fc9216x4096",
                    choices=["fc9216x4096", "fc784x300", "mlp784", "conv2", "fc4096_sweep",
                             "fc9216x4096_adaptive", "lenet5_inference", "conv2_direct", "hbm_kernels", "all"],
                    help="fc9216x4096 (default): the metric's workload, one JSON line; the others "
                         "print one informational JSON line each (no CPU baseline)")
    return ap.parse_args()


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_1905_07931_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_traffic(kernel_file, src_hash):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it
    was taken on the current kernel source (else None)."""
    path = os.path.join(PROFILES, kernel_file)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic_json:"):
                d = json.loads(line.split(":", 1)[1])
                if d.get("source_hash") == src_hash:
                    return d.get("bytes_per_launch")
    return None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the hot path is "
              "built and measured on a single MI355X, multi-GPU sharding is not part of it.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L1.lib()  # fail loudly if the HIP library is missing

    if args.workload != "fc9216x4096":
        import bench_workloads
        names = (["fc784x300", "mlp784", "conv2", "conv2_direct", "fc4096_sweep", "fc9216x4096_adaptive",
                  "lenet5_inference", "hbm_kernels"]
                 if args.workload == "all"
                 else [args.workload])
        for n in names:
            for line in bench_workloads.run(n, args, dev):
                print(json.dumps(line), flush=True)
        return

    t0 = time.time()
    Lr = synth.fc9216_4096(seed=0)
    gen_s = time.time() - t0
    N, K, B, nnz = Lr.N, Lr.K, Lr.B, Lr.nnz
    eta, lam = Lr.eta, Lr.lam

    W = L1.CSR.from_host(Lr.row_ptr, Lr.col_idx, Lr.vals, K, device=dev)
    X = torch.from_numpy(Lr.X).to(dev)
    dY = torch.from_numpy(Lr.dY).to(dev)
    Y = torch.empty((N, B), dtype=torch.float32, device=dev)
    dX = torch.empty((K, B), dtype=torch.float32, device=dev)
    dW = torch.empty((N, K), dtype=torch.float32, device=dev)
    csc = L1.CSC.empty(K, nnz, dev)
    Wout = L1.CSR(N, K, torch.empty(N + 1, dtype=torch.int32, device=dev),
                  torch.empty(N * K, dtype=torch.int32, device=dev),
                  torch.empty(N * K, dtype=torch.float32, device=dev), None)

    bm = L1.Bitmap.empty(N, K, dev)
    names = ["csr_spmm_fwd", "csr_bitmap_build", "csc_build", "csr_spmm_bwd_t", "dense_wgrad_prox",
             "csr_recompress_counted"]

    def step(ev=None, prec=L1.F32):
        """The step as a training loop runs it (L1.l1_step, two streams), all
        outputs ready on the current stream at the end; ev: {call: (start,
        end)} events recorded around calls on the stream they run on."""
        L1.l1_step(W, X, dY, eta, lam, Y=Y, dX=dX, dW=dW, csc=csc, out=Wout, precision=prec, bitmap=bm,
                   events=ev, schedule="two_stream")

    def update(prec=L1.F32):
        Z, wc = L1.dense_wgrad_prox(W, dY, X, eta, lam, bm, Z=dW, precision=prec)
        L1.csr_recompress_counted(Z, wc, out=Wout)

    calls = {
        "csr_spmm_fwd": lambda: L1.csr_spmm_fwd(W, X, Y),
        "csc_build": lambda: L1.csc_build(W, csc, bitmap=bm),
        "csr_bitmap_build": lambda: L1.csr_bitmap_build(W, bm),
        "csr_spmm_bwd_t": lambda: L1.csr_spmm_bwd_t(W, dY, csc, dX),
    }
    wc_buf = {}
    calls["dense_wgrad_prox"] = lambda: wc_buf.__setitem__(
        "wc", L1.dense_wgrad_prox(W, dY, X, eta, lam, bm, Z=dW)[1])
    calls["csr_recompress_counted"] = lambda: L1.csr_recompress_counted(dW, wc_buf["wc"], out=Wout)

    def serial_step(ev=None):
        """The same calls one after another on one stream (events between them
        give the per-call split)."""
        for i, n in enumerate(names):
            if ev is not None:
                ev[i].record()
            calls[n]()
        if ev is not None:
            ev[len(names)].record()

    def ev_pair():
        return (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

    def timed_steps(fn, watch=("dense_wgrad_prox", "csr_recompress_counted")):
        """K back-to-back steps; an event on the current stream between steps
        gives each step's time, events around the watched calls (on their own
        stream) their live durations."""
        bound = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        evs = [{w: ev_pair() for w in watch} for _ in range(args.steps)]
        torch.cuda.synchronize()
        bound[0].record()
        for s_ in range(args.steps):
            fn(evs[s_])
            bound[s_ + 1].record()
        torch.cuda.synchronize()
        each = [bound[i].elapsed_time(bound[i + 1]) for i in range(args.steps)]
        live = {w: float(np.mean([e[w][0].elapsed_time(e[w][1]) for e in evs])) for w in watch}
        return bound[0].elapsed_time(bound[-1]) / args.steps, each, live

    for _ in range(args.warmup):
        step()
        serial_step()
    torch.cuda.synchronize()

    # whole-step timing of the two-stream step; the dominant launch (the
    # weight-gradient GEMM with the prox epilogue, alone on the main stream)
    # and the recompression timed live inside it
    ms_per_step, step_each, live = timed_steps(lambda ev: step(ev))
    step_pct = [round(float(np.percentile(step_each, q)), 4) for q in (10, 50, 90)]
    wg_live_ms, rc_live_ms = live["dense_wgrad_prox"], live["csr_recompress_counted"]

    # the serial schedule, and per-call durations from events between its calls
    ms_serial, _, _ = timed_steps(lambda ev: serial_step(), watch=())
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s_ in range(args.steps):
        serial_step(evs[s_])
    torch.cuda.synchronize()
    per = {n: float(np.mean([evs[s_][i].elapsed_time(evs[s_][i + 1]) for s_ in range(args.steps)]))
           for i, n in enumerate(names)}
    nnz_out = int(Wout.row_ptr[-1].item())

    # each call cold: a 1 GiB write evicts L2 and the 256 MB MALL before it
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    cold = {}
    for n in names:
        ts = []
        for _ in range(max(3, min(args.steps, 10))):
            flush.fill_(1.0)
            a_, b_ = ev_pair()
            a_.record()
            calls[n]()
            b_.record()
            torch.cuda.synchronize()
            ts.append(a_.elapsed_time(b_))
        cold[n] = float(np.median(ts))
    del flush

    # the unfused weight update (dense_wgrad, then prox_l1_recompress reading
    # dW twice) on the same inputs, for comparison
    for _ in range(2):
        L1.dense_wgrad(dY, X, dW)
        L1.prox_l1_recompress(W, dW, eta, lam, out=Wout)
    ue = [ev_pair() for _ in range(args.steps)]
    pe = [ev_pair() for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s_ in range(args.steps):
        ue[s_][0].record()
        L1.dense_wgrad(dY, X, dW)
        pe[s_][0].record()
        L1.prox_l1_recompress(W, dW, eta, lam, out=Wout)
        pe[s_][1].record()
        ue[s_][1].record()
    torch.cuda.synchronize()
    unfused_ms = float(np.mean([a_.elapsed_time(b_) for a_, b_ in ue]))
    unfused_prox_ms = float(np.mean([a_.elapsed_time(b_) for a_, b_ in pe]))

    # dense dW with bf16 operands: reported beside the step, not part of it
    dWb = torch.empty_like(dW)
    L1.dense_wgrad(dY, X, dWb, precision=L1.BF16)
    evb = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evb[0].record()
    for s_ in range(args.steps):
        L1.dense_wgrad(dY, X, dWb, precision=L1.BF16)
        evb[s_ + 1].record()
    torch.cuda.synchronize()
    bf16_ms = float(np.mean([evb[i].elapsed_time(evb[i + 1]) for i in range(args.steps)]))
    del dWb

    # the same step with the weight gradient split into bf16 hi + lo on the
    # bf16 matrix cores (BF16X3: inside the 1e-4 contract)
    for _ in range(2):
        step(prec=L1.BF16X3)
    ms_x3, _, live_x3 = timed_steps(lambda ev: step(ev, prec=L1.BF16X3))
    wg_x3_ms = live_x3["dense_wgrad_prox"]

    # both steps captured once into a HIP graph and replayed: the same kernels
    # without the host's per-launch cost (every call is capture-safe here)
    import bench_workloads
    Wout.nnz = nnz_out  # the host count, as under capture
    ms_graph = bench_workloads._graph_timed(torch, step, args.steps)
    ms_graph_x3 = bench_workloads._graph_timed(torch, lambda: step(prec=L1.BF16X3), args.steps)

    flops_step = 2.0 * nnz * B * 2 + 2.0 * N * K * B          # fwd + bwd + dense dW
    flops_nnz_only = 6.0 * nnz * B
    gflops = flops_step / (ms_per_step * 1e-3) / 1e9

    # algorithmic bytes of the recompression (each operand once): Z and its
    # word counts in, W' out; and of the unfused prox + recompression: dW in,
    # W in (CSR), W' out
    kw = (K + 31) // 32
    csr_in = 8.0 * nnz + 4.0 * (N + 1)
    csr_out = 8.0 * nnz_out + 4.0 * (N + 1)
    bytes_recompress = 4.0 * N * K + 4.0 * N * kw + csr_out
    bytes_prox = 4.0 * N * K + csr_in + csr_out
    rc_ms = per["csr_recompress_counted"]  # the call alone (serial schedule)
    rc_gbs = bytes_recompress / (rc_ms * 1e-3) / 1e9

    wg_flops = 2.0 * N * K * B
    wg_tflops = wg_flops / (wg_live_ms * 1e-3) / 1e12  # live, inside the timed steps
    traffic = counter_traffic("dense_wgrad_prox_fc9216x4096_pmc.txt",
                              source_hash("gemm.hip", "prox_epilogue.hpp"))
    roof = {"kernel": "dense_wgrad_prox (wgrad_f32_dma_kernel<true>: direct global->LDS tiles, prox epilogue)", "bound": "mfma",
            "achieved": round(wg_tflops, 2), "peak": PEAK_MFMA_F32_TFLOPS, "unit": "TFLOP/s",
            "frac": round(wg_tflops / PEAK_MFMA_F32_TFLOPS, 4), "traffic": traffic,
            "algorithmic_flops": wg_flops, "launch_ms": round(wg_live_ms, 4)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(Lr, args.cpu_seconds)

    out = {
        "metric": METRIC, "value": round(gflops, 1), "unit": "GFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "fc9216x4096_b1024_d9_zipf_l1_step", "N": N, "K": K, "B": B,
                   "nnz": nnz, "density": 0.09, "row_lengths": "zipf s=1.1", "eta": eta,
                   "lambda": lam, "phase": "l1 (fwd, csc, bwd, dense dW + prox, recompress)"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernels_ms": {k: round(v, 4) for k, v in per.items()},
        "kernels_ms_cold": {k: round(v, 4) for k, v in cold.items()},
        "ms_per_step_p10_p50_p90": step_pct,
        "schedule": "two streams (bitmap index and CSC build beside the forward SpMM; backward SpMM beside "
                    "the weight update); kernels_ms from the serial schedule, kernels_ms_cold with a 1 GiB "
                    "write before each call",
        "ms_per_step_serial": round(ms_serial, 4),
        "ms_per_step_graph": round(ms_graph, 4),
        "value_graph": round(flops_step / (ms_graph * 1e-3) / 1e9, 1),
        "gflops_nnz_only": round(flops_nnz_only / (ms_per_step * 1e-3) / 1e9, 1),
        "recompress": {"ms": round(rc_ms, 4), "ms_cold": round(cold["csr_recompress_counted"], 4),
                       "ms_live_in_step": round(rc_live_ms, 4), "algorithmic_bytes": bytes_recompress,
                       "hbm_gbs": round(rc_gbs, 1), "hbm_frac": round(rc_gbs / PEAK_HBM_GBS, 4),
                       "hbm_frac_cold": round(bytes_recompress / (cold["csr_recompress_counted"] * 1e-3) / 1e9
                                              / PEAK_HBM_GBS, 4),
                       "note": "csr_recompress_counted (row and row-block totals of the word counts, then the compaction of Z, which adds up its row starts): Z and its word counts "
                               "read once, W' written; ms is the call alone, ms_live_in_step shares the GPU with "
                               "the backward SpMM on the other stream"},
        "weight_update_ms": round(per["dense_wgrad_prox"] + rc_ms, 4),
        "weight_update_unfused": {"ms": round(unfused_ms, 4), "prox_l1_recompress_ms": round(unfused_prox_ms, 4),
                                  "prox_recompress_hbm_frac": round(bytes_prox / (unfused_prox_ms * 1e-3) / 1e9
                                                                    / PEAK_HBM_GBS, 4),
                                  "note": "dense_wgrad then prox_l1_recompress (two passes over dW and W), "
                                          "the same result bit for bit"},
        "nnz_out": nnz_out,
        "dense_wgrad_bf16": {"ms": round(bf16_ms, 4),
                             "tflops": round(wg_flops / (bf16_ms * 1e-3) / 1e12, 1),
                             "peak": PEAK_MFMA_BF16_TFLOPS,
                             "frac": round(wg_flops / (bf16_ms * 1e-3) / 1e12 / PEAK_MFMA_BF16_TFLOPS, 4),
                             "note": "operands rounded to bf16, exact products, fp32 sums; outside the "
                                     "1e-4 fp32 contract and not part of the step"},
        "step_bf16x3": {"ms_per_step": round(ms_x3, 4),
                        "value": round(flops_step / (ms_x3 * 1e-3) / 1e9, 1),
                        "ms_per_step_graph": round(ms_graph_x3, 4),
                        "value_graph": round(flops_step / (ms_graph_x3 * 1e-3) / 1e9, 1),
                        "dense_wgrad_prox_ms": round(wg_x3_ms, 4),
                        "dense_wgrad_tflops": round(wg_flops / (wg_x3_ms * 1e-3) / 1e12, 1),
                        "bf16_mfma_frac": round(3 * wg_flops / (wg_x3_ms * 1e-3) / 1e12 / PEAK_MFMA_BF16_TFLOPS, 4),
                        "note": "the same step with dense_wgrad precision BF16X3: operands split into bf16 "
                                "hi + lo, hi.hi + hi.lo + lo.hi exact on the bf16 matrix cores, fp32 sums; "
                                "within the 1e-4 contract (per-product error < 4.7e-5); tflops counts the "
                                "2NKB fp32-equivalent flops, bf16_mfma_frac the 3x executed ones"},
        "input_gen_s": round(gen_s, 2),
    }
    print(json.dumps(out), flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def oracle_step(oracle, rp, ci, v, X, dY, K, eta, lam):
    oracle.spmm_fwd(rp, ci, v, X)
    oracle.spmm_bwd_t(rp, ci, v, dY, K)
    dW = oracle.dense_wgrad(dY, X)
    Z, _ = oracle.prox_dense(rp, ci, v, dW, eta, lam, K)
    oracle.recompress(Z)


def cpu_baseline(Lr, min_seconds):
    """The oracle timed on the host cores on the same step: the whole layer
    (fwd, bwd, dense dW, prox, recompression) with the OpenMP threads the
    oracle uses, repeated until at least `min_seconds` have elapsed (at most
    12 runs), the median run reported; and once with one thread on a bounded
    sample (the first 256 rows with their columns, the same batch)."""
    import oracle

    N, K, B = Lr.N, Lr.K, Lr.B
    times = []
    while len(times) < 12 and (sum(times) < min_seconds or len(times) < 1):
        t0 = time.perf_counter()
        oracle_step(oracle, Lr.row_ptr, Lr.col_idx, Lr.vals, Lr.X, Lr.dY, K, Lr.eta, Lr.lam)
        times.append(time.perf_counter() - t0)
    sec = float(np.median(times))
    flops = 2.0 * Lr.nnz * B * 2 + 2.0 * N * K * B
    threads = oracle.num_threads()
    # one thread, rows 0..255 (every call scales with the rows)
    R = 256
    rp = np.ascontiguousarray(Lr.row_ptr[:R + 1])
    n_s = int(rp[-1])
    ci, v, dYs = Lr.col_idx[:n_s], Lr.vals[:n_s], np.ascontiguousarray(Lr.dY[:R])
    oracle.set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oracle_step(oracle, rp, ci, v, Lr.X, dYs, K, Lr.eta, Lr.lam)
        sec1 = time.perf_counter() - t0
    finally:
        oracle.set_num_threads(threads)
    flops1 = 2.0 * n_s * B * 2 + 2.0 * R * K * B
    return {"value": round(flops / sec / 1e9, 3), "unit": "GFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"the full step ({N}x{K} CSR, {Lr.nnz} nnz, B={B}): fwd, bwd, dense dW, prox, "
                      f"recompress; median of {len(times)} runs, {sec:.2f} s each",
            "value_1thread": round(flops1 / sec1 / 1e9, 3),
            "sample_1thread": f"rows 0-{R - 1} ({n_s} nnz, B={B}), the same five calls on one thread, "
                              f"{sec1:.2f} s",
            "host_cpu": cpu_model(), "host_logical_cpus": os.cpu_count()}


if __name__ == "__main__":
    main()
