"""The other layer shapes of the method, timed the way bench.py times the
9216 -> 4096 step (inputs resident in HBM, warm-up, back-to-back steps between
two events, per-call events in a second pass).  Each workload yields one
informational JSON line; bench.py's default line is the metric.

    fc784x300     l1 step of the 784 -> 300 layer, batch 64, 10% density
    mlp784        MLP 784-300-100-10, batch 256: l1 step then a debiasing step
    conv2         LeNet-5 conv2 as im2col, 50 x 500 CSR, batch 16384:
                  fwd, CSC, bwd, masked dW (SDDMM), support-restricted prox, compaction
    fc4096_sweep  4096 x 4096, batch 512, densities 1/5/20/50%: 20 alternating
                  l1 / debiasing iterations with the CSR rebuilt after every l1 step
                  (the l1 update fused: dense_wgrad_prox + csr_recompress_counted)
    fc9216x4096_adaptive
                  the 9216 -> 4096 l1 step with Prox-ADAM (Algorithm 2) and with
                  Prox-RMSProp (Algorithm 1) in place of the plain proximal step
    lenet5_inference
                  forward-only compressed LeNet-5 (Table A1 nonzero counts),
                  batch sweep, beside the same network with every weight stored
    conv2_direct  LeNet-5 conv2 from real 20 x 12 x 12 maps, batch 256: direct
                  sparse conv forward and input gradient, im2col + filter
                  gradient (dense and pattern-sampled), prox + recompression
    hbm_kernels   one line per call of the memory-bound shapes (conv2 as im2col,
                  4096 x 4096 at 1% density): warm and cold-cache (1 GiB
                  written before each call) time, algorithmic bytes, their
                  rate against 8 TB/s and against a measured device copy
"""
from __future__ import annotations

import json
import os

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "sparse train-step GFLOP/s (nnz-effective) and achieved HBM GB/s vs peak"


def _timed(torch, step, steps, warmup, names):
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    per = None
    if names:
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(steps)]
        for s in range(steps):
            step(evs[s])
        torch.cuda.synchronize()
        per = {n: round(float(np.mean([evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(steps)])), 4)
               for i, n in enumerate(names)}
    return ms, per


def _graph_timed(torch, step, steps):
    """The same step captured once into a HIP graph (torch.cuda.CUDAGraph) and
    replayed back to back: the GPU time without the host's per-launch cost."""
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # workspaces for the capture stream are allocated here
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def _line(workload, flops, ms, cfg, per=None, **extra):
    out = {"metric": METRIC, "value": round(flops / (ms * 1e-3) / 1e9, 1), "unit": "GFLOP/s",
           "n_gpus": 1, "ms_per_step": round(ms, 4), "higher_is_better": True, "dtype": "f32",
           "data": "synthetic", "config": dict(workload=workload, **cfg), "informational": True}
    if per:
        out["kernels_ms"] = per
    out.update(extra)
    return out


def _csr_out(L1, torch, N, K, dev):
    return L1.CSR(N, K, torch.empty(N + 1, dtype=torch.int32, device=dev),
                  torch.empty(N * K, dtype=torch.int32, device=dev),
                  torch.empty(N * K, dtype=torch.float32, device=dev), None)


def fc784x300(args, dev):
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    L = synth.fc784_300(seed=0)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    X, dY = torch.from_numpy(L.X).to(dev), torch.from_numpy(L.dY).to(dev)
    Y = torch.empty((L.N, L.B), dtype=torch.float32, device=dev)
    dX = torch.empty((L.K, L.B), dtype=torch.float32, device=dev)
    dW = torch.empty((L.N, L.K), dtype=torch.float32, device=dev)
    csc = L1.CSC.empty(L.K, L.nnz, dev)
    Wout = _csr_out(L1, torch, L.N, L.K, dev)
    names = ["csr_spmm_fwd", "csc_build", "csr_spmm_bwd_t", "dense_wgrad", "prox_l1_recompress"]

    def step(ev=None):
        mark = (lambda i: ev[i].record()) if ev else (lambda i: None)
        mark(0); L1.csr_spmm_fwd(W, X, Y)
        mark(1); L1.csc_build(W, csc)
        mark(2); L1.csr_spmm_bwd_t(W, dY, csc, dX)
        mark(3); L1.dense_wgrad(dY, X, dW)
        mark(4); L1.prox_l1_recompress(W, dW, L.eta, L.lam, out=Wout)
        mark(5)
    ms, per = _timed(torch, step, max(args.steps, 20), max(args.warmup, 5), names)
    nnz_out = int(Wout.row_ptr[-1].item())
    Wout.nnz = nnz_out
    ms_graph = _graph_timed(torch, step, max(args.steps, 20))

    def step2(ev=None):  # the two-stream schedule of L1.l1_step
        L1.l1_step(W, X, dY, L.eta, L.lam, Y=Y, dX=dX, dW=dW, csc=csc, out=Wout, schedule="two_stream")
    ms2, _ = _timed(torch, step2, max(args.steps, 20), max(args.warmup, 5), None)
    ms2_graph = _graph_timed(torch, step2, max(args.steps, 20))
    flops = 4.0 * L.nnz * L.B + 2.0 * L.N * L.K * L.B
    yield _line("fc784x300_b64_d10_l1_step", flops, ms,
                dict(N=L.N, K=L.K, B=L.B, nnz=L.nnz, density=0.10), per,
                nnz_out=nnz_out, ms_per_step_graph=round(ms_graph, 4),
                value_graph=round(flops / (ms_graph * 1e-3) / 1e9, 1),
                ms_per_step_two_stream=round(ms2, 4), ms_per_step_two_stream_graph=round(ms2_graph, 4),
                note="ms_per_step: the calls one after another on one stream (what L1.l1_step "
                     "picks for this layer); two_stream: L1.l1_step forced onto two streams")


def mlp784(args, dev):
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    layers, Xh, labels = synth.mlp_784_300_100_10(seed=0)
    B = Xh.shape[1]
    eta, lam = 0.01, 1e-4
    W0 = [L1.CSR.from_host(l.row_ptr, l.col_idx, l.vals, l.K, device=dev) for l in layers]
    W1 = [_csr_out(L1, torch, l.N, l.K, dev) for l in layers]
    X, lab = torch.from_numpy(Xh).to(dev), torch.from_numpy(labels).to(dev)
    shapes = [(l.N, l.K) for l in layers]
    A = [torch.empty((n, B), dtype=torch.float32, device=dev) for n, _ in shapes]
    H = [torch.empty((n, B), dtype=torch.float32, device=dev) for n, _ in shapes[:2]]
    D = [torch.empty((n, B), dtype=torch.float32, device=dev) for n, _ in shapes]
    dH = [torch.empty((k, B), dtype=torch.float32, device=dev) for _, k in shapes]
    dW = [torch.empty((n, k), dtype=torch.float32, device=dev) for n, k in shapes]
    cscs = [L1.CSC.empty(k, n * k, dev) for n, k in shapes]
    gvs = [torch.empty(n * k, dtype=torch.float32, device=dev) for n, k in shapes]

    def fwd_bwd(Ws):
        inp = [X, None, None]
        for j in range(3):
            L1.csr_spmm_fwd(Ws[j], inp[j], A[j])
            if j < 2:
                L1.relu_fwd(A[j], H[j])
                inp[j + 1] = H[j]
        L1.softmax_xent(A[2], lab, dlogits=D[2])
        for j in (2, 1):
            csc = L1.csc_build(Ws[j], cscs[j])
            L1.csr_spmm_bwd_t(Ws[j], D[j], csc, dH[j])
            L1.relu_bwd(A[j - 1], dH[j], D[j - 1])
        return inp

    known = [None, None, None]  # nnz of the l1 step's output, learned once

    def step(ev=None):
        mark = (lambda i: ev[i].record()) if ev else (lambda i: None)
        mark(0)
        inp = fwd_bwd(W0)
        for j in range(3):
            L1.dense_wgrad(D[j], inp[j], dW[j])
            L1.prox_l1_recompress(W0[j], dW[j], eta, lam, out=W1[j])
            W1[j].nnz = known[j]
        mark(1)
        inp = fwd_bwd(W1)
        for j in range(3):
            L1.sddmm_masked_wgrad(W1[j], D[j], inp[j], gvs[j])
            L1.prox_l1_step(L1.PROX_CSR, W1[j], gvs[j], eta, 0.0)
        mark(2)
    # the debiasing step runs on the l1 step's output structure: learn its size once
    step()
    torch.cuda.synchronize()
    for j, w in enumerate(W1):
        w.nnz = None
        known[j] = w.host_nnz()
    ms, per = _timed(torch, step, max(args.steps, 20), max(args.warmup, 5), ["l1_step", "debias_step"])
    ms_graph = _graph_timed(torch, step, max(args.steps, 20))
    nnz0 = [l.nnz for l in layers]
    nnz1 = [w.nnz for w in W1]
    flops = sum(4.0 * a * B + 2.0 * n * k * B for a, (n, k) in zip(nnz0, shapes)) + \
        sum(6.0 * a * B for a in nnz1)
    yield _line("mlp784_300_100_10_b256_l1_then_debias", flops, ms,
                dict(B=B, nnz=nnz0, nnz_after_l1=nnz1), per, ms_per_step_graph=round(ms_graph, 4),
                value_graph=round(flops / (ms_graph * 1e-3) / 1e9, 1))


def conv2(args, dev):
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    L = synth.conv2_im2col(seed=0)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    vals0 = W.vals.clone()
    X, dY = torch.from_numpy(L.X).to(dev), torch.from_numpy(L.dY).to(dev)
    Y = torch.empty((L.N, L.B), dtype=torch.float32, device=dev)
    dX = torch.empty((L.K, L.B), dtype=torch.float32, device=dev)
    gv = torch.empty(L.nnz, dtype=torch.float32, device=dev)
    csc = L1.CSC.empty(L.K, L.nnz, dev)
    Wc = L1.CSR(L.N, L.K, torch.empty(L.N + 1, dtype=torch.int32, device=dev),
                torch.empty(L.nnz, dtype=torch.int32, device=dev),
                torch.empty(L.nnz, dtype=torch.float32, device=dev), None)
    names = ["csr_spmm_fwd", "csc_build", "csr_spmm_bwd_t", "sddmm_masked_wgrad", "prox_l1_step_csr",
             "csr_compact"]

    def step(ev=None):
        mark = (lambda i: ev[i].record()) if ev else (lambda i: None)
        W.vals.copy_(vals0)  # every step starts from the same weights
        mark(0); L1.csr_spmm_fwd(W, X, Y)
        mark(1); L1.csc_build(W, csc)
        mark(2); L1.csr_spmm_bwd_t(W, dY, csc, dX)
        mark(3); L1.sddmm_masked_wgrad(W, dY, X, gv)
        mark(4); L1.prox_l1_step(L1.PROX_CSR, W, gv, L.eta, L.lam)
        mark(5); L1.csr_compact(W, Wc)
        mark(6)
    ms, per = _timed(torch, step, max(args.steps, 20), max(args.warmup, 5), names)
    ms_graph = _graph_timed(torch, step, max(args.steps, 20))
    flops = 6.0 * L.nnz * L.B
    # SDDMM reads X and dY once at least: the HBM roof of this shape
    sddmm_bytes = 4.0 * (L.K + L.N) * L.B + 12.0 * L.nnz
    yield _line("conv2_im2col_50x500_b16384_d10", flops, ms, dict(N=L.N, K=L.K, B=L.B, nnz=L.nnz), per,
                ms_per_step_graph=round(ms_graph, 4), value_graph=round(flops / (ms_graph * 1e-3) / 1e9, 1),
                sddmm_hbm_gbs=round(sddmm_bytes / (per["sddmm_masked_wgrad"] * 1e-3) / 1e9, 1),
                spmm_fwd_hbm_gbs=round((4.0 * (L.K + L.N) * L.B + 8.0 * L.nnz) /
                                       (per["csr_spmm_fwd"] * 1e-3) / 1e9, 1))


def fc4096_sweep(args, dev):
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    cal = json.load(open(os.path.join(ROOT, "tests", "golden", "fc4096_lambda.json")))
    iters = 20
    batches = [synth.fc4096_batch(t) for t in range(iters)]
    Xs = [torch.from_numpy(x).to(dev) for x, _ in batches]
    dYs = [torch.from_numpy(d).to(dev) for _, d in batches]
    del batches
    for pct in (1, 5, 20, 50):
        L = synth.fc4096_sweep(pct / 100)
        lam = cal["lambda"][str(pct)]
        N, K, B = L.N, L.K, L.B
        W0 = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, K, device=dev)
        bufs = [_csr_out(L1, torch, N, K, dev) for _ in range(2)]
        Y = torch.empty((N, B), dtype=torch.float32, device=dev)
        dX = torch.empty((K, B), dtype=torch.float32, device=dev)
        dW = torch.empty((N, K), dtype=torch.float32, device=dev)
        gv = torch.empty(N * K, dtype=torch.float32, device=dev)
        csc = L1.CSC.empty(K, N * K, dev)
        bm = L1.Bitmap.empty(N, K, dev)
        wcs = torch.empty((N, (K + 31) // 32), dtype=torch.int32, device=dev)
        # one untimed pass learns the nnz of every iteration (the host passes it
        # to the calls, as a training loop that sizes its buffers would)
        nnz_seq = []

        def run(timed_nnz=None):
            W = W0
            k = 0
            for t in range(iters):
                if t % 2 == 0:
                    if W is not W0:
                        L1.csc_update_vals(W, csc)
                    else:
                        L1.csc_build(W, csc)
                    L1.csr_spmm_fwd(W, Xs[t], Y)
                    L1.csr_spmm_bwd_t(W, dYs[t], csc, dX)
                    out = bufs[k % 2]
                    k += 1
                    # the l1 update as the step makes it: Z = prox(W - eta dY X^T) from
                    # the GEMM's epilogue, then Z -> CSR (the bits of dense_wgrad +
                    # prox_l1_recompress)
                    L1.csr_bitmap_build(W, bm)
                    _, wc = L1.dense_wgrad_prox(W, dYs[t], Xs[t], L.eta, lam, bm, Z=dW, word_counts=wcs)
                    L1.csr_recompress_counted(dW, wc, out=out, capacity=N * K)
                    W = out
                    if timed_nnz is None:
                        nnz_seq.append(W.host_nnz())
                    else:
                        W.nnz = timed_nnz[t // 2]
                else:
                    L1.csc_build(W, csc)
                    L1.csr_spmm_fwd(W, Xs[t], Y)
                    L1.csr_spmm_bwd_t(W, dYs[t], csc, dX)
                    L1.sddmm_masked_wgrad(W, dYs[t], Xs[t], gv)
                    L1.prox_l1_step(L1.PROX_CSR, W, gv, L.eta, 0.0)
        run()
        torch.cuda.synchronize()
        reps = 3
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            run(nnz_seq)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / (reps * iters)
        flops = 0.0
        prev = L.nnz
        for t in range(iters):
            if t % 2 == 0:
                flops += 4.0 * prev * B + 2.0 * N * K * B
                prev = nnz_seq[t // 2]
            else:
                flops += 6.0 * prev * B
        flops /= iters
        # the debiasing gradient alone, on the layer's starting pattern
        # (median of 10 event-timed calls)
        evs = []
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            L1.sddmm_masked_wgrad(W0, dYs[1], Xs[1], gv)
            e1.record()
            evs.append((e0, e1))
        torch.cuda.synchronize()
        sd_us = float(np.median([e0.elapsed_time(e1) * 1e3 for e0, e1 in evs]))
        yield _line(f"fc4096_b512_d{pct}_alternating_l1_debias", flops, ms,
                    dict(N=N, K=K, B=B, nnz=L.nnz, density=pct / 100, lam=lam, iterations=iters),
                    None, nnz_after_l1_steps=nnz_seq, debias_sddmm_us=round(sd_us, 1),
                    debias_sddmm_tflops=round(2.0 * L.nnz * B / (sd_us * 1e-6) / 1e12, 2))


def fc9216x4096_adaptive(args, dev):
    """One line per solver: fwd, CSC, bwd, dense dW, then the fused adaptive
    prox + recompression over all N*K weights (L1.l1_step with the adaptive
    state, on two streams; the serial calls beside it) with dense m, v state (which
    advances every step; the work per step is the same).  eta = 1e-3 (the usual
    ADAM step), lambda = 1e-4 as for the plain step: almost every weight
    survives, the largest output the step can have."""
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    L = synth.fc9216_4096(seed=0)
    N, K, B, nnz = L.N, L.K, L.B, L.nnz
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, K, device=dev)
    X, dY = torch.from_numpy(L.X).to(dev), torch.from_numpy(L.dY).to(dev)
    Y = torch.empty((N, B), dtype=torch.float32, device=dev)
    dX = torch.empty((K, B), dtype=torch.float32, device=dev)
    dW = torch.empty((N, K), dtype=torch.float32, device=dev)
    csc = L1.CSC.empty(K, nnz, dev)
    Wout = _csr_out(L1, torch, N, K, dev)
    eta, lam = 1e-3, L.lam
    for solver, tag in [(L1.SOLVER_ADAM, "adam"), (L1.SOLVER_RMSPROP, "rmsprop")]:
        st = L1.AdaptiveState.zeros(solver, (N, K), dev)
        names = ["csr_spmm_fwd", "csc_build", "csr_spmm_bwd_t", "dense_wgrad", f"prox_{tag}_recompress"]

        def step(ev=None, prec=L1.F32):
            mark = (lambda i: ev[i].record()) if ev else (lambda i: None)
            mark(0); L1.csr_spmm_fwd(W, X, Y)
            mark(1); L1.csc_build(W, csc)
            mark(2); L1.csr_spmm_bwd_t(W, dY, csc, dX)
            mark(3); L1.dense_wgrad(dY, X, dW, precision=prec)
            mark(4); L1.prox_adaptive_recompress(W, dW, st, eta, lam, out=Wout)
            mark(5)
        def step2(ev=None, prec=L1.F32):  # the two-stream schedule of L1.l1_step
            L1.l1_step(W, X, dY, eta, lam, Y=Y, dX=dX, dW=dW, csc=csc, out=Wout, precision=prec,
                       schedule="two_stream", adaptive=st)
        # serial calls (per-call split), then the two-stream step (the line's value)
        ms_serial, per = _timed(torch, step, max(args.steps, 10), max(args.warmup, 3), names)
        ms, _ = _timed(torch, step2, max(args.steps, 10), max(args.warmup, 3), None)
        nnz_out = int(Wout.row_ptr[-1].item())
        # the same step with the split-bf16 weight gradient (inside the 1e-4 contract)
        ms_x3, _ = _timed(torch, lambda ev=None: step2(ev, prec=L1.BF16X3), max(args.steps, 10),
                          max(args.warmup, 3), None)
        state_bytes = (16.0 if solver == L1.SOLVER_ADAM else 8.0) * N * K  # read and write m, v / v
        alg = 4.0 * N * K + state_bytes + (8.0 * nnz + 4 * (N + 1)) + (8.0 * nnz_out + 4 * (N + 1))
        # the two-pass kernels also re-read m', v' (ADAM) or G, v' (RMSProp)
        moved = alg + 8.0 * N * K
        kms = per[f"prox_{tag}_recompress"]
        flops = 4.0 * nnz * B + 2.0 * N * K * B
        yield _line(f"fc9216x4096_b1024_d9_zipf_l1_step_prox_{tag}", flops, ms,
                    dict(N=N, K=K, B=B, nnz=nnz, density=0.09, solver=tag, eta=eta, lam=lam,
                         eps=st.eps, beta1=st.beta1 if tag == "adam" else None, beta2=st.beta2), per,
                    nnz_out=nnz_out,
                    prox_hbm_algorithmic_bytes=alg, prox_hbm_gbs=round(alg / (kms * 1e-3) / 1e9, 1),
                    prox_hbm_frac=round(alg / (kms * 1e-3) / 1e9 / 8000.0, 4),
                    prox_bytes_moved_two_pass=moved,
                    prox_moved_gbs=round(moved / (kms * 1e-3) / 1e9, 1),
                    ms_per_step_bf16x3=round(ms_x3, 4),
                    value_bf16x3=round(flops / (ms_x3 * 1e-3) / 1e9, 1),
                    ms_per_step_serial=round(ms_serial, 4),
                    note="ms_per_step: L1.l1_step on two streams (fp32 and BF16X3 dW); "
                         "ms_per_step_serial and kernels_ms: the calls one after another on one stream")
        del st


LENET_G1 = (1, 28, 28, 5, 5, 1, 1, 0, 0)
LENET_P1 = (20, 24, 24, 2, 2, 2, 2, 0, 0)
LENET_G2 = (20, 12, 12, 5, 5, 1, 1, 0, 0)
LENET_P2 = (50, 8, 8, 2, 2, 2, 2, 0, 0)


def _dense_lenet(layers):
    """The same network with every weight stored (the uncompressed model)."""
    out = {}
    rng = np.random.default_rng(123)
    for k, (n_out, fan_in, _, _, _) in layers.items():
        rp = (np.arange(n_out + 1) * fan_in).astype(np.int32)
        ci = np.tile(np.arange(fan_in, dtype=np.int32), n_out)
        v = (rng.standard_normal(n_out * fan_in) * np.sqrt(2.0 / fan_in)).astype(np.float32)
        v[v == 0] = 1e-3
        out[k] = (n_out, fan_in, rp, ci, v)
    return out


def lenet5_inference(args, dev):
    """Forward-only LeNet-5: conv1 20@5x5 -> max pool 2 -> conv2 50@5x5 -> max
    pool 2 -> fc1 500 -> ReLU -> fc2 10, weights with the Table A1 SpC(Retrain)
    nonzero counts (12,217 of 430,500), inputs 28 x 28 maps, batch-contiguous.
    One line per batch size: images/s eager and replayed from a HIP graph, the
    per-layer times, and the same network with all weights stored."""
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    from paper_1905_07931_amd.metrics import compression_label
    g1, p1, g2, p2 = (L1.ConvGeom(*x) for x in (LENET_G1, LENET_P1, LENET_G2, LENET_P2))
    names = ["conv1", "pool1", "conv2", "pool2", "fc1", "relu", "fc2"]
    for B in (1, 64, 256, 1024, 10000):
        layers, Xh = synth.lenet5_compressed(seed=0, B=B)
        X = torch.from_numpy(Xh).to(dev)
        res = {}
        for tag, ls in (("compressed", layers), ("all_weights", _dense_lenet(layers))):
            W = {k: L1.CSR.from_host(v[2], v[3], v[4], v[1], device=dev) for k, v in ls.items()}
            y1 = torch.empty((20 * 576, B), dtype=torch.float32, device=dev)
            q1 = torch.empty((20 * 144, B), dtype=torch.float32, device=dev)
            y2 = torch.empty((50 * 64, B), dtype=torch.float32, device=dev)
            q2 = torch.empty((800, B), dtype=torch.float32, device=dev)
            h1 = torch.empty((500, B), dtype=torch.float32, device=dev)
            r1 = torch.empty_like(h1)
            z = torch.empty((10, B), dtype=torch.float32, device=dev)

            def step(ev=None):
                mark = (lambda i: ev[i].record()) if ev else (lambda i: None)
                mark(0); L1.csr_conv_fwd(g1, W["conv1"], X, y1)
                mark(1); L1.maxpool_fwd(p1, y1, q1)
                mark(2); L1.csr_conv_fwd(g2, W["conv2"], q1, y2)
                mark(3); L1.maxpool_fwd(p2, y2, q2)
                mark(4); L1.csr_spmm_fwd(W["fc1"], q2, h1)
                mark(5); L1.relu_fwd(h1, r1)
                mark(6); L1.csr_spmm_fwd(W["fc2"], r1, z)
                mark(7)
            ms, per = _timed(torch, step, max(args.steps, 20), max(args.warmup, 5), names)
            ms_graph = _graph_timed(torch, step, max(args.steps, 20))
            nnz = {k: int(v[2][-1]) for k, v in ls.items()}
            macs = nnz["conv1"] * 576 + nnz["conv2"] * 64 + nnz["fc1"] + nnz["fc2"]
            res[tag] = dict(ms=ms, ms_graph=ms_graph, per=per, nnz=sum(nnz.values()), macs=macs)
            del W, y1, q1, y2, q2, h1, r1, z
        c, d = res["compressed"], res["all_weights"]
        best = min(c["ms"], c["ms_graph"])
        yield _line(f"lenet5_inference_b{B}", 2.0 * c["macs"] * B, best,
                    dict(model="LeNet-5 (Table A1 SpC(Retrain) nonzeros)", B=B, nnz=c["nnz"],
                         weights=430500), c["per"],
                    images_per_s=round(B / (best * 1e-3), 1),
                    ms_per_batch_eager=round(c["ms"], 4), ms_per_batch_graph=round(c["ms_graph"], 4),
                    all_weights_ms=round(min(d["ms"], d["ms_graph"]), 4),
                    all_weights_kernels_ms=d["per"],
                    speedup_vs_all_weights=round(min(d["ms"], d["ms_graph"]) / best, 2),
                    compression=compression_label(c["nnz"], 430500),
                    note="value = 2 * (nonzero MACs per image) * B / time")


def conv2_direct(args, dev):
    """LeNet-5 conv2 (20 -> 50 channels, 5x5, 12x12 maps, batch 256, 10%
    density) from the maps: the l1-phase step with the direct sparse products."""
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    L = synth.lenet5_conv2(seed=0)
    g = L1.ConvGeom(*L.geom)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    X, dY = torch.from_numpy(L.X).to(dev), torch.from_numpy(L.dY).to(dev)
    F = L.OH * L.OW * L.B
    Y = torch.empty((L.n_out * L.OH * L.OW, L.B), dtype=torch.float32, device=dev)
    dX = torch.empty_like(X)
    Xc = torch.empty((L.K, F), dtype=torch.float32, device=dev)
    dW = torch.empty((L.n_out, L.K), dtype=torch.float32, device=dev)
    gv = torch.empty(max(L.nnz, 1), dtype=torch.float32, device=dev)
    dYm = dY.view(L.n_out, F)
    csc = L1.CSC.empty(L.K, L.nnz, dev)
    Wout = _csr_out(L1, torch, L.n_out, L.K, dev)
    names = ["csr_conv_fwd", "csc_build", "csr_conv_bwd_data", "conv_im2col", "dense_wgrad",
             "prox_l1_recompress", "sddmm_masked_wgrad"]

    def step(ev=None):
        mark = (lambda i: ev[i].record()) if ev else (lambda i: None)
        mark(0); L1.csr_conv_fwd(g, W, X, Y)
        mark(1); L1.csc_build(W, csc)
        mark(2); L1.csr_conv_bwd_data(g, L.n_out, csc, dY, dX, nnz=L.nnz)
        mark(3); L1.conv_im2col(g, X, Xc)
        mark(4); L1.dense_wgrad(dYm, Xc, dW)
        mark(5); L1.prox_l1_recompress(W, dW, L.eta, L.lam, out=Wout)
        mark(6); L1.sddmm_masked_wgrad(W, dYm, Xc, gv)
        mark(7)
    ms, per = _timed(torch, step, max(args.steps, 20), max(args.warmup, 5), names)
    ms_graph = _graph_timed(torch, step, max(args.steps, 20))
    # the l1 step proper (fwd, CSC, input gradient, im2col, dense filter
    # gradient, prox); the sampled gradient of the debiasing phase is timed beside it
    l1_ms = sum(v for k, v in per.items() if k != "sddmm_masked_wgrad")
    flops = 2.0 * L.nnz * F * 2 + 2.0 * L.n_out * L.K * F
    im2col_bytes = 4.0 * L.K * F + 4.0 * L.C * L.H * L.W * L.B
    yield _line("lenet5_conv2_direct_b256_d10_l1_step", flops, l1_ms,
                dict(n_out=L.n_out, C=L.C, H=L.H, W=L.W, KH=L.KH, KW=L.KW, B=L.B, nnz=L.nnz, density=0.10),
                per, ms_all_calls_eager=round(ms, 4), ms_all_calls_graph=round(ms_graph, 4),
                im2col_hbm_gbs=round(im2col_bytes / (per["conv_im2col"] * 1e-3) / 1e9, 1),
                note="value over the l1-step calls; the sampled filter gradient is the debiasing phase's")


PEAK_HBM_GBS = 8000.0
HBM_COUNTERS = os.path.join(ROOT, "profiles", "hbm_kernels_conv2_fc4096d1_counters.txt")


def csrc_hash():
    """Hash of every kernel source: counter bytes are used only if they were
    taken on the current sources."""
    import hashlib
    d = os.path.join(ROOT, "paper_1905_07931_amd", "csrc")
    h = hashlib.sha256()
    for n in sorted(os.listdir(d)):
        if n.endswith((".hip", ".hpp")):
            with open(os.path.join(d, n), "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def _counter_bytes():
    """{"workload/call": FETCH+WRITE bytes per call} from the committed counter
    summary, or {} if it is missing or was taken on other sources."""
    if not os.path.exists(HBM_COUNTERS):
        return {}
    with open(HBM_COUNTERS) as f:
        for line in f:
            if line.startswith("counters_json:"):
                d = json.loads(line.split(":", 1)[1])
                if d.get("source_hash") == csrc_hash():
                    return d.get("bytes_per_call", {})
    return {}


def _copy_ceiling(torch, dev):
    """Bytes moved (read + write) per second by a 1 GiB device-to-device copy."""
    x = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        y.copy_(x)
    b.record()
    torch.cuda.synchronize()
    gbs = 2.0 * (1 << 30) / (a.elapsed_time(b) / 5 * 1e-3) / 1e9
    del x, y
    return gbs


def _call_times(torch, call, reps, flush, order, tag):
    """Median event time of `call` warm (back-to-back calls) and cold (a 1 GiB
    write before each call, so neither L2 nor the 256 MB MALL holds its
    operands).  The warm calls are queued behind a spin kernel of a few ms, so
    they run back to back however long the host takes to enqueue them (a call
    of a few us is shorter than its Python launch).  Cold calls are appended
    to `order` (the counter summary maps the kernels between two flushes to
    that call)."""
    call()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda._sleep(int(2.4e9 * 300e-6 * reps))  # ~300 us of GPU clock per queued call
    for a, b in ev:
        a.record()
        call()
        b.record()
    torch.cuda.synchronize()
    warm = float(np.median([a.elapsed_time(b) for a, b in ev]))
    for a, b in ev:
        flush.fill_(1.0)
        order.append(tag)
        a.record()
        call()
        b.record()
    torch.cuda.synchronize()
    cold = float(np.median([a.elapsed_time(b) for a, b in ev]))
    return warm, cold


def hbm_kernels(args, dev):
    import torch
    import paper_1905_07931_amd as L1
    from paper_1905_07931_amd import synth
    copy_gbs = _copy_ceiling(torch, dev)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
    counted = _counter_bytes()
    order = []
    reps = max(args.steps, 10)
    lines = []

    def emit(workload, cfg, call, ms_warm, ms_cold, alg, note):
        tag = f"{workload}/{call}"
        cb = counted.get(tag)
        g_cold = alg / (ms_cold * 1e-3) / 1e9
        g_warm = alg / (ms_warm * 1e-3) / 1e9
        lines.append({"metric": "achieved HBM GB/s (algorithmic bytes)", "value": round(g_cold, 1), "unit": "GB/s",
                      "n_gpus": 1, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
                      "config": dict(workload=workload, call=call, **cfg), "informational": True,
                      "ms_cold": round(ms_cold, 4), "ms_warm": round(ms_warm, 4), "algorithmic_bytes": alg,
                      "hbm_gbs_cold": round(g_cold, 1), "hbm_gbs_warm": round(g_warm, 1),
                      "frac_of_8tbs_cold": round(g_cold / PEAK_HBM_GBS, 4),
                      "frac_of_copy_cold": round(g_cold / copy_gbs, 4), "copy_ceiling_gbs": round(copy_gbs, 1),
                      "counter_bytes": cb, "counter_over_alg": round(cb / alg, 3) if cb else None,
                      "note": note})

    # LeNet-5 conv2 lowered by im2col: W 50 x 500 at 10%, X[500][16384]
    L = synth.conv2_im2col(seed=0)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    vals0 = W.vals.clone()
    X, dY = torch.from_numpy(L.X).to(dev), torch.from_numpy(L.dY).to(dev)
    Y = torch.empty((L.N, L.B), dtype=torch.float32, device=dev)
    dX = torch.empty((L.K, L.B), dtype=torch.float32, device=dev)
    gv = torch.empty(L.nnz, dtype=torch.float32, device=dev)
    csc = L1.CSC.empty(L.K, L.nnz, dev)
    L1.csc_build(W, csc)
    Wc = L1.CSR(L.N, L.K, torch.empty(L.N + 1, dtype=torch.int32, device=dev),
                torch.empty(L.nnz, dtype=torch.int32, device=dev),
                torch.empty(L.nnz, dtype=torch.float32, device=dev), None)
    N, K, B, nnz = L.N, L.K, L.B, L.nnz
    wl, cfg = "conv2_im2col_50x500_b16384_d10", dict(N=N, K=K, B=B, nnz=nnz)
    csr_b = 8.0 * nnz + 4.0 * (N + 1)
    calls = [
        ("csr_spmm_fwd", lambda: L1.csr_spmm_fwd(W, X, Y), csr_b + 4.0 * (K + N) * B, "CSR + X in, Y out"),
        ("csc_build", lambda: L1.csc_build(W, csc), csr_b + 12.0 * nnz + 4.0 * (K + 1),
         "CSR in; col_ptr, row_idx, perm, vals_t out"),
        ("csr_spmm_bwd_t", lambda: L1.csr_spmm_bwd_t(W, dY, csc, dX), 8.0 * nnz + 4.0 * (K + 1) + 4.0 * (K + N) * B,
         "CSC + dY in, dX out"),
        ("sddmm_masked_wgrad", lambda: L1.sddmm_masked_wgrad(W, dY, X, gv), csr_b + 4.0 * (K + N) * B + 4.0 * nnz,
         "pattern + dY + X in, gv out"),
        ("prox_l1_step_csr", lambda: L1.prox_l1_step(L1.PROX_CSR, W, gv, L.eta, L.lam), 12.0 * nnz,
         "vals and gv in, vals out (support-restricted prox)"),
        ("csr_compact", lambda: L1.csr_compact(W, Wc), csr_b + 8.0 * nnz + 4.0 * (N + 1),
         "CSR in, CSR without stored zeros out"),
    ]
    for name, fn, alg, note in calls:
        def fnr(fn=fn):
            fn()
        w, c = _call_times(torch, fnr, reps, flush, order, f"{wl}/{name}")
        W.vals.copy_(vals0)
        emit(wl, cfg, name, w, c, alg, note)
    del X, dY, Y, dX

    # the 4096 x 4096 layer at 1% density, batch 512 (one l1 iteration's calls)
    L = synth.fc4096_sweep(0.01)
    lam = json.load(open(os.path.join(ROOT, "tests", "golden", "fc4096_lambda.json")))["lambda"]["1"]
    x_, d_ = synth.fc4096_batch(0)
    X, dY = torch.from_numpy(x_).to(dev), torch.from_numpy(d_).to(dev)
    N, K, B, nnz = L.N, L.K, L.B, L.nnz
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, K, device=dev)
    Y = torch.empty((N, B), dtype=torch.float32, device=dev)
    dX = torch.empty((K, B), dtype=torch.float32, device=dev)
    gv = torch.empty(nnz, dtype=torch.float32, device=dev)
    dW = torch.empty((N, K), dtype=torch.float32, device=dev)
    Z = torch.empty((N, K), dtype=torch.float32, device=dev)
    csc = L1.CSC.empty(K, nnz, dev)
    L1.csc_build(W, csc)
    bm = L1.csr_bitmap_build(W)
    L1.dense_wgrad(dY, X, dW)
    out = _csr_out(L1, torch, N, K, dev)
    _, wc = L1.dense_wgrad_prox(W, dY, X, L.eta, lam, bm, Z=Z)
    L1.csr_recompress_counted(Z, wc, out=out)
    nnz_out = out.host_nnz()
    wl, cfg = "fc4096_b512_d1", dict(N=N, K=K, B=B, nnz=nnz, nnz_out=nnz_out)
    csr_b = 8.0 * nnz + 4.0 * (N + 1)
    kw = (K + 31) // 32
    calls = [
        ("csr_spmm_fwd", lambda: L1.csr_spmm_fwd(W, X, Y), csr_b + 4.0 * (K + N) * B, "CSR + X in, Y out"),
        ("csr_spmm_bwd_t", lambda: L1.csr_spmm_bwd_t(W, dY, csc, dX), 8.0 * nnz + 4.0 * (K + 1) + 4.0 * (K + N) * B,
         "CSC + dY in, dX out"),
        ("sddmm_masked_wgrad", lambda: L1.sddmm_masked_wgrad(W, dY, X, gv), csr_b + 4.0 * (K + N) * B + 4.0 * nnz,
         "pattern + dY + X in, gv out"),
        ("prox_l1_recompress", lambda: L1.prox_l1_recompress(W, dW, L.eta, lam, out=out, capacity=N * K),
         4.0 * N * K + csr_b + 8.0 * nnz_out + 4.0 * (N + 1), "dW + CSR in (dW once), CSR' out"),
        ("csr_recompress_counted", lambda: L1.csr_recompress_counted(Z, wc, out=out, capacity=N * K),
         4.0 * N * K + 4.0 * N * kw + 8.0 * nnz_out + 4.0 * (N + 1), "Z + word counts in, CSR' out"),
        ("csr_bitmap_build", lambda: L1.csr_bitmap_build(W, bm), csr_b + 8.0 * N * kw, "CSR in, mask + pos out"),
    ]
    for name, fn, alg, note in calls:
        w, c = _call_times(torch, fn, reps, flush, order, f"{wl}/{name}")
        emit(wl, cfg, name, w, c, alg, note)
    lines.append({"hbm_kernels_cold_order": order, "source_hash": csrc_hash(), "informational": True})
    yield from lines


def run(name, args, dev):
    return {"fc784x300": fc784x300, "mlp784": mlp784, "conv2": conv2, "fc4096_sweep": fc4096_sweep,
            "fc9216x4096_adaptive": fc9216x4096_adaptive, "lenet5_inference": lenet5_inference,
            "conv2_direct": conv2_direct, "hbm_kernels": hbm_kernels}[name](args, dev)
