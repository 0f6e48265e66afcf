"""One l1-phase training step of a CSR layer on two HIP streams.

The step of Sections 2.3 and 3.1-3.2 for a layer Y = W X with W stored
compressed (CSR) and activations batch-contiguous:

    Y  = W X                      forward product
    CSC(W)                        column-major copy of W for the transposed product
    dX = W^T dY                   backward product (gradient to the layer below)
    G  = dY X^T                   dense weight gradient (every weight, zero or not)
    W' = prox_{eta*lambda}(W - eta G), recompressed to CSR   (Eq. (prox))

The last two run as dense_wgrad_prox (the GEMM's epilogue applies the soft
threshold to its own result and counts the survivors per 32-column word) and
csr_recompress_counted, so the dense Z = S_t(W - eta G) is written once and
read once by the recompression, and G itself is never stored.  With an adaptive solver
(Algorithms 1-2) G is stored and the preconditioned step is fused with the
recompression instead (prox_adaptive_recompress).

Only the forward product has to finish before the rest: dY is the upstream
gradient of Y.  The calls keep the dependencies of a training loop and run on
two streams of equal (default) priority:

    main:  fwd ─────────────────────┬── dW GEMM + prox ──── recompress ───┐
    side:  bitmap ─┴─ CSC ─ bwd plan ─┴─ bwd (W^T dY) ─────────────────────┴─ join

W's bitmap index (read by the GEMM's prox epilogue and by the CSC build),
the CSC copy and the backward product's plan (csr_spmm_plan over the CSC)
depend on W only, so they fill the gaps of the forward product's planning
launches; the backward product itself needs dY and runs beside the weight
update.  Every launch is deterministic, so the outputs equal those
of the same calls made one after another on one stream, bit for bit.

The overlap pays where a product takes the tiled path (a workspace for its
plan and pair stream).  Small layers run the rows kernel, a few short launches
with no planning to hide; there the waits between the streams cost more than
they save (at 784 -> 300, batch 64: 180 us on two streams against 100 us on
one), so the default schedule ("auto") makes the calls one after another on
the caller's stream unless one of the two products is tiled.

Each entry point keeps its own workspace per stream, so the two streams never
share scratch memory.  The function is capture-safe: it forks the side stream
from the caller's stream and joins it back before returning, so it records
into a HIP graph (torch.cuda.CUDAGraph) like a single-stream sequence.  As
for every entry point under capture, W's nnz must be known on the host
(W.nnz set): reading it from the device is a host wait.
"""
from __future__ import annotations

from . import (CSC, CSR, F32, OP_SPMM, AdaptiveState, Bitmap, SpmmPlan, csc_build, csr_bitmap_build,
               csr_recompress_counted, csr_spmm_bwd_t, csr_spmm_bwd_t_plan, csr_spmm_bwd_t_planned, csr_spmm_fwd,
               dense_wgrad, dense_wgrad_prox, prox_adaptive_recompress, workspace_bytes)

_side_streams: dict = {}
_plans: dict = {}


def _bwd_plan(W: CSR, csc: CSC, B: int, side) -> SpmmPlan:
    """The backward product's plan buffer of this side stream, taken for this
    shape (one buffer per side stream, grown when a larger plan needs it and
    never freed, so its memory is not handed to other work while the side
    stream may still use it; the steps on one side stream use it in order)."""
    import torch
    key = (side.cuda_stream, csc.col_ptr.device)
    p = _plans.get(key)
    # allocated with the side stream current, like the call workspaces: a
    # replaced buffer goes back to the caching allocator in that stream's order
    with torch.cuda.stream(side):
        if p is None:
            p = SpmmPlan(W.n_cols, W.n_rows, W.host_nnz(), B, csc.col_ptr.device)
            _plans[key] = p
        else:
            p.reshape(W.n_cols, W.n_rows, W.host_nnz(), B)
    return p


def side_stream(device):
    """The side stream used for `device` (created once, default priority)."""
    import torch
    idx = torch.device(device).index
    if idx is None:
        idx = torch.cuda.current_device()
    s = _side_streams.get(idx)
    if s is None:
        s = torch.cuda.Stream(device=idx)
        _side_streams[idx] = s
    return s


def two_stream_pays(W: CSR, B: int) -> bool:
    """True if either product of W at batch B takes the tiled path."""
    nnz = W.host_nnz()
    return (workspace_bytes(OP_SPMM, W.n_rows, W.n_cols, nnz, B) > 0
            or workspace_bytes(OP_SPMM, W.n_cols, W.n_rows, nnz, B) > 0)


def l1_step(W: CSR, X, dY, eta: float, lam: float, *, Y, dX, dW, csc: CSC, out: CSR,
            precision: int = F32, side=None, events: dict | None = None,
            schedule: str = "auto", adaptive: AdaptiveState | None = None,
            bitmap: Bitmap | None = None) -> CSR:
    """Run one l1 step on the caller's current stream plus a side stream.

    W is the N x K layer (CSR, nnz known on the host or read from the device),
    X the K x B input, dY the N x B upstream gradient.  Results go to the
    caller's buffers: Y (N x B), dX (K x B), dW (N x K: the dense prox result
    Z = S_t(W - eta G) of the plain step, the gradient G of an adaptive one),
    csc (the CSC copy of W, capacity >= nnz) and out (W' in CSR, capacity N*K).
    precision selects the dense weight gradient's arithmetic (F32 or BF16X3).
    side: the stream to fork onto (default: one per device).  events: optional
    {call name: (start, end)} torch events, recorded around that call on the
    stream it runs on ("csr_bitmap_build", "csc_build", "csr_spmm_fwd",
    "csr_spmm_bwd_t_plan" (two streams only), "csr_spmm_bwd_t",
    "dense_wgrad_prox", "csr_recompress_counted"; adaptive:
    "dense_wgrad",
    "prox_adaptive_recompress").  schedule: "two_stream", "serial" (every call on the
    caller's stream) or "auto" (two_stream where a product is tiled).
    adaptive: Prox-RMSProp / Prox-ADAM state with dense [N][K] m, v; the step
    then ends with prox_adaptive_recompress (state updated in place, t
    advanced) instead of dense_wgrad_prox + csr_recompress_counted.  bitmap: buffers for
    W's bitmap index (Bitmap.empty(N, K), shared by the CSC build and the weight
    update); allocated per call if None.  All
    outputs are ready on the
    caller's stream when the call returns.  Returns out.
    """
    import torch
    if schedule not in ("auto", "two_stream", "serial"):
        raise ValueError(f"unknown schedule {schedule!r}")
    main = torch.cuda.current_stream(X.device)
    if schedule == "auto":
        schedule = "two_stream" if two_stream_pays(W, X.shape[1]) else "serial"
    if schedule == "serial":
        side = main
    elif side is None:
        side = side_stream(X.device)
    elif side.cuda_stream == main.cuda_stream:
        raise ValueError("the side stream must differ from the current stream")

    def call(name, stream, fn):
        ev = events.get(name) if events else None
        if ev is not None:
            ev[0].record(stream)
        fn()
        if ev is not None:
            ev[1].record(stream)

    fork = side is not main
    if bitmap is None:
        bitmap = Bitmap.empty(W.n_rows, W.n_cols, X.device)  # on the caller's stream
    if fork:
        side.wait_stream(main)  # W, X, dY as the caller left them
    # the forward product is enqueued first, so its launches reach the GPU first
    call("csr_spmm_fwd", main, lambda: csr_spmm_fwd(W, X, Y, stream=main))
    call("csr_bitmap_build", side, lambda: csr_bitmap_build(W, bitmap, stream=side))
    if fork:
        indexed = torch.cuda.Event()
        indexed.record(side)
    call("csc_build", side, lambda: csc_build(W, csc, bitmap=bitmap, stream=side))
    plan = None
    if fork and not torch.cuda.is_current_stream_capturing():
        # the backward product's planning needs W (its CSC) only: it runs here,
        # beside the forward product's planning, not behind the weight-gradient
        # GEMM (whose workgroups fill every CU once it starts).  A captured
        # graph keeps the whole call after the forward product: there the
        # runtime orders the two branches' launches itself, and planning ahead
        # measured slower (1.53 against 1.48 ms at 9216 -> 4096).
        plan = _bwd_plan(W, csc, dY.shape[1], side)
        call("csr_spmm_bwd_t_plan", side, lambda: csr_spmm_bwd_t_plan(W, csc, dY.shape[1], plan, stream=side))
        side.wait_stream(main)  # dY follows Y; the CSC and the plan are on side already
        call("csr_spmm_bwd_t", side, lambda: csr_spmm_bwd_t_planned(W, dY, csc, plan, dX, stream=side))
    else:
        if fork:
            side.wait_stream(main)  # dY follows Y; the CSC is on side already
        call("csr_spmm_bwd_t", side, lambda: csr_spmm_bwd_t(W, dY, csc, dX, stream=side))
    if adaptive is None:
        if fork:
            main.wait_event(indexed)
        counts = {}
        call("dense_wgrad_prox", main,
             lambda: counts.setdefault("wc", dense_wgrad_prox(W, dY, X, eta, lam, bitmap, Z=dW, precision=precision,
                                                              stream=main)[1]))
        call("csr_recompress_counted", main, lambda: csr_recompress_counted(dW, counts["wc"], out=out, stream=main))
    else:
        call("dense_wgrad", main, lambda: dense_wgrad(dY, X, dW, precision=precision, stream=main))
        call("prox_adaptive_recompress", main,
             lambda: prox_adaptive_recompress(W, dW, adaptive, eta, lam, out=out, stream=main))
    if fork:
        main.wait_stream(side)
    return out
