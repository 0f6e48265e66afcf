"""l1csr: the training hot path of l1-regularised compressed learning on MI355X.

A thin ctypes binding over ``libl1csr.so`` (built by
``python -m paper_1905_07931_amd.build``).  The functions keep the names of
the C ABI in ``include/l1csr.h``; they only check and marshal arguments
(torch tensors on the GPU -> device pointers, torch's current HIP stream) and
raise :class:`L1CSRError` on a non-zero status.  Every computation runs in the
library's HIP kernels; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

__all__ = [
    "CSR", "CSC", "L1CSRError", "lib", "status_str", "workspace_bytes",
    "csr_spmm_fwd", "csc_build", "csc_update_vals", "csr_spmm_bwd_t", "dense_wgrad", "sddmm_masked_wgrad",
    "prox_l1_step", "csr_recompress", "prox_l1_recompress", "csr_compact", "csr_validate", "relu_fwd", "relu_bwd",
    "softmax_xent", "PROX_DENSE", "PROX_CSR", "F32", "BF16", "BF16X3",
    "prox_adaptive_step", "prox_adaptive_recompress", "SOLVER_RMSPROP", "SOLVER_ADAM", "AdaptiveState",
    "ConvGeom", "csr_conv_fwd", "csr_conv_bwd_data", "conv_im2col", "maxpool_fwd",
    "l1_step", "side_stream", "prox_l1_recompress_noalloc", "dense_wgrad_prox", "csr_recompress_counted",
    "dense_wgrad_prox_recompress", "csr_bitmap_build", "Bitmap", "SpmmPlan", "csr_spmm_plan", "csr_spmm_planned",
    "csr_spmm_bwd_t_plan", "csr_spmm_bwd_t_planned",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libl1csr.so")

OK, EINVAL, ECAPACITY, EBADCSR, EHIP, EUNSUPPORTED, ESCRATCH = 0, -1, -2, -3, -4, -5, -6
NOALLOC_SCRATCH_BYTES = 16 << 20  # L1CSR_NOALLOC_SCRATCH_BYTES
PROX_DENSE, PROX_CSR = 0, 1
F32, BF16, BF16X3 = 0, 1, 2
SOLVER_RMSPROP, SOLVER_ADAM = 1, 2
OP_CSC_BUILD, OP_RECOMPRESS, OP_SDDMM, OP_SPMM, OP_COMPACT, OP_SOFTMAX_XENT = 1, 2, 3, 4, 5, 6
OP_PROX_RECOMPRESS = 7
OP_DENSE_WGRAD = 8
OP_WGRAD_PROX = 9


class L1CSRError(RuntimeError):
    def __init__(self, name, status):
        self.status = status
        super().__init__(f"{name} failed: {status_str(status)} ({status})")


_lib = None


def lib():
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_1905_07931_amd.build`")
        # torch ships its own libamdhip64.so.7; loaded first, it is the copy the
        # dynamic linker hands the library, so the process holds one HIP
        # runtime and torch's streams and memory are valid in the library's
        # launches (loaded the other way round, the library would bind the
        # system runtime and torch a second one)
        import torch  # noqa: F401
        L = C.CDLL(LIB_PATH)
        i32, i64, f32, vp, sz = C.c_int32, C.c_int64, C.c_float, C.c_void_p, C.c_size_t
        L.l1csr_status_str.argtypes = [C.c_int]
        L.l1csr_status_str.restype = C.c_char_p
        L.l1csr_workspace_bytes.argtypes = [C.c_int, i32, i32, i64, i32]
        L.l1csr_workspace_bytes.restype = sz
        L.l1csr_host_alloc_mapped.argtypes = [sz, C.POINTER(vp), C.POINTER(vp)]
        L.l1csr_host_free_mapped.argtypes = [vp]
        L.csr_spmm_fwd.argtypes = [i32, i32, i64, vp, vp, vp, vp, i64, i32, vp, i64, vp, sz, vp]
        L.csr_spmm_plan.argtypes = [i32, i32, i64, vp, vp, vp, i32, vp, sz, vp]
        L.csr_spmm_planned.argtypes = [i32, i32, i64, vp, vp, vp, vp, i64, i32, vp, i64, vp, sz, vp]
        L.csc_build.argtypes = [i32, i32, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.csc_update_vals.argtypes = [i32, i64, vp, vp, vp, vp, vp]
        L.csr_spmm_bwd_t.argtypes = [i32, i32, i64, vp, vp, vp, vp, vp, vp, vp, i64, i32, vp, i64,
                                     vp, sz, vp]
        L.dense_wgrad.argtypes = [i32, i32, i32, vp, i64, vp, i64, vp, i64, C.c_int, vp, sz, vp]
        L.sddmm_masked_wgrad.argtypes = [i32, i32, i64, vp, vp, vp, i64, vp, i64, i32, vp, vp, sz, vp]
        L.prox_l1_step.argtypes = [C.c_int, i32, i32, i64, vp, vp, vp, vp, i64, f32, f32, vp, i64,
                                   vp, vp]
        L.csr_recompress.argtypes = [i32, i32, vp, i64, f32, vp, vp, vp, vp, i64, vp,
                                     C.POINTER(C.c_int64), vp, sz, vp]
        L.prox_l1_recompress.argtypes = [i32, i32, i64, vp, vp, vp, vp, i64, f32, f32, vp, vp, vp,
                                         i64, vp, C.POINTER(C.c_int64), vp, sz, vp]
        L.prox_l1_recompress_noalloc.argtypes = [i32, i32, i64, vp, vp, vp, vp, i64, f32, f32, vp, vp,
                                                 vp, i64, vp, C.POINTER(C.c_int64), vp]
        L.dense_wgrad_prox.argtypes = [i32, i32, i32, vp, i64, vp, i64, C.c_int, i64, vp, vp, vp, vp, vp, f32, f32,
                                       vp, i64, vp, vp, sz, vp]
        L.csr_recompress_counted.argtypes = [i32, i32, vp, i64, vp, vp, vp, vp, i64, vp, C.POINTER(C.c_int64),
                                             vp, sz, vp]
        L.csr_bitmap_build.argtypes = [i32, i32, i64, vp, vp, vp, vp, vp]
        L.prox_adaptive_step.argtypes = [C.c_int, C.c_int, i32, i32, i64, vp, vp, vp, vp, i64, vp, vp,
                                         i64, f32, f32, f32, f32, f32, i64, vp, i64, vp, vp, sz, vp]
        L.prox_adaptive_recompress.argtypes = [C.c_int, i32, i32, i64, vp, vp, vp, vp, i64, vp, vp, i64,
                                               f32, f32, f32, f32, f32, i64, vp, vp, vp, i64, vp,
                                               C.POINTER(C.c_int64), vp, sz, vp]
        L.csr_compact.argtypes = [i32, i64, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.csr_conv_fwd.argtypes = [vp, i32, i64, vp, vp, vp, vp, i64, i32, vp, i64, vp]
        L.csr_conv_bwd_data.argtypes = [vp, i32, i64, vp, vp, vp, vp, i64, i32, vp, i64, vp]
        L.conv_im2col.argtypes = [vp, vp, i64, i32, vp, i64, vp]
        L.l1csr_maxpool_fwd.argtypes = [vp, vp, i64, i32, vp, i64, vp]
        L.csr_validate.argtypes = [i32, i32, i64, vp, vp, vp, vp]
        L.l1csr_relu_fwd.argtypes = [i64, vp, vp, vp]
        L.l1csr_relu_bwd.argtypes = [i64, vp, vp, vp, vp]
        L.l1csr_softmax_xent.argtypes = [i32, i32, vp, i64, vp, vp, vp, vp, sz, vp]
        for name in ("csr_spmm_fwd", "csr_spmm_plan", "csr_spmm_planned", "csc_build", "csc_update_vals", "csr_spmm_bwd_t", "dense_wgrad",
                     "sddmm_masked_wgrad", "prox_l1_step", "csr_recompress", "prox_l1_recompress",
                     "prox_l1_recompress_noalloc", "dense_wgrad_prox", "csr_recompress_counted", "csr_bitmap_build",
                     "csr_compact", "csr_validate", "l1csr_relu_fwd", "l1csr_relu_bwd", "l1csr_softmax_xent",
                     "prox_adaptive_step", "prox_adaptive_recompress", "csr_conv_fwd",
                     "csr_conv_bwd_data", "conv_im2col", "l1csr_maxpool_fwd"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().l1csr_status_str(int(status)).decode()


def workspace_bytes(op: int, n_rows: int, n_cols: int, nnz: int, B: int) -> int:
    return int(lib().l1csr_workspace_bytes(op, n_rows, n_cols, nnz, B))


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _check(rc, name):
    if rc != OK:
        raise L1CSRError(name, rc)


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


class _HostWord:
    """One int32 of pinned host memory that kernels write directly
    (l1csr_host_alloc_mapped), as a call's d_nnz_out: the count reaches the
    host with the call's own kernels, and no copy is queued behind it."""

    def __init__(self, host: int, dev: int):
        self.host, self.dev, self.event = host, dev, None

    def value(self) -> int:
        return C.c_int32.from_address(self.host).value


class _HostWords:
    """A CSR holds one word for its lifetime; when it goes, the word returns
    here and is handed out again only after the event recorded behind its
    last write has completed.  Pages are never freed (queued work may still
    write them)."""
    PAGE = 1024  # words per page

    def __init__(self):
        self.free: list = []
        self.disabled = False

    def acquire(self):
        for i, w in enumerate(self.free):
            if w.event is None or w.event.query():
                return self.free.pop(i)
        if self.disabled:
            return None
        h, d = C.c_void_p(), C.c_void_p()
        if lib().l1csr_host_alloc_mapped(4 * self.PAGE, C.byref(h), C.byref(d)) != 0:
            self.disabled = True  # the runtime refused: the calls fall back to a queued copy
            return None
        words = [_HostWord(h.value + 4 * i, d.value + 4 * i) for i in range(self.PAGE)]
        self.free.extend(words[1:])
        return words[0]

    def release(self, w):
        self.free.append(w)


_words = _HostWords()


def _nnz_word(out):
    """The word `out` has kernels write its nnz into (acquired on first use),
    or None under graph capture or where no mapped memory is available."""
    import weakref
    torch = _torch()
    if torch.cuda.is_current_stream_capturing():
        return None
    w = getattr(out, "_word", None)
    if w is None:
        w = _words.acquire()
        if w is not None:
            out._word = w
            weakref.finalize(out, _words.release, w)
    return w


def _nnz_dev(out):
    w = _nnz_word(out)
    return None if w is None else C.c_void_p(w.dev)


def _set_nnz(out, need, stream):
    """The host count a call returned (>= 0), else the count its kernels
    wrote into out's host word (an event behind them), else a queued copy.
    Whenever the call was given the word, the event goes behind it even if
    the host count is known: its kernels write the word all the same, and the
    pool hands the word to another CSR only once that write is done."""
    torch = _torch()
    w = getattr(out, "_word", None)
    capturing = torch.cuda.is_current_stream_capturing()
    ev = None
    if w is not None and not capturing:
        s = torch.cuda.current_stream(out.row_ptr.device) if stream is None else stream
        ev = torch.cuda.Event()
        ev.record(s)
        w.event = ev
    if need >= 0:
        out.nnz = int(need)
        out._pending = None
        return
    if ev is None:
        out.track_nnz(stream)
        return
    out.nnz = None
    out._pending = (w, ev)


def _stream(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _dev(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on the GPU (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    return t


def _vec(t, dtype, name):
    _dev(t, dtype, name)
    if t.dim() != 1 or (t.numel() > 1 and t.stride(0) != 1):
        raise ValueError(f"{name} must be a contiguous 1-D tensor")
    return t


def _mat(t, name):
    """A [rows][ld] float32 matrix with unit column stride; returns (rows, cols, ld)."""
    torch = _torch()
    _dev(t, torch.float32, name)
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    rows, cols = t.shape
    if cols > 1 and t.stride(1) != 1:
        raise ValueError(f"{name} must have a contiguous last dimension")
    ld = t.stride(0) if rows > 1 else max(cols, 1)
    return rows, cols, ld


_ws_cache: dict = {}


def _workspace(nbytes, device, stream=None):
    """Scratch for one call, cached per (device, stream the call runs on): calls
    on one stream run in order and may share it, calls on two streams never do.
    A buffer is allocated with its stream current, so the caching allocator
    reuses it only in that stream's order once it is replaced."""
    if nbytes == 0:
        return None, 0
    torch = _torch()
    s = torch.cuda.current_stream(device) if stream is None else stream
    key = (device.index, s.cuda_stream)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < nbytes:
        with torch.cuda.stream(s):
            buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    return buf, nbytes


@dataclass
class CSR:
    """An N x K CSR matrix in device memory (int32 indices, float32 values).

    ``nnz`` is the host-side count when known.  A call that writes a CSR
    without waiting (:func:`csr_recompress`, :func:`prox_l1_recompress`, ...
    at full capacity) leaves it ``None``: ``row_ptr[-1]`` holds it on the
    device, and the call's own kernels have also written it into a word of
    mapped pinned host memory that the CSR keeps (or, where the runtime gives
    no such memory, the call has queued a copy behind its last kernel).  The
    first use of the matrix then waits for that call only (an event), not for
    the whole device; set ``nnz`` beforehand (e.g. under graph capture) to
    avoid the wait.
    ``col_idx``/``vals`` may be longer than nnz (capacity).
    """
    n_rows: int
    n_cols: int
    row_ptr: "object"
    col_idx: "object"
    vals: "object"
    nnz: int | None = None
    _pending: "object" = None  # (pinned int32 holding nnz (a copy or a word kernels write), its event)

    def host_nnz(self) -> int:
        if self.nnz is None:
            if self._pending is not None:
                host, ev = self._pending
                ev.synchronize()
                self.nnz = host.value() if isinstance(host, _HostWord) else int(host[0])
            else:
                self.nnz = int(self.row_ptr[-1].item())
        self._pending = None
        return self.nnz

    def track_nnz(self, stream=None):
        """Queue the copy of row_ptr[-1] to pinned host memory on `stream`
        (after the kernels that wrote it) and forget the host count."""
        torch = _torch()
        s = torch.cuda.current_stream(self.row_ptr.device) if stream is None else stream
        self.nnz = None
        self._pending = None
        if torch.cuda.is_current_stream_capturing():
            return  # a captured graph has no host copy to wait for: the caller sets nnz
        host = torch.empty(1, dtype=torch.int32, pin_memory=True)
        with torch.cuda.stream(s):
            host.copy_(self.row_ptr[-1:], non_blocking=True)
            ev = torch.cuda.Event()
            ev.record(s)
        self._pending = (host, ev)

    def validate_shapes(self):
        torch = _torch()
        _vec(self.row_ptr, torch.int32, "row_ptr")
        _vec(self.col_idx, torch.int32, "col_idx")
        _vec(self.vals, torch.float32, "vals")
        if self.row_ptr.numel() != self.n_rows + 1:
            raise ValueError("row_ptr must have n_rows + 1 entries")
        # the stored count sizes plans and workspaces: never guess it from the capacity
        nnz = self.host_nnz()
        if self.col_idx.numel() < nnz or self.vals.numel() < nnz:
            raise ValueError("col_idx/vals shorter than nnz")
        return nnz

    @staticmethod
    def from_host(row_ptr, col_idx, vals, n_cols, device="cuda", capacity=None):
        torch = _torch()
        import numpy as np
        rp = torch.as_tensor(np.ascontiguousarray(row_ptr, dtype=np.int32), device=device)
        nnz = int(rp[-1].item()) if rp.numel() else 0
        cap = max(nnz if capacity is None else capacity, 1)
        ci = torch.zeros(cap, dtype=torch.int32, device=device)
        v = torch.zeros(cap, dtype=torch.float32, device=device)
        if nnz:
            ci[:nnz] = torch.as_tensor(np.ascontiguousarray(col_idx[:nnz], dtype=np.int32), device=device)
            v[:nnz] = torch.as_tensor(np.ascontiguousarray(vals[:nnz], dtype=np.float32), device=device)
        return CSR(rp.numel() - 1, n_cols, rp, ci, v, nnz)

    def to_host(self):
        nnz = self.host_nnz()
        return (self.row_ptr.cpu().numpy(), self.col_idx[:nnz].cpu().numpy(),
                self.vals[:nnz].cpu().numpy())


@dataclass
class CSC:
    """Column-major copy of a CSR matrix: col_ptr, row_idx, perm (CSR position of
    each entry) and vals_t (its value)."""
    col_ptr: "object"
    row_idx: "object"
    perm: "object"
    vals_t: "object"

    @staticmethod
    def empty(n_cols, capacity, device):
        torch = _torch()
        cap = max(int(capacity), 1)
        return CSC(torch.empty(n_cols + 1, dtype=torch.int32, device=device),
                   torch.empty(cap, dtype=torch.int32, device=device),
                   torch.empty(cap, dtype=torch.int32, device=device),
                   torch.empty(cap, dtype=torch.float32, device=device))


# ---------------------------------------------------------------------------
# the ABI, one function per entry point
# ---------------------------------------------------------------------------

def csr_spmm_fwd(W: CSR, X, Y=None, stream=None):
    """Y = W . X  (X [K][B], Y [N][B], batch contiguous)."""
    torch = _torch()
    nnz = W.validate_shapes()
    K, B, ldx = _mat(X, "X")
    if K != W.n_cols:
        raise ValueError(f"X has {K} rows, W has {W.n_cols} columns")
    if Y is None:
        Y = torch.empty((W.n_rows, B), dtype=torch.float32, device=X.device)
    N, By, ldy = _mat(Y, "Y")
    if N != W.n_rows or By != B:
        raise ValueError("Y must be [n_rows][B]")
    ws, wsb = _workspace(workspace_bytes(OP_SPMM, W.n_rows, W.n_cols, nnz, B), X.device, stream)
    _check(lib().csr_spmm_fwd(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals),
                              _p(X), ldx, B, _p(Y), ldy, _p(ws), wsb, _stream(stream)),
           "csr_spmm_fwd")
    return Y


class SpmmPlan:
    """A caller-owned plan of a tiled product (csr_spmm_plan): its device
    buffer and the (n_rows, n_cols, nnz, B) it was made for."""

    def __init__(self, n_rows, n_cols, nnz, B, device):
        self.buf = None
        self.device = device
        self.reshape(n_rows, n_cols, nnz, B)

    def reshape(self, n_rows, n_cols, nnz, B):
        """Take this buffer for another shape, growing it if it is too small
        (the caller orders the reuse after the last use of the old plan)."""
        torch = _torch()
        self.key = (n_rows, n_cols, nnz, B)
        self.nbytes = workspace_bytes(OP_SPMM, n_rows, n_cols, nnz, B)
        if self.nbytes and (self.buf is None or self.buf.numel() < self.nbytes):
            self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=self.device)
        return self


def _plan_args(plan, key):
    if plan.key != key:
        raise ValueError(f"plan made for (n_rows, n_cols, nnz, B) = {plan.key}, used for {key}")
    return _p(plan.buf), plan.nbytes


def csr_spmm_plan(W: CSR, B: int, plan: SpmmPlan | None = None, stream=None) -> SpmmPlan:
    """The planning launches of Y = W . X for a batch of B columns (no X needed)."""
    nnz = W.validate_shapes()
    key = (W.n_rows, W.n_cols, nnz, int(B))
    if plan is None:
        plan = SpmmPlan(*key, W.row_ptr.device)
    pp, pb = _plan_args(plan, key)
    _check(lib().csr_spmm_plan(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), int(B), pp, pb,
                               _stream(stream)), "csr_spmm_plan")
    return plan


def csr_spmm_planned(W: CSR, X, plan: SpmmPlan, Y=None, stream=None):
    """Y = W . X from a plan made by csr_spmm_plan(W, B)."""
    torch = _torch()
    nnz = W.validate_shapes()
    K, B, ldx = _mat(X, "X")
    if K != W.n_cols:
        raise ValueError(f"X has {K} rows, W has {W.n_cols} columns")
    if Y is None:
        Y = torch.empty((W.n_rows, B), dtype=torch.float32, device=X.device)
    N, By, ldy = _mat(Y, "Y")
    if N != W.n_rows or By != B:
        raise ValueError("Y must be [n_rows][B]")
    pp, pb = _plan_args(plan, (W.n_rows, W.n_cols, nnz, B))
    _check(lib().csr_spmm_planned(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), _p(X), ldx, B,
                                  _p(Y), ldy, pp, pb, _stream(stream)), "csr_spmm_planned")
    return Y


def _csc_as_csr(W: CSR, csc: CSC) -> CSR:
    """W^T in CSR form: the CSC copy's arrays (for the planned backward product)."""
    return CSR(W.n_cols, W.n_rows, csc.col_ptr, csc.row_idx, csc.vals_t, W.host_nnz())


def csr_spmm_bwd_t_plan(W: CSR, csc: CSC, B: int, plan: SpmmPlan | None = None, stream=None) -> SpmmPlan:
    """The planning launches of dX = W^T . dY over the CSC copy (needs W's pattern and values only)."""
    return csr_spmm_plan(_csc_as_csr(W, csc), B, plan, stream)


def csr_spmm_bwd_t_planned(W: CSR, dY, csc: CSC, plan: SpmmPlan, dX=None, stream=None):
    """dX = W^T . dY from a plan made by csr_spmm_bwd_t_plan (the same bits as csr_spmm_bwd_t)."""
    return csr_spmm_planned(_csc_as_csr(W, csc), dY, plan, dX, stream)


def csc_build(W: CSR, out: CSC | None = None, bitmap: "Bitmap | None" = None, stream=None) -> CSC:
    """Deterministic CSC copy of W (col_ptr, row_idx, perm, vals_t), built from
    W's bitmap index (given, or built by the call)."""
    nnz = W.validate_shapes()
    dev = W.row_ptr.device
    if out is None:
        out = CSC.empty(W.n_cols, max(nnz, 1), dev)
    ws, wsb = _workspace(workspace_bytes(OP_CSC_BUILD, W.n_rows, W.n_cols, nnz, 0), dev, stream)
    mask = None if bitmap is None else _p(bitmap.mask)
    pos = None if bitmap is None else _p(bitmap.pos)
    _check(lib().csc_build(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), mask, pos,
                           _p(out.col_ptr), _p(out.row_idx), _p(out.perm), _p(out.vals_t), _p(ws),
                           wsb, _stream(stream)), "csc_build")
    return out


def csc_update_vals(W: CSR, csc: CSC, stream=None) -> CSC:
    """vals_t <- vals[perm] after a values-only update of W."""
    nnz = W.validate_shapes()
    _check(lib().csc_update_vals(W.n_cols, nnz, _p(csc.col_ptr), _p(csc.perm), _p(W.vals),
                                 _p(csc.vals_t), _stream(stream)), "csc_update_vals")
    return csc


def csr_spmm_bwd_t(W: CSR, dY, csc: CSC | None = None, dX=None, stream=None):
    """dX = W^T . dY through the CSC copy (deterministic) or, with csc=None, float atomics."""
    torch = _torch()
    nnz = W.validate_shapes()
    N, B, ldy = _mat(dY, "dY")
    if N != W.n_rows:
        raise ValueError("dY must be [n_rows][B]")
    if dX is None:
        dX = torch.empty((W.n_cols, B), dtype=torch.float32, device=dY.device)
    K, Bx, ldx = _mat(dX, "dX")
    if K != W.n_cols or Bx != B:
        raise ValueError("dX must be [n_cols][B]")
    cp = ri = vt = ws = None
    wsb = 0
    if csc is not None:
        cp, ri, vt = csc.col_ptr, csc.row_idx, csc.vals_t
        ws, wsb = _workspace(workspace_bytes(OP_SPMM, W.n_cols, W.n_rows, nnz, B), dY.device, stream)
    _check(lib().csr_spmm_bwd_t(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals),
                                _p(cp), _p(ri), _p(vt), _p(dY), ldy, B, _p(dX), ldx, _p(ws), wsb,
                                _stream(stream)), "csr_spmm_bwd_t")
    return dX


def dense_wgrad(dY, X, dW=None, precision=F32, stream=None):
    """dW = dY . X^T on the matrix cores: fp32 operands (F32); operands
    rounded to bf16 with exact products and fp32 sums (BF16); or operands split
    into bf16 hi + lo with three exact products per pair and fp32 sums (BF16X3,
    inside the fp32 contract)."""
    torch = _torch()
    N, B, ldy = _mat(dY, "dY")
    K, Bx, ldx = _mat(X, "X")
    if Bx != B:
        raise ValueError("dY and X must share the batch dimension")
    if dW is None:
        dW = torch.empty((N, K), dtype=torch.float32, device=dY.device)
    Nw, Kw, ldw = _mat(dW, "dW")
    if (Nw, Kw) != (N, K):
        raise ValueError("dW must be [N][K]")
    ws, wsb = _workspace(workspace_bytes(OP_DENSE_WGRAD, N, K, 0, B), dY.device, stream)
    _check(lib().dense_wgrad(N, K, B, _p(dY), ldy, _p(X), ldx, _p(dW), ldw, int(precision), _p(ws), wsb,
                             _stream(stream)), "dense_wgrad")
    return dW


def sddmm_masked_wgrad(W: CSR, dY, X, gv=None, stream=None):
    """gv[p] = (dY . X^T)[row(p), col(p)] on W's pattern."""
    torch = _torch()
    nnz = W.validate_shapes()
    N, B, ldy = _mat(dY, "dY")
    K, Bx, ldx = _mat(X, "X")
    if N != W.n_rows or K != W.n_cols or Bx != B:
        raise ValueError("shape mismatch")
    if gv is None:
        gv = torch.empty(max(nnz, 1), dtype=torch.float32, device=dY.device)
    ws, wsb = _workspace(workspace_bytes(OP_SDDMM, W.n_rows, W.n_cols, nnz, B), dY.device, stream)
    _check(lib().sddmm_masked_wgrad(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(dY),
                                    ldy, _p(X), ldx, B, _p(gv), _p(ws), wsb, _stream(stream)),
           "sddmm_masked_wgrad")
    return gv


def prox_l1_step(mode, W: CSR, G, eta, lam, Z=None, row_counts=None, stream=None):
    """Eq. (prox).  Dense mode returns Z (may be G itself); CSR mode updates W.vals in place."""
    torch = _torch()
    nnz = W.validate_shapes()
    if mode == PROX_CSR:
        _vec(G, torch.float32, "G")
        if G.numel() < nnz:
            raise ValueError("G must hold one gradient per stored entry")
        _check(lib().prox_l1_step(PROX_CSR, W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx),
                                  _p(W.vals), _p(G), 0, float(eta), float(lam), None, 0, None,
                                  _stream(stream)), "prox_l1_step")
        return W
    N, K, ldg = _mat(G, "G")
    if (N, K) != (W.n_rows, W.n_cols):
        raise ValueError("G must be [n_rows][n_cols]")
    if Z is None:
        Z = torch.empty((N, K), dtype=torch.float32, device=G.device)
    Nz, Kz, ldz = _mat(Z, "Z")
    if (Nz, Kz) != (N, K):
        raise ValueError("Z must be [n_rows][n_cols]")
    if row_counts is not None:
        _vec(row_counts, torch.int32, "row_counts")
    _check(lib().prox_l1_step(PROX_DENSE, W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx),
                              _p(W.vals), _p(G), ldg, float(eta), float(lam), _p(Z), ldz,
                              _p(row_counts), _stream(stream)), "prox_l1_step")
    return Z


def csr_recompress(Z, t=0.0, row_counts=None, capacity=None, out: CSR | None = None, stream=None):
    """Dense Z -> canonical CSR keeping |Z| > t.

    With the default capacity (N*K) the call never waits and the result's
    ``nnz`` is None (read ``row_ptr[-1]``).  With a smaller capacity it waits
    and raises L1CSRError(ECAPACITY) if the result does not fit.
    """
    torch = _torch()
    N, K, ldz = _mat(Z, "Z")
    dev = Z.device
    if out is None:
        cap = N * K if capacity is None else int(capacity)
        out = CSR(N, K, torch.empty(N + 1, dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.float32, device=dev), None)
    cap = min(out.col_idx.numel(), out.vals.numel()) if capacity is None else int(capacity)
    ws, wsb = _workspace(workspace_bytes(OP_RECOMPRESS, N, K, 0, 0), dev, stream)
    need = C.c_int64(-1)
    _check(lib().csr_recompress(N, K, _p(Z), ldz, float(t), _p(row_counts), _p(out.row_ptr),
                                _p(out.col_idx), _p(out.vals), cap, _nnz_dev(out), C.byref(need), _p(ws), wsb,
                                _stream(stream)), "csr_recompress")
    _set_nnz(out, need.value, stream)
    return out


@dataclass
class Bitmap:
    """Bitmap index of a CSR pattern, word-major: mask / pos
    [ceil(n_cols / 32)][n_rows] (csr_bitmap_build)."""
    mask: "object"
    pos: "object"

    @staticmethod
    def empty(n_rows, n_cols, device):
        torch = _torch()
        kw = max((n_cols + 31) // 32, 1)  # word-major: [kw][n_rows]
        return Bitmap(torch.empty((kw, max(n_rows, 1)), dtype=torch.int32, device=device),
                      torch.empty((kw, max(n_rows, 1)), dtype=torch.int32, device=device))


def csr_bitmap_build(W: CSR, bm: Bitmap | None = None, stream=None) -> Bitmap:
    """W's bitmap index for dense_wgrad_prox_recompress (depends on the pattern only)."""
    nnz = W.validate_shapes()
    if bm is None:
        bm = Bitmap.empty(W.n_rows, W.n_cols, W.row_ptr.device)
    kw = (W.n_cols + 31) // 32
    for t_ in (bm.mask, bm.pos):
        if not t_.is_contiguous() or t_.numel() < W.n_rows * kw:
            raise ValueError("bitmap arrays must be contiguous with n_rows * ceil(n_cols / 32) entries")
    _check(lib().csr_bitmap_build(W.n_rows, W.n_cols, nnz, _p(W.row_ptr), _p(W.col_idx), _p(bm.mask),
                                  _p(bm.pos), _stream(stream)), "csr_bitmap_build")
    return bm


def dense_wgrad_prox(W: CSR, dY, X, eta, lam, bitmap: Bitmap, Z=None, word_counts=None, precision=F32,
                     stream=None):
    """Z = S_{eta*lam}(W - eta * dY.X^T) ([N][K], dW never stored) and the
    nonzero count of every 32-column word of Z's rows ([N][ceil(K/32)]), one
    GEMM launch; W read through its bitmap index.  Returns (Z, word_counts)."""
    torch = _torch()
    nnz = W.validate_shapes()
    N, B, ldy = _mat(dY, "dY")
    K, Bx, ldx = _mat(X, "X")
    if (N, K) != (W.n_rows, W.n_cols) or Bx != B:
        raise ValueError("dY must be [N][B] and X [K][B] for an N x K layer")
    dev = dY.device
    if Z is None:
        Z = torch.empty((N, K), dtype=torch.float32, device=dev)
    rz, cz, ldz = _mat(Z, "Z")
    if (rz, cz) != (N, K):
        raise ValueError("Z must be [N][K]")
    kw = (K + 31) // 32
    if word_counts is None:
        word_counts = torch.empty((max(N, 1), max(kw, 1)), dtype=torch.int32, device=dev)
    if not word_counts.is_contiguous() or word_counts.numel() < N * kw:
        raise ValueError("word_counts must be contiguous with N * ceil(K/32) entries")
    ws, wsb = (None, 0)
    if precision == F32:
        ws, wsb = _workspace(workspace_bytes(OP_WGRAD_PROX, N, K, nnz, B), dev, stream)
    _check(lib().dense_wgrad_prox(N, K, B, _p(dY), ldy, _p(X), ldx, int(precision), nnz, _p(W.row_ptr),
                                  _p(W.col_idx), _p(W.vals), _p(bitmap.mask), _p(bitmap.pos), float(eta), float(lam),
                                  _p(Z), ldz, _p(word_counts), _p(ws), wsb, _stream(stream)), "dense_wgrad_prox")
    return Z, word_counts


def csr_recompress_counted(Z, word_counts, out: CSR | None = None, capacity=None, stream=None) -> CSR:
    """Z -> CSR of its nonzeros using dense_wgrad_prox's word counts (Z read once)."""
    torch = _torch()
    N, K, ldz = _mat(Z, "Z")
    dev = Z.device
    if out is None:
        cap = N * K if capacity is None else int(capacity)
        out = CSR(N, K, torch.empty(N + 1, dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.float32, device=dev), None)
    cap = min(out.col_idx.numel(), out.vals.numel()) if capacity is None else int(capacity)
    ws, wsb = _workspace(workspace_bytes(OP_RECOMPRESS, N, K, 0, 0), dev, stream)
    need = C.c_int64(-1)
    _check(lib().csr_recompress_counted(N, K, _p(Z), ldz, _p(word_counts), _p(out.row_ptr), _p(out.col_idx),
                                        _p(out.vals), cap, _nnz_dev(out), C.byref(need), _p(ws), wsb, _stream(stream)),
           "csr_recompress_counted")
    _set_nnz(out, need.value, stream)
    return out


def dense_wgrad_prox_recompress(W: CSR, dY, X, eta, lam, Z=None, out: CSR | None = None,
                                precision=F32, capacity=None, bitmap: Bitmap | None = None, stream=None):
    """The whole l1 update: csr_bitmap_build (unless `bitmap` is given),
    dense_wgrad_prox and csr_recompress_counted, in that order on `stream`.
    Z = S_{eta*lam}(W - eta * dY.X^T) and W' = CSR(Z), bit for bit as
    dense_wgrad + prox_l1_step + csr_recompress.  Returns (Z, out)."""
    if bitmap is None:
        bitmap = csr_bitmap_build(W, stream=stream)
    Z, wc = dense_wgrad_prox(W, dY, X, eta, lam, bitmap, Z=Z, precision=precision, stream=stream)
    out = csr_recompress_counted(Z, wc, out=out, capacity=capacity, stream=stream)
    return Z, out


def prox_l1_recompress_noalloc(W: CSR, G, eta, lam, out: CSR, capacity=None, stream=None):
    """prox_l1_recompress without a workspace: the library's static per-device
    scratch (L1CSR_NOALLOC_SCRATCH_BYTES) serves the call, which allocates
    nothing; `out` must be given.  Calls of it that overlap on one GPU race."""
    nnz = W.validate_shapes()
    N, K, ldg = _mat(G, "G")
    if (N, K) != (W.n_rows, W.n_cols):
        raise ValueError("G must be [n_rows][n_cols]")
    cap = min(out.col_idx.numel(), out.vals.numel()) if capacity is None else int(capacity)
    need = C.c_int64(-1)
    _check(lib().prox_l1_recompress_noalloc(N, K, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), _p(G),
                                            ldg, float(eta), float(lam), _p(out.row_ptr), _p(out.col_idx),
                                            _p(out.vals), cap, _nnz_dev(out), C.byref(need), _stream(stream)),
           "prox_l1_recompress_noalloc")
    _set_nnz(out, need.value, stream)
    return out


def prox_l1_recompress(W: CSR, G, eta, lam, capacity=None, out: CSR | None = None, stream=None):
    """W' = CSR(S_{eta*lam}(W - eta*G)) in one call (same bits as prox + recompress)."""
    torch = _torch()
    nnz = W.validate_shapes()
    N, K, ldg = _mat(G, "G")
    if (N, K) != (W.n_rows, W.n_cols):
        raise ValueError("G must be [n_rows][n_cols]")
    dev = G.device
    if out is None:
        cap = N * K if capacity is None else int(capacity)
        out = CSR(N, K, torch.empty(N + 1, dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.float32, device=dev), None)
    cap = min(out.col_idx.numel(), out.vals.numel()) if capacity is None else int(capacity)
    ws, wsb = _workspace(workspace_bytes(OP_PROX_RECOMPRESS, N, K, nnz, 0), dev, stream)
    need = C.c_int64(-1)
    _check(lib().prox_l1_recompress(N, K, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), _p(G), ldg,
                                    float(eta), float(lam), _p(out.row_ptr), _p(out.col_idx),
                                    _p(out.vals), cap, _nnz_dev(out), C.byref(need), _p(ws), wsb,
                                    _stream(stream)), "prox_l1_recompress")
    _set_nnz(out, need.value, stream)
    return out


@dataclass
class AdaptiveState:
    """Hyper-parameters and per-weight state of Prox-RMSProp / Prox-ADAM
    (Algorithms 1-2).  m (ADAM only) and v are float32 device tensors: [N][K]
    (a leading dimension >= K is allowed) for the dense form, [nnz] for the
    stored-entry form; both start at zero.  t is the step number of the next
    call (from 1); the binding increments it after each call."""
    solver: int
    v: object
    m: object = None
    eps: float = 1e-8
    beta1: float = 0.9
    beta2: float = 0.999
    t: int = 1

    @staticmethod
    def zeros(solver, shape, device, **kw):
        torch = _torch()
        v = torch.zeros(shape, dtype=torch.float32, device=device)
        m = torch.zeros(shape, dtype=torch.float32, device=device) if solver == SOLVER_ADAM else None
        return AdaptiveState(solver, v, m, **kw)


def _state_mat(st: AdaptiveState, N, K):
    n, k, lds = _mat(st.v, "v")
    if (n, k) != (N, K):
        raise ValueError("state v must be [n_rows][n_cols]")
    if st.solver == SOLVER_ADAM:
        if st.m is None:
            raise ValueError("Prox-ADAM needs the first-moment state m")
        nm, km, ldm = _mat(st.m, "m")
        if (nm, km, ldm) != (N, K, lds):
            raise ValueError("m and v must have the same shape and leading dimension")
    return lds


def prox_adaptive_step(mode, W: CSR, G, st: AdaptiveState, eta, lam, Z=None, row_counts=None,
                       stream=None):
    """One Prox-RMSProp / Prox-ADAM step (Algorithms 1-2).  Dense mode returns Z
    (may be G itself) and updates st.m, st.v in place; CSR mode updates W.vals
    and the per-entry state in place.  st.t advances by one."""
    torch = _torch()
    nnz = W.validate_shapes()
    m = st.m if st.solver == SOLVER_ADAM else None
    if mode == PROX_CSR:
        _vec(G, torch.float32, "G")
        _vec(st.v, torch.float32, "v")
        if m is not None:
            _vec(m, torch.float32, "m")
        if G.numel() < nnz or st.v.numel() < nnz or (m is not None and m.numel() < nnz):
            raise ValueError("G and the state must hold one entry per stored weight")
        _check(lib().prox_adaptive_step(PROX_CSR, st.solver, W.n_rows, W.n_cols, nnz, _p(W.row_ptr),
                                        _p(W.col_idx), _p(W.vals), _p(G), 0, _p(m), _p(st.v), 0,
                                        float(eta), float(lam), float(st.eps), float(st.beta1),
                                        float(st.beta2), int(st.t), None, 0, None, None, 0,
                                        _stream(stream)), "prox_adaptive_step")
        st.t += 1
        return W
    N, K, ldg = _mat(G, "G")
    if (N, K) != (W.n_rows, W.n_cols):
        raise ValueError("G must be [n_rows][n_cols]")
    lds = _state_mat(st, N, K)
    if Z is None:
        Z = torch.empty((N, K), dtype=torch.float32, device=G.device)
    Nz, Kz, ldz = _mat(Z, "Z")
    if (Nz, Kz) != (N, K):
        raise ValueError("Z must be [n_rows][n_cols]")
    if row_counts is not None:
        _vec(row_counts, torch.int32, "row_counts")
    ws, wsb = _workspace(workspace_bytes(OP_PROX_RECOMPRESS, N, K, nnz, 0), G.device, stream)
    _check(lib().prox_adaptive_step(PROX_DENSE, st.solver, N, K, nnz, _p(W.row_ptr), _p(W.col_idx),
                                    _p(W.vals), _p(G), ldg, _p(m), _p(st.v), lds, float(eta),
                                    float(lam), float(st.eps), float(st.beta1), float(st.beta2),
                                    int(st.t), _p(Z), ldz, _p(row_counts), _p(ws), wsb,
                                    _stream(stream)), "prox_adaptive_step")
    st.t += 1
    return Z


def prox_adaptive_recompress(W: CSR, G, st: AdaptiveState, eta, lam, capacity=None,
                             out: CSR | None = None, stream=None):
    """W' = CSR of the Prox-RMSProp / Prox-ADAM step over all N*K weights, in
    one call (same bits as prox_adaptive_step + csr_recompress); st.m, st.v are
    updated in place and st.t advances by one (not on a capacity error)."""
    torch = _torch()
    nnz = W.validate_shapes()
    N, K, ldg = _mat(G, "G")
    if (N, K) != (W.n_rows, W.n_cols):
        raise ValueError("G must be [n_rows][n_cols]")
    lds = _state_mat(st, N, K)
    m = st.m if st.solver == SOLVER_ADAM else None
    dev = G.device
    if out is None:
        cap = N * K if capacity is None else int(capacity)
        out = CSR(N, K, torch.empty(N + 1, dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
                  torch.empty(max(cap, 1), dtype=torch.float32, device=dev), None)
    cap = min(out.col_idx.numel(), out.vals.numel()) if capacity is None else int(capacity)
    ws, wsb = _workspace(workspace_bytes(OP_PROX_RECOMPRESS, N, K, nnz, 0), dev, stream)
    need = C.c_int64(-1)
    _check(lib().prox_adaptive_recompress(st.solver, N, K, nnz, _p(W.row_ptr), _p(W.col_idx),
                                          _p(W.vals), _p(G), ldg, _p(m), _p(st.v), lds, float(eta),
                                          float(lam), float(st.eps), float(st.beta1),
                                          float(st.beta2), int(st.t), _p(out.row_ptr),
                                          _p(out.col_idx), _p(out.vals), cap, _nnz_dev(out), C.byref(need),
                                          _p(ws), wsb, _stream(stream)), "prox_adaptive_recompress")
    st.t += 1
    _set_nnz(out, need.value, stream)
    return out


@dataclass
class ConvGeom:
    """Convolution geometry: input channels C, maps H x W, filters KH x KW,
    stride SH x SW, zero padding PH x PW."""
    C: int
    H: int
    W: int
    KH: int
    KW: int
    SH: int = 1
    SW: int = 1
    PH: int = 0
    PW: int = 0

    @property
    def out_hw(self):
        return ((self.H + 2 * self.PH - self.KH) // self.SH + 1,
                (self.W + 2 * self.PW - self.KW) // self.SW + 1)

    @property
    def in_rows(self):
        return self.C * self.H * self.W

    @property
    def filter_cols(self):
        return self.C * self.KH * self.KW

    def _arr(self):
        return (C.c_int32 * 9)(self.C, self.H, self.W, self.KH, self.KW, self.SH, self.SW, self.PH, self.PW)


def csr_conv_fwd(g: ConvGeom, W: CSR, X, Y=None, stream=None):
    """Output maps [n_out*OH*OW][B] of the CSR filter bank W on maps X [C*H*W][B]."""
    torch = _torch()
    nnz = W.validate_shapes()
    rows, B, ldx = _mat(X, "X")
    if rows != g.in_rows or W.n_cols != g.filter_cols:
        raise ValueError("X must be [C*H*W][B] and W must have C*KH*KW columns")
    OH, OW = g.out_hw
    if Y is None:
        Y = torch.empty((W.n_rows * OH * OW, B), dtype=torch.float32, device=X.device)
    ry, by, ldy = _mat(Y, "Y")
    if (ry, by) != (W.n_rows * OH * OW, B):
        raise ValueError("Y must be [n_out*OH*OW][B]")
    _check(lib().csr_conv_fwd(g._arr(), W.n_rows, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), _p(X), ldx,
                              B, _p(Y), ldy, _stream(stream)), "csr_conv_fwd")
    return Y


def csr_conv_bwd_data(g: ConvGeom, n_out: int, csc: CSC, dY, dX=None, nnz=None, stream=None):
    """Input-map gradient [C*H*W][B] from dY [n_out*OH*OW][B] and the CSC copy
    of the filter bank (csc_build of the n_out x C*KH*KW CSR)."""
    torch = _torch()
    rows, B, ldy = _mat(dY, "dY")
    OH, OW = g.out_hw
    if rows != n_out * OH * OW:
        raise ValueError("dY must be [n_out*OH*OW][B]")
    if csc.col_ptr.numel() != g.filter_cols + 1:
        raise ValueError("the CSC must have C*KH*KW columns")
    n = csc.row_idx.numel() if nnz is None else int(nnz)
    if dX is None:
        dX = torch.empty((g.in_rows, B), dtype=torch.float32, device=dY.device)
    rx, bx, ldx = _mat(dX, "dX")
    if (rx, bx) != (g.in_rows, B):
        raise ValueError("dX must be [C*H*W][B]")
    _check(lib().csr_conv_bwd_data(g._arr(), n_out, n, _p(csc.col_ptr), _p(csc.row_idx), _p(csc.vals_t),
                                   _p(dY), ldy, B, _p(dX), ldx, _stream(stream)), "csr_conv_bwd_data")
    return dX


def conv_im2col(g: ConvGeom, X, Xcol=None, stream=None):
    """The lowered operand [C*KH*KW][OH*OW*B] of maps X [C*H*W][B]."""
    torch = _torch()
    rows, B, ldx = _mat(X, "X")
    if rows != g.in_rows:
        raise ValueError("X must be [C*H*W][B]")
    OH, OW = g.out_hw
    if Xcol is None:
        Xcol = torch.empty((g.filter_cols, OH * OW * B), dtype=torch.float32, device=X.device)
    rc, cc, ldc = _mat(Xcol, "Xcol")
    if (rc, cc) != (g.filter_cols, OH * OW * B):
        raise ValueError("Xcol must be [C*KH*KW][OH*OW*B]")
    _check(lib().conv_im2col(g._arr(), _p(X), ldx, B, _p(Xcol), ldc, _stream(stream)), "conv_im2col")
    return Xcol


def maxpool_fwd(g: ConvGeom, X, Y=None, stream=None):
    """Max pooling (KH x KW windows, stride SH x SW, no padding) of [C*H*W][B] maps."""
    torch = _torch()
    rows, B, ldx = _mat(X, "X")
    if rows != g.in_rows:
        raise ValueError("X must be [C*H*W][B]")
    OH, OW = g.out_hw
    if Y is None:
        Y = torch.empty((g.C * OH * OW, B), dtype=torch.float32, device=X.device)
    ry, by, ldy = _mat(Y, "Y")
    if (ry, by) != (g.C * OH * OW, B):
        raise ValueError("Y must be [C*OH*OW][B]")
    _check(lib().l1csr_maxpool_fwd(g._arr(), _p(X), ldx, B, _p(Y), ldy, _stream(stream)), "l1csr_maxpool_fwd")
    return Y


def csr_compact(W: CSR, out: CSR | None = None, stream=None) -> CSR:
    """Copy of W without its stored zeros (out of place)."""
    torch = _torch()
    nnz = W.validate_shapes()
    dev = W.row_ptr.device
    if out is None:
        cap = max(nnz, 1)
        out = CSR(W.n_rows, W.n_cols, torch.empty(W.n_rows + 1, dtype=torch.int32, device=dev),
                  torch.empty(cap, dtype=torch.int32, device=dev),
                  torch.empty(cap, dtype=torch.float32, device=dev), None)
    ws, wsb = _workspace(workspace_bytes(OP_COMPACT, W.n_rows, 0, nnz, 0), dev, stream)
    _check(lib().csr_compact(W.n_rows, nnz, _p(W.row_ptr), _p(W.col_idx), _p(W.vals), _p(out.row_ptr),
                             _p(out.col_idx), _p(out.vals), _nnz_dev(out), _p(ws), wsb, _stream(stream)),
           "csr_compact")
    _set_nnz(out, -1, stream)
    return out


def csr_validate(W: CSR, nnz: int | None = None, stream=None) -> bool:
    """Check on the device that W is a canonical CSR (row_ptr[0] = 0,
    non-decreasing, row_ptr[N] = nnz, columns in range and strictly increasing
    in each row).  Waits for the device status and returns True if well formed."""
    torch = _torch()
    _vec(W.row_ptr, torch.int32, "row_ptr")
    _vec(W.col_idx, torch.int32, "col_idx")
    if W.row_ptr.numel() != W.n_rows + 1:
        raise ValueError("row_ptr must hold n_rows + 1 entries")
    n = W.nnz if nnz is None else int(nnz)
    if n is None:
        n = W.host_nnz()
    if n < 0 or n > W.col_idx.numel():
        raise ValueError("nnz must lie within col_idx")
    status = torch.empty(1, dtype=torch.int32, device=W.row_ptr.device)
    _check(lib().csr_validate(W.n_rows, W.n_cols, n, _p(W.row_ptr), _p(W.col_idx), _p(status),
                              _stream(stream)), "csr_validate")
    return int(status.item()) == OK


def relu_fwd(x, y=None, stream=None):
    torch = _torch()
    _dev(x, torch.float32, "x")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    y = torch.empty_like(x) if y is None else y
    _check(lib().l1csr_relu_fwd(x.numel(), _p(x), _p(y), _stream(stream)), "l1csr_relu_fwd")
    return y


def relu_bwd(x, dy, dx=None, stream=None):
    torch = _torch()
    _dev(x, torch.float32, "x")
    _dev(dy, torch.float32, "dy")
    if not (x.is_contiguous() and dy.is_contiguous()) or x.shape != dy.shape:
        raise ValueError("x and dy must be contiguous and of the same shape")
    dx = torch.empty_like(x) if dx is None else dx
    _check(lib().l1csr_relu_bwd(x.numel(), _p(x), _p(dy), _p(dx), _stream(stream)), "l1csr_relu_bwd")
    return dx


def softmax_xent(logits, labels, dlogits=None, loss=None, stream=None):
    """Mean softmax cross-entropy over batch columns; returns (loss[1], dlogits)."""
    torch = _torch()
    Cn, B, ld = _mat(logits, "logits")
    _vec(labels, torch.int32, "labels")
    if dlogits is None:
        dlogits = torch.empty_like(logits)
    _, _, ldd = _mat(dlogits, "dlogits")
    if ldd != ld:
        raise ValueError("dlogits must share the leading dimension of logits")
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=logits.device)
    ws, wsb = _workspace(workspace_bytes(OP_SOFTMAX_XENT, Cn, 0, 0, B), logits.device, stream)
    _check(lib().l1csr_softmax_xent(Cn, B, _p(logits), ld, _p(labels), _p(dlogits), _p(loss),
                                    _p(ws), wsb, _stream(stream)), "l1csr_softmax_xent")
    return loss, dlogits


# the two-stream l1 step over the entry points above
from .step import l1_step, side_stream  # noqa: E402
