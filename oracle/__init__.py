"""CPU oracle for the l1-compressed CSR training step.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import this
package.  It shares no code with the HIP implementation; it wraps the plain C
definitions in ``l1csr_oracle.c`` (fp64 accumulation, no fused products).

Every function takes and returns numpy arrays in the library's layout:
CSR ``row_ptr`` (int32, N+1), ``col_idx`` (int32), ``vals`` (float32); dense
operands batch-contiguous (``X[K][B]``, ``Y[N][B]``), ``dW``/``Z`` as ``[N][K]``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "l1csr_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no fused multiply-add, OpenMP over rows)."""
    if force or not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC):
        tmp = LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-fopenmp", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def build_sanitized(out_path: str) -> str:
    """The same source built with AddressSanitizer and UndefinedBehaviorSanitizer
    (any report aborts), for the sanitizer run of the oracle's pins."""
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
           "-fopenmp", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", _SRC, "-o", out_path, "-lm"]
    subprocess.run(cmd, check=True)
    return out_path


def lib():
    global _lib
    if _lib is None:
        # ORACLE_LIB names another build of the same source (the sanitizer run)
        path = os.environ.get("ORACLE_LIB") or LIB_PATH
        if path == LIB_PATH and not os.path.exists(LIB_PATH):
            build()
        L = C.CDLL(path)
        i32, i64, f32 = C.c_int32, C.c_int64, C.c_float
        L.orc_spmm_fwd.argtypes = [i32, i32, i32, _i32p, _i32p, _f32p, _f32p, i64, _f32p, i64]
        L.orc_spmm_bwd_t.argtypes = [i32, i32, i32, _i32p, _i32p, _f32p, _f32p, i64, _f32p, i64]
        L.orc_dense_wgrad.argtypes = [i32, i32, i32, _f32p, i64, _f32p, i64, _f32p, i64]
        L.orc_dense_wgrad_bf16.argtypes = [i32, i32, i32, _f32p, i64, _f32p, i64, _f32p, i64]
        L.orc_dense_wgrad_bf16x3.argtypes = [i32, i32, i32, _f32p, i64, _f32p, i64, _f32p, i64]
        L.orc_bf16_round.argtypes = [f32]
        L.orc_bf16_round.restype = f32
        L.orc_sddmm.argtypes = [i32, i32, i32, _i32p, _i32p, _f32p, i64, _f32p, i64, _f32p]
        L.orc_soft_threshold.argtypes = [C.c_double, C.c_double]
        L.orc_soft_threshold.restype = C.c_double
        L.orc_threshold.argtypes = [f32, f32]
        L.orc_threshold.restype = C.c_double
        L.orc_prox_arg.argtypes = [f32, f32, f32]
        L.orc_prox_arg.restype = C.c_double
        L.orc_prox_dense.argtypes = [i32, i32, _i32p, _i32p, _f32p, _f32p, i64, f32, f32,
                                     _f32p, i64, C.c_void_p]
        L.orc_prox_csr.argtypes = [i32, _f32p, _f32p, f32, f32, _f32p]
        L.orc_prox_adaptive_dense.argtypes = [i32, i32, i32, _i32p, _i32p, _f32p, _f32p, i64,
                                              _f32p, _f32p, i64, f32, f32, f32, f32, f32, i64,
                                              _f32p, i64, C.c_void_p]
        L.orc_prox_adaptive_csr.argtypes = [i32, i32, _f32p, _f32p, _f32p, _f32p, f32, f32, f32,
                                            f32, f32, i64, _f32p]
        conv = [i32] * 9
        L.orc_conv_fwd.argtypes = [i32] + conv + [i32, _i32p, _i32p, _f32p, _f32p, i64, _f32p, i64]
        L.orc_conv_bwd_data.argtypes = [i32] + conv + [i32, _i32p, _i32p, _f32p, _f32p, i64, _f32p, i64]
        L.orc_im2col.argtypes = conv + [i32, _f32p, i64, _f32p, i64]
        L.orc_maxpool_fwd.argtypes = [i32] * 7 + [i32, _f32p, i64, _f32p, i64]
        L.orc_recompress.argtypes = [i32, i32, _f32p, i64, f32, _i32p, _i32p, _f32p, i64,
                                     C.POINTER(C.c_int64)]
        L.orc_compact.argtypes = [i32, _i32p, _i32p, _f32p, _i32p, _i32p, _f32p,
                                  C.POINTER(C.c_int64)]
        L.orc_csc.argtypes = [i32, i32, _i32p, _i32p, _f32p, _i32p, _i32p, _i32p, _f32p]
        L.orc_relu_fwd.argtypes = [i64, _f32p, _f32p]
        L.orc_relu_bwd.argtypes = [i64, _f32p, _f32p, _f32p]
        L.orc_softmax_xent.argtypes = [i32, i32, _f32p, i64, _i32p, _f32p,
                                       C.POINTER(C.c_double)]
        L.orc_num_threads.restype = C.c_int
        L.orc_set_num_threads.argtypes = [C.c_int]
        _lib = L
    return _lib


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with status {rc}")


def num_threads() -> int:
    return lib().orc_num_threads()


def set_num_threads(n: int) -> None:
    lib().orc_set_num_threads(int(n))


def _csr(row_ptr, col_idx, vals):
    return _c(row_ptr, np.int32), _c(col_idx, np.int32), _c(vals, np.float32)


def spmm_fwd(row_ptr, col_idx, vals, X, n_cols=None):
    """Y = W.X (forward product)."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    X = _c(X, np.float32)
    N = rp.shape[0] - 1
    K = X.shape[0] if n_cols is None else n_cols
    B = X.shape[1]
    Y = np.empty((N, B), np.float32)
    _check(lib().orc_spmm_fwd(N, K, B, rp, ci, v, X, B, Y, B), "spmm_fwd")
    return Y


def spmm_bwd_t(row_ptr, col_idx, vals, dY, n_cols):
    """dX = W^T.dY (backward product for the data gradient)."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    dY = _c(dY, np.float32)
    N = rp.shape[0] - 1
    B = dY.shape[1]
    dX = np.empty((n_cols, B), np.float32)
    _check(lib().orc_spmm_bwd_t(N, n_cols, B, rp, ci, v, dY, B, dX, B), "spmm_bwd_t")
    return dX


def dense_wgrad(dY, X):
    """dW = dY.X^T (dense weight gradient of the l1 phase)."""
    dY = _c(dY, np.float32)
    X = _c(X, np.float32)
    N, B = dY.shape
    K = X.shape[0]
    dW = np.empty((N, K), np.float32)
    _check(lib().orc_dense_wgrad(N, K, B, dY, B, X, B, dW, K), "dense_wgrad")
    return dW


def bf16_round(x):
    """Each element rounded to bf16 (8 significant bits, nearest even), as float32."""
    x = _c(np.asarray(x, np.float32).reshape(-1), np.float32)
    f = lib().orc_bf16_round
    return np.array([f(float(v)) for v in x], np.float32)


def dense_wgrad_bf16(dY, X):
    """dW = bf16(dY).bf16(X)^T with exact products summed in double."""
    dY = _c(dY, np.float32)
    X = _c(X, np.float32)
    N, B = dY.shape
    K = X.shape[0]
    dW = np.empty((N, K), np.float32)
    _check(lib().orc_dense_wgrad_bf16(N, K, B, dY, B, X, B, dW, K), "dense_wgrad_bf16")
    return dW


def dense_wgrad_bf16x3(dY, X):
    """dW with each operand split into bf16 hi = bf16(x), lo = bf16(x - hi) and
    each product taken as hi hi + hi lo + lo hi, exact products summed in double."""
    dY = _c(dY, np.float32)
    X = _c(X, np.float32)
    N, B = dY.shape
    K = X.shape[0]
    dW = np.empty((N, K), np.float32)
    _check(lib().orc_dense_wgrad_bf16x3(N, K, B, dY, B, X, B, dW, K), "dense_wgrad_bf16x3")
    return dW


def sddmm(row_ptr, col_idx, dY, X):
    """gv[p] = (dY.X^T)[row(p), col(p)] (masked weight gradient of debiasing)."""
    rp = _c(row_ptr, np.int32)
    ci = _c(col_idx, np.int32)
    dY = _c(dY, np.float32)
    X = _c(X, np.float32)
    N = rp.shape[0] - 1
    B = dY.shape[1]
    gv = np.empty(ci.shape[0], np.float32)
    _check(lib().orc_sddmm(N, X.shape[0], B, rp, ci, dY, B, X, B, gv), "sddmm")
    return gv


def soft_threshold(z: float, t: float) -> float:
    return lib().orc_soft_threshold(float(z), float(t))


def threshold(eta: float, lam: float) -> float:
    return lib().orc_threshold(eta, lam)


def prox_dense(row_ptr, col_idx, vals, G, eta, lam, n_cols):
    """Z = S_{eta*lam}(dense(W) - eta*G) as float32, plus per-row nonzero counts."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    G = _c(G, np.float32)
    N = rp.shape[0] - 1
    Z = np.empty((N, n_cols), np.float32)
    cnt = np.empty(N, np.int32)
    _check(lib().orc_prox_dense(N, n_cols, rp, ci, v, G, n_cols, eta, lam, Z, n_cols,
                                cnt.ctypes.data_as(C.c_void_p)), "prox_dense")
    return Z, cnt


def prox_csr(vals, gv, eta, lam):
    """vals' = S_{eta*lam}(vals - eta*gv) on the stored entries only."""
    v = _c(vals, np.float32)
    g = _c(gv, np.float32)
    out = np.empty_like(v)
    _check(lib().orc_prox_csr(v.shape[0], v, g, eta, lam, out), "prox_csr")
    return out


RMSPROP = 1
ADAM = 2


def _state(x, shape):
    """A fresh float32 copy of a solver state (zeros when x is None)."""
    if x is None:
        return np.zeros(shape, np.float32)
    return np.array(x, dtype=np.float32, copy=True, order="C").reshape(shape)


def prox_adaptive_dense(solver, row_ptr, col_idx, vals, G, m, v, eta, lam, eps, beta1, beta2,
                        t, n_cols):
    """One Prox-RMSProp (solver=RMSPROP, Algorithm 1) or Prox-ADAM (solver=ADAM,
    Algorithm 2) step over all N*K weights.  m, v are [N][K] states (None =
    zeros; m is ignored for RMSProp).  Returns (Z, row_counts, m', v') with Z
    the new dense weights; the inputs are not modified."""
    rp, ci, w = _csr(row_ptr, col_idx, vals)
    G = _c(G, np.float32)
    N = rp.shape[0] - 1
    m2 = _state(m, (N, n_cols))
    v2 = _state(v, (N, n_cols))
    Z = np.empty((N, n_cols), np.float32)
    cnt = np.empty(N, np.int32)
    _check(lib().orc_prox_adaptive_dense(int(solver), N, n_cols, rp, ci, w, G, n_cols, m2, v2,
                                         n_cols, eta, lam, eps, beta1, beta2, int(t), Z, n_cols,
                                         cnt.ctypes.data_as(C.c_void_p)), "prox_adaptive_dense")
    return Z, cnt, m2, v2


def prox_adaptive_recompress(solver, row_ptr, col_idx, vals, G, m, v, eta, lam, eps, beta1,
                             beta2, t, n_cols):
    """prox_adaptive_dense followed by recompress: returns ((row_ptr', col_idx',
    vals'), m', v')."""
    Z, _, m2, v2 = prox_adaptive_dense(solver, row_ptr, col_idx, vals, G, m, v, eta, lam, eps,
                                       beta1, beta2, t, n_cols)
    return recompress(Z, 0.0), m2, v2


def prox_adaptive_csr(solver, vals, gv, m, v, eta, lam, eps, beta1, beta2, t):
    """The adaptive step on the stored entries only (state per entry).
    Returns (vals', m', v')."""
    w = _c(vals, np.float32)
    g = _c(gv, np.float32)
    m2 = _state(m, w.shape)
    v2 = _state(v, w.shape)
    out = np.empty_like(w)
    _check(lib().orc_prox_adaptive_csr(int(solver), w.shape[0], w, g, m2, v2, eta, lam, eps,
                                       beta1, beta2, int(t), out), "prox_adaptive_csr")
    return out, m2, v2


def conv_out_size(H, Wd, KH, KW, SH=1, SW=1, PH=0, PW=0):
    """(OH, OW) of a convolution (floor division), as the oracle computes them."""
    return (H + 2 * PH - KH) // SH + 1, (Wd + 2 * PW - KW) // SW + 1


def conv_fwd(row_ptr, col_idx, vals, X, C, H, Wd, KH, KW, SH=1, SW=1, PH=0, PW=0):
    """Direct sparse convolution: X is [C*H*W][B] maps, W an N x (C*KH*KW) CSR
    filter bank; returns the [N*OH*OW][B] output maps."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    X = _c(X, np.float32)
    B = X.shape[1]
    N = rp.shape[0] - 1
    OH, OW = conv_out_size(H, Wd, KH, KW, SH, SW, PH, PW)
    Y = np.empty((N * OH * OW, B), np.float32)
    _check(lib().orc_conv_fwd(N, C, H, Wd, KH, KW, SH, SW, PH, PW, B, rp, ci, v, X, B, Y, B), "conv_fwd")
    return Y


def conv_bwd_data(row_ptr, col_idx, vals, dY, C, H, Wd, KH, KW, SH=1, SW=1, PH=0, PW=0):
    """The adjoint of conv_fwd: [N*OH*OW][B] output gradients -> [C*H*W][B]."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    dY = _c(dY, np.float32)
    B = dY.shape[1]
    N = rp.shape[0] - 1
    dX = np.empty((C * H * Wd, B), np.float32)
    _check(lib().orc_conv_bwd_data(N, C, H, Wd, KH, KW, SH, SW, PH, PW, B, rp, ci, v, dY, B, dX, B),
           "conv_bwd_data")
    return dX


def im2col(X, C, H, Wd, KH, KW, SH=1, SW=1, PH=0, PW=0):
    """The lowered operand: [C*KH*KW][OH*OW*B]."""
    X = _c(X, np.float32)
    B = X.shape[1]
    OH, OW = conv_out_size(H, Wd, KH, KW, SH, SW, PH, PW)
    out = np.empty((C * KH * KW, OH * OW * B), np.float32)
    _check(lib().orc_im2col(C, H, Wd, KH, KW, SH, SW, PH, PW, B, X, B, out, OH * OW * B), "im2col")
    return out


def maxpool_fwd(X, C, H, Wd, KH=2, KW=2, SH=2, SW=2):
    """Max pooling of [C*H*W][B] maps -> [C*OH*OW][B]."""
    X = _c(X, np.float32)
    B = X.shape[1]
    OH, OW = conv_out_size(H, Wd, KH, KW, SH, SW)
    Y = np.empty((C * OH * OW, B), np.float32)
    _check(lib().orc_maxpool_fwd(C, H, Wd, KH, KW, SH, SW, B, X, B, Y, B), "maxpool_fwd")
    return Y


def recompress(Z, t=0.0):
    """Dense Z -> canonical CSR keeping |Z| > t.  Returns (row_ptr, col_idx, vals)."""
    Z = _c(Z, np.float32)
    N, K = Z.shape
    rp = np.empty(N + 1, np.int32)
    nnz = C.c_int64(0)
    cap = int(np.count_nonzero(np.abs(Z) > np.float32(t)))
    ci = np.empty(max(cap, 1), np.int32)
    v = np.empty(max(cap, 1), np.float32)
    _check(lib().orc_recompress(N, K, Z, K, t, rp, ci, v, cap, C.byref(nnz)), "recompress")
    return rp, ci[: nnz.value].copy(), v[: nnz.value].copy()


def csc(row_ptr, col_idx, vals, n_cols):
    """The canonical CSC of an N x n_cols CSR matrix (Section 3.2's column-wise
    copy): (col_ptr, row_idx, perm, vals_t), the entries of each column in
    ascending row order, perm[q] the CSR position of CSC entry q."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    N = rp.shape[0] - 1
    n = ci.shape[0]
    cp = np.empty(n_cols + 1, np.int32)
    ri = np.empty(max(n, 1), np.int32)
    pm = np.empty(max(n, 1), np.int32)
    vt = np.empty(max(n, 1), np.float32)
    _check(lib().orc_csc(N, n_cols, rp, ci, v, cp, ri, pm, vt), "csc")
    return cp, ri[:n].copy(), pm[:n].copy(), vt[:n].copy()


def compact(row_ptr, col_idx, vals):
    """Drop the stored zeros of a CSR matrix."""
    rp, ci, v = _csr(row_ptr, col_idx, vals)
    N = rp.shape[0] - 1
    rpo = np.empty(N + 1, np.int32)
    cio = np.empty(max(ci.shape[0], 1), np.int32)
    vo = np.empty(max(ci.shape[0], 1), np.float32)
    nnz = C.c_int64(0)
    _check(lib().orc_compact(N, rp, ci, v, rpo, cio, vo, C.byref(nnz)), "compact")
    return rpo, cio[: nnz.value].copy(), vo[: nnz.value].copy()


def relu_fwd(x):
    x = _c(x, np.float32)
    y = np.empty_like(x)
    lib().orc_relu_fwd(x.size, x.reshape(-1), y.reshape(-1))
    return y


def relu_bwd(x, dy):
    x = _c(x, np.float32)
    dy = _c(dy, np.float32)
    dx = np.empty_like(x)
    lib().orc_relu_bwd(x.size, x.reshape(-1), dy.reshape(-1), dx.reshape(-1))
    return dx


def softmax_xent(logits, labels):
    """Mean softmax cross-entropy over batch columns; returns (loss, dlogits)."""
    z = _c(logits, np.float32)
    lab = _c(labels, np.int32)
    Cn, B = z.shape
    dz = np.empty_like(z)
    loss = C.c_double(0.0)
    _check(lib().orc_softmax_xent(Cn, B, z, B, lab, dz, C.byref(loss)), "softmax_xent")
    return loss.value, dz


def densify(row_ptr, col_idx, vals, n_cols):
    """Dense [N][K] float32 copy of a CSR matrix (test helper, no arithmetic)."""
    rp = np.asarray(row_ptr)
    N = rp.shape[0] - 1
    D = np.zeros((N, n_cols), np.float32)
    rows = np.repeat(np.arange(N), np.diff(rp))
    D[rows, np.asarray(col_idx)] = np.asarray(vals, np.float32)
    return D
