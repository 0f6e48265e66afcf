"""Shared helpers of the GPU parity tests (no method arithmetic here)."""
import numpy as np

TOL = 1e-4  # fp32 value tolerance, relative to the order-independent scale m


def cuda():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU (run with -m 'not gpu' on a CPU machine)")
    return torch.device("cuda")


def t(a, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    out = torch.from_numpy(a)
    if dtype is not None:
        out = out.to(dtype)
    return out.to(cuda())


def h(x):
    return x.detach().cpu().numpy()


def assert_scaled_close(got, ref, m, tol=TOL, what=""):
    """|got - ref| <= tol * m elementwise, where m = sum |a_k b_k| of each output.

    m is the scale of the rounding error of an fp32 sum in any order; an entry
    with m = 0 is an empty sum and must be exactly 0.
    """
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    m = np.asarray(m, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    err = np.abs(got - ref)
    bad = err > tol * m
    bad |= (m == 0) & (got != 0)
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} entries off; first at {tuple(i)}: "
                             f"got {got[tuple(i)]!r} ref {ref[tuple(i)]!r} m {m[tuple(i)]!r}")


def bits_equal(a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    return a.shape == b.shape and a.dtype == b.dtype and a.tobytes() == b.tobytes()


def csc_reference(row_ptr, col_idx, n_cols):
    """CSC of a CSR structure by a stable sort on (column, row): col_ptr, row_idx, perm."""
    rp = np.asarray(row_ptr, np.int64)
    rows = np.repeat(np.arange(rp.shape[0] - 1), np.diff(rp))
    cols = np.asarray(col_idx, np.int64)
    order = np.lexsort((rows, cols))
    col_ptr = np.zeros(n_cols + 1, np.int64)
    np.cumsum(np.bincount(cols, minlength=n_cols), out=col_ptr[1:])
    return col_ptr.astype(np.int32), rows[order].astype(np.int32), order.astype(np.int32)
