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
    """The oracle's canonical CSC of a CSR structure: col_ptr, row_idx, perm
    (pinned against scipy's CSR -> CSC conversion in the oracle pins)."""
    import oracle
    ci = np.asarray(col_idx, np.int32)
    cp, ri, pm, _ = oracle.csc(row_ptr, ci, np.zeros(ci.shape[0], np.float32), n_cols)
    return cp, ri, pm
