"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: the arrays
the paper prints for its worked example (Fig. 1), the closed form and the
listing form of the soft-threshold (Section 2.2, Fig. 4), library routines
(numpy / scipy dense and sparse products), invariants (adjoint identity), exact
integer brute force on a dyadic grid, and the textbook LASSO solution that the
proximal gradient step (Eq. (prox)) must converge to.
"""
import os

import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from paper_1905_07931_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split(":", 1)
            out[k.strip()] = [int(t) for t in v.split()]
    return out


@pytest.fixture(scope="module")
def fig1():
    g = _read_golden("fig1_csr.txt")
    A = np.array([g[f"A_row{i}"] for i in range(4)], np.float32)
    return A, g


def _dense(L):
    return oracle.densify(L.row_ptr, L.col_idx, L.vals, L.K).astype(np.float64)


def _layers():
    out = []
    for (N, K, B, nnz, seed) in [(1, 1, 1, 1, 0), (7, 5, 3, 12, 1), (64, 65, 63, 700, 2),
                                 (33, 90, 17, 0, 3), (20, 20, 9, 400, 4)]:
        out.append(synth.fc_layer(N, K, B, nnz, seed=seed))
    # forced empty and full rows
    out.append(synth.dyadic_layer(40, 70, 33, 600, seed=5, empty_rows=(0, 3, 39), full_rows=(7,)))
    return out


# --------------------------------------------------------------------------
# Fig. 1: CSR and COO of the worked example
# --------------------------------------------------------------------------

def test_fig1_recompress_matches_printed_csr(fig1):
    A, g = fig1
    rp, ci, v = oracle.recompress(A, 0.0)
    assert rp.tolist() == g["row_ptrs"]
    assert ci.tolist() == g["col_indices"]
    assert v.astype(np.int64).tolist() == g["elements"]
    # COO row array = CSR row pointers expanded (Fig. 1 (iv))
    assert np.repeat(np.arange(4), np.diff(rp)).tolist() == g["coo_row"]


def test_fig1_products_with_identity(fig1):
    A, g = fig1
    rp = np.array(g["row_ptrs"], np.int32)
    ci = np.array(g["col_indices"], np.int32)
    v = np.array(g["elements"], np.float32)
    I4 = np.eye(4, dtype=np.float32)
    # W.I = W and W^T.I = W^T: catches a transposed operand or a wrong index
    assert np.array_equal(oracle.spmm_fwd(rp, ci, v, I4), A)
    assert np.array_equal(oracle.spmm_bwd_t(rp, ci, v, I4, 4), A.T)
    # a hand-computed product: A . [1,2,3,4]^T = [15, 28, 50, 28]
    x = np.array([[1], [2], [3], [4]], np.float32)
    assert oracle.spmm_fwd(rp, ci, v, x)[:, 0].tolist() == [15.0, 28.0, 50.0, 28.0]
    # A^T . [1,2,3,4]^T = [16, 35, 25, 43]
    assert oracle.spmm_bwd_t(rp, ci, v, x, 4)[:, 0].tolist() == [16.0, 35.0, 25.0, 43.0]


# --------------------------------------------------------------------------
# Soft-threshold: closed form (Section 2.2) and Fig. 4's min/max form
# --------------------------------------------------------------------------

@pytest.mark.parametrize("z,t,expect", [
    (2.0, 0.5, 1.5), (-2.0, 0.5, -1.5), (0.3, 0.5, 0.0), (-0.3, 0.5, 0.0),
    (0.5, 0.5, 0.0), (-0.5, 0.5, 0.0), (0.0, 0.5, 0.0), (3.0, 0.0, 3.0),
    (-3.0, 0.0, -3.0), (1e-30, 1e-31, 9e-31),
])
def test_soft_threshold_table(z, t, expect):
    r = oracle.soft_threshold(z, t)
    assert r == pytest.approx(expect, rel=1e-15, abs=0)
    if expect == 0.0:
        assert np.signbit(r) == False  # canonical +0


def test_soft_threshold_equals_fig4_form():
    rng = np.random.default_rng(7)
    z = np.concatenate([rng.standard_normal(20000) * s for s in (1e-6, 1e-3, 1.0, 1e3)])
    z = z.astype(np.float32)
    for eta, lam in [(0.01, 1e-4), (0.5, 0.5), (2.0 ** -7, 2.0 ** -4), (0.01, 0.0)]:
        t = np.float64(np.float32(eta)) * np.float64(np.float32(lam))
        # prox_csr with a zero gradient applies S_t to z itself
        got = oracle.prox_csr(z, np.zeros_like(z), eta, lam)
        zd = z.astype(np.float64)
        fig4 = np.minimum(np.maximum(zd - t, 0.0), zd + t).astype(np.float32)
        assert np.array_equal(got.view(np.uint32), fig4.view(np.uint32))


def test_threshold_is_eta_times_lambda():
    assert oracle.threshold(0.01, 1e-4) == float(np.float32(0.01)) * float(np.float32(1e-4))
    assert oracle.threshold(0.5, 0.25) == 0.125


def test_prox_lambda_zero_is_sgd():
    rng = np.random.default_rng(3)
    w = rng.standard_normal(5000).astype(np.float32)
    g = rng.standard_normal(5000).astype(np.float32)
    got = oracle.prox_csr(w, g, 0.01, 0.0)
    ref = (w.astype(np.float64) - np.float64(np.float32(0.01)) * g.astype(np.float64)).astype(np.float32)
    assert np.array_equal(got, ref)


def test_prox_dense_off_pattern_small_gradient_stays_zero():
    # w = 0 and |g| <= lam  =>  |eta*g| <= eta*lam  =>  S_t(-eta*g) = 0
    L = synth.fc_layer(30, 40, 8, 200, seed=11)
    rng = np.random.default_rng(11)
    G = (rng.random((30, 40)) * 2 - 1).astype(np.float32) * np.float32(1e-4)
    Z, cnt = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, G, 0.01, 1e-4, 40)
    D = _dense(L)
    assert np.all(Z[D == 0] == 0)
    # stored weights move by -eta*g then shrink by t: check against the formula by hand
    on = D != 0
    z = D[on] - np.float64(np.float32(0.01)) * G[on].astype(np.float64)
    t = np.float64(np.float32(0.01)) * np.float64(np.float32(1e-4))
    ref = (np.sign(z) * np.maximum(np.abs(z) - t, 0.0)).astype(np.float32)
    assert np.array_equal(Z[on], ref)
    assert cnt.tolist() == np.count_nonzero(Z, axis=1).tolist()


def test_prox_large_threshold_empties_matrix():
    L = synth.fc_layer(12, 9, 4, 50, seed=2)
    G = np.ones((12, 9), np.float32)
    Z, cnt = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, G, 1.0, 100.0, 9)
    assert not Z.any() and not np.signbit(Z).any() and cnt.sum() == 0
    rp, ci, v = oracle.recompress(Z)
    assert rp.tolist() == [0] * 13 and ci.size == 0


# --------------------------------------------------------------------------
# Products against library routines, the adjoint identity and brute force
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L", _layers(), ids=lambda L: f"{L.N}x{L.K}b{L.B}nnz{L.nnz}")
def test_spmm_fwd_matches_dense_and_scipy(L):
    Y = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    ref = _dense(L) @ L.X.astype(np.float64)
    m = np.abs(_dense(L)) @ np.abs(L.X.astype(np.float64))
    assert np.all(np.abs(Y - ref) <= 1e-7 * m + 1e-30)
    S = sp.csr_matrix((L.vals, L.col_idx, L.row_ptr), shape=(L.N, L.K))
    ref2 = S.astype(np.float64) @ L.X.astype(np.float64)
    assert np.all(np.abs(Y - ref2) <= 1e-7 * m + 1e-30)


@pytest.mark.parametrize("L", _layers(), ids=lambda L: f"{L.N}x{L.K}b{L.B}nnz{L.nnz}")
def test_spmm_bwd_matches_transpose_and_adjoint(L):
    dX = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)
    D = _dense(L)
    ref = D.T @ L.dY.astype(np.float64)
    m = np.abs(D.T) @ np.abs(L.dY.astype(np.float64))
    assert np.all(np.abs(dX - ref) <= 1e-7 * m + 1e-30)
    # the backward product is the forward product of the transposed CSR
    St = sp.csr_matrix((L.vals, L.col_idx, L.row_ptr), shape=(L.N, L.K)).T.tocsr()
    St.sort_indices()
    dX2 = oracle.spmm_fwd(St.indptr.astype(np.int32), St.indices.astype(np.int32),
                          St.data.astype(np.float32), L.dY)
    assert np.array_equal(dX, dX2)
    # <dY, W X> = <W^T dY, X>
    Y = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    lhs = np.sum(L.dY.astype(np.float64) * Y)
    rhs = np.sum(dX.astype(np.float64) * L.X)
    scale = np.sum(np.abs(L.dY) @ np.abs(L.X.T.astype(np.float64)) * np.abs(D)) + 1e-30
    assert abs(lhs - rhs) <= 1e-6 * scale


@pytest.mark.parametrize("L", _layers(), ids=lambda L: f"{L.N}x{L.K}b{L.B}nnz{L.nnz}")
def test_dense_wgrad_and_sddmm(L):
    dW = oracle.dense_wgrad(L.dY, L.X)
    ref = L.dY.astype(np.float64) @ L.X.T.astype(np.float64)
    m = np.abs(L.dY.astype(np.float64)) @ np.abs(L.X.T.astype(np.float64))
    assert dW.shape == (L.N, L.K)
    assert np.all(np.abs(dW - ref) <= 1e-7 * m + 1e-30)
    gv = oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X)
    rows = np.repeat(np.arange(L.N), np.diff(L.row_ptr))
    assert np.array_equal(gv, dW[rows, L.col_idx])


def test_dense_wgrad_batch_one_is_exact_outer_product():
    rng = np.random.default_rng(5)
    dy = rng.standard_normal((37, 1)).astype(np.float32)
    x = rng.standard_normal((53, 1)).astype(np.float32)
    dW = oracle.dense_wgrad(dy, x)
    assert np.array_equal(dW, dy * x.T)  # float32 products are correctly rounded


def test_bf16_rounding_closed_forms():
    # bf16 keeps 8 significant bits; the IEEE rule is round to nearest, ties to
    # the even kept last bit.  Each case is fixed by that definition alone.
    cases = [
        (1 + 2 ** -8, 1.0),                  # halfway, kept last bit 0 -> down
        (1 + 2 ** -7 + 2 ** -8, 1 + 2 ** -6),  # halfway, kept last bit 1 -> up to even
        (1 + 2 ** -8 + 2 ** -20, 1 + 2 ** -7),  # just above halfway -> up
        (1 + 2 ** -8 - 2 ** -20, 1.0),        # just below halfway -> down
        (-(1 + 2 ** -8), -1.0),               # symmetric in the sign
        (2 - 2 ** -9, 2.0),                   # carries into the next binade
        (3.0, 3.0), (0.0, 0.0), (-0.5, -0.5),
        (0.1, 205 * 2.0 ** -11),              # 0x3DCCCCCD -> 0x3DCD = (1 + 77/128) 2^-4
    ]
    got = oracle.bf16_round(np.array([c[0] for c in cases], np.float32))
    for (x, want), g in zip(cases, got):
        assert float(g) == want, (x, float(g), want)
    # every output has at most 8 significant bits and lies within half a bf16
    # ulp (2^-8 relative) of its input
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    r = oracle.bf16_round(x)
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    assert np.all(np.abs(r.astype(np.float64) - x) <= 2.0 ** -8 * np.abs(x.astype(np.float64)))


def test_dense_wgrad_bf16_pins():
    rng = np.random.default_rng(11)
    # operands already on the bf16 grid: the same numbers as the fp32 definition
    dY = oracle.bf16_round(rng.standard_normal(37 * 19)).reshape(37, 19)
    X = oracle.bf16_round(rng.random(23 * 19)).reshape(23, 19)
    assert np.array_equal(oracle.dense_wgrad_bf16(dY, X), oracle.dense_wgrad(dY, X))
    # B = 1: one product of the rounded operands, exact in float32
    dy = rng.standard_normal((29, 1)).astype(np.float32)
    x = rng.standard_normal((31, 1)).astype(np.float32)
    want = oracle.bf16_round(dy).reshape(29, 1) * oracle.bf16_round(x).reshape(1, 31)
    assert np.array_equal(oracle.dense_wgrad_bf16(dy, x), want)
    # within the rounding bound of the fp32 result: each operand moves by at most
    # 2^-8 relative, so |d(ab)| <= (2^-7 + 2^-16)|ab|
    dY = rng.standard_normal((40, 300)).astype(np.float32)
    X = rng.random((50, 300)).astype(np.float32)
    m = np.abs(dY.astype(np.float64)) @ np.abs(X.T.astype(np.float64))
    d = np.abs(oracle.dense_wgrad_bf16(dY, X).astype(np.float64) - oracle.dense_wgrad(dY, X))
    assert np.all(d <= (2.0 ** -7 + 2.0 ** -16) * m + 2.0 ** -23 * m)
    assert np.max(d / m) > 2.0 ** -14  # and the rounding does show


def _bf16_bits(x):
    """bf16 rounding by integer arithmetic on the float32 bit pattern (add half
    an ulp of the 16 dropped bits, plus the kept lsb for ties to even, then
    truncate): independent of the oracle's frexp-based definition."""
    u = np.asarray(x, np.float32).reshape(-1).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return r.astype(np.uint32).view(np.float32)


def test_bf16_rounding_matches_bit_arithmetic():
    rng = np.random.default_rng(21)
    x = (rng.standard_normal(4000) * np.exp2(rng.integers(-60, 60, 4000))).astype(np.float32)
    # exact ties: the 16 dropped bits are 0x8000, kept lsb even and odd
    t = rng.integers(0x3F000000, 0x4F000000, 400, dtype=np.uint64) & 0xFFFF0000
    ties = np.concatenate([(t | 0x8000), (t | 0x18000)]).astype(np.uint32).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    assert np.array_equal(oracle.bf16_round(x), _bf16_bits(x))


def test_dense_wgrad_bf16x3_pins():
    rng = np.random.default_rng(12)
    # the split: hi + lo is within 2^-16 |x| of x, both parts on the bf16 grid
    x = rng.standard_normal(3000).astype(np.float32)
    hi = _bf16_bits(x)
    lo = _bf16_bits(x - hi)
    assert np.all(np.abs(x.astype(np.float64) - hi - lo) <= 2.0 ** -16 * np.abs(x))
    assert np.array_equal(_bf16_bits(lo), lo)
    # B = 1: hi hi + hi lo + lo hi of the independently split operands, exact in
    # double, rounded once
    dy = rng.standard_normal((29, 1)).astype(np.float32)
    xx = rng.standard_normal((31, 1)).astype(np.float32)
    ha, hb = _bf16_bits(dy).astype(np.float64), _bf16_bits(xx).astype(np.float64)
    la = _bf16_bits(dy.reshape(-1) - ha.astype(np.float32)).astype(np.float64)
    lb = _bf16_bits(xx.reshape(-1) - hb.astype(np.float32)).astype(np.float64)
    want = (np.outer(ha, hb) + np.outer(ha, lb) + np.outer(la, hb)).astype(np.float32)
    assert np.array_equal(oracle.dense_wgrad_bf16x3(dy, xx), want)
    # the lo lo term is dropped: x = 1 + 2^-8 + 2^-9 splits into hi = 1 + 2^-7,
    # lo = -2^-9, so x x comes out 2^-18 short (visible in float32 at 1)
    v = np.array([[1.0 + 2.0 ** -8 + 2.0 ** -9]], np.float32)
    got = float(oracle.dense_wgrad_bf16x3(v, v)[0, 0])
    assert got == float(np.float32(float(v[0, 0]) ** 2 - 2.0 ** -18)) and got != float(np.float32(float(v[0, 0]) ** 2))
    # operands on the bf16 grid: lo = 0, the fp32 definition itself
    dY = oracle.bf16_round(rng.standard_normal(37 * 19)).reshape(37, 19)
    X = oracle.bf16_round(rng.random(23 * 19)).reshape(23, 19)
    assert np.array_equal(oracle.dense_wgrad_bf16x3(dY, X), oracle.dense_wgrad(dY, X))
    # within 3 (1 + 2^-7) 2^-16 of sum |dY X| of the exact product (plus the two
    # float32 output roundings), and the dropped terms do show
    dY = rng.standard_normal((40, 300)).astype(np.float32)
    X = rng.random((50, 300)).astype(np.float32)
    m = np.abs(dY.astype(np.float64)) @ np.abs(X.T.astype(np.float64))
    d = np.abs(oracle.dense_wgrad_bf16x3(dY, X).astype(np.float64) - oracle.dense_wgrad(dY, X))
    assert np.all(d <= 3 * (1 + 2.0 ** -7) * 2.0 ** -16 * m + 2.0 ** -23 * m)
    assert np.max(d / m) > 2.0 ** -22


def test_dyadic_exact_integer_brute_force():
    L = synth.dyadic_layer(23, 41, 19, 300, seed=9, empty_rows=(2,), full_rows=(5,))
    Wi = np.rint(_dense(L) * 16).astype(np.int64)
    Xi = np.rint(L.X.astype(np.float64) * 16).astype(np.int64)
    Di = np.rint(L.dY.astype(np.float64) * 16).astype(np.int64)
    Y = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    assert np.array_equal(np.rint(Y.astype(np.float64) * 256).astype(np.int64), Wi @ Xi)
    dX = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)
    assert np.array_equal(np.rint(dX.astype(np.float64) * 256).astype(np.int64), Wi.T @ Di)
    dW = oracle.dense_wgrad(L.dY, L.X)
    assert np.array_equal(np.rint(dW.astype(np.float64) * 256).astype(np.int64), Di @ Xi.T)


# --------------------------------------------------------------------------
# Dense -> CSR
# --------------------------------------------------------------------------

def test_recompress_structure_cases():
    rng = np.random.default_rng(1)
    Z = rng.standard_normal((9, 13)).astype(np.float32)
    Z[rng.random((9, 13)) < 0.6] = 0
    Z[3, :] = 0
    Z[4, :] = 1
    Z[0, 5] = -0.0
    rp, ci, v = oracle.recompress(Z)
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0)
    assert np.diff(rp).tolist() == np.count_nonzero(Z, axis=1).tolist()
    for i in range(9):
        seg = ci[rp[i]:rp[i + 1]]
        assert np.all(np.diff(seg) > 0)
        assert np.array_equal(v[rp[i]:rp[i + 1]], Z[i, seg])
    assert np.array_equal(oracle.densify(rp, ci, v, 13), Z + 0.0)
    # threshold t keeps |Z| > t only
    rp2, ci2, v2 = oracle.recompress(Z, 0.5)
    assert rp2[-1] == np.count_nonzero(np.abs(Z) > 0.5)
    # all zero and all dense
    assert oracle.recompress(np.zeros((3, 4), np.float32))[0].tolist() == [0, 0, 0, 0]
    rp3, ci3, _ = oracle.recompress(np.ones((3, 4), np.float32))
    assert rp3.tolist() == [0, 4, 8, 12] and ci3.tolist() == [0, 1, 2, 3] * 3


def test_compact_drops_stored_zeros():
    rp = np.array([0, 3, 3, 5], np.int32)
    ci = np.array([0, 2, 4, 1, 3], np.int32)
    v = np.array([1.0, 0.0, -2.0, -0.0, 5.0], np.float32)
    rpo, cio, vo = oracle.compact(rp, ci, v)
    assert rpo.tolist() == [0, 2, 2, 3] and cio.tolist() == [0, 4, 3] and vo.tolist() == [1, -2, 5]


# --------------------------------------------------------------------------
# CSC: the column-wise copy the backward product reads (Section 3.2)
# --------------------------------------------------------------------------

def _csc_layers():
    out = _layers()
    rng = np.random.default_rng(6)
    rp, ci = synth.zipf_pattern(rng, 300, 257, 9000, 1.1)  # power-law rows, some full
    out.append(synth.Layer(300, 257, 1, rp, ci, rng.standard_normal(ci.shape[0]).astype(np.float32),
                           np.zeros((257, 1), np.float32), np.zeros((300, 1), np.float32), 0.0, 0.0, "zipf"))
    return out


@pytest.mark.parametrize("L", _csc_layers(), ids=lambda L: f"N{L.N}K{L.K}nnz{L.col_idx.shape[0]}")
def test_csc_matches_scipy_and_transposes_back(L):
    cp, ri, pm, vt = oracle.csc(L.row_ptr, L.col_idx, L.vals, L.K)
    n = L.col_idx.shape[0]
    # scipy's CSR -> CSC conversion (sorted indices) is the canonical CSC
    A = sp.csr_matrix((np.arange(1, n + 1, dtype=np.int64), L.col_idx, L.row_ptr), shape=(L.N, L.K)).tocsc()
    A.sort_indices()
    assert cp.tolist() == A.indptr.tolist()
    assert ri.tolist() == A.indices.tolist()
    assert (pm + 1).tolist() == A.data.tolist()  # the data carried the CSR positions
    # perm is a bijection onto the CSR positions, and every field follows it
    assert sorted(pm.tolist()) == list(range(n))
    rows = np.repeat(np.arange(L.N), np.diff(L.row_ptr))
    assert np.array_equal(ri, rows[pm]) and np.array_equal(L.col_idx[pm], np.repeat(np.arange(L.K), np.diff(cp)))
    assert np.array_equal(vt.view(np.int32), L.vals[pm].view(np.int32))
    # the CSC read as the CSR of W^T, transposed once more, gives W back
    cp2, ri2, pm2, vt2 = oracle.csc(cp, ri, vt, L.N)
    assert np.array_equal(cp2, L.row_ptr) and np.array_equal(ri2, L.col_idx)
    assert np.array_equal(vt2.view(np.int32), L.vals.view(np.int32))
    assert np.array_equal(oracle.densify(cp, ri, vt, L.N), _dense(L).T.astype(np.float32))


def test_csc_of_fig1(fig1):
    # the worked example's matrix, column by column: rows in ascending order
    A, g = fig1
    rp, ci, v = oracle.recompress(A)
    cp, ri, pm, vt = oracle.csc(rp, ci, v, A.shape[1])
    for k in range(A.shape[1]):
        rows = ri[cp[k]:cp[k + 1]]
        assert rows.tolist() == np.flatnonzero(A[:, k]).tolist()
        assert vt[cp[k]:cp[k + 1]].tolist() == A[rows, k].tolist()


# --------------------------------------------------------------------------
# The proximal gradient step converges to the textbook LASSO solution
# --------------------------------------------------------------------------

def test_prox_gradient_converges_to_lasso_closed_form():
    # One output row, squared loss 0.5*||W X - T||^2 with orthonormal rows of X
    # (X X^T = I): the minimiser of loss + lam*||w||_1 is S_lam(T X^T).
    K, B = 24, 64
    rng = np.random.default_rng(4)
    Q, _ = np.linalg.qr(rng.standard_normal((B, K)))
    X = Q.T.astype(np.float32)                       # [K][B], rows orthonormal
    T = rng.standard_normal((1, B)).astype(np.float32)
    lam, eta = 0.3, 0.5
    rp = np.array([0, 0], np.int32)
    ci = np.zeros(0, np.int32)
    v = np.zeros(0, np.float32)
    for _ in range(80):
        Y = oracle.spmm_fwd(rp, ci, v, X)
        dW = oracle.dense_wgrad(Y - T, X)
        Z, _ = oracle.prox_dense(rp, ci, v, dW, eta, lam, K)
        rp, ci, v = oracle.recompress(Z)
    w = oracle.densify(rp, ci, v, K)[0].astype(np.float64)
    ols = (T.astype(np.float64) @ X.T.astype(np.float64))[0]
    lasso = np.sign(ols) * np.maximum(np.abs(ols) - lam, 0.0)
    assert np.max(np.abs(w - lasso)) < 1e-5
    assert 0 < np.count_nonzero(lasso) < K           # the case is really sparse
    assert np.array_equal(w != 0, lasso != 0)


# --------------------------------------------------------------------------
# Layer glue (ReLU, softmax cross-entropy)
# --------------------------------------------------------------------------

def test_relu():
    x = np.array([-1.0, 0.0, -0.0, 2.5, 1e-40], np.float32)
    y = oracle.relu_fwd(x)
    assert y.tolist() == [0.0, 0.0, 0.0, 2.5, np.float32(1e-40)] and not np.signbit(y).any()
    dx = oracle.relu_bwd(x, np.full(5, 3.0, np.float32))
    assert dx.tolist() == [0.0, 0.0, 0.0, 3.0, 3.0]


def test_softmax_xent_uniform_and_finite_difference():
    C, B = 10, 6
    lab = np.arange(B, dtype=np.int32) % C
    loss, dz = oracle.softmax_xent(np.zeros((C, B), np.float32), lab)
    assert loss == pytest.approx(np.log(10.0), rel=1e-12)
    onehot = np.zeros((C, B))
    onehot[lab, np.arange(B)] = 1
    assert np.allclose(dz, (0.1 - onehot) / B, atol=1e-8)
    rng = np.random.default_rng(0)
    z = rng.standard_normal((C, B)).astype(np.float32) * 3
    loss, dz = oracle.softmax_xent(z, lab)
    assert np.allclose(dz.sum(axis=0), 0, atol=1e-7)
    h = 1e-2
    for (c, b) in [(0, 0), (3, 2), (9, 5), (lab[4], 4)]:
        zp = z.copy(); zp[c, b] += h
        zm = z.copy(); zm[c, b] -= h
        fd = (oracle.softmax_xent(zp, lab)[0] - oracle.softmax_xent(zm, lab)[0]) / (2 * h)
        assert fd == pytest.approx(dz[c, b], rel=2e-3, abs=2e-6)
    # shift invariance of the column softmax
    l2, dz2 = oracle.softmax_xent(z + 7.0, lab)
    assert l2 == pytest.approx(loss, rel=1e-6) and np.allclose(dz2, dz, atol=1e-7)
