"""Each ABI call on the GPU against the CPU oracle, on the same seeded inputs.

Bar: bit-exact for structure (row pointers, column indices, CSC, masks, prox
outputs, recompression) and for any sum on the dyadic grid; within 1e-4 of
the order-independent scale m = sum |a_k b_k| for fp32 sums of real data.
"""
import numpy as np
import pytest

import oracle
import paper_1905_07931_amd as L1
from paper_1905_07931_amd import synth

from _helpers import TOL, assert_scaled_close, bits_equal, csc_reference, cuda, h, t

pytestmark = pytest.mark.gpu

SHAPES = [  # (N, K, B, nnz, seed)
    (1, 1, 1, 1, 0), (7, 5, 3, 12, 1), (64, 65, 63, 700, 2), (65, 64, 64, 2000, 3),
    (33, 90, 17, 0, 4), (300, 784, 64, 23520, 0), (130, 257, 65, 9000, 5), (40, 300, 256, 5000, 6),
    (16, 20, 1, 120, 7), (3, 4100, 129, 6000, 8),
    (51, 500, 130, 2550, 9),          # conv2-like rows (mean 50), VEC 2, the last row block one row
]


def _ids(s):
    return "N{}K{}B{}nnz{}".format(*s[:4])


def _layer(shape):
    N, K, B, nnz, seed = shape
    return synth.fc_layer(N, K, B, nnz, seed=seed)


def _W(L):
    return L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())


def _absL(L):
    return np.abs(L.vals), np.abs(L.X), np.abs(L.dY)


# ----------------------------------------------------------------------------
# forward product
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
def test_spmm_fwd(shape):
    L = _layer(shape)
    Y = h(L1.csr_spmm_fwd(_W(L), t(L.X)))
    ref = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    av, ax, _ = _absL(L)
    m = oracle.spmm_fwd(L.row_ptr, L.col_idx, av, ax)
    assert_scaled_close(Y, ref, m, what="Y")


# Shapes that drive the LDS-tiled kernel through each vector width (the width
# follows from the batch: 64*VEC columns per workgroup), several X tiles, a
# ragged batch tail, ragged row blocks and both rows-per-wave plans.  The tiled
# kernel is chosen from nnz*B >= 1.7e8 products on (smaller products take the
# rows kernel, covered by SHAPES).
TILED = [  # (N, K, B, nnz, seed)
    (300, 784, 64, 23520, 20),        # B < 128: the rows kernel, VEC 1
    (8000, 1000, 128, 1400000, 21),   # VEC 2
    (4096, 300, 1024, 200000, 22),    # VEC 4
    (4096, 300, 1020, 200000, 23),    # VEC 4, ragged last batch chunk
    (9000, 333, 1024, 200000, 24),    # VEC 4, ragged tile and row block
    (60000, 300, 256, 900000, 28),    # 6000 waves: the stream offsets come from a scan launch
]


@pytest.mark.parametrize("shape", TILED, ids=_ids)
def test_spmm_fwd_tiled_widths(shape):
    L = _layer(shape)
    Y = h(L1.csr_spmm_fwd(_W(L), t(L.X)))
    ref = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    m = oracle.spmm_fwd(L.row_ptr, L.col_idx, np.abs(L.vals), L.X)
    assert_scaled_close(Y, ref, m, what="Y")


@pytest.mark.parametrize("shape", [(300, 4096, 1024, 200000, 25), (64, 8192, 1024, 200000, 26)],
                         ids=_ids)
def test_spmm_bwd_tiled_widths(shape):
    L = _layer(shape)
    W = _W(L)
    dX = h(L1.csr_spmm_bwd_t(W, t(L.dY), L1.csc_build(W)))
    ref = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)
    m = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, np.abs(L.vals), np.abs(L.dY), L.K)
    assert_scaled_close(dX, ref, m, what="dX")


def test_spmm_power_law_rows_dyadic_bit_exact():
    # Zipf row lengths (a few full rows, many short ones) through the tiled
    # kernel on the dyadic grid: every sum is exact, so the bits must match
    import numpy as np_
    rng = np_.random.default_rng(27)
    N, K, B = 4096, 512, 512
    rp, ci = synth.zipf_pattern(rng, N, K, 400000, 1.1)
    vals = (rng.integers(1, 17, ci.shape[0]) * rng.choice([-1.0, 1.0], ci.shape[0]) / 16).astype(np_.float32)
    X = (rng.integers(0, 17, (K, B)) / 16).astype(np_.float32)
    W = L1.CSR.from_host(rp, ci, vals, K, device=cuda())
    assert bits_equal(h(L1.csr_spmm_fwd(W, t(X))), oracle.spmm_fwd(rp, ci, vals, X))


@pytest.mark.parametrize("case", ["zipf_steep", "mostly_empty_rows"])
def test_spmm_tiled_skewed_patterns_both_directions(case):
    # the planner's pieces, deal and bucketing on skewed patterns: a steep
    # power law (a few rows split into many strided pieces, most rows short)
    # and a layer whose rows are three quarters empty, through the tiled
    # kernel forward and backward, against the oracle
    rng = np.random.default_rng(29 if case == "zipf_steep" else 30)
    if case == "zipf_steep":
        N, K, B = 4096, 2048, 512
        rp, ci = synth.zipf_pattern(rng, N, K, 400000, 1.5)
    else:
        N, K, B = 8192, 1000, 1024
        dense = rng.random((N, K)) < 0.15
        dense[rng.random(N) < 0.75] = False
        rp, ci = synth.pattern_from_positions(N, K, np.flatnonzero(dense.reshape(-1)))
    vals = rng.standard_normal(ci.shape[0]).astype(np.float32)
    X = rng.random((K, B), dtype=np.float32)
    dY = rng.standard_normal((N, B)).astype(np.float32)
    assert L1.workspace_bytes(L1.OP_SPMM, N, K, len(ci), B) > 0  # the tiled path
    W = L1.CSR.from_host(rp, ci, vals, K, device=cuda())
    Y = h(L1.csr_spmm_fwd(W, t(X)))
    assert_scaled_close(Y, oracle.spmm_fwd(rp, ci, vals, X), oracle.spmm_fwd(rp, ci, np.abs(vals), X), what="Y")
    dX = h(L1.csr_spmm_bwd_t(W, t(dY), L1.csc_build(W)))
    assert_scaled_close(dX, oracle.spmm_bwd_t(rp, ci, vals, dY, K),
                        oracle.spmm_bwd_t(rp, ci, np.abs(vals), np.abs(dY), K), what="dX")


# The tiled product split into its planning launches and the product from
# the plan: the same bits as the one-call form, forward and backward, on the
# half-wave, full-wave and VEC-2 plans and a shape with no plan; the plan is
# made before the dense operand is written.
PLANNED = [  # (N, K, B, nnz, seed)
    (4096, 300, 1024, 200000, 70),    # VEC 4 half-wave (forward), full-wave (backward over 300 CSC rows)
    (8000, 1000, 128, 1400000, 71),   # VEC 2
    (9000, 333, 1020, 200000, 72),    # ragged tile, row block and batch chunk
    (300, 784, 64, 23520, 73),        # no tiled plan: the rows kernel
]


@pytest.mark.parametrize("shape", PLANNED, ids=_ids)
def test_planned_product_equals_one_call(shape):
    import torch
    L = _layer(shape)
    W = _W(L)
    csc = L1.csc_build(W)
    X = torch.empty((L.K, L.B), dtype=torch.float32, device=cuda())
    dY = torch.empty((L.N, L.B), dtype=torch.float32, device=cuda())
    pf = L1.csr_spmm_plan(W, L.B)           # before X and dY hold anything
    pb = L1.csr_spmm_bwd_t_plan(W, csc, L.B)
    X.copy_(t(L.X))
    dY.copy_(t(L.dY))
    Yp = h(L1.csr_spmm_planned(W, X, pf))
    dXp = h(L1.csr_spmm_bwd_t_planned(W, dY, csc, pb))
    assert bits_equal(Yp, h(L1.csr_spmm_fwd(W, X)))
    assert bits_equal(dXp, h(L1.csr_spmm_bwd_t(W, dY, csc)))
    ref = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    assert_scaled_close(Yp, ref, oracle.spmm_fwd(L.row_ptr, L.col_idx, np.abs(L.vals), np.abs(L.X)), what="Y")
    # operands the tiled kernel cannot take (ld not a multiple of 4): the plan
    # is ignored and the rows kernel gives the one-call result
    if L.B % 4 == 0:
        Xs = torch.zeros((L.K, L.B + 1), dtype=torch.float32, device=cuda())
        Xs[:, :L.B] = X
        Xv = Xs[:, :L.B]
        assert bits_equal(h(L1.csr_spmm_planned(W, Xv, pf)), h(L1.csr_spmm_fwd(W, Xv)))


def test_plan_is_checked_against_its_shape():
    L = _layer((4096, 300, 1024, 200000, 74))
    W = _W(L)
    p = L1.csr_spmm_plan(W, 1024)
    with pytest.raises(ValueError):
        L1.csr_spmm_planned(W, t(L.X[:, :512]), p)  # made for B = 1024


def _banded_dyadic(seed):
    """4096 x 9216 at batch 1024 with every row dense over the first 128
    columns, two fully dense rows, and uniform entries elsewhere (~2.9 M in
    all), on the dyadic grid.  The mean load per (wave, X tile) keeps the
    forward product on the tiled path with half-wave units (B >= 256 and a
    mean chunk below 0.75 of the 1 KB LDS slot), while the first X tile holds
    about 1000 pairs per wave, far beyond the slot, so the loop's reads of a
    run from the stream in global memory are exercised; the full rows are cut
    into strided pieces (a split row summed by the fix-up pass)."""
    N, K, B = 4096, 9216, 1024
    rng = np.random.default_rng(seed)
    dense = np.zeros((N, K), bool)
    dense[:, :128] = True
    flat = rng.choice(N * (K - 128), 2_400_000, replace=False)
    dense[flat // (K - 128), 128 + flat % (K - 128)] = True
    dense[[17, 3001], :] = True
    rp, ci = synth.pattern_from_positions(N, K, np.flatnonzero(dense.reshape(-1)))
    return synth.dyadic_layer(N, K, B, 0, seed=seed, pattern=(rp, ci))


def test_spmm_chunks_beyond_lds_slot_dyadic_bit_exact():
    L = _banded_dyadic(41)
    W = _W(L)
    assert L1.workspace_bytes(L1.OP_SPMM, L.N, L.K, L.nnz, L.B) > 0  # the tiled path
    Y = h(L1.csr_spmm_fwd(W, t(L.X)))
    assert bits_equal(Y, oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)), "Y"
    dX = h(L1.csr_spmm_bwd_t(W, t(L.dY), L1.csc_build(W)))
    assert bits_equal(dX, oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)), "dX"


def test_spmm_fwd_padded_leading_dimension():
    L = synth.fc_layer(50, 70, 37, 900, seed=11)
    import torch
    Xp = torch.zeros((70, 41), dtype=torch.float32, device=cuda())
    Xp[:, :37] = t(L.X)
    Yp = torch.full((50, 43), 7.0, dtype=torch.float32, device=cuda())
    L1.csr_spmm_fwd(_W(L), Xp[:, :37], Yp[:, :37])
    ref = oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)
    m = oracle.spmm_fwd(L.row_ptr, L.col_idx, np.abs(L.vals), L.X)
    assert_scaled_close(h(Yp)[:, :37], ref, m, what="Y")
    assert np.all(h(Yp)[:, 37:] == 7.0)  # padding untouched


def test_spmm_fwd_dyadic_bit_exact():
    L = synth.dyadic_layer(70, 300, 256, 6000, seed=3, empty_rows=(0, 5, 69), full_rows=(10,))
    Y = h(L1.csr_spmm_fwd(_W(L), t(L.X)))
    assert bits_equal(Y, oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X))


# ----------------------------------------------------------------------------
# CSC copy and backward product
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
def test_csc_build_bit_exact(shape):
    L = _layer(shape)
    csc = L1.csc_build(_W(L))
    cp, ri, pm = csc_reference(L.row_ptr, L.col_idx, L.K)
    assert bits_equal(h(csc.col_ptr), cp)
    assert bits_equal(h(csc.row_idx)[: L.nnz], ri)
    assert bits_equal(h(csc.perm)[: L.nnz], pm)
    assert bits_equal(h(csc.vals_t)[: L.nnz], L.vals[pm])


def test_csc_build_wide_matrix_column_tiles():
    # many 32-column words, a ragged last word
    L = synth.fc_layer(45, 40000, 1, 30000, seed=12)
    csc = L1.csc_build(_W(L))
    cp, ri, pm = csc_reference(L.row_ptr, L.col_idx, L.K)
    assert bits_equal(h(csc.col_ptr), cp)
    assert bits_equal(h(csc.row_idx)[: L.nnz], ri)
    assert bits_equal(h(csc.perm)[: L.nnz], pm)


@pytest.mark.parametrize("shape", [(10000, 70, 1, 300000, 14), (9216, 4096, 1, 3397386, 15), (12289, 1, 1, 9000, 16)],
                         ids=_ids)
def test_csc_build_tall_matrices_row_blocks(shape):
    # several 4096-row blocks per word (ragged last block), a one-column
    # matrix, and the transposed shape of the 9216 -> 4096 layer; built with
    # a bitmap index from csr_bitmap_build (as the step does) and without
    N, K, B, nnz, seed = shape
    L = synth.fc_layer(N, K, B, nnz, seed=seed)
    W = _W(L)
    cp, ri, pm = csc_reference(L.row_ptr, L.col_idx, L.K)
    for csc in (L1.csc_build(W), L1.csc_build(W, bitmap=L1.csr_bitmap_build(W))):
        assert bits_equal(h(csc.col_ptr), cp)
        assert bits_equal(h(csc.row_idx)[: L.nnz], ri)
        assert bits_equal(h(csc.perm)[: L.nnz], pm)
        assert bits_equal(h(csc.vals_t)[: L.nnz], L.vals[pm])


@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
@pytest.mark.parametrize("path", ["csc", "atomic"])
def test_spmm_bwd_t(shape, path):
    L = _layer(shape)
    W = _W(L)
    csc = L1.csc_build(W) if path == "csc" else None
    dX = h(L1.csr_spmm_bwd_t(W, t(L.dY), csc))
    ref = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)
    av, _, ady = _absL(L)
    m = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, av, ady, L.K)
    assert_scaled_close(dX, ref, m, what="dX")


def test_spmm_bwd_dyadic_bit_exact_and_deterministic():
    L = synth.dyadic_layer(90, 200, 128, 5000, seed=4, empty_rows=(1,), full_rows=(3, 4))
    W = _W(L)
    csc = L1.csc_build(W)
    ref = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)
    a = h(L1.csr_spmm_bwd_t(W, t(L.dY), csc))
    assert bits_equal(a, ref)
    assert bits_equal(h(L1.csr_spmm_bwd_t(W, t(L.dY), None)), ref)


def test_spmm_bwd_csc_stays_valid_after_value_update():
    # debiasing changes values only: the CSC structure is kept, values refreshed through perm
    L = synth.fc_layer(60, 80, 32, 1500, seed=13)
    W = _W(L)
    csc = L1.csc_build(W)
    W.vals.mul_(-0.5)
    L1.csc_update_vals(W, csc)
    dX = h(L1.csr_spmm_bwd_t(W, t(L.dY), csc))
    v2 = (L.vals * np.float32(-0.5)).astype(np.float32)
    ref = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, v2, L.dY, L.K)
    m = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, np.abs(v2), np.abs(L.dY), L.K)
    assert_scaled_close(dX, ref, m, what="dX")


# ----------------------------------------------------------------------------
# dense weight gradient (fp32 matrix cores)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("NKB", [(1, 1, 1), (7, 5, 3), (129, 130, 33), (300, 784, 64),
                                 (257, 1000, 100), (128, 128, 32), (64, 300, 256), (5, 9, 0)])
def test_dense_wgrad(NKB):
    N, K, B = NKB
    rng = np.random.default_rng(N * 7 + K)
    dY = rng.standard_normal((N, B)).astype(np.float32)
    X = rng.random((K, B)).astype(np.float32)
    dW = h(L1.dense_wgrad(t(dY), t(X)))
    ref = oracle.dense_wgrad(dY, X)
    m = oracle.dense_wgrad(np.abs(dY), X)
    assert_scaled_close(dW, ref, m, what="dW")


def test_dense_wgrad_batch_one_bit_exact_and_padded():
    rng = np.random.default_rng(1)
    dY = rng.standard_normal((70, 1)).astype(np.float32)
    X = rng.standard_normal((150, 1)).astype(np.float32)
    assert bits_equal(h(L1.dense_wgrad(t(dY), t(X))), oracle.dense_wgrad(dY, X))
    # leading dimensions not a multiple of 4 (scalar loads)
    import torch
    dY2 = rng.standard_normal((33, 45)).astype(np.float32)
    X2 = rng.random((66, 45)).astype(np.float32)
    dYp = torch.zeros((33, 47), device=cuda()); dYp[:, :45] = t(dY2)
    Xp = torch.zeros((66, 51), device=cuda()); Xp[:, :45] = t(X2)
    dWp = torch.full((33, 70), 3.0, device=cuda())
    L1.dense_wgrad(dYp[:, :45], Xp[:, :45], dWp[:, :66])
    assert_scaled_close(h(dWp)[:, :66], oracle.dense_wgrad(dY2, X2),
                        oracle.dense_wgrad(np.abs(dY2), X2), what="dW")
    assert np.all(h(dWp)[:, 66:] == 3.0)


@pytest.mark.parametrize("NKB", [(50, 500, 16384), (7, 130, 9001), (20, 25, 147456), (129, 257, 2080),
                                 (300, 784, 256 * 8)])
def test_dense_wgrad_split_reduction(NKB):
    # few output tiles and a long batch: the reduction is split into ranges
    # (ragged last range when B is not a multiple of the range length) and the
    # partials are added in a fixed order
    N, K, B = NKB
    assert L1.workspace_bytes(L1.OP_DENSE_WGRAD, N, K, 0, B) > 0
    rng = np.random.default_rng(N + K + B)
    dY = rng.standard_normal((N, B)).astype(np.float32)
    X = rng.random((K, B)).astype(np.float32)
    dW1 = h(L1.dense_wgrad(t(dY), t(X)))
    assert_scaled_close(dW1, oracle.dense_wgrad(dY, X), oracle.dense_wgrad(np.abs(dY), X), what="dW split")
    assert bits_equal(h(L1.dense_wgrad(t(dY), t(X))), dW1)  # reproducible


@pytest.mark.parametrize("NKB", [(257, 10999, 370), (130, 38400, 300), (200, 32768, 96),
                                 (2048, 9216, 64), (2000, 9000, 70)])
def test_dense_wgrad_many_tiles(NKB):
    # at least 256 output tiles (no split of the reduction): 258 ragged tiles
    # with scalar loads (B % 4 != 0), 600 tiles, 512 tiles (whole rounds of
    # two workgroups per CU); the last two take the 256 x 288 shape (whole
    # float4 loads, then ragged tiles with scalar loads)
    N, K, B = NKB
    assert L1.workspace_bytes(L1.OP_DENSE_WGRAD, N, K, 0, B) == 0
    rng = np.random.default_rng(N + K + B)
    dY = rng.standard_normal((N, B)).astype(np.float32)
    X = rng.random((K, B)).astype(np.float32)
    dW1 = h(L1.dense_wgrad(t(dY), t(X)))
    assert_scaled_close(dW1, oracle.dense_wgrad(dY, X), oracle.dense_wgrad(np.abs(dY), X), what="dW")
    assert bits_equal(h(L1.dense_wgrad(t(dY), t(X))), dW1)  # reproducible


@pytest.mark.parametrize("precision", [L1.F32, L1.BF16X3])
def test_dense_wgrad_empty_batch_large_shape(precision):
    # B = 0 on a shape that takes the 256 x 288 tiles: no reduction step at
    # all, every entry of dW written as an exact zero (padded ld, garbage before)
    import torch
    dY = torch.zeros((2048, 0), device=cuda())
    X = torch.zeros((9216, 0), device=cuda())
    dW = torch.full((2048, 9220), 5.0, device=cuda())
    L1.dense_wgrad(dY, X, dW[:, :9216], precision=precision)
    out = h(dW)
    assert not out[:, :9216].any() and np.all(out[:, 9216:] == 5.0)


def test_dense_wgrad_many_tiles_dyadic_bit_exact():
    L = synth.dyadic_layer(257, 10999, 370, 10, seed=7)
    assert bits_equal(h(L1.dense_wgrad(t(L.dY), t(L.X))), oracle.dense_wgrad(L.dY, L.X))


def test_dense_wgrad_split_reduction_dyadic_bit_exact():
    L = synth.dyadic_layer(50, 500, 16384, 10, seed=6)
    assert L1.workspace_bytes(L1.OP_DENSE_WGRAD, 50, 500, 0, 16384) > 0
    assert bits_equal(h(L1.dense_wgrad(t(L.dY), t(L.X))), oracle.dense_wgrad(L.dY, L.X))


def test_dense_wgrad_dyadic_bit_exact():
    L = synth.dyadic_layer(200, 300, 256, 10, seed=5)
    assert bits_equal(h(L1.dense_wgrad(t(L.dY), t(L.X))), oracle.dense_wgrad(L.dY, L.X))


# bf16 operands: against the oracle that rounds the operands to bf16 first
# (products exact, so only fp32 summation separates the two: the 1e-4 bar),
# and within the bf16 rounding bound of the fp32 result
@pytest.mark.parametrize("NKB", [(1, 1, 1), (7, 5, 3), (129, 130, 33), (300, 784, 64),
                                 (257, 1000, 100), (64, 300, 256), (256, 384, 1024), (5, 9, 0)])
def test_dense_wgrad_bf16(NKB):
    N, K, B = NKB
    rng = np.random.default_rng(N * 11 + K)
    dY = rng.standard_normal((N, B)).astype(np.float32)
    X = rng.random((K, B)).astype(np.float32)
    dW = h(L1.dense_wgrad(t(dY), t(X), precision=L1.BF16))
    ref = oracle.dense_wgrad_bf16(dY, X)
    m = oracle.dense_wgrad_bf16(np.abs(dY), X)
    assert_scaled_close(dW, ref, m, what="dW bf16")
    m32 = oracle.dense_wgrad(np.abs(dY), X).astype(np.float64)
    d32 = np.abs(dW.astype(np.float64) - oracle.dense_wgrad(dY, X))
    assert np.all(d32 <= (2.0 ** -7 + 2.0 ** -16 + 1e-4) * m32 + 1e-30)


def test_dense_wgrad_bf16_batch_one_bit_exact_and_padded():
    # B = 1: each entry is one exact product of the rounded operands, so the
    # rounding of every operand is checked bit for bit
    rng = np.random.default_rng(2)
    dY = rng.standard_normal((70, 1)).astype(np.float32)
    X = rng.standard_normal((150, 1)).astype(np.float32)
    assert bits_equal(h(L1.dense_wgrad(t(dY), t(X), precision=L1.BF16)), oracle.dense_wgrad_bf16(dY, X))
    import torch
    dY2 = rng.standard_normal((33, 45)).astype(np.float32)
    X2 = rng.random((66, 45)).astype(np.float32)
    dYp = torch.zeros((33, 47), device=cuda()); dYp[:, :45] = t(dY2)
    Xp = torch.zeros((66, 51), device=cuda()); Xp[:, :45] = t(X2)
    dWp = torch.full((33, 70), 3.0, device=cuda())
    L1.dense_wgrad(dYp[:, :45], Xp[:, :45], dWp[:, :66], precision=L1.BF16)
    assert_scaled_close(h(dWp)[:, :66], oracle.dense_wgrad_bf16(dY2, X2),
                        oracle.dense_wgrad_bf16(np.abs(dY2), X2), what="dW bf16")
    assert np.all(h(dWp)[:, 66:] == 3.0)


# bf16 hi + lo split, three products: against the oracle of the same split
# (exact products, so only fp32 summation separates the two), and against the
# exact fp32 definition within the 1e-4 contract itself
@pytest.mark.parametrize("NKB", [(1, 1, 1), (7, 5, 3), (129, 130, 33), (300, 784, 64),
                                 (257, 1000, 100), (64, 300, 256), (256, 384, 1024), (130, 2600, 300),
                                 (5, 9, 0),
                                 # many tiles: the 256 x 288 shape (ragged, scalar loads; whole float4)
                                 (1000, 12700, 70), (1024, 12800, 64)])
def test_dense_wgrad_bf16x3(NKB):
    N, K, B = NKB
    rng = np.random.default_rng(N * 13 + K)
    dY = rng.standard_normal((N, B)).astype(np.float32)
    X = rng.random((K, B)).astype(np.float32)
    dW = h(L1.dense_wgrad(t(dY), t(X), precision=L1.BF16X3))
    m = oracle.dense_wgrad(np.abs(dY), X)
    assert_scaled_close(dW, oracle.dense_wgrad_bf16x3(dY, X), m, what="dW bf16x3 vs its split")
    assert_scaled_close(dW, oracle.dense_wgrad(dY, X), m, what="dW bf16x3 vs fp32")
    assert bits_equal(h(L1.dense_wgrad(t(dY), t(X), precision=L1.BF16X3)), dW)  # reproducible


def test_dense_wgrad_bf16x3_batch_one_dyadic_and_padded():
    rng = np.random.default_rng(3)
    # B = 1: three exact products added in fp32 (two roundings at most)
    dY = rng.standard_normal((70, 1)).astype(np.float32)
    X = rng.standard_normal((150, 1)).astype(np.float32)
    m = np.abs(dY.astype(np.float64)) @ np.abs(X.T.astype(np.float64))
    assert_scaled_close(h(L1.dense_wgrad(t(dY), t(X), precision=L1.BF16X3)), oracle.dense_wgrad_bf16x3(dY, X),
                        m, tol=2.0 ** -22, what="dW bf16x3, B = 1")
    # dyadic operands sit on the bf16 grid (lo = 0) and every sum is exact
    L = synth.dyadic_layer(200, 300, 256, 10, seed=5)
    assert bits_equal(h(L1.dense_wgrad(t(L.dY), t(L.X), precision=L1.BF16X3)), oracle.dense_wgrad(L.dY, L.X))
    # leading dimensions not a multiple of 4 (scalar loads), ragged tiles
    import torch
    dY2 = rng.standard_normal((33, 45)).astype(np.float32)
    X2 = rng.random((66, 45)).astype(np.float32)
    dYp = torch.zeros((33, 47), device=cuda()); dYp[:, :45] = t(dY2)
    Xp = torch.zeros((66, 51), device=cuda()); Xp[:, :45] = t(X2)
    dWp = torch.full((33, 70), 3.0, device=cuda())
    L1.dense_wgrad(dYp[:, :45], Xp[:, :45], dWp[:, :66], precision=L1.BF16X3)
    assert_scaled_close(h(dWp)[:, :66], oracle.dense_wgrad(dY2, X2), oracle.dense_wgrad(np.abs(dY2), X2),
                        what="dW bf16x3, padded")
    assert np.all(h(dWp)[:, 66:] == 3.0)


def test_dense_wgrad_bf16x3_full_size_sampled():
    # the 9216 -> 4096 layer's gradient at batch 1024, in the launch the step
    # uses; sampled rows and columns against the exact fp32 definition
    L = synth.fc9216_4096(seed=0)
    dW = L1.dense_wgrad(t(L.dY), t(L.X), precision=L1.BF16X3)
    rng = np.random.default_rng(94)
    rows = np.sort(rng.choice(L.N, 48, replace=False))
    cols = np.sort(rng.choice(L.K, 64, replace=False))
    got = h(dW)[np.ix_(rows, cols)]
    ref = oracle.dense_wgrad(L.dY[rows], L.X[cols])
    m = oracle.dense_wgrad(np.abs(L.dY[rows]), np.abs(L.X[cols]))
    assert_scaled_close(got, ref, m, what="dW bf16x3 full size")


# ----------------------------------------------------------------------------
# CSR well-formedness check
# ----------------------------------------------------------------------------

def test_csr_validate():
    import torch
    L = synth.fc_layer(300, 784, 1, 23520, seed=0)
    good = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    assert L1.csr_validate(good)
    empty = L1.CSR.from_host(np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), 9,
                             device=cuda())
    assert L1.csr_validate(empty)
    none = L1.CSR(0, 5, torch.zeros(1, dtype=torch.int32, device=cuda()),
                  torch.zeros(1, dtype=torch.int32, device=cuda()),
                  torch.zeros(1, dtype=torch.float32, device=cuda()), 0)
    assert L1.csr_validate(none)

    def broken(edit):
        rp, ci = L.row_ptr.copy(), L.col_idx.copy()
        edit(rp, ci)
        W = L1.CSR(L.N, L.K, t(rp), t(ci), t(L.vals), L.nnz)
        return L1.csr_validate(W, nnz=L.nnz)

    r5 = int(L.row_ptr[5])
    assert not broken(lambda rp, ci: rp.__setitem__(0, 1))                        # row_ptr[0] != 0
    assert not broken(lambda rp, ci: rp.__setitem__(7, rp[6] - 1))                # decreasing
    assert not broken(lambda rp, ci: rp.__setitem__(L.N, L.nnz - 1))              # last != nnz
    assert not broken(lambda rp, ci: ci.__setitem__(r5, L.K))                      # column out of range
    assert not broken(lambda rp, ci: ci.__setitem__(r5, -1))                       # negative column
    assert not broken(lambda rp, ci: ci.__setitem__(r5 + 1, ci[r5]))               # duplicate
    assert not broken(lambda rp, ci: ci.__setitem__(slice(r5, r5 + 2), ci[r5:r5 + 2][::-1].copy()))  # unsorted
    # a column order that only breaks across a row boundary is fine
    assert broken(lambda rp, ci: None)
    bad0 = L1.CSR(0, 5, torch.full((1,), 2, dtype=torch.int32, device=cuda()),
                  torch.zeros(1, dtype=torch.int32, device=cuda()),
                  torch.zeros(1, dtype=torch.float32, device=cuda()), 0)
    assert not L1.csr_validate(bad0)


# ----------------------------------------------------------------------------
# masked weight gradient
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("shape", SHAPES + [(20, 30, 5000, 300, 9), (50, 500, 2048, 2500, 10)],
                         ids=_ids)
def test_sddmm(shape):
    L = _layer(shape)
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    ref = oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X)
    m = oracle.sddmm(L.row_ptr, L.col_idx, np.abs(L.dY), L.X)
    assert_scaled_close(gv, ref, m, what="gv")


# dense patterns (50 % and 93 % of the entries stored) through the gather
# kernel, with vector and scalar operand loads and ragged column ranges
@pytest.mark.parametrize("shape", [(2048, 2048, 256, 2097152, 11), (1100, 1030, 333, 1050000, 12)],
                         ids=_ids)
def test_sddmm_dense_patterns(shape):
    L = _layer(shape)
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    ref = oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X)
    m = oracle.sddmm(L.row_ptr, L.col_idx, np.abs(L.dY), L.X)
    assert_scaled_close(gv, ref, m, what="gv")


# X larger than one XCD's L2 (4096 or 4000 columns by a batch of 512 or 500:
# 8 MB) with many entries per row: the planner cuts the columns into 8 ranges,
# one per XCD, instead of 4; ragged columns and batch in the second shape, a
# batch of 513 (scalar loads, three batch ranges, the last one column wide) in
# the third
@pytest.mark.parametrize("shape", [(1024, 4096, 512, 838861, 13), (700, 4000, 500, 600000, 14),
                                   (600, 4096, 513, 400000, 16)], ids=_ids)
def test_sddmm_xcd_column_split(shape):
    L = _layer(shape)
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    ref = oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X)
    m = oracle.sddmm(L.row_ptr, L.col_idx, np.abs(L.dY), L.X)
    assert_scaled_close(gv, ref, m, what="gv")


def test_sddmm_xcd_column_split_dyadic_bit_exact():
    L = synth.dyadic_layer(512, 4096, 512, 419430, seed=15, empty_rows=(5,), full_rows=(9,))
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    assert bits_equal(gv, oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X))


# a third of the entries stored or more, with vector loads: the row-block
# kernel (8-row blocks, 64-column windows); rows not a multiple of 8, columns
# not a multiple of 64, a batch whose last range is partial
@pytest.mark.parametrize("shape", [(300, 1000, 260, 150000, 17), (1027, 4096, 512, 2400000, 18)], ids=_ids)
def test_sddmm_row_blocks(shape):
    L = _layer(shape)
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    ref = oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X)
    m = oracle.sddmm(L.row_ptr, L.col_idx, np.abs(L.dY), L.X)
    assert_scaled_close(gv, ref, m, what="gv")


def test_sddmm_row_blocks_dyadic_bit_exact():
    L = synth.dyadic_layer(301, 1000, 516, 120000, seed=19, empty_rows=(4,), full_rows=(0, 300))
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    assert bits_equal(gv, oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X))


def test_sddmm_dyadic_bit_exact():
    L = synth.dyadic_layer(40, 60, 1100, 900, seed=6, empty_rows=(2,), full_rows=(7,))
    gv = h(L1.sddmm_masked_wgrad(_W(L), t(L.dY), t(L.X)))[: L.nnz]
    assert bits_equal(gv, oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X))


# ----------------------------------------------------------------------------
# prox, recompression, compaction (bit-exact)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
@pytest.mark.parametrize("eta,lam", [(0.01, 1e-4), (0.5, 0.3), (2.0 ** -7, 2.0 ** -4)])
def test_prox_dense_and_recompress_bit_exact(shape, eta, lam):
    L = _layer(shape)
    rng = np.random.default_rng(shape[-1])
    G = (rng.standard_normal((L.N, L.K)) * 0.05).astype(np.float32)
    W = _W(L)
    cnt = t(np.zeros(L.N, np.int32))
    Z = L1.prox_l1_step(L1.PROX_DENSE, W, t(G), eta, lam, row_counts=cnt)
    Zr, cr = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, G, eta, lam, L.K)
    assert bits_equal(h(Z), Zr)
    assert bits_equal(h(cnt), cr)
    out = L1.csr_recompress(Z, 0.0, row_counts=cnt)
    rp, ci, v = oracle.recompress(Zr, 0.0)
    assert bits_equal(h(out.row_ptr), rp)
    nnz = int(rp[-1])
    assert bits_equal(h(out.col_idx)[:nnz], ci)
    assert bits_equal(h(out.vals)[:nnz], v)


@pytest.mark.parametrize("NK", [(7, 5), (64, 300), (33, 1031), (40, 9000), (5, 20000)])
def test_prox_l1_recompress_fused_bit_exact(NK):
    # one call: W - eta*G -> soft threshold -> CSR, against the oracle's prox + recompress;
    # covers ragged rows (K % 4 != 0) and rows longer than one LDS pass (K > 8192)
    N, K = NK
    L = synth.fc_layer(N, K, 4, int(0.1 * N * K), seed=N + K)
    rng = np.random.default_rng(N * K)
    G = (rng.standard_normal((N, K)) * 0.05).astype(np.float32)
    G[0, : min(K, 7)] = 0.0  # zero gradient on some (maybe stored) weights
    for eta, lam in [(0.01, 1e-4), (0.5, 0.3)]:
        out = L1.prox_l1_recompress(_W(L), t(G), eta, lam)
        Zr, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, G, eta, lam, K)
        rp, ci, v = oracle.recompress(Zr)
        n = int(rp[-1])
        assert bits_equal(h(out.row_ptr), rp)
        assert bits_equal(h(out.col_idx)[:n], ci) and bits_equal(h(out.vals)[:n], v)


@pytest.mark.parametrize("NK", [(9000, 333), (2000, 9217), (4096, 4096), (700, 20001), (1, 1)])
def test_prox_l1_recompress_large_shapes_both_capacity_paths(NK):
    # thousands of slabs (ragged last slab when K % 2048 != 0): the no-wait call
    # (capacity N*K) and the checked call (capacity N*K - 1: count, wait, fill)
    # must both equal the oracle bit for bit
    N, K = NK
    L = synth.fc_layer(N, K, 4, int(0.05 * N * K), seed=N ^ K)
    rng = np.random.default_rng(N + K)
    G = (rng.standard_normal((N, K)) * 0.05).astype(np.float32)
    eta, lam = 0.5, 0.05
    one = L1.prox_l1_recompress(_W(L), t(G), eta, lam)
    Zr, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, G, eta, lam, K)
    rp, ci, v = oracle.recompress(Zr)
    n = int(rp[-1])
    assert 0 < n < N * K or N * K == 1
    assert bits_equal(h(one.row_ptr), rp)
    assert bits_equal(h(one.col_idx)[:n], ci) and bits_equal(h(one.vals)[:n], v)
    if n < N * K:
        two = L1.prox_l1_recompress(_W(L), t(G), eta, lam, capacity=N * K - 1)
        assert two.nnz == n
        assert bits_equal(h(two.row_ptr), rp)
        assert bits_equal(h(two.col_idx)[:n], ci) and bits_equal(h(two.vals)[:n], v)


def test_prox_l1_recompress_capacity():
    L = synth.fc_layer(30, 50, 4, 150, seed=3)
    rng = np.random.default_rng(3)
    G = (rng.standard_normal((30, 50)) * 0.05).astype(np.float32)
    Zr, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, G, 0.5, 0.05, 50)
    need = int(np.count_nonzero(Zr))
    with pytest.raises(L1.L1CSRError) as ei:
        L1.prox_l1_recompress(_W(L), t(G), 0.5, 0.05, capacity=need - 1)
    assert ei.value.status == L1.ECAPACITY
    out = L1.prox_l1_recompress(_W(L), t(G), 0.5, 0.05, capacity=need)
    assert out.nnz == need
    rp, ci, v = oracle.recompress(Zr)
    assert bits_equal(h(out.col_idx)[:need], ci) and bits_equal(h(out.vals)[:need], v)


def test_prox_dense_in_place_and_threshold_ties():
    L = synth.dyadic_layer(64, 300, 64, 4000, seed=7, empty_rows=(3,), full_rows=(9,))
    dW = oracle.dense_wgrad(L.dY, L.X)
    G = t(dW)
    Z = L1.prox_l1_step(L1.PROX_DENSE, _W(L), G, L.eta, L.lam, Z=G)  # Z aliases G
    Zr, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, dW, L.eta, L.lam, L.K)
    assert bits_equal(h(Z), Zr)
    # the dyadic grid produces exact ties |z| == t, which must give +0
    t_ = np.float64(np.float32(L.eta)) * np.float64(np.float32(L.lam))
    D = oracle.densify(L.row_ptr, L.col_idx, L.vals, L.K).astype(np.float64)
    z = D - np.float64(np.float32(L.eta)) * dW.astype(np.float64)
    assert np.any(np.abs(z) == t_)


def test_recompress_without_counts_threshold_and_capacity():
    rng = np.random.default_rng(3)
    Zh = rng.standard_normal((37, 301)).astype(np.float32)
    Zh[rng.random(Zh.shape) < 0.7] = 0
    Zh[4] = 0
    Zh[5] = 1
    Zh[6, 10] = -0.0
    for thr in (0.0, 0.5):
        out = L1.csr_recompress(t(Zh), thr)
        rp, ci, v = oracle.recompress(Zh, thr)
        nnz = int(rp[-1])
        assert bits_equal(h(out.row_ptr), rp)
        assert bits_equal(h(out.col_idx)[:nnz], ci) and bits_equal(h(out.vals)[:nnz], v)
    need = int(np.count_nonzero(Zh))
    with pytest.raises(L1.L1CSRError) as ei:
        L1.csr_recompress(t(Zh), 0.0, capacity=need - 1)
    assert ei.value.status == L1.ECAPACITY
    out = L1.csr_recompress(t(Zh), 0.0, capacity=need)
    assert out.nnz == need
    rp, ci, v = oracle.recompress(Zh, 0.0)
    assert bits_equal(h(out.col_idx)[:need], ci)


def test_recompress_fig1_example():
    A = np.array([[1, 7, 0, 0], [0, 2, 8, 0], [5, 0, 3, 9], [0, 6, 0, 4]], np.float32)
    out = L1.csr_recompress(t(A), 0.0)
    assert h(out.row_ptr).tolist() == [0, 2, 4, 7, 9]
    assert h(out.col_idx)[:9].tolist() == [0, 1, 1, 2, 0, 2, 3, 1, 3]
    assert h(out.vals)[:9].tolist() == [1, 7, 2, 8, 5, 3, 9, 6, 4]


def test_prox_csr_and_compact_bit_exact():
    L = synth.fc_layer(80, 120, 16, 3000, seed=14)
    gv = oracle.sddmm(L.row_ptr, L.col_idx, L.dY, L.X)
    for lam in (0.0, 0.05):
        W = _W(L)
        L1.prox_l1_step(L1.PROX_CSR, W, t(gv), 0.01, lam)
        ref = oracle.prox_csr(L.vals, gv, 0.01, lam)
        assert bits_equal(h(W.vals)[: L.nnz], ref)
        assert bits_equal(h(W.row_ptr), L.row_ptr) and bits_equal(h(W.col_idx)[: L.nnz], L.col_idx)
        if lam > 0:
            assert np.count_nonzero(ref == 0) > 0
            C = L1.csr_compact(W)
            rp, ci, v = oracle.compact(L.row_ptr, L.col_idx, ref)
            assert bits_equal(h(C.row_ptr), rp)
            assert bits_equal(h(C.col_idx)[: rp[-1]], ci) and bits_equal(h(C.vals)[: rp[-1]], v)


# ----------------------------------------------------------------------------
# layer glue
# ----------------------------------------------------------------------------

def test_relu_bit_exact():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(10007).astype(np.float32)
    x[:3] = [0.0, -0.0, 1e-40]
    dy = rng.standard_normal(10007).astype(np.float32)
    assert bits_equal(h(L1.relu_fwd(t(x))), oracle.relu_fwd(x))
    assert bits_equal(h(L1.relu_bwd(t(x), t(dy))), oracle.relu_bwd(x, dy))


@pytest.mark.parametrize("C,B", [(10, 256), (10, 1), (3, 1000), (10, 16384)])
def test_softmax_xent(C, B):
    rng = np.random.default_rng(C + B)
    z = (rng.standard_normal((C, B)) * 4).astype(np.float32)
    lab = rng.integers(0, C, size=B).astype(np.int32)
    loss, dz = L1.softmax_xent(t(z), t(lab))
    lr, dzr = oracle.softmax_xent(z, lab)
    assert abs(float(h(loss)[0]) - lr) <= 1e-5 * max(1.0, abs(lr))
    assert np.max(np.abs(h(dz) - dzr)) <= 1e-6 / B * 10
