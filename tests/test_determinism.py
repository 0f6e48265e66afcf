"""Run-twice determinism of the hot path.

Every call except the atomic transposed product takes a fixed summation order
(per-row or per-tile loops, fixed-order reductions of split partials, ballots
and scans for the structure), so two runs on the same inputs must agree bit
for bit.  Each run starts from buffers filled with different garbage.  The
float-atomic backward (csr_spmm_bwd_t without a CSC) is the labelled
exception: its order of additions depends on scheduling, so it is only
required to stay within the 1e-4 bar of the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_1905_07931_amd as L1
from paper_1905_07931_amd import synth

from _helpers import assert_scaled_close, cuda, h, t

pytestmark = pytest.mark.gpu


def _bits(a):
    a = h(a)
    return a.view(np.int32) if a.dtype == np.float32 else a


def _step(L, W, fill):
    """An l1 step and a debiasing step on its output; returns every output."""
    import torch
    dev = cuda()
    X, dY = t(L.X), t(L.dY)
    Y = torch.full((L.N, L.B), fill, device=dev)
    dX = torch.full((L.K, L.B), fill, device=dev)
    dW = torch.full((L.N, L.K), fill, device=dev)
    dW3 = torch.full((L.N, L.K), fill, device=dev)
    L1.csr_spmm_fwd(W, X, Y)
    csc = L1.csc_build(W)
    L1.csr_spmm_bwd_t(W, dY, csc, dX)
    L1.dense_wgrad(dY, X, dW)
    L1.dense_wgrad(dY, X, dW3, precision=L1.BF16X3)
    W1 = L1.prox_l1_recompress(W, dW, L.eta, L.lam)
    gv = L1.sddmm_masked_wgrad(W1, dY, X)
    n1 = W1.host_nnz()
    L1.prox_l1_step(L1.PROX_CSR, W1, gv, L.eta, 0.0)
    return [Y, dX, dW, dW3, csc.col_ptr, csc.row_idx[: L.nnz], csc.perm[: L.nnz], csc.vals_t[: L.nnz],
            W1.row_ptr, W1.col_idx[:n1], W1.vals[:n1], gv[:n1]]


@pytest.mark.parametrize("shape", [(2000, 3000, 256, 0.05, "zipf"), (300, 784, 64, 0.10, "uniform")])
def test_l1_and_debias_steps_bitwise_reproducible(shape):
    N, K, B, d, pattern = shape
    L = synth.fc_layer(N, K, B, synth.nnz_for(N, K, d), seed=17, pattern=pattern)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    a = [_bits(x) for x in _step(L, W, 7.0)]
    b = [_bits(x) for x in _step(L, W, -3.0)]
    for i, (x, y) in enumerate(zip(a, b)):
        assert np.array_equal(x, y), i


def test_split_reduction_and_conv_reproducible():
    # dense gradient with few tiles and a long batch (split reduction), and
    # the direct convolution of LeNet-5 conv2
    rng = np.random.default_rng(5)
    dY = t(rng.standard_normal((50, 16384)).astype(np.float32))
    X = t(rng.random((500, 16384)).astype(np.float32))
    assert np.array_equal(_bits(L1.dense_wgrad(dY, X)), _bits(L1.dense_wgrad(dY, X)))
    C = synth.lenet5_conv2(seed=3)
    g = L1.ConvGeom(*C.geom)
    W = L1.CSR.from_host(C.row_ptr, C.col_idx, C.vals, C.K, device=cuda())
    Xc = t(C.X)
    assert np.array_equal(_bits(L1.csr_conv_fwd(g, W, Xc)), _bits(L1.csr_conv_fwd(g, W, Xc)))
    csc = L1.csc_build(W)
    dYc = t(C.dY)
    a = L1.csr_conv_bwd_data(g, C.n_out, csc, dYc, nnz=C.nnz)
    b = L1.csr_conv_bwd_data(g, C.n_out, csc, dYc, nnz=C.nnz)
    assert np.array_equal(_bits(a), _bits(b))


def test_atomic_backward_is_the_labelled_exception():
    L = synth.fc_layer(2000, 3000, 256, synth.nnz_for(2000, 3000, 0.05), seed=18, pattern="zipf")
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    ref = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)
    m = oracle.spmm_bwd_t(L.row_ptr, L.col_idx, np.abs(L.vals), np.abs(L.dY), L.K)
    for _ in range(2):
        assert_scaled_close(h(L1.csr_spmm_bwd_t(W, t(L.dY), None)), ref, m, what="dX atomics")
