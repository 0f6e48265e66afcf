"""Every product and the l1 update on randomly drawn small layers (hypothesis).

Shapes from N, K in {1, 2, 7, 64, 65, 300}, batch in {1, 63, 64, 65, 256},
density in {0, 0.01, 0.1, 0.5, 1}, optionally a forced empty first row and a
forced full last row; values N(0, 0.05), X ~ U[0,1), dY ~ N(0,1).  The draws
are derandomized, so the same examples run every time.  Checked against the
oracle: SpMM forward, the CSC copy (bit for bit), the backward through the CSC
and through atomics, the dense gradient in fp32 and in split bf16, the
sampled gradient, and prox + recompression of the GPU's own gradient (bit
for bit).
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
import paper_1905_07931_amd as L1
from paper_1905_07931_amd import synth

from _helpers import assert_scaled_close, bits_equal, csc_reference, cuda, h, t

pytestmark = pytest.mark.gpu

DIMS = [1, 2, 7, 64, 65, 300]
BATCH = [1, 63, 64, 65, 256]
DENSITY = [0.0, 0.01, 0.1, 0.5, 1.0]


@st.composite
def layers(draw):
    N, K = draw(st.sampled_from(DIMS)), draw(st.sampled_from(DIMS))
    B, d = draw(st.sampled_from(BATCH)), draw(st.sampled_from(DENSITY))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    return N, K, B, d, seed, draw(st.booleans()), draw(st.booleans())


def _layer(N, K, B, d, seed, empty_first, full_last):
    L = synth.fc_layer(N, K, B, int(round(d * N * K)), seed=seed)
    if not (empty_first or full_last):
        return L.row_ptr, L.col_idx, L.vals, L.X, L.dY
    mask = np.zeros((N, K), bool)
    mask[np.repeat(np.arange(N), np.diff(L.row_ptr)), L.col_idx] = True
    if full_last:
        mask[N - 1, :] = True
    if empty_first:
        mask[0, :] = False
    rp, ci = synth.pattern_from_positions(N, K, np.flatnonzero(mask.reshape(-1)))
    vals = (np.random.default_rng(seed + 1).standard_normal(ci.shape[0]) * 0.05).astype(np.float32)
    return rp, ci, vals, L.X, L.dY


@settings(max_examples=60, deadline=None, derandomize=True, database=None,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(layers())
def test_products_and_update_on_random_layers(p):
    N, K, B, d, seed, empty_first, full_last = p
    rp, ci, v, X, dY = _layer(*p)
    W = L1.CSR.from_host(rp, ci, v, K, device=cuda())
    Xg, dYg = t(X), t(dY)
    av, ax, ady = np.abs(v), np.abs(X), np.abs(dY)

    Y = L1.csr_spmm_fwd(W, Xg)
    assert_scaled_close(h(Y), oracle.spmm_fwd(rp, ci, v, X), oracle.spmm_fwd(rp, ci, av, ax), what="Y")

    csc = L1.csc_build(W)
    col_ptr, row_idx, perm = csc_reference(rp, ci, K)
    n = int(rp[-1])
    assert bits_equal(h(csc.col_ptr), col_ptr)
    assert bits_equal(h(csc.row_idx)[:n], row_idx) and bits_equal(h(csc.perm)[:n], perm)

    ref_dx = oracle.spmm_bwd_t(rp, ci, v, dY, K)
    m_dx = oracle.spmm_bwd_t(rp, ci, av, ady, K)
    assert_scaled_close(h(L1.csr_spmm_bwd_t(W, dYg, csc)), ref_dx, m_dx, what="dX (CSC)")
    assert_scaled_close(h(L1.csr_spmm_bwd_t(W, dYg, None)), ref_dx, m_dx, what="dX (atomics)")

    m_dw = oracle.dense_wgrad(ady, ax)
    ref_dw = oracle.dense_wgrad(dY, X)
    dW = L1.dense_wgrad(dYg, Xg)
    assert_scaled_close(h(dW), ref_dw, m_dw, what="dW")
    assert_scaled_close(h(L1.dense_wgrad(dYg, Xg, precision=L1.BF16X3)), ref_dw, m_dw, what="dW bf16x3")

    gv = L1.sddmm_masked_wgrad(W, dYg, Xg)
    assert_scaled_close(h(gv)[:n], oracle.sddmm(rp, ci, dY, X), oracle.sddmm(rp, ci, ady, ax), what="gv")

    eta, lam = 0.01, 1e-4
    out = L1.prox_l1_recompress(W, dW, eta, lam)
    Z, _ = oracle.prox_dense(rp, ci, v, h(dW), eta, lam, K)
    rpn, cin, vn = oracle.recompress(Z)
    m2 = int(rpn[-1])
    assert bits_equal(h(out.row_ptr), rpn)
    assert bits_equal(h(out.col_idx)[:m2], cin) and bits_equal(h(out.vals)[:m2], vn)
