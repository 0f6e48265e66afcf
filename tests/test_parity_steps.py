"""Whole training steps of the paper's layer shapes on the GPU, against the oracle.

Each step chains the ABI calls the way a training loop does (forward, CSC,
backward, weight gradient, proximal step, recompression, and the debiasing
step on a fixed pattern, Sections 2.3-2.4 and 3.1-3.3).  Every stage is
compared with the oracle applied to that stage's GPU inputs:
  - sums (products, gradients): |gpu - oracle| <= 1e-4 * m, m = sum |a_k b_k|;
  - prox / recompression / compaction / ReLU: bit-exact (fed the GPU's own
    gradient, so the comparison is well posed);
  - structure (row pointers, column indices, CSC): bit-exact.
For the single-layer l1 steps the fully independent oracle step (its own
gradient) is also run: every entry where its new pattern differs from the
GPU's must lie in the rounding band of the threshold, | |z| - eta*lambda | <=
eta * 1e-4 * m_ik, with z = w - eta*g and m_ik = sum_b |dY[i,b] X[k,b]|.

At the full size of the 9216 -> 4096 layer (batch 1024) every output is
compared in full: all of Y, dX and dW against the oracle, the CSC and the new
CSR bit for bit, and the same step on the dyadic grid through the two-stream
l1_step bit for bit end to end.  The 20-iteration 4096 x 4096 sweep compares
every output in full at its first l1 and first debiasing iteration and a
seeded sample of rows / columns (computed one by one by the oracle) after
that.
"""
import json
import os

import numpy as np
import pytest

import oracle
import paper_1905_07931_amd as L1
from paper_1905_07931_amd import synth

from _helpers import TOL, assert_scaled_close, bits_equal, csc_reference, cuda, h, t

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------
# oracle-side checks of one stage
# ----------------------------------------------------------------------------

def rows_of(rp, ci, v, rows):
    """The CSR of a subset of rows (in the given order)."""
    rp = np.asarray(rp, np.int64)
    lens = np.array([rp[r + 1] - rp[r] for r in rows], np.int64)
    sub_rp = np.zeros(len(rows) + 1, np.int32)
    sub_rp[1:] = np.cumsum(lens)
    if lens.sum() == 0:
        return sub_rp, np.zeros(0, np.int32), np.zeros(0, np.float32)
    sub_ci = np.concatenate([ci[rp[r]:rp[r + 1]] for r in rows]).astype(np.int32)
    sub_v = np.concatenate([v[rp[r]:rp[r + 1]] for r in rows]).astype(np.float32)
    return sub_rp, sub_ci, sub_v


def check_fwd(W, X, Y, rows=None, what="Y"):
    rp, ci, v = W
    if rows is not None:
        rp, ci, v = rows_of(rp, ci, v, rows)
        Y = Y[rows]
    ref = oracle.spmm_fwd(rp, ci, v, X)
    m = oracle.spmm_fwd(rp, ci, np.abs(v), np.abs(X))
    assert_scaled_close(Y, ref, m, what=what)


def transposed_rows(rp, ci, v, cols):
    """Rows `cols` of W^T as a CSR (each in ascending row order of W)."""
    ci = np.asarray(ci)
    flag = np.zeros(int(ci.max()) + 1 if len(ci) else 1, bool)
    flag[[c for c in cols if c < len(flag)]] = True
    sel = np.nonzero(flag[ci])[0] if len(ci) else np.zeros(0, np.int64)
    r = np.searchsorted(np.asarray(rp, np.int64), sel, side="right") - 1
    c = ci[sel]
    sub_rp = np.zeros(len(cols) + 1, np.int32)
    parts_r, parts_v = [], []
    for j, k in enumerate(cols):
        m = c == k
        parts_r.append(r[m])
        parts_v.append(np.asarray(v)[sel[m]])
        sub_rp[j + 1] = sub_rp[j] + int(m.sum())
    return (sub_rp, np.concatenate(parts_r).astype(np.int32) if parts_r else np.zeros(0, np.int32),
            np.concatenate(parts_v).astype(np.float32) if parts_v else np.zeros(0, np.float32))


def check_bwd(W, K, dY, dX, cols=None, what="dX"):
    rp, ci, v = W
    if cols is None:
        ref = oracle.spmm_bwd_t(rp, ci, v, dY, K)
        m = oracle.spmm_bwd_t(rp, ci, np.abs(v), np.abs(dY), K)
        assert_scaled_close(dX, ref, m, what=what)
        return
    WT = transposed_rows(rp, ci, v, cols)
    ref = oracle.spmm_fwd(*WT, dY)
    m = oracle.spmm_fwd(WT[0], WT[1], np.abs(WT[2]), np.abs(dY))
    assert_scaled_close(dX[cols], ref, m, what=what)


def check_dw(dY, X, dW, rows=None, what="dW"):
    """dW against the oracle (all rows, or the given ones); returns the oracle's dW."""
    if rows is not None:
        dY, dW = dY[rows], dW[rows]
    ref = oracle.dense_wgrad(dY, X)
    m = oracle.dense_wgrad(np.abs(dY), np.abs(X))
    assert_scaled_close(dW, ref, m, what=what)
    return ref


def check_sddmm(W, dY, X, gv, rows=None, what="gv"):
    rp, ci, _ = W
    if rows is not None:
        rp64 = np.asarray(rp, np.int64)
        gv = np.concatenate([gv[rp64[r]:rp64[r + 1]] for r in rows]) if len(rows) else gv[:0]
        rp, ci, _ = rows_of(rp, ci, np.zeros(len(ci), np.float32), rows)
        dY = dY[rows]
    ref = oracle.sddmm(rp, ci, dY, X)
    m = oracle.sddmm(rp, ci, np.abs(dY), np.abs(X))
    assert_scaled_close(gv, ref, m, what=what)


def check_prox_recompress(W, dW, eta, lam, K, out):
    """The GPU's new CSR equals the oracle's prox + recompression of the GPU's dW, bit for bit."""
    rp, ci, v = W
    Z, _ = oracle.prox_dense(rp, ci, v, dW, eta, lam, K)
    rpn, cin, vn = oracle.recompress(Z)
    n = int(rpn[-1])
    assert out.host_nnz() == n
    assert bits_equal(h(out.row_ptr), rpn), "row_ptr"
    assert bits_equal(h(out.col_idx)[:n], cin), "col_idx"
    assert bits_equal(h(out.vals)[:n], vn), "vals"
    return rpn, cin, vn


def independent_band_check(W, dY, X, eta, lam, K, new_W, dWr=None):
    """Pattern of the fully independent oracle step vs the GPU's: every
    difference lies in the rounding band of the threshold.  Returns the count.
    dWr: the oracle's full dense gradient if already computed."""
    rp, ci, v = W
    if dWr is None:
        dWr = oracle.dense_wgrad(dY, X)
    Zi, _ = oracle.prox_dense(rp, ci, v, dWr, eta, lam, K)
    mask_i = Zi != 0
    N = len(rp) - 1
    mask_g = np.zeros((N, K), bool)
    rows_g = np.repeat(np.arange(N), np.diff(np.asarray(new_W[0], np.int64)))
    mask_g[rows_g, new_W[1]] = True
    diff = np.argwhere(mask_i != mask_g)
    if len(diff):
        Wd = oracle.densify(rp, ci, v, K)
        thr = np.float64(eta) * np.float64(lam)
        for i, k in diff:
            z = np.float64(Wd[i, k]) - np.float64(eta) * np.float64(dWr[i, k])
            m = np.sum(np.abs(dY[i].astype(np.float64)) * np.abs(X[k].astype(np.float64)))
            assert abs(abs(z) - thr) <= eta * TOL * m, (int(i), int(k), z, thr, m)
    return len(diff)


# ----------------------------------------------------------------------------
# single-layer l1 steps
# ----------------------------------------------------------------------------

def l1_step(L, W, host, rows=None, cols=None, band=True, precision=L1.F32):
    """fwd, CSC, bwd, dense dW, prox + recompress; every stage checked."""
    X, dY = L.X, L.dY
    Xg, dYg = t(X), t(dY)
    Y = L1.csr_spmm_fwd(W, Xg)
    csc = L1.csc_build(W)
    dX = L1.csr_spmm_bwd_t(W, dYg, csc)
    dW = L1.dense_wgrad(dYg, Xg, precision=precision)
    out = L1.prox_l1_recompress(W, dW, L.eta, L.lam)
    dWh = h(dW)
    check_fwd(host, X, h(Y), rows)
    col_ptr, row_idx, perm = csc_reference(host[0], host[1], L.K)
    n = int(host[0][-1])
    assert bits_equal(h(csc.col_ptr), col_ptr)
    assert bits_equal(h(csc.row_idx)[:n], row_idx) and bits_equal(h(csc.perm)[:n], perm)
    check_bwd(host, L.K, dY, h(dX), cols)
    dWr = check_dw(dY, X, dWh, rows)
    new = check_prox_recompress(host, dWh, L.eta, L.lam, L.K, out)
    n_band = None
    if band:
        n_band = independent_band_check(host, dY, X, L.eta, L.lam, L.K, new,
                                        dWr=dWr if rows is None else None)
    return out, new, n_band


def test_fc784x300_l1_step():
    L = synth.fc784_300(seed=0)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    out, new, n_band = l1_step(L, W, (L.row_ptr, L.col_idx, L.vals))
    # almost every zero weight has |dW| > lambda here, so the layer regrows nearly dense
    assert int(new[0][-1]) > 0.99 * L.N * L.K
    assert n_band <= 10


def test_fc9216x4096_zipf_l1_step_full_size():
    # every entry of Y (4096 x 1024), dX (9216 x 1024) and dW (4096 x 9216)
    # against the oracle; the CSC and the new CSR bit for bit
    L = synth.fc9216_4096(seed=0)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    out, new, n_band = l1_step(L, W, (L.row_ptr, L.col_idx, L.vals))
    assert n_band <= 1e-5 * L.N * L.K


def test_fc9216x4096_zipf_dyadic_two_stream_step_bit_exact():
    """The 9216 -> 4096 layer with Zipf rows, batch 1024, on the dyadic grid
    (values +-k/16, X j/16, dY +-k/16, eta 2^-7, lambda 2^-4): every fp32
    product and partial sum of the step is exact (|Y|, |dX|, |dW| stay below
    2^24 units of 2^-8), and the prox's z and S_t(z) are exact on a grid of
    2^-15, so the two-stream l1_step -- the launch configuration the bench
    times -- must equal the fully independent oracle step bit for bit: Y, dX,
    dW, the CSC (col_ptr, row_idx, perm, vals_t) and the new CSR."""
    import torch
    L = synth.dyadic_layer(4096, 9216, 1024, synth.nnz_for(4096, 9216, 0.09), seed=0,
                           pattern="zipf")
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    W.nnz = L.nnz
    X, dY = t(L.X), t(L.dY)
    o = _step_buffers(L, dev)
    L1.l1_step(W, X, dY, L.eta, L.lam, Y=o["Y"], dX=o["dX"], dW=o["dW"], csc=o["csc"], out=o["out"],
               schedule="two_stream")
    torch.cuda.synchronize()
    assert bits_equal(h(o["Y"]), oracle.spmm_fwd(L.row_ptr, L.col_idx, L.vals, L.X)), "Y"
    assert bits_equal(h(o["dX"]), oracle.spmm_bwd_t(L.row_ptr, L.col_idx, L.vals, L.dY, L.K)), "dX"
    dWr = oracle.dense_wgrad(L.dY, L.X)  # exact on the grid: the step's products must give it
    col_ptr, row_idx, perm = csc_reference(L.row_ptr, L.col_idx, L.K)
    c = o["csc"]
    assert bits_equal(h(c.col_ptr), col_ptr), "col_ptr"
    assert bits_equal(h(c.row_idx)[:L.nnz], row_idx), "row_idx"
    assert bits_equal(h(c.perm)[:L.nnz], perm), "perm"
    assert bits_equal(h(c.vals_t)[:L.nnz], L.vals[perm]), "vals_t"
    Z, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, dWr, L.eta, L.lam, L.K)
    assert bits_equal(h(o["dW"]), Z), "Z = S_t(W - eta dW)"  # the step's dense buffer holds Z
    rpn, cin, vn = oracle.recompress(Z)
    n = int(rpn[-1])
    # the grid produces exact ties |z| == t (deleted) as well as survivors
    assert 0 < n < L.N * L.K
    assert bits_equal(h(o["out"].row_ptr), rpn), "row_ptr'"
    assert bits_equal(h(o["out"].col_idx)[:n], cin), "col_idx'"
    assert bits_equal(h(o["out"].vals)[:n], vn), "vals'"


@pytest.mark.parametrize("which", ["fc784x300", "fc9216x4096"])
def test_l1_step_with_split_bf16_gradient(which):
    # the same steps with the weight gradient in BF16X3 (inside the contract):
    # dW within 1e-4 of the exact product, the prox + recompression of the
    # GPU's dW bit for bit, and every mask difference from the fully
    # independent oracle step inside the rounding band of the threshold
    if which == "fc784x300":
        L = synth.fc784_300(seed=0)
        rows = cols = None
    else:
        L = synth.fc9216_4096(seed=0)
        rng = np.random.default_rng(91)
        rows = np.sort(rng.choice(L.N, 48, replace=False))
        cols = rng.choice(L.K, 64, replace=False)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    out, new, n_band = l1_step(L, W, (L.row_ptr, L.col_idx, L.vals), rows=rows, cols=cols,
                               precision=L1.BF16X3)
    assert n_band <= 1e-4 * L.N * L.K


def test_empty_layer_regrows_then_empties():
    """nnz = 0: the products are zero; the prox grows entries with |eta*g| > eta*lambda.
    A lambda above every |g| then deletes the whole layer (an empty CSR)."""
    L = synth.fc_layer(70, 90, 33, 0, seed=31)
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())
    out, new, _ = l1_step(L, W, (L.row_ptr, L.col_idx, L.vals))
    assert 0 < int(new[0][-1]) <= L.N * L.K
    big = synth.fc_layer(70, 90, 33, 0, seed=31)
    big.lam = 1e6
    out2, new2, _ = l1_step(big, out, new)
    assert int(new2[0][-1]) == 0 and not np.any(new2[0])
    # and a step on the empty result works again
    out3, new3, _ = l1_step(L, out2, new2)
    assert int(new3[0][-1]) == int(new[0][-1])


# ----------------------------------------------------------------------------
# MLP 784-300-100-10: l1-phase step, then a debiasing step
# ----------------------------------------------------------------------------

def test_mlp_784_300_100_10_l1_then_debias_step():
    layers, X, labels = synth.mlp_784_300_100_10(seed=0)
    B = X.shape[1]
    eta, lam = 0.01, 1e-4
    dev = cuda()
    Ws = [L1.CSR.from_host(Lj.row_ptr, Lj.col_idx, Lj.vals, Lj.K, device=dev) for Lj in layers]
    host = [(Lj.row_ptr, Lj.col_idx, Lj.vals) for Lj in layers]
    Xg, lab = t(X), t(labels)

    def forward():
        inputs, pre = [Xg], []
        for j, W in enumerate(Ws):
            A = L1.csr_spmm_fwd(W, inputs[-1])
            check_fwd(host[j], h(inputs[-1]), h(A), what=f"A{j + 1}")
            pre.append(A)
            if j < 2:
                H = L1.relu_fwd(A)
                assert bits_equal(h(H), oracle.relu_fwd(h(A)))
                inputs.append(H)
        return inputs, pre

    def backward(inputs, pre):
        loss, dZ = L1.softmax_xent(pre[2], lab)
        lr, dzr = oracle.softmax_xent(h(pre[2]), labels)
        assert abs(float(h(loss)[0]) - lr) <= 1e-5 * max(1.0, abs(lr))
        assert np.max(np.abs(h(dZ) - dzr)) <= 1e-5 / B
        deltas = [None, None, dZ]
        for j in (2, 1):
            csc = L1.csc_build(Ws[j])
            dH = L1.csr_spmm_bwd_t(Ws[j], deltas[j], csc)
            check_bwd(host[j], Ws[j].n_cols, h(deltas[j]), h(dH), what=f"dH{j}")
            dA = L1.relu_bwd(pre[j - 1], dH)
            assert bits_equal(h(dA), oracle.relu_bwd(h(pre[j - 1]), h(dH)))
            deltas[j - 1] = dA
        return lr, deltas

    # l1 phase
    inputs, pre = forward()
    loss0, deltas = backward(inputs, pre)
    assert np.isfinite(loss0)
    for j in range(3):
        dW = L1.dense_wgrad(deltas[j], inputs[j])
        dWh = h(dW)
        check_dw(h(deltas[j]), h(inputs[j]), dWh, what=f"dW{j + 1}")
        out = L1.prox_l1_recompress(Ws[j], dW, eta, lam)
        host[j] = check_prox_recompress(host[j], dWh, eta, lam, Ws[j].n_cols, out)
        Ws[j] = out
    # debiasing: gradient on the pattern, SGD, pattern unchanged
    inputs, pre = forward()
    loss1, deltas = backward(inputs, pre)
    assert np.isfinite(loss1)
    for j in range(3):
        W = Ws[j]
        nnz = W.host_nnz()
        gv = L1.sddmm_masked_wgrad(W, deltas[j], inputs[j])
        gvh = h(gv)[:nnz]
        check_sddmm(host[j], h(deltas[j]), h(inputs[j]), gvh, what=f"gv{j + 1}")
        L1.prox_l1_step(L1.PROX_CSR, W, gv, eta, 0.0)
        ref = oracle.prox_csr(host[j][2], gvh, eta, 0.0)
        assert bits_equal(h(W.vals)[:nnz], ref)
        assert bits_equal(h(W.row_ptr), host[j][0]) and bits_equal(h(W.col_idx)[:nnz], host[j][1])
        host[j] = (host[j][0], host[j][1], ref)


# ----------------------------------------------------------------------------
# LeNet-5 conv2 lowered by im2col: masked gradient over 16384 columns, CSR prox
# ----------------------------------------------------------------------------

def test_conv2_im2col_step():
    L = synth.conv2_im2col(seed=0)
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    host = (L.row_ptr, L.col_idx, L.vals)
    Xg, dYg = t(L.X), t(L.dY)
    Y = L1.csr_spmm_fwd(W, Xg)
    check_fwd(host, L.X, h(Y))
    csc = L1.csc_build(W)
    dX = L1.csr_spmm_bwd_t(W, dYg, csc)
    check_bwd(host, L.K, L.dY, h(dX))
    gv = L1.sddmm_masked_wgrad(W, dYg, Xg)
    gvh = h(gv)[: L.nnz]
    check_sddmm(host, L.dY, L.X, gvh)
    L1.prox_l1_step(L1.PROX_CSR, W, gv, L.eta, L.lam)
    ref = oracle.prox_csr(L.vals, gvh, L.eta, L.lam)
    assert bits_equal(h(W.vals)[: L.nnz], ref)
    C = L1.csr_compact(W)
    rp, ci, v = oracle.compact(L.row_ptr, L.col_idx, ref)
    assert bits_equal(h(C.row_ptr), rp)
    assert bits_equal(h(C.col_idx)[: rp[-1]], ci) and bits_equal(h(C.vals)[: rp[-1]], v)


# ----------------------------------------------------------------------------
# FC 4096 x 4096, batch 512: 20 alternating l1 / debiasing iterations
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("pct", [1, 5, 20, 50])
def test_fc4096_density_sweep_alternating_steps(pct):
    cal = json.load(open(os.path.join(GOLDEN, "fc4096_lambda.json")))
    lam = cal["lambda"][str(pct)]
    L = synth.fc4096_sweep(pct / 100)
    eta, N, K = L.eta, L.N, L.K
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, K, device=cuda())
    host = (L.row_ptr, L.col_idx, L.vals)
    rng = np.random.default_rng(4096 + pct)
    csc = None
    history = []
    for it in range(20):
        X, dY = synth.fc4096_batch(it)
        Xg, dYg = t(X), t(dY)
        rows = rng.choice(N, 32, replace=False)
        cols = rng.choice(K, 32, replace=False)
        if it < 2:  # the first l1 and the first debiasing iteration: every output in full
            rows = cols = None
        if it % 2 == 0:
            # l1 step; the CSC of this pattern was built at the previous (debiasing) step
            csc = L1.csc_build(W) if csc is None else L1.csc_update_vals(W, csc)
            Y = L1.csr_spmm_fwd(W, Xg)
            dX = L1.csr_spmm_bwd_t(W, dYg, csc)
            dW = L1.dense_wgrad(dYg, Xg)
            out = L1.prox_l1_recompress(W, dW, eta, lam)
            dWh = h(dW)
            check_fwd(host, X, h(Y), rows, what=f"Y it{it}")
            check_bwd(host, K, dY, h(dX), cols, what=f"dX it{it}")
            check_dw(dY, X, dWh, rows, what=f"dW it{it}")
            new = check_prox_recompress(host, dWh, eta, lam, K, out)
            if it == 0:
                old = oracle.densify(*host, K) != 0
                flips = np.count_nonzero((oracle.densify(*new, K) != 0) != old)
                assert abs(flips / L.nnz - 0.02) < 0.002, flips / L.nnz
            W, host = out, new
        else:
            # debiasing step on the new pattern: CSC rebuilt, masked gradient, SGD
            csc = L1.csc_build(W)
            nnz = W.host_nnz()
            if it == 1:
                col_ptr, row_idx, perm = csc_reference(host[0], host[1], K)
                assert bits_equal(h(csc.col_ptr), col_ptr) and bits_equal(h(csc.perm)[:nnz], perm)
            Y = L1.csr_spmm_fwd(W, Xg)
            dX = L1.csr_spmm_bwd_t(W, dYg, csc)
            gv = L1.sddmm_masked_wgrad(W, dYg, Xg)
            gvh = h(gv)[:nnz]
            check_fwd(host, X, h(Y), rows, what=f"Y it{it}")
            check_bwd(host, K, dY, h(dX), cols, what=f"dX it{it}")
            check_sddmm(host, dY, X, gvh, rows, what=f"gv it{it}")
            L1.prox_l1_step(L1.PROX_CSR, W, gv, eta, 0.0)
            ref = oracle.prox_csr(host[2], gvh, eta, 0.0)
            assert bits_equal(h(W.vals)[:nnz], ref)
            assert bits_equal(h(W.col_idx)[:nnz], host[1])
            host = (host[0], host[1], ref)
        history.append(int(host[0][-1]))
    # the pattern changes by a few percent per l1 step, not wholesale
    for a, b in zip(history[::2], history[2::2]):
        assert abs(b - a) <= 0.25 * max(a, 1)


@pytest.mark.parametrize("precision", [L1.F32, L1.BF16X3])
def test_graph_replays_match_eager(precision):
    """The l1 step of the 784 -> 300 layer followed by a debiasing step on its
    output, captured once into a HIP graph (torch.cuda.CUDAGraph) and replayed
    three times with eager work and host waits in between: every replay gives
    the eager result bit for bit (all the kernels are deterministic), after
    the outputs were overwritten with garbage.  With the fp32 and the split
    bf16 weight gradient."""
    import torch
    L = synth.fc784_300(seed=0)
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    X, dY = t(L.X), t(L.dY)
    X2 = t(np.flip(L.X, 1).copy())
    Y = torch.empty((L.N, L.B), device=dev)
    dX = torch.empty((L.K, L.B), device=dev)
    dW = torch.empty((L.N, L.K), device=dev)
    gv = torch.empty(L.N * L.K, device=dev)
    csc = L1.CSC.empty(L.K, L.nnz, dev)
    W1 = L1.CSR(L.N, L.K, torch.empty(L.N + 1, dtype=torch.int32, device=dev),
                torch.empty(L.N * L.K, dtype=torch.int32, device=dev),
                torch.empty(L.N * L.K, dtype=torch.float32, device=dev), None)
    def step(x, nnz1=None):
        L1.csr_spmm_fwd(W, x, Y)
        L1.csc_build(W, csc)
        L1.csr_spmm_bwd_t(W, dY, csc, dX)
        L1.dense_wgrad(dY, x, dW, precision=precision)
        L1.prox_l1_recompress(W, dW, L.eta, L.lam, out=W1)
        W1.nnz = nnz1  # None: the binding reads it from the device (a host wait)
        L1.sddmm_masked_wgrad(W1, dY, x, gv)
        L1.prox_l1_step(L1.PROX_CSR, W1, gv, L.eta, 0.0)

    step(X)
    torch.cuda.synchronize()
    n = W1.host_nnz()
    outs = lambda: [Y, dX, dW, W1.row_ptr, W1.col_idx[:n], W1.vals[:n], gv[:n]]
    ref = [o.clone() for o in outs()]

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(X, n)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step(X, n)  # captured with the structure size known: no host wait inside

    for r in range(3):
        step(X2)  # eager work on the same buffers between replays
        torch.cuda.synchronize()
        for o in outs():
            o.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs(), ref):
            assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                               b.view(torch.int32) if b.dtype == torch.float32 else b), r


# ----------------------------------------------------------------------------
# the two-stream step (L1.l1_step) and calls on several streams
# ----------------------------------------------------------------------------

def _step_buffers(L, dev):
    import torch
    return dict(Y=torch.empty((L.N, L.B), device=dev), dX=torch.empty((L.K, L.B), device=dev),
                dW=torch.empty((L.N, L.K), device=dev), csc=L1.CSC.empty(L.K, L.nnz, dev),
                out=L1.CSR(L.N, L.K, torch.empty(L.N + 1, dtype=torch.int32, device=dev),
                           torch.empty(L.N * L.K, dtype=torch.int32, device=dev),
                           torch.empty(L.N * L.K, dtype=torch.float32, device=dev), None))


def _step_outputs(o, nnz_in):
    n = int(o["out"].row_ptr[-1].item())
    c = o["csc"]
    return [o["Y"], o["dX"], o["dW"], c.col_ptr, c.row_idx[:nnz_in], c.perm[:nnz_in], c.vals_t[:nnz_in],
            o["out"].row_ptr, o["out"].col_idx[:n], o["out"].vals[:n]]


def _same_bits(a, b):
    import torch
    as_int = lambda x: x.view(torch.int32) if x.dtype == torch.float32 else x
    return a.shape == b.shape and torch.equal(as_int(a), as_int(b))


@pytest.mark.parametrize("precision", [L1.F32, L1.BF16X3])
@pytest.mark.parametrize("which", ["fc784x300", "fc9216x4096"])
def test_two_stream_step_matches_serial_calls(which, precision):
    """L1.l1_step (CSC build and backward product on a side stream, forced,
    and its automatic choice: two streams for the tiled 9216 -> 4096 products,
    one for the 784 -> 300 layer; the weight update as the fused
    dense_wgrad_prox_recompress) gives the outputs of the unfused calls made
    one after another on one stream, bit for bit (its dense buffer holds Z =
    S_t(W - eta dW)), on four calls in a row with the outputs overwritten in
    between; the serial calls are checked against the oracle by the step
    tests above."""
    import torch
    L = synth.fc784_300(seed=0) if which == "fc784x300" else synth.fc9216_4096(seed=0)
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    X, dY = t(L.X), t(L.dY)
    a, b = _step_buffers(L, dev), _step_buffers(L, dev)
    L1.csr_spmm_fwd(W, X, a["Y"])
    L1.csc_build(W, a["csc"])
    L1.csr_spmm_bwd_t(W, dY, a["csc"], a["dX"])
    L1.dense_wgrad(dY, X, a["dW"], precision=precision)
    L1.prox_l1_recompress(W, a["dW"], L.eta, L.lam, out=a["out"])
    L1.prox_l1_step(L1.PROX_DENSE, W, a["dW"], L.eta, L.lam, Z=a["dW"])  # the step leaves Z in dW
    ref = _step_outputs(a, L.nnz)
    for r, schedule in enumerate(("two_stream", "auto", "two_stream", "serial")):
        for x in (b["Y"], b["dX"], b["dW"], b["out"].vals, b["csc"].vals_t):
            x.fill_(-7)
        got = L1.l1_step(W, X, dY, L.eta, L.lam, Y=b["Y"], dX=b["dX"], dW=b["dW"], csc=b["csc"],
                         out=b["out"], precision=precision, schedule=schedule)
        assert got is b["out"]
        for i, (x, y) in enumerate(zip(_step_outputs(b, L.nnz), ref)):
            assert _same_bits(x, y), (r, i)
    torch.cuda.synchronize()


def test_two_stream_step_graph_replays_match_eager():
    """L1.l1_step on two streams captured into a HIP graph (the side stream forked from and
    joined to the capture stream) and replayed three times, with eager steps
    on other inputs and garbage written to the outputs in between: every
    replay gives the eager result bit for bit."""
    import torch
    L = synth.fc784_300(seed=0)
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    X, dY = t(L.X), t(L.dY)
    X2 = t(np.flip(L.X, 1).copy())
    o = _step_buffers(L, dev)
    run = lambda x: L1.l1_step(W, x, dY, L.eta, L.lam, Y=o["Y"], dX=o["dX"], dW=o["dW"], csc=o["csc"],
                               out=o["out"], schedule="two_stream")
    run(X)
    torch.cuda.synchronize()
    ref = [x.clone() for x in _step_outputs(o, L.nnz)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(X)
    for r in range(3):
        run(X2)
        torch.cuda.synchronize()
        for x in (o["Y"], o["dX"], o["dW"], o["out"].vals, o["csc"].vals_t):
            x.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        for i, (x, y) in enumerate(zip(_step_outputs(o, L.nnz), ref)):
            assert _same_bits(x, y), (r, i)


def test_calls_on_two_streams_use_separate_workspaces():
    """Tiled forward products (plan, pair stream and partial rows in the
    call's workspace) issued alternately on two streams with no wait between
    them: each stream's calls use their own workspace, so every result equals
    the one-stream result bit for bit."""
    import torch
    L = synth.fc9216_4096(seed=0)
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    assert L1.workspace_bytes(L1.OP_SPMM, L.N, L.K, L.nnz, L.B) > 0  # the tiled path
    rng = np.random.default_rng(5)
    Xs = [t(L.X), t(rng.standard_normal(L.X.shape).astype(np.float32))]
    ref = [L1.csr_spmm_fwd(W, x) for x in Xs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[torch.full_like(ref[0], -7.0) for _ in range(3)] for _ in range(2)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for r in range(3):
        for i in range(2):
            L1.csr_spmm_fwd(W, Xs[i], outs[i][r], stream=streams[i])
    for s in streams:
        torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for i in range(2):
        for r in range(3):
            assert _same_bits(outs[i][r], ref[i]), (i, r)


def test_l1_step_schedule_choice():
    """"auto" forks only where a product takes the tiled path, and a bad
    schedule name is rejected before anything is enqueued."""
    from paper_1905_07931_amd.step import two_stream_pays
    dev = cuda()
    small, big = synth.fc784_300(seed=0), synth.fc9216_4096(seed=0)
    Ws = L1.CSR.from_host(small.row_ptr, small.col_idx, small.vals, small.K, device=dev)
    Wb = L1.CSR.from_host(big.row_ptr, big.col_idx, big.vals, big.K, device=dev)
    assert not two_stream_pays(Ws, small.B)
    assert two_stream_pays(Wb, big.B)
    o = _step_buffers(small, dev)
    with pytest.raises(ValueError):
        L1.l1_step(Ws, t(small.X), t(small.dY), small.eta, small.lam, Y=o["Y"], dX=o["dX"], dW=o["dW"],
                   csc=o["csc"], out=o["out"], schedule="parallel")


@pytest.mark.parametrize("solver", [L1.SOLVER_ADAM, L1.SOLVER_RMSPROP])
@pytest.mark.parametrize("which,schedule", [("fc784x300", "two_stream"), ("fc9216x4096", "auto")])
def test_two_stream_adaptive_step_matches_serial_calls(which, schedule, solver):
    """L1.l1_step with a Prox-ADAM / Prox-RMSProp state (Algorithms 1-2) on two
    streams gives, over two carried steps, the outputs, the state m, v and the
    step counter of the same calls made one after another on one stream, bit
    for bit (the adaptive calls are checked against the oracle in their own
    tests)."""
    import torch
    L = synth.fc784_300(seed=0) if which == "fc784x300" else synth.fc9216_4096(seed=0)
    dev = cuda()
    W = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=dev)
    X, dY = t(L.X), t(L.dY)
    a, b = _step_buffers(L, dev), _step_buffers(L, dev)
    sa = L1.AdaptiveState.zeros(solver, (L.N, L.K), dev)
    sb = L1.AdaptiveState.zeros(solver, (L.N, L.K), dev)
    eta = 1e-3
    for r in range(2):
        L1.csr_spmm_fwd(W, X, a["Y"])
        L1.csc_build(W, a["csc"])
        L1.csr_spmm_bwd_t(W, dY, a["csc"], a["dX"])
        L1.dense_wgrad(dY, X, a["dW"])
        L1.prox_adaptive_recompress(W, a["dW"], sa, eta, L.lam, out=a["out"])
        for x in (b["Y"], b["dX"], b["dW"], b["out"].vals):
            x.fill_(-7)
        L1.l1_step(W, X, dY, eta, L.lam, Y=b["Y"], dX=b["dX"], dW=b["dW"], csc=b["csc"], out=b["out"],
                   schedule=schedule, adaptive=sb)
        for i, (x, y) in enumerate(zip(_step_outputs(b, L.nnz), _step_outputs(a, L.nnz))):
            assert _same_bits(x, y), (r, i)
        assert _same_bits(sb.v, sa.v), r
        if solver == L1.SOLVER_ADAM:
            assert _same_bits(sb.m, sa.m), r
        assert sb.t == sa.t == r + 2
    torch.cuda.synchronize()


@pytest.mark.parametrize("which", ["fc784x300", "fc4096_d5"])
def test_l1_step_loop_carries_W_forward(which):
    """A training loop feeds each step's new CSR back in as the next W
    (ping-pong buffers) without ever setting nnz itself.  Each output's count
    is queued to pinned host memory behind the call that wrote it, and the
    next step takes it from there (a wait on that copy alone), so products,
    CSC and plans are sized for the stored entries, never for the N*K
    capacity.  Three steps through l1_step (auto schedule) equal the same
    calls made one after another on one stream, bit for bit."""
    import torch
    dev = cuda()
    if which == "fc784x300":
        L = synth.fc784_300(seed=0)
        lam = L.lam
        batches = [(L.X, L.dY)] * 3
    else:
        L = synth.fc4096_sweep(0.05)
        lam = json.load(open(os.path.join(GOLDEN, "fc4096_lambda.json")))["lambda"]["5"]
        batches = [synth.fc4096_batch(2 * it) for it in range(3)]
    N, K, eta = L.N, L.K, L.eta
    Wa = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, K, device=dev)
    Wb = L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, K, device=dev)
    bufs_a = [_step_buffers(L, dev)["out"] for _ in range(2)]
    bufs_b = [_step_buffers(L, dev)["out"] for _ in range(2)]
    Y, dX = torch.empty((N, L.B), device=dev), torch.empty((K, L.B), device=dev)
    Yb, dXb = torch.empty_like(Y), torch.empty_like(dX)
    dW, dWb = torch.empty((N, K), device=dev), torch.empty((N, K), device=dev)
    csc_a, csc_b = L1.CSC.empty(K, N * K, dev), L1.CSC.empty(K, N * K, dev)
    for it, (Xh, dYh) in enumerate(batches):
        X, dY = t(Xh), t(dYh)
        if it > 0:
            assert Wb.nnz is None and Wb._pending is not None  # count still on its way to the host
        outa, outb = bufs_a[it % 2], bufs_b[it % 2]
        L1.csr_spmm_fwd(Wa, X, Y)
        L1.csc_build(Wa, csc_a)
        L1.csr_spmm_bwd_t(Wa, dY, csc_a, dX)
        L1.dense_wgrad(dY, X, dW)
        L1.prox_l1_recompress(Wa, dW, eta, lam, out=outa)
        L1.prox_l1_step(L1.PROX_DENSE, Wa, dW, eta, lam, Z=dW)  # as the step leaves its dense buffer
        L1.l1_step(Wb, X, dY, eta, lam, Y=Yb, dX=dXb, dW=dWb, csc=csc_b, out=outb, schedule="auto")
        n_in = Wb.host_nnz()
        assert n_in == int(Wb.row_ptr[-1].item())
        n = outb.host_nnz()
        assert n == outa.host_nnz() == int(outb.row_ptr[-1].item())
        for x, y in ((Yb, Y), (dXb, dX), (dWb, dW), (outb.row_ptr, outa.row_ptr),
                     (outb.col_idx[:n], outa.col_idx[:n]), (outb.vals[:n], outa.vals[:n]),
                     (csc_b.col_ptr, csc_a.col_ptr), (csc_b.row_idx[:n_in], csc_a.row_idx[:n_in])):
            assert _same_bits(x, y), it
        outb.nnz = None  # as the step left it: the count comes from the queued copy
        outb.track_nnz()
        Wa, Wb = outa, outb
    torch.cuda.synchronize()
    # the backward plans of steps with different nnz share one buffer per side stream
    from paper_1905_07931_amd import step as step_mod
    side = step_mod.side_stream(dev)
    assert sum(1 for k in step_mod._plans if k[0] == side.cuda_stream) <= 1
