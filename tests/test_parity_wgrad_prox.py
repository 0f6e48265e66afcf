"""The fused l1 update dense_wgrad_prox_recompress on the GPU.

Z = S_t(W - eta * dY.X^T) (Eq. (prox) with the minibatch gradient, the
closed form of Section 2.2) and W' = CSR(Z) (Section 3.1) must equal, bit for
bit:
  - the unfused calls dense_wgrad (same precision) + prox_l1_step (dense
    mode) + prox_l1_recompress, and
  - the oracle's prox and recompression applied to that dense_wgrad result
    (the products themselves are checked against the oracle by the
    dense_wgrad tests; on the dyadic grid the whole update is compared with
    the fully independent oracle step).
Shapes cover both GEMM tile shapes (256 x 288 and 128 x 128), ragged tiles in
both dimensions, the split-reduction and bf16-operand fallbacks, empty
layers, rows and batches, and the capacity paths.
"""
import numpy as np
import pytest

import oracle
import paper_1905_07931_amd as L1
from paper_1905_07931_amd import synth

from _helpers import bits_equal, cuda, h, t

pytestmark = pytest.mark.gpu


def _W(L):
    return L1.CSR.from_host(L.row_ptr, L.col_idx, L.vals, L.K, device=cuda())


def _fused_vs_unfused(L, precision, lam=None, eta=None):
    import torch
    lam = L.lam if lam is None else lam
    eta = L.eta if eta is None else eta
    W = _W(L)
    X, dY = t(L.X), t(L.dY)
    Z, out = L1.dense_wgrad_prox_recompress(W, dY, X, eta, lam, precision=precision)
    dW = L1.dense_wgrad(dY, X, precision=precision)
    dWh = h(dW)
    ref_out = L1.prox_l1_recompress(W, dW, eta, lam)
    Zr = L1.prox_l1_step(L1.PROX_DENSE, W, dW.clone(), eta, lam)
    torch.cuda.synchronize()
    assert bits_equal(h(Z), h(Zr)), "Z vs prox_l1_step"
    n = out.host_nnz()
    assert n == ref_out.host_nnz()
    assert bits_equal(h(out.row_ptr), h(ref_out.row_ptr)), "row_ptr"
    assert bits_equal(h(out.col_idx)[:n], h(ref_out.col_idx)[:n]), "col_idx"
    assert bits_equal(h(out.vals)[:n], h(ref_out.vals)[:n]), "vals"
    # and the oracle's prox + recompression of the same gradient
    Zo, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, dWh, eta, lam, L.K)
    assert bits_equal(h(Z), Zo), "Z vs oracle"
    rp, ci, v = oracle.recompress(Zo)
    assert int(rp[-1]) == n
    assert bits_equal(h(out.row_ptr), rp) and bits_equal(h(out.col_idx)[:n], ci) and bits_equal(h(out.vals)[:n], v)
    return n


SHAPES = [  # (N, K, B, nnz, seed): tile shapes and ragged edges
    (300, 784, 64, 23520, 0),        # the 784 -> 300 layer
    (1000, 1000, 100, 90000, 1),     # ragged 128- and 288-wide tiles
    (257, 10999, 37, 200000, 2),     # ragged rows, many column tiles
    (64, 33, 5, 300, 3),             # narrower than one 32-column word
    (1, 1, 1, 1, 4), (1, 700, 3, 10, 5), (700, 1, 3, 10, 6),
    (130, 257, 65, 0, 7),            # empty layer: only regrowth
]


def _ids(s):
    return "N{}K{}B{}nnz{}".format(*s[:4])


@pytest.mark.parametrize("precision", [L1.F32, L1.BF16X3, L1.BF16])
@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
def test_fused_update_equals_unfused_calls(shape, precision):
    N, K, B, nnz, seed = shape
    L = synth.fc_layer(N, K, B, nnz, seed=seed)
    _fused_vs_unfused(L, precision)


@pytest.mark.parametrize("precision", [L1.F32, L1.BF16X3])
def test_fused_update_full_size_9216x4096(precision):
    # the 256 x 288 tiles (two rounds of the chip), Zipf rows; a lambda that
    # deletes part of the layer as well as regrowing it
    L = synth.fc9216_4096(seed=0)
    n = _fused_vs_unfused(L, precision, lam=0.5)
    assert 0 < n < L.N * L.K


def test_fused_update_direct_load_tiles_with_ragged_edges():
    # 4036 x 9116 at batch 64: the 256 x 288 direct-load tiles (512 of them,
    # two rounds), the last row block 196 rows high and the last column block
    # 188 wide, so the epilogue's row and column bounds and its double-buffered
    # gathers meet partial tiles
    L = synth.fc_layer(4036, 9116, 64, synth.nnz_for(4036, 9116, 0.09), seed=14)
    n = _fused_vs_unfused(L, L1.F32, lam=0.5)
    assert 0 < n < L.N * L.K


def test_fused_update_split_reduction_fallback():
    # 50 x 500 with a reduction of 16384: the fp32 product splits its batch
    # (no fused epilogue there), so dW goes through Z and the prox runs after
    L = synth.conv2_im2col(seed=0)
    _fused_vs_unfused(L, L1.F32)


def test_fused_update_dyadic_full_size_bit_exact_with_independent_oracle():
    # every fp32 sum of dW is exact on the dyadic grid, so the update must
    # equal the fully independent oracle step (its own dW) bit for bit
    import torch
    L = synth.dyadic_layer(4096, 9216, 1024, synth.nnz_for(4096, 9216, 0.09), seed=1, pattern="zipf")
    W = _W(L)
    Z, out = L1.dense_wgrad_prox_recompress(W, t(L.dY), t(L.X), L.eta, L.lam)
    torch.cuda.synchronize()
    dWr = oracle.dense_wgrad(L.dY, L.X)
    Zo, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, dWr, L.eta, L.lam, L.K)
    assert bits_equal(h(Z), Zo)
    rp, ci, v = oracle.recompress(Zo)
    n = int(rp[-1])
    assert 0 < n < L.N * L.K  # the grid makes exact ties |z| == t, deleted
    assert bits_equal(h(out.row_ptr), rp) and bits_equal(h(out.col_idx)[:n], ci) and bits_equal(h(out.vals)[:n], v)


def test_fused_update_empty_batch_and_huge_threshold():
    # B = 0: dW = 0, so Z = S_t(W) (stored weights shrink by t); then a
    # threshold above every |w - eta g| deletes the whole layer
    L = synth.fc_layer(300, 784, 0, 23520, seed=8)
    _fused_vs_unfused(L, L1.F32)
    L2 = synth.fc_layer(300, 784, 16, 23520, seed=9)
    assert _fused_vs_unfused(L2, L1.F32, lam=1e6) == 0


def test_fused_update_capacity_paths():
    import torch
    L = synth.fc_layer(200, 300, 32, 6000, seed=10)
    W = _W(L)
    X, dY = t(L.X), t(L.dY)
    Z, full = L1.dense_wgrad_prox_recompress(W, dY, X, L.eta, 0.05)
    n = full.host_nnz()
    assert 0 < n < L.N * L.K
    # exactly enough room: the call waits, fills and reports the count on the host
    Z2, exact = L1.dense_wgrad_prox_recompress(W, dY, X, L.eta, 0.05, capacity=n)
    assert exact.nnz == n
    assert bits_equal(h(exact.row_ptr), h(full.row_ptr)) and bits_equal(h(exact.vals)[:n], h(full.vals)[:n])
    # one short: L1CSR_ECAPACITY, row pointers valid, nothing else written
    out = L1.CSR(L.N, L.K, torch.empty(L.N + 1, dtype=torch.int32, device=cuda()),
                 torch.full((n - 1,), -7, dtype=torch.int32, device=cuda()),
                 torch.full((n - 1,), -7.0, dtype=torch.float32, device=cuda()), None)
    with pytest.raises(L1.L1CSRError) as ei:
        L1.dense_wgrad_prox_recompress(W, dY, X, L.eta, 0.05, out=out, capacity=n - 1)
    assert ei.value.status == L1.ECAPACITY
    torch.cuda.synchronize()
    assert bits_equal(h(out.row_ptr), h(full.row_ptr))
    assert bool((out.col_idx == -7).all()) and bool((out.vals == -7.0).all())


@pytest.mark.parametrize("N", [64, 4097, 16384, 16385])
def test_counted_recompress_row_prefix_paths(N):
    # each row's start is added up inside the compaction (up to 256 blocks of
    # 16, 32 or 64 rows, capacity >= N * K) or written by a scan first (more
    # rows than 256 blocks of 64 hold, or a smaller capacity whose check needs
    # nnz' on the host): the same CSR as the oracle's recompression on every
    # path, nnz' in d_nnz_out
    import ctypes as C
    import torch
    rng = np.random.default_rng(N)
    K = 40
    Zh = np.where(rng.random((N, K)) < 0.3, rng.standard_normal((N, K)), 0.0).astype(np.float32)
    Zh[::7] = 0.0  # empty rows, also the first
    Zh[-1] = np.where(np.arange(K) % 3 == 0, 1.5, 0.0)  # the last row's entries close the count
    kw = (K + 31) // 32
    pad = np.zeros((N, kw * 32), bool)
    pad[:, :K] = Zh != 0
    wc = t(pad.reshape(N, kw, 32).sum(2).astype(np.int32))
    Z = t(Zh)
    rp, ci, v = oracle.recompress(Zh)
    n = int(rp[-1])
    ws = torch.empty(L1.workspace_bytes(L1.OP_RECOMPRESS, N, K, 0, 0), dtype=torch.uint8, device=cuda())
    for cap in (N * K, n):
        rpo = torch.full((N + 1,), -3, dtype=torch.int32, device=cuda())
        cio = torch.full((cap,), -3, dtype=torch.int32, device=cuda())
        vo = torch.full((cap,), -3.0, dtype=torch.float32, device=cuda())
        dn = torch.full((1,), -3, dtype=torch.int32, device=cuda())
        hw = L1._words.acquire()  # and a word of mapped host memory the kernels write
        assert hw is not None
        C.c_int32.from_address(hw.host).value = -3
        for sink in (L1._p(dn), C.c_void_p(hw.dev)):
            need = C.c_int64(-5)
            st = L1.lib().csr_recompress_counted(N, K, L1._p(Z), K, L1._p(wc), L1._p(rpo), L1._p(cio), L1._p(vo),
                                                 cap, sink, C.byref(need), L1._p(ws), ws.numel(), L1._stream())
            torch.cuda.synchronize()
            assert st == 0, (cap, st)
            assert need.value == (-1 if cap >= N * K else n)
        assert int(h(dn)[0]) == n and hw.value() == n
        L1._words.release(hw)
        assert bits_equal(h(rpo), rp), cap
        assert bits_equal(h(cio)[:n], ci) and bits_equal(h(vo)[:n], v), cap
        if cap > n:
            assert bool((cio[n:] == -3).all()) and bool((vo[n:] == -3.0).all())


def test_counts_reach_the_host_through_mapped_words():
    # a call at full capacity leaves nnz' in pinned host memory written by its
    # own kernels (no copy queued behind it); the word stays with its CSR and
    # later calls into the same CSR overwrite it in stream order; when the CSR
    # goes, the word is handed out again only after its last write is done
    import gc
    import torch
    L = synth.fc_layer(257, 1000, 70, 30000, seed=13)
    W = _W(L)
    bm = L1.csr_bitmap_build(W)
    out = None
    for lam in (0.02, 0.5, 0.0, 1e6):
        Z, wc = L1.dense_wgrad_prox(W, t(L.dY), t(L.X), L.eta, lam, bm)
        out = L1.csr_recompress_counted(Z, wc, out=out)
        assert out.nnz is None and isinstance(out._pending[0], L1._HostWord)
        n = out.host_nnz()
        assert n == int(out.row_ptr[-1].item()) == int((h(Z) != 0).sum())
        assert out._pending is None and out.nnz == n
    assert n == 0  # the last threshold deletes every weight
    w = out._word
    del out
    gc.collect()
    assert w in L1._words.free
    torch.cuda.synchronize()
    again = [L1._words.acquire() for _ in range(len(L1._words.free))]
    assert w in again  # its event has completed
    for x in again:
        L1._words.release(x)


def test_word_of_a_call_with_a_host_count_waits_for_its_kernels():
    # a call that returns nnz' on the host (a capacity below N*K) still hands
    # its kernels the CSR's host word: the word gets an event behind the call,
    # so the pool cannot give it to another CSR while that write is queued
    import torch
    rng = np.random.default_rng(14)
    Zh = (rng.standard_normal((64, 300)) * (rng.random((64, 300)) < 0.3)).astype(np.float32)
    out = L1.csr_recompress(t(Zh), capacity=64 * 300 - 1)
    assert out.nnz == int((Zh != 0).sum())
    w = getattr(out, "_word", None)
    if w is None:
        pytest.skip("no mapped host memory on this runtime")
    assert w.event is not None
    torch.cuda.synchronize()
    assert w.event.query()


def test_counts_fall_back_to_a_queued_copy_without_mapped_memory(monkeypatch):
    # where the runtime gives no mapped host memory, the binding queues a
    # copy of row_ptr[-1] behind the call instead: the same counts
    import torch
    words = L1._HostWords()
    words.disabled = True
    monkeypatch.setattr(L1, "_words", words)
    L = synth.fc_layer(257, 1000, 70, 30000, seed=13)
    W = _W(L)
    Z, wc = L1.dense_wgrad_prox(W, t(L.dY), t(L.X), L.eta, 0.02, L1.csr_bitmap_build(W))
    out = L1.csr_recompress_counted(Z, wc)
    assert getattr(out, "_word", None) is None and out.nnz is None
    assert not isinstance(out._pending[0], L1._HostWord)
    torch.cuda.synchronize()
    assert out.host_nnz() == int(out.row_ptr[-1].item()) == int((h(Z) != 0).sum())


def test_fused_update_padded_leading_dimensions():
    import torch
    L = synth.fc_layer(130, 300, 40, 4000, seed=11)
    W = _W(L)
    dev = cuda()
    Xp = torch.zeros((L.K, 44), device=dev)
    Xp[:, :40] = t(L.X)
    dYp = torch.zeros((L.N, 48), device=dev)
    dYp[:, :40] = t(L.dY)
    Zp = torch.full((L.N, 304), 5.0, device=dev)
    Z, out = L1.dense_wgrad_prox_recompress(W, dYp[:, :40], Xp[:, :40], L.eta, L.lam, Z=Zp[:, :300])
    Zr, ref = L1.dense_wgrad_prox_recompress(W, t(L.dY), t(L.X), L.eta, L.lam)
    torch.cuda.synchronize()
    assert bits_equal(h(Zp)[:, :300], h(Zr)) and np.all(h(Zp)[:, 300:] == 5.0)
    n = ref.host_nnz()
    assert out.host_nnz() == n and bits_equal(h(out.col_idx)[:n], h(ref.col_idx)[:n])


def _bitmap_reference(row_ptr, col_idx, N, K):
    """mask[i][w] bit c = (i, 32w + c) stored; pos[i][w] = first CSR position
    of row i with column >= 32w (numpy: bit arithmetic and a sorted search)."""
    kw = (K + 31) // 32
    rp = np.asarray(row_ptr, np.int64)
    ci = np.asarray(col_idx, np.int64)
    rows = np.repeat(np.arange(N), np.diff(rp))
    mask = np.zeros((N, kw), np.uint64)
    np.bitwise_or.at(mask, (rows, ci >> 5), np.left_shift(np.uint64(1), (ci & 31).astype(np.uint64)))
    pos = np.empty((N, kw), np.int64)
    for i in range(N):
        seg = ci[rp[i]:rp[i + 1]]
        pos[i] = rp[i] + np.searchsorted(seg, 32 * np.arange(kw), side="left")
    return mask.astype(np.uint32).view(np.int32), pos.astype(np.int32)


@pytest.mark.parametrize("case", ["zipf", "banded", "narrow", "empty_rows", "wide", "block_edge"])
def test_bitmap_index_bit_exact(case):
    # long rows cross the 512-entry spans of the build (words straddling a
    # span boundary), dense rows fill every word, empty rows and columns that
    # are not a multiple of 32; up to 320 words a row block is built in LDS
    # (a partial last block of 16 rows), wider rows go word by word to memory
    rng = np.random.default_rng(61)
    if case == "zipf":
        N, K = 700, 9216
        rp, ci = synth.zipf_pattern(rng, N, K, 600000, 1.1)
    elif case == "banded":
        N, K = 300, 2000
        dense = np.zeros((N, K), bool)
        dense[:, 500:1700] = rng.random((N, 1200)) < 0.7
        dense[[3, 77], :] = True
        rp, ci = synth.pattern_from_positions(N, K, np.flatnonzero(dense.reshape(-1)))
    elif case == "narrow":
        N, K = 1000, 45
        rp, ci = synth.uniform_pattern(rng, N, K, 20000)
    elif case == "wide":
        N, K = 90, 20000  # 625 words: past the LDS block
        rp, ci = synth.zipf_pattern(rng, N, K, 150000, 1.1)
    elif case == "block_edge":
        N, K = 33, 10240  # 320 words: the LDS block's limit; 33 rows: two full blocks and one row
        dense = rng.random((N, K)) < 0.05
        dense[[0, 31, 32], :] = True
        dense[5] = False
        rp, ci = synth.pattern_from_positions(N, K, np.flatnonzero(dense.reshape(-1)))
    else:
        N, K = 200, 1001
        dense = rng.random((N, K)) < 0.3
        dense[::3] = False
        rp, ci = synth.pattern_from_positions(N, K, np.flatnonzero(dense.reshape(-1)))
    vals = np.ones(len(ci), np.float32)
    W = L1.CSR.from_host(rp, ci, vals, K, device=cuda())
    bm = L1.csr_bitmap_build(W)
    mask, pos = _bitmap_reference(rp, ci, N, K)
    kw = (K + 31) // 32  # word-major on the device: [kw][N]
    assert bits_equal(np.ascontiguousarray(h(bm.mask).reshape(-1)[: N * kw].reshape(kw, N).T), mask)
    assert bits_equal(np.ascontiguousarray(h(bm.pos).reshape(-1)[: N * kw].reshape(kw, N).T), pos)


def test_fused_update_with_prebuilt_bitmap():
    # the bitmap built by the caller (as l1_step does on its side stream)
    # gives the same result as the one the call builds itself
    import torch
    L = synth.fc_layer(1000, 1000, 100, 90000, seed=12)
    W = _W(L)
    bm = L1.csr_bitmap_build(W)
    Z1, o1 = L1.dense_wgrad_prox_recompress(W, t(L.dY), t(L.X), L.eta, L.lam, bitmap=bm)
    Z2, o2 = L1.dense_wgrad_prox_recompress(W, t(L.dY), t(L.X), L.eta, L.lam)
    torch.cuda.synchronize()
    n = o2.host_nnz()
    assert bits_equal(h(Z1), h(Z2)) and o1.host_nnz() == n
    assert bits_equal(h(o1.col_idx)[:n], h(o2.col_idx)[:n]) and bits_equal(h(o1.vals)[:n], h(o2.vals)[:n])


@pytest.mark.parametrize("precision", [L1.F32, L1.BF16X3, L1.BF16])
def test_word_counts_and_counted_recompress(precision):
    # the two calls the step makes: dense_wgrad_prox's per-word counts are the
    # nonzeros of Z per 32 columns, and csr_recompress_counted gives the
    # canonical CSR of Z (as csr_recompress with t = 0)
    import torch
    L = synth.fc_layer(257, 1000, 70, 30000, seed=13)
    W = _W(L)
    bm = L1.csr_bitmap_build(W)
    Z, wc = L1.dense_wgrad_prox(W, t(L.dY), t(L.X), L.eta, 0.02, bm, precision=precision)
    out = L1.csr_recompress_counted(Z, wc)
    ref = L1.csr_recompress(Z.clone(), 0.0)
    torch.cuda.synchronize()
    Zh = h(Z)
    kw = (L.K + 31) // 32
    pad = np.zeros((L.N, kw * 32), bool)
    pad[:, :L.K] = Zh != 0
    assert bits_equal(h(wc).reshape(-1)[: L.N * kw].reshape(L.N, kw), pad.reshape(L.N, kw, 32).sum(2).astype(np.int32))
    n = ref.host_nnz()
    assert out.host_nnz() == n and 0 < n < L.N * L.K
    assert bits_equal(h(out.row_ptr), h(ref.row_ptr))
    assert bits_equal(h(out.col_idx)[:n], h(ref.col_idx)[:n]) and bits_equal(h(out.vals)[:n], h(ref.vals)[:n])
