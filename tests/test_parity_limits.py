"""The largest layer the int32 CSR layout holds: N = K = 46340, so a full
result has N*K = 2,147,395,600 entries, just below 2^31.  Row pointers and
output positions then come within 0.01 % of the int32 range; the whole row
pointer array and the entries at both ends of the output (positions near 0
and near 2^31) are checked exactly.  About 26 GB of device memory each."""
import numpy as np
import pytest

import oracle
import paper_1905_07931_amd as L1

from _helpers import cuda, h

pytestmark = pytest.mark.gpu

N = K = 46340
ZEROS = [(0, 0), (1, K - 1), (N // 2, 123), (N - 1, K - 1)]


def _expected_row_ptr():
    cnt = np.full(N, K, np.int64)
    for i, _ in ZEROS:
        cnt[i] -= 1
    return np.concatenate([[0], np.cumsum(cnt)])


def _check_structure(out, val):
    rp = h(out.row_ptr).astype(np.int64)
    exp = _expected_row_ptr()
    assert np.array_equal(rp, exp)
    assert rp[-1] == N * K - len(ZEROS) and rp[-1] < 2 ** 31
    for i, k0 in ZEROS:
        ci = h(out.col_idx[int(rp[i]):int(rp[i + 1])])
        assert np.array_equal(ci, np.delete(np.arange(K, dtype=np.int32), k0)), i
        assert np.all(h(out.vals[int(rp[i]):int(rp[i + 1])]) == val), i
    # a full row in the middle of the array
    i = N // 3
    assert np.array_equal(h(out.col_idx[int(rp[i]):int(rp[i + 1])]), np.arange(K, dtype=np.int32))


def test_recompress_at_the_int32_limit():
    import torch
    Z = torch.full((N, K), 0.5, device=cuda())
    for i, k in ZEROS:
        Z[i, k] = 0.0
    out = L1.csr_recompress(Z)
    torch.cuda.synchronize()
    del Z
    _check_structure(out, np.float32(0.5))
    del out
    torch.cuda.empty_cache()


def test_prox_recompress_at_the_int32_limit():
    # an empty W and G = -1 everywhere: z = eta, kept with value S_t(eta), t = eta*lam;
    # G = 0 at the chosen positions gives z = 0 there, dropped
    import torch
    eta, lam = 0.01, 0.5
    W = L1.CSR.from_host(np.zeros(N + 1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), K,
                         device=cuda())
    G = torch.full((N, K), -1.0, device=cuda())
    for i, k in ZEROS:
        G[i, k] = 0.0
    out = L1.prox_l1_recompress(W, G, eta, lam)
    torch.cuda.synchronize()
    del G
    Zr, _ = oracle.prox_dense(np.zeros(2, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32),
                              np.full((1, 1), -1.0, np.float32), eta, lam, 1)
    _check_structure(out, Zr[0, 0])
    del out
    torch.cuda.empty_cache()
