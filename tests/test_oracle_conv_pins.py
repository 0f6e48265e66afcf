"""Pins of the oracle's convolution layers (CPU only).

The convolution with CSR filters, its adjoint, the im2col lowering and max
pooling are checked against things other than themselves: scipy's 2-D
cross-correlation (single and multi channel, padding and stride through an
explicitly padded input and slicing), a hand-written im2col of a 3 x 3 map, the
adjoint identity <dY, conv(X)> = <conv_T(dY), X>, delta filters that shift
the map, and numpy's window maxima.
"""
import numpy as np
import pytest
from scipy.signal import correlate2d

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def dense_to_csr(Wd):
    """CSR of a dense [N][K] filter bank (zeros not stored)."""
    N, K = Wd.shape
    rp = np.zeros(N + 1, np.int32)
    ci, v = [], []
    for i in range(N):
        nz = np.nonzero(Wd[i])[0]
        ci.extend(nz.tolist())
        v.extend(Wd[i, nz].tolist())
        rp[i + 1] = len(ci)
    return rp, np.array(ci, np.int32), np.array(v, np.float32)


def maps(rng, C, H, Wd, B):
    return rng.standard_normal((C * H * Wd, B)).astype(np.float32)


def to_nchw(X, C, H, Wd):
    """[C*H*W][B] -> [B][C][H][W] (a view change only)."""
    return np.ascontiguousarray(X.T.reshape(-1, C, H, Wd))


@pytest.mark.parametrize("C,N,H,Wd,KH,KW", [(1, 1, 7, 9, 3, 2), (3, 4, 12, 12, 5, 5), (20, 2, 12, 12, 5, 5)])
def test_conv_fwd_equals_scipy_correlate2d(C, N, H, Wd, KH, KW):
    rng = np.random.default_rng(C * 100 + N)
    B = 3
    Wdn = rng.standard_normal((N, C * KH * KW)).astype(np.float32)
    Wdn[rng.random(Wdn.shape) < 0.6] = 0.0
    X = maps(rng, C, H, Wd, B)
    Y = oracle.conv_fwd(*dense_to_csr(Wdn), X, C, H, Wd, KH, KW)
    OH, OW = H - KH + 1, Wd - KW + 1
    Xb = to_nchw(X, C, H, Wd).astype(np.float64)
    k = Wdn.astype(np.float64).reshape(N, C, KH, KW)
    for b in range(B):
        for co in range(N):
            ref = sum(correlate2d(Xb[b, ci], k[co, ci], mode="valid") for ci in range(C))
            got = Y[:, b].reshape(N, OH, OW)[co]
            np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("SH,SW,PH,PW", [(2, 2, 1, 1), (1, 2, 2, 0), (3, 1, 0, 2)])
def test_conv_fwd_stride_and_padding_equal_padded_correlation_sliced(SH, SW, PH, PW):
    rng = np.random.default_rng(SH * 10 + PH)
    C, N, H, Wd, KH, KW, B = 2, 3, 9, 8, 3, 4, 2
    Wdn = rng.standard_normal((N, C * KH * KW)).astype(np.float32)
    X = maps(rng, C, H, Wd, B)
    Y = oracle.conv_fwd(*dense_to_csr(Wdn), X, C, H, Wd, KH, KW, SH, SW, PH, PW)
    OH, OW = oracle.conv_out_size(H, Wd, KH, KW, SH, SW, PH, PW)
    Xb = np.pad(to_nchw(X, C, H, Wd).astype(np.float64), ((0, 0), (0, 0), (PH, PH), (PW, PW)))
    k = Wdn.astype(np.float64).reshape(N, C, KH, KW)
    for b in range(B):
        for co in range(N):
            full = sum(correlate2d(Xb[b, ci], k[co, ci], mode="valid") for ci in range(C))
            ref = full[::SH, ::SW][:OH, :OW]
            np.testing.assert_allclose(Y[:, b].reshape(N, OH, OW)[co], ref, rtol=1e-5, atol=1e-5)


def test_im2col_of_a_3x3_map_by_hand():
    # one channel, maps 1..9 (row-major), 2 x 2 windows, stride 1: the four
    # windows in (oh, ow) order, batch of one
    X = np.arange(1, 10, dtype=np.float32).reshape(9, 1)
    Xc = oracle.im2col(X, 1, 3, 3, 2, 2)
    expect = np.array([[1, 2, 4, 5],    # (kh, kw) = (0, 0)
                       [2, 3, 5, 6],    # (0, 1)
                       [4, 5, 7, 8],    # (1, 0)
                       [5, 6, 8, 9]],   # (1, 1)
                      np.float32)
    assert np.array_equal(Xc, expect)
    # padding 1: the corner window sees zeros above and to the left
    Xp = oracle.im2col(X, 1, 3, 3, 2, 2, 1, 1, 1, 1)
    assert Xp.shape == (4, 16)
    assert np.array_equal(Xp[:, 0], np.array([0, 0, 0, 1], np.float32))
    # batch-contiguous columns: each column block of B copies the B samples
    X2 = np.stack([np.arange(9), 100 + np.arange(9)], axis=1).astype(np.float32)
    Xc2 = oracle.im2col(X2, 1, 3, 3, 2, 2)
    assert np.array_equal(Xc2[:, 0::2], expect - 1) and np.array_equal(Xc2[:, 1::2], expect + 99)


def test_conv_fwd_equals_filter_bank_times_im2col():
    rng = np.random.default_rng(5)
    C, N, H, Wd, KH, KW, B = 4, 6, 10, 7, 3, 3, 5
    Wdn = rng.standard_normal((N, C * KH * KW)).astype(np.float32)
    Wdn[rng.random(Wdn.shape) < 0.7] = 0.0
    rp, ci, v = dense_to_csr(Wdn)
    X = maps(rng, C, H, Wd, B)
    for geo in [(1, 1, 0, 0), (2, 1, 1, 2)]:
        Y = oracle.conv_fwd(rp, ci, v, X, C, H, Wd, KH, KW, *geo)
        Xc = oracle.im2col(X, C, H, Wd, KH, KW, *geo)
        ref = Wdn.astype(np.float64) @ Xc.astype(np.float64)  # [N][OH*OW*B]
        np.testing.assert_allclose(Y.reshape(N, -1), ref, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("geo", [(1, 1, 0, 0), (2, 2, 1, 1), (1, 3, 2, 1)])
def test_conv_bwd_data_is_the_adjoint(geo):
    rng = np.random.default_rng(7)
    C, N, H, Wd, KH, KW, B = 5, 4, 11, 9, 3, 5, 3
    Wdn = rng.standard_normal((N, C * KH * KW)).astype(np.float32)
    Wdn[rng.random(Wdn.shape) < 0.5] = 0.0
    rp, ci, v = dense_to_csr(Wdn)
    X = maps(rng, C, H, Wd, B)
    OH, OW = oracle.conv_out_size(H, Wd, KH, KW, *geo)
    dY = rng.standard_normal((N * OH * OW, B)).astype(np.float32)
    Y = oracle.conv_fwd(rp, ci, v, X, C, H, Wd, KH, KW, *geo)
    dX = oracle.conv_bwd_data(rp, ci, v, dY, C, H, Wd, KH, KW, *geo)
    lhs = float(np.sum(dY.astype(np.float64) * Y.astype(np.float64)))
    rhs = float(np.sum(dX.astype(np.float64) * X.astype(np.float64)))
    assert abs(lhs - rhs) <= 1e-5 * (abs(lhs) + 1.0)


def test_conv_delta_filter_shifts_the_map():
    # one entry at (kh, kw) = (1, 2) of a 3 x 4 filter: Y[oh][ow] = X[oh+1][ow+2]
    rng = np.random.default_rng(9)
    C, H, Wd, KH, KW, B = 1, 6, 8, 3, 4, 4
    rp, ci, v = np.array([0, 1], np.int32), np.array([1 * KW + 2], np.int32), np.array([1.0], np.float32)
    X = maps(rng, C, H, Wd, B)
    Y = oracle.conv_fwd(rp, ci, v, X, C, H, Wd, KH, KW)
    OH, OW = H - KH + 1, Wd - KW + 1
    Xm = X.reshape(H, Wd, B)
    assert np.array_equal(Y.reshape(OH, OW, B), Xm[1:1 + OH, 2:2 + OW])
    # its adjoint puts dY back at the shifted positions and zeros elsewhere
    dY = rng.standard_normal((OH * OW, B)).astype(np.float32)
    dX = oracle.conv_bwd_data(rp, ci, v, dY, C, H, Wd, KH, KW).reshape(H, Wd, B)
    assert np.array_equal(dX[1:1 + OH, 2:2 + OW], dY.reshape(OH, OW, B))
    mask = np.ones((H, Wd), bool)
    mask[1:1 + OH, 2:2 + OW] = False
    assert not dX[mask].any()


@pytest.mark.parametrize("K,S", [(2, 2), (3, 2), (2, 1)])
def test_maxpool_equals_window_maxima(K, S):
    rng = np.random.default_rng(K * 10 + S)
    C, H, Wd, B = 3, 9, 8, 4
    X = maps(rng, C, H, Wd, B)
    Y = oracle.maxpool_fwd(X, C, H, Wd, K, K, S, S)
    OH, OW = (H - K) // S + 1, (Wd - K) // S + 1
    win = np.lib.stride_tricks.sliding_window_view(to_nchw(X, C, H, Wd), (K, K), axis=(2, 3))
    ref = win.max(axis=(-1, -2))[:, :, ::S, ::S][:, :, :OH, :OW]  # [B][C][OH][OW]
    assert np.array_equal(to_nchw(Y, C, OH, OW), ref)
