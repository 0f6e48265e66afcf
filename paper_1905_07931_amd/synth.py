"""Seeded synthetic inputs shaped like the layers the paper trains.

This module only draws random numbers; it holds none of the method's
arithmetic and imports nothing else from the package, so both the HIP path and
the CPU oracle can be fed from it.

Conventions: CSR int32 ``row_ptr``/``col_idx`` (columns sorted inside a row),
float32 ``vals``; dense operands batch-contiguous (``X[K][B]``, ``dY[N][B]``).
Random streams come from ``SeedSequence(seed).spawn(4)`` in the order
(pattern, values, X, dY/labels); every draw is made in float64 and cast to
float32.  The paper's datasets (MNIST, CIFAR-10) are not used: uniform[0,1)
inputs stand in for pixel intensities scaled to [0,1].
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class Layer:
    """One CSR layer plus a batch of input and upstream gradient."""
    N: int
    K: int
    B: int
    row_ptr: np.ndarray
    col_idx: np.ndarray
    vals: np.ndarray
    X: np.ndarray            # [K][B]
    dY: np.ndarray | None    # [N][B]
    eta: float = 0.01
    lam: float = 1e-4
    name: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])


def streams(seed: int):
    ss = np.random.SeedSequence(seed).spawn(4)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss]


def pattern_from_positions(N: int, K: int, pos: np.ndarray):
    """Sorted flat positions (row-major) -> CSR row_ptr, col_idx."""
    pos = np.sort(np.asarray(pos, dtype=np.int64))
    rows = pos // K
    cols = (pos % K).astype(np.int32)
    counts = np.bincount(rows, minlength=N)
    row_ptr = np.zeros(N + 1, np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    return row_ptr.astype(np.int32), cols


def uniform_pattern(rng, N: int, K: int, nnz: int):
    """Exactly nnz distinct positions drawn uniformly without replacement."""
    if nnz == 0:
        return np.zeros(N + 1, np.int32), np.zeros(0, np.int32)
    pos = rng.choice(N * K, size=nnz, replace=False)
    return pattern_from_positions(N, K, pos)


def zipf_row_lengths(N: int, K: int, total: int, s: float) -> np.ndarray:
    """Deterministic power-law row lengths L_i ~ (i+1)^-s, capped at K, sum = total.

    The scale c is found by bisection so that sum(min(K, floor(c r_i))) is the
    largest value <= total; the remainder goes +1 to uncapped rows with the
    largest fractional part of c*r_i (ties to the lower index).
    """
    if total > N * K:
        raise ValueError("more nonzeros than entries")
    r = (np.arange(N, dtype=np.float64) + 1.0) ** (-s)

    def lengths(c):
        return np.minimum(K, np.floor(c * r)).astype(np.int64)

    lo, hi = 0.0, 1.0
    while lengths(hi).sum() <= total and hi < 1e30:
        hi *= 2.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if lengths(mid).sum() <= total:
            lo = mid
        else:
            hi = mid
    L = lengths(lo)
    rem = int(total - L.sum())
    if rem > 0:
        frac = lo * r - np.floor(lo * r)
        cand = np.nonzero(L < K)[0]
        order = cand[np.lexsort((cand, -frac[cand]))]
        L[order[:rem]] += 1
    assert L.sum() == total and L.max() <= K
    return L


def zipf_pattern(rng, N: int, K: int, nnz: int, s: float = 1.1):
    L = zipf_row_lengths(N, K, nnz, s)
    L = L[rng.permutation(N)]
    row_ptr = np.zeros(N + 1, np.int64)
    np.cumsum(L, out=row_ptr[1:])
    cols = np.empty(int(row_ptr[-1]), np.int32)
    for i in range(N):
        if L[i]:
            cols[row_ptr[i]:row_ptr[i + 1]] = np.sort(rng.choice(K, size=int(L[i]), replace=False))
    return row_ptr.astype(np.int32), cols


def fc_layer(N, K, B, nnz, seed=0, w_std=0.05, pattern="uniform", zipf_s=1.1,
             dy_scale=1.0, eta=0.01, lam=1e-4, name="") -> Layer:
    """A CSR layer with N(0, w_std) values, X ~ U[0,1), dY ~ N(0,1)*dy_scale."""
    rp_rng, v_rng, x_rng, dy_rng = streams(seed)
    if pattern == "uniform":
        row_ptr, col_idx = uniform_pattern(rp_rng, N, K, nnz)
    elif pattern == "zipf":
        row_ptr, col_idx = zipf_pattern(rp_rng, N, K, nnz, zipf_s)
    else:
        raise ValueError(pattern)
    vals = (v_rng.standard_normal(col_idx.shape[0]) * w_std).astype(np.float32)
    X = x_rng.random((K, B)).astype(np.float32)
    dY = (dy_rng.standard_normal((N, B)) * dy_scale).astype(np.float32)
    return Layer(N, K, B, row_ptr, col_idx, vals, X, dY, eta, lam, name)


def dyadic_layer(N, K, B, nnz, seed=0, empty_rows=(), full_rows=(), pattern="uniform",
                 zipf_s=1.1) -> Layer:
    """Inputs on a coarse dyadic grid: every float32 product and partial sum of
    the hot path is then exact, so any summation order gives the same bits.

    vals = +-k/16 (k in 1..16), X = j/16 (j in 0..16), dY = +-k/16; eta = 2^-7.
    ``pattern`` is "uniform", "zipf" (power-law row lengths, as fc_layer) or
    an explicit (row_ptr, col_idx) pair (nnz is then ignored).  Rows listed in
    ``empty_rows`` get no entries, rows in ``full_rows`` all K.
    """
    rp_rng, v_rng, x_rng, dy_rng = streams(seed)
    if isinstance(pattern, tuple):
        row_ptr = np.asarray(pattern[0], np.int32)
        col_idx = np.asarray(pattern[1], np.int32)
    elif pattern == "zipf":
        row_ptr, col_idx = zipf_pattern(rp_rng, N, K, nnz, zipf_s)
    elif pattern == "uniform":
        row_ptr, col_idx = uniform_pattern(rp_rng, N, K, nnz)
    else:
        raise ValueError(pattern)
    if len(empty_rows) or len(full_rows):
        dense = np.zeros((N, K), bool)
        rows = np.repeat(np.arange(N), np.diff(row_ptr))
        dense[rows, col_idx] = True
        for i in empty_rows:
            dense[i, :] = False
        for i in full_rows:
            dense[i, :] = True
        pos = np.flatnonzero(dense.reshape(-1))
        row_ptr, col_idx = pattern_from_positions(N, K, pos)
    n = col_idx.shape[0]
    mag = v_rng.integers(1, 17, size=n)
    sign = np.where(v_rng.random(n) < 0.5, -1.0, 1.0)
    vals = (sign * mag / 16.0).astype(np.float32)
    X = (x_rng.integers(0, 17, size=(K, B)) / 16.0).astype(np.float32)
    dY = (dy_rng.integers(-16, 17, size=(N, B)) / 16.0).astype(np.float32)
    return Layer(N, K, B, row_ptr, col_idx, vals, X, dY, eta=2.0 ** -7, lam=2.0 ** -4,
                 name="dyadic")


# ---------------------------------------------------------------------------
# The five synthetic workloads (sizes and distributions of the paper's layers)
# ---------------------------------------------------------------------------

def nnz_for(N, K, density):
    return int(round(density * N * K))


def fc784_300(seed=0) -> Layer:
    """Single FC layer 784->300 (LeNet-300 first layer shape), 10% density, B = 64."""
    return fc_layer(300, 784, 64, nnz_for(300, 784, 0.10), seed=seed, w_std=0.05,
                    name="fc784x300_b64_d10")


def mlp_784_300_100_10(seed=0, B=256):
    """MLP 784-300-100-10, densities 8%/9%/26%, He-initialised values, B = 256.

    Returns (layers, X, labels): layers[j] holds layer j's CSR (its X/dY fields
    are unused), X[784][B] ~ U[0,1), labels uniform over 10 classes.
    """
    rp_rng, v_rng, x_rng, lab_rng = streams(seed)
    shapes = [(300, 784, 0.08), (100, 300, 0.09), (10, 100, 0.26)]
    layers = []
    for (N, K, d) in shapes:
        row_ptr, col_idx = uniform_pattern(rp_rng, N, K, nnz_for(N, K, d))
        vals = (v_rng.standard_normal(col_idx.shape[0]) * np.sqrt(2.0 / K)).astype(np.float32)
        layers.append(Layer(N, K, B, row_ptr, col_idx, vals, None, None, 0.01, 1e-4,
                            name=f"mlp_{N}x{K}"))
    X = x_rng.random((784, B)).astype(np.float32)
    labels = lab_rng.integers(0, 10, size=B).astype(np.int32)
    return layers, X, labels


def conv2_im2col(seed=0) -> Layer:
    """LeNet-5 conv2 (20->50 channels, 5x5, 12x12 maps, batch 256) lowered by
    im2col: W 50x500 at 10% density, X[500][256*64] ~ U[0,1) drawn directly."""
    return fc_layer(50, 500, 256 * 64, nnz_for(50, 500, 0.10), seed=seed, w_std=0.05,
                    name="conv2_im2col_50x500_b16384_d10")


def fc9216_4096(seed=0) -> Layer:
    """Large FC layer 9216->4096 (AlexNet fc6 shape), 9% density with Zipf(1.1)
    row lengths, values N(0, 0.01), B = 1024."""
    N, K = 4096, 9216
    return fc_layer(N, K, 1024, nnz_for(N, K, 0.09), seed=seed, w_std=0.01,
                    pattern="zipf", zipf_s=1.1, name="fc9216x4096_b1024_d9_zipf")


def fc4096_sweep(density, seed=0) -> Layer:
    """FC 4096->4096, batch 512, uniform pattern, values N(0, 0.1)."""
    N = K = 4096
    L = fc_layer(N, K, 512, nnz_for(N, K, density), seed=seed, w_std=0.1,
                 dy_scale=1.0 / 512, name=f"fc4096_b512_d{int(round(density * 100))}")
    return L


def fc4096_batch(t, seed=0, K=4096, N=4096, B=512):
    """Fresh (X, dY) for iteration t of the density sweep (own spawned stream)."""
    ss = np.random.SeedSequence([seed, 1000 + t])
    rng = np.random.Generator(np.random.PCG64(ss))
    X = rng.random((K, B)).astype(np.float32)
    dY = (rng.standard_normal((N, B)) / B).astype(np.float32)
    return X, dY


# ---------------------------------------------------------------------------
# Convolution layers (the conv rows of the paper's networks)
# ---------------------------------------------------------------------------

@dataclass
class ConvLayer:
    """A CSR filter bank (n_out x C*KH*KW, column (ci*KH + kh)*KW + kw) with a
    batch of input maps X [C*H*W][B] and output-map gradients dY [n_out*OH*OW][B]."""
    n_out: int
    C: int
    H: int
    W: int
    KH: int
    KW: int
    SH: int
    SW: int
    PH: int
    PW: int
    B: int
    row_ptr: np.ndarray
    col_idx: np.ndarray
    vals: np.ndarray
    X: np.ndarray
    dY: np.ndarray
    eta: float = 0.01
    lam: float = 1e-4
    name: str = ""

    @property
    def OH(self) -> int:
        return (self.H + 2 * self.PH - self.KH) // self.SH + 1

    @property
    def OW(self) -> int:
        return (self.W + 2 * self.PW - self.KW) // self.SW + 1

    @property
    def K(self) -> int:
        return self.C * self.KH * self.KW

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    @property
    def geom(self):
        """(C, H, W, KH, KW, SH, SW, PH, PW)"""
        return (self.C, self.H, self.W, self.KH, self.KW, self.SH, self.SW, self.PH, self.PW)


def conv_layer(n_out, C, H, W, KH, KW, B, nnz, seed=0, SH=1, SW=1, PH=0, PW=0, w_std=0.05,
               dyadic=False, name="") -> ConvLayer:
    """Uniform random filter pattern with exactly nnz entries; values
    N(0, w_std), maps U[0,1), dY N(0,1) -- or, with dyadic=True, values
    +-k/16, maps j/16 and dY +-k/16 (every fp32 partial sum exact)."""
    rp_rng, v_rng, x_rng, dy_rng = streams(seed)
    K = C * KH * KW
    row_ptr, col_idx = uniform_pattern(rp_rng, n_out, K, nnz)
    OH = (H + 2 * PH - KH) // SH + 1
    OW = (W + 2 * PW - KW) // SW + 1
    n = col_idx.shape[0]
    if dyadic:
        sign = np.where(v_rng.random(n) < 0.5, -1.0, 1.0)
        vals = (sign * v_rng.integers(1, 17, size=n) / 16.0).astype(np.float32)
        X = (x_rng.integers(0, 17, size=(C * H * W, B)) / 16.0).astype(np.float32)
        dY = (dy_rng.integers(-16, 17, size=(n_out * OH * OW, B)) / 16.0).astype(np.float32)
    else:
        vals = (v_rng.standard_normal(n) * w_std).astype(np.float32)
        X = x_rng.random((C * H * W, B)).astype(np.float32)
        dY = dy_rng.standard_normal((n_out * OH * OW, B)).astype(np.float32)
    return ConvLayer(n_out, C, H, W, KH, KW, SH, SW, PH, PW, B, row_ptr, col_idx, vals, X, dY,
                     name=name or f"conv{n_out}x{C}x{KH}x{KW}_{H}x{W}_b{B}")


def lenet5_conv2(seed=0, B=256, density=0.10) -> ConvLayer:
    """LeNet-5 conv2: 20 -> 50 channels, 5x5 filters on 12x12 maps, batch 256
    (the lowered shape is the 50 x 500 by 500 x (256*64) product)."""
    return conv_layer(50, 20, 12, 12, 5, 5, B, nnz_for(50, 500, density), seed=seed, w_std=0.05,
                      name=f"lenet5_conv2_b{B}_d{int(round(density * 100))}")


# LeNet-5 layer shapes and the nonzeros kept after compression and retraining
# (Table A1, SpC(Retrain) column): conv1 142/500, conv2 1750/25000,
# fc1 10045/400000, fc2 280/5000.
LENET5_NNZ = {"conv1": 142, "conv2": 1750, "fc1": 10045, "fc2": 280}


def lenet5_compressed(seed=0, B=256):
    """Synthetic compressed LeNet-5 for inference: uniform random patterns with
    the Table A1 nonzero counts, He-initialised values N(0, sqrt(2/fan_in)),
    inputs X [784][B] ~ U[0,1) (28 x 28 single-channel maps).  Returns a dict
    name -> (n_out, fan_in, row_ptr, col_idx, vals) and X."""
    rp_rng, v_rng, x_rng, _ = streams(seed)
    shapes = {"conv1": (20, 25), "conv2": (50, 500), "fc1": (500, 800), "fc2": (10, 500)}
    layers = {}
    for name, (n_out, fan_in) in shapes.items():
        row_ptr, col_idx = uniform_pattern(rp_rng, n_out, fan_in, LENET5_NNZ[name])
        vals = (v_rng.standard_normal(col_idx.shape[0]) * np.sqrt(2.0 / fan_in)).astype(np.float32)
        layers[name] = (n_out, fan_in, row_ptr, col_idx, vals)
    X = x_rng.random((784, B)).astype(np.float32)
    return layers, X
