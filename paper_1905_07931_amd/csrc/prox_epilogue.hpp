// The proximal step of Eq. (prox) applied in a weight-gradient GEMM's
// epilogue: instead of dW the kernel writes
//     Z[i][k] = S_t(w_ik - eta * dW[i][k]),  t = eta * lambda,
// and the number of nonzero Z entries of every 32-column word of every row,
// so that the recompression that follows reads Z once and never W.
//
// W's value at (i, k) comes from a bitmap index of its CSR built before the
// GEMM: for every row and 32-column word, mask (bit c set iff column 32w + c
// is stored) and pos (CSR position of the row's first entry with column >=
// 32w), so w_ik = vals[pos + popcount(mask & below(c))] if the bit is set,
// else 0.  The tile's mask/pos words are staged in LDS once the reduction is
// done, and the stored values are gathered straight into LDS.
//
// The arithmetic is that of the prox kernels (prox.hip): double, eta*g exact,
// z rounds once, S_t(z) once more to float; zero results are +0.0; an entry
// is kept iff its float result is nonzero.
#pragma once

#include "common.hpp"

namespace l1csr {

// S_t(z) = z - t for z > t, z + t for z < -t, else 0, written as
// z - min(max(z, -t), t): the same single rounding of z - t or z + t, and
// z - z = +-0 in between.  Adding +0.0f after the conversion makes every
// zero +0.0 whatever the signs of the zeros min/max return.
__device__ __forceinline__ float soft_threshold(float w, float g, double eta, double t) {
    const double z = (double)w - eta * (double)g;
    const double c = fmin(fmax(z, -t), t);
    return (float)(z - c) + 0.0f;
}

// kernel argument of a GEMM with the prox epilogue
struct prox_epi {
    const unsigned *mask;  // [kw][M] (word-major)
    const int *pos;        // [kw][M]
    const float *vals;     // W's values (CSR order)
    double eta, t;
    int kw;                // 32-column words per row, ceil(Nn / 32)
    int *counts;           // [M][kw] nonzero Z entries per (row, word)
};

typedef float floatx16 __attribute__((ext_vector_type(16)));

// Stage the tile's mask/pos words (rows m0 .. m0+BM, words n0/32 .. n0/32 +
// BN/32) into LDS; all NT threads of the workgroup call it (it ends with a
// barrier).  stage holds BM * BN / 32 int2.
template <int BM, int BN, int NT>
__device__ __forceinline__ void prox_stage(const prox_epi &P, int M, int m0, int n0, int2 *stage) {
    constexpr int WPT = BN / 32;
    const int w0 = n0 >> 5;
    for (int i = threadIdx.x; i < BM * WPT; i += NT) {
        const int w = i / BM, r = i - w * BM;  // consecutive threads: consecutive rows of a word
        const int row = m0 + r, gw = w0 + w;
        int2 v = make_int2(0, 0);
        if (row < M && gw < P.kw) {
            const int64_t o = (int64_t)gw * M + row;
            v = make_int2((int)P.mask[o], P.pos[o]);
        }
        stage[r * WPT + w] = v;
    }
    __syncthreads();
}

typedef __attribute__((address_space(3))) void prox_lds_void;

// A zero in device memory: the gather's source for the positions W does not
// store, so every lane loads (no branch per register) and the loaded value is
// w itself.
static __device__ float kProxZero = 0.f;

// The epilogue of one wave holding a (2*32) x (TN*32) block of the tile at
// (m0 + wm, n0 + wn) in the D layout of the 32x32 MFMAs: lane l, register r
// of MFMA tile (a, b) holds row 32a + 8(r/4) + 4(l/32) + r%4, column
// 32b + l%32.  W's values are gathered TPB MFMA tiles (16*TPB registers) at a
// time with direct global->LDS loads into this wave's buffer gbuf (lane l's
// value of register j of the batch at gbuf[j*64 + l]; lanes at positions W
// does not store load a zero), so a batch costs one memory round trip and no
// registers; then the batch is thresholded, stored and counted (ballots over
// the lanes of each row half; lane l holds the counts of the wave's row l,
// one per 32-column word).  NBUF = 2: gbuf holds two batches, and the next
// batch's gather is in flight while the current one is thresholded.
template <int TN, int BN, int TPB, int NBUF = 1>
__device__ __forceinline__ void prox_store(const floatx16 (&acc)[2][TN], int M, int Nn, int m0, int n0,
                                           int wm, int wn, const int2 *stage, float *gbuf,
                                           float *__restrict__ C, int64_t ldc, const prox_epi &P) {
    constexpr int WPT = BN / 32, NTILE = 2 * TN;
    static_assert(NTILE % TPB == 0, "batches of whole MFMA tiles");
    static_assert(NBUF == 1 || NBUF == 2, "one or two gather buffers");
    const int lane = threadIdx.x & 63;
    const int lr = lane & 31, lh = lane >> 5;
    const unsigned below = (1u << lr) - 1u;
    int mine[TN] = {};  // this lane's counts (wave row `lane`) per word of the block
    // the wave's gather buffer as one wave-uniform LDS address; the zero's
    // address taken once (kept in registers rather than rebuilt per load)
    const unsigned gb = (unsigned)uniform((int)(uintptr_t)(prox_lds_void *)gbuf);
    const uint64_t zero = (uint64_t)(uintptr_t)&kProxZero;
    // this lane's output column per word of the block, whether it is inside
    // the matrix (as a wave mask), and its first row: register r of MFMA tile
    // (a, b) is row rbase + ro(a, r), ro(a, r) = 32a + 8(r/4) + r%4 (the same
    // for the whole wave), so its address is cb[b] + ro * ldc
    const int rbase = m0 + wm + 4 * lh;
    float *cb[TN];
    bool colok[TN];
#pragma unroll
    for (int b = 0; b < TN; ++b) {
        const int col = n0 + wn + b * 32 + lr;
        colok[b] = col < Nn;
        cb[b] = C + (int64_t)rbase * ldc + col;
    }
    auto gather = [&](int q0, unsigned base) {  // issue the loads of batch q0 into the buffer at base
#pragma unroll
        for (int j = 0; j < 16 * TPB; ++j) {
            const int q = q0 + j / 16, a = q / TN, b = q % TN, r = j % 16;
            const int rt = a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
            const int2 mp = stage[(wm + rt) * WPT + ((wn >> 5) + b)];
            const unsigned m = (unsigned)mp.x;
            const uint64_t stored = (uint64_t)(uintptr_t)(P.vals + mp.y + __popc(m & below));
            const uint64_t src = (m >> lr) & 1u ? stored : zero;
            __builtin_amdgcn_global_load_lds((const void *)(uintptr_t)src,
                                             (prox_lds_void *)(uintptr_t)(base + 4u * j * kWave), 4, 0, 0);
        }
    };
    auto threshold = [&](int q0, const float *gv) {  // prox, store and count batch q0 (values in gv)
#pragma unroll
        for (int j = 0; j < 16 * TPB; ++j) {
            const int q = q0 + j / 16, a = q / TN, b = q % TN, r = j % 16;
            const int ro = a * 32 + 8 * (r >> 2) + (r & 3);
            const float w = gv[j * kWave + lane];
            const float o = soft_threshold(w, acc[a][b][r], P.eta, P.t);
            const bool valid = rbase + ro < M && colok[b];
            if (valid) cb[b][(int64_t)ro * ldc] = o;
            const uint64_t k = __ballot(valid && o != 0.f);
            // row ro (lanes 0-31) and row ro + 4 (lanes 32-63) of the wave block:
            // their nonzero counts in word b go to the lanes of those rows
            const int c_lo = __popcll(k & 0xffffffffull), c_hi = __popcll(k >> 32);
            asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(mine[b]) : "s"(c_lo), "I"(ro));
            asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(mine[b]) : "s"(c_hi), "I"(ro + 4));
        }
    };
    constexpr unsigned kBatchBytes = 4u * 16 * TPB * kWave;
    if constexpr (NBUF == 1) {
#pragma unroll
        for (int q0 = 0; q0 < NTILE; q0 += TPB) {
            gather(q0, gb);
            __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): the gathered values are in LDS
            threshold(q0, gbuf);
        }
    } else {
        gather(0, gb);
#pragma unroll
        for (int q0 = 0; q0 < NTILE; q0 += TPB) {
            const int cur = (q0 / TPB) & 1;
            // vmcnt(0): batch q0's values are in LDS (and the previous batch's
            // stores are done); the other buffer was read by that batch
            __builtin_amdgcn_s_waitcnt(0x0f70);
            if (q0 + TPB < NTILE) gather(q0 + TPB, gb + (cur ^ 1) * kBatchBytes);
            threshold(q0, gbuf + cur * 16 * TPB * kWave);
        }
    }
    const int row = m0 + wm + lane;
#pragma unroll
    for (int b = 0; b < TN; ++b) {
        const int word = ((n0 + wn) >> 5) + b;
        if (row < M && word < P.kw) P.counts[(int64_t)row * P.kw + word] = mine[b];
    }
}

}  // namespace l1csr
