// Dense weight gradient dW[N][K] = dY[N][B] . X[K][B]^T on the fp32 matrix
// cores (v_mfma_f32_32x32x2_f32).
//
// Both operands keep the reduction index (the batch) contiguous, the natural
// layout for the matrix-core operand fragments.  A 256-thread workgroup owns a
// 128x128 tile of dW as 2x2 waves of 64x64, each wave 2x2 MFMA tiles of 32x32.
// Reduction chunks of 32 are staged through LDS (double buffered; the next
// chunk's global loads are in flight during the current chunk's MFMAs).
//
// Reduction-index assignment: an MFMA step multiplies the pairs k in {0, 1}
// held by lane halves 0 and 1.  Any bijection between the chunk's 32 batch
// indices and (step, half) gives the same sum as long as the A and B fragments
// use the same one; lane half h takes batch indices [16h, 16h + 16) of the
// chunk, step s index 16h + s, so each lane reads its fragments as contiguous
// float4s from LDS.
//
// Outputs with many tiles also have a 256x288 shape: 4x3 waves of 64x96 (2x3
// MFMA tiles each), K-step 32, one 12-wave workgroup per CU (153 KB of LDS).
// Per MFMA it stages fewer bytes and spends fewer barriers, and 4096 x 9216
// is 512 tiles, two whole rounds of the 256 CUs.  The host takes the shape
// with the shorter modelled time: the tiles per CU, ceil(tiles / 256), times
// the tile's flops at the shape's measured rate.
#include <cmath>

#include "common.hpp"
#include "launch.hpp"
#include "prox_epilogue.hpp"

namespace l1csr {

namespace {

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDS_STRIDE = BK + 4;  // 36 floats: conflict-free 16-byte fragment reads
constexpr int kThreads = 256;
constexpr int kLoadsPerThread = (BM * BK / 4) / kThreads;  // float4 loads per operand: 4

template <bool V4>
__device__ __forceinline__ void load_tile(const float *__restrict__ src, int64_t ld, int rows,
                                          int kred, int row0, int k0, float4 (&r)[kLoadsPerThread]) {
#pragma unroll
    for (int i = 0; i < kLoadsPerThread; ++i) {
        const int f = threadIdx.x + i * kThreads;  // float4 index inside the tile
        const int rr = f >> 3;                      // 8 float4 per tile row
        const int kk = (f & 7) * 4;
        const int grow = row0 + rr;
        const int gk = k0 + kk;
        if (V4 && grow < rows && gk + 3 < kred) {
            r[i] = *reinterpret_cast<const float4 *>(src + (int64_t)grow * ld + gk);
        } else {
            const float *p = src + (int64_t)grow * ld + gk;
            const bool rv = grow < rows;
            r[i].x = (rv && gk + 0 < kred) ? p[0] : 0.f;
            r[i].y = (rv && gk + 1 < kred) ? p[1] : 0.f;
            r[i].z = (rv && gk + 2 < kred) ? p[2] : 0.f;
            r[i].w = (rv && gk + 3 < kred) ? p[3] : 0.f;
        }
    }
}

__device__ __forceinline__ void store_tile(float *lds, const float4 (&r)[kLoadsPerThread]) {
#pragma unroll
    for (int i = 0; i < kLoadsPerThread; ++i) {
        const int f = threadIdx.x + i * kThreads;
        const int rr = f >> 3;
        const int kk = (f & 7) * 4;
        *reinterpret_cast<float4 *>(lds + rr * LDS_STRIDE + kk) = r[i];
    }
}

// double-buffered operand tiles
union tile_smem {
    struct {
        float As[2][BM * LDS_STRIDE];
        float Bs[2][BN * LDS_STRIDE];
    } ab;
};

// acc = the 128x128 tile (m0, n0) of A . Bt^T (A [M][lda], Bt [Nn][ldb], both
// with the reduction index contiguous).
template <bool V4>
__device__ __forceinline__ void mfma_tile(int M, int Nn, int Kr, const float *__restrict__ A,
                                          int64_t lda, const float *__restrict__ Bt, int64_t ldb,
                                          int m0, int n0, tile_smem &sm, floatx16 (&acc)[2][2]) {
    auto &As = sm.ab.As;
    auto &Bs = sm.ab.Bs;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
    const int lr = lane & 31;  // row inside a 32x32 tile (A) / column (B)
    const int lh = lane >> 5;  // lane half: which 16 reduction indices

#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    const int nchunks = (Kr + BK - 1) / BK;
    float4 ra[kLoadsPerThread], rb[kLoadsPerThread];
    load_tile<V4>(A, lda, M, Kr, m0, 0, ra);
    load_tile<V4>(Bt, ldb, Nn, Kr, n0, 0, rb);
    store_tile(As[0], ra);
    store_tile(Bs[0], rb);
    __syncthreads();

    for (int c = 0; c < nchunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunks) {
            load_tile<V4>(A, lda, M, Kr, m0, (c + 1) * BK, ra);
            load_tile<V4>(Bt, ldb, Nn, Kr, n0, (c + 1) * BK, rb);
        }
        const float *as0 = As[buf] + (wm + lr) * LDS_STRIDE + lh * 16;
        const float *as1 = as0 + 32 * LDS_STRIDE;
        const float *bs0 = Bs[buf] + (wn + lr) * LDS_STRIDE + lh * 16;
        const float *bs1 = bs0 + 32 * LDS_STRIDE;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 a0 = *reinterpret_cast<const float4 *>(as0 + 4 * q);
            const float4 a1 = *reinterpret_cast<const float4 *>(as1 + 4 * q);
            const float4 b0 = *reinterpret_cast<const float4 *>(bs0 + 4 * q);
            const float4 b1 = *reinterpret_cast<const float4 *>(bs1 + 4 * q);
            const float av0[4] = {a0.x, a0.y, a0.z, a0.w};
            const float av1[4] = {a1.x, a1.y, a1.z, a1.w};
            const float bv0[4] = {b0.x, b0.y, b0.z, b0.w};
            const float bv1[4] = {b1.x, b1.y, b1.z, b1.w};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av0[s], bv0[s], acc[0][0], 0, 0, 0);
                acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(av0[s], bv1[s], acc[0][1], 0, 0, 0);
                acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av1[s], bv0[s], acc[1][0], 0, 0, 0);
                acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(av1[s], bv1[s], acc[1][1], 0, 0, 0);
            }
        }
        if (c + 1 < nchunks) {
            store_tile(As[buf ^ 1], ra);
            store_tile(Bs[buf ^ 1], rb);
        }
        __syncthreads();
    }
}

// D layout of v_mfma_f32_32x32x2_f32: lane l, register r holds
// row 8*(r/4) + 4*(l/32) + r%4, column l%32 of the 32x32 tile.
__device__ __forceinline__ int acc_row(int a, int r) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return (wave >> 1) * 64 + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
__device__ __forceinline__ int acc_col(int b) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return (wave & 1) * 64 + b * 32 + (lane & 31);
}

// PROX: the epilogue writes Z = S_t(W - eta*dW) and the per-(row, 64-column
// slab) counts instead of dW (prox_epilogue.hpp)
template <bool V4, bool PROX>
__global__ __launch_bounds__(kThreads, 2) void wgrad_f32_mfma_kernel(
    int M, int Nn, int Kr, const float *__restrict__ A, int64_t lda, const float *__restrict__ Bt,
    int64_t ldb, float *__restrict__ C, int64_t ldc, prox_epi P) {
    __shared__ __attribute__((aligned(16))) tile_smem sm;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    floatx16 acc[2][2];
    mfma_tile<V4>(M, Nn, Kr, A, lda, Bt, ldb, m0, n0, sm, acc);
    if constexpr (PROX) {
        // the tile loop ended with a barrier: the operand buffers are free
        static_assert(sizeof(sm.ab.As) >= sizeof(int2) * BM * (BN / 32), "staging space");
        int2 *stage = reinterpret_cast<int2 *>(sm.ab.As);
        prox_stage<BM, BN, kThreads>(P, M, m0, n0, stage);
        const int wave = threadIdx.x >> 6;
        constexpr int TPB = 2;  // MFMA tiles per gather batch: 8 KB of LDS per wave
        static_assert(sizeof(sm.ab.Bs) >= sizeof(float) * 16 * TPB * kThreads, "gather space");
        float *gbuf = &sm.ab.Bs[0][0] + wave * 16 * TPB * kWave;
        prox_store<2, BN, TPB>(acc, M, Nn, m0, n0, (wave >> 1) * 64, (wave & 1) * 64, stage, gbuf, C, ldc, P);
        return;
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int col = n0 + acc_col(b);
            if (col >= Nn) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + acc_row(a, r);
                if (row < M) C[(int64_t)row * ldc + col] = acc[a][b][r];
            }
        }
}

// The 256x288 shape (see the file comment); load and stage helpers generic in
// the tile height, the tile loop as in mfma_tile.
constexpr int LBM = 256, LBN = 288, LWM = 4, LWN = 3;
constexpr int kLargeThreads = 64 * LWM * LWN;

template <bool V4, int ROWS>
__device__ __forceinline__ void load_rows(const float *__restrict__ src, int64_t ld, int rows, int kred, int row0,
                                          int k0, float4 (&r)[(ROWS * BK / 4 + kLargeThreads - 1) / kLargeThreads]) {
    constexpr int LPT = (ROWS * BK / 4 + kLargeThreads - 1) / kLargeThreads;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
        const int f = threadIdx.x + i * kLargeThreads;  // float4 index inside the tile
        const int rr = f >> 3;                           // 8 float4 per tile row
        const int kk = (f & 7) * 4;
        const int grow = row0 + rr, gk = k0 + kk;
        const bool rv = rr < ROWS && grow < rows;
        if (V4 && rv && gk + 3 < kred) {
            r[i] = *reinterpret_cast<const float4 *>(src + (int64_t)grow * ld + gk);
        } else {
            const float *p = src + (int64_t)grow * ld + gk;
            r[i].x = (rv && gk + 0 < kred) ? p[0] : 0.f;
            r[i].y = (rv && gk + 1 < kred) ? p[1] : 0.f;
            r[i].z = (rv && gk + 2 < kred) ? p[2] : 0.f;
            r[i].w = (rv && gk + 3 < kred) ? p[3] : 0.f;
        }
    }
}

template <int ROWS>
__device__ __forceinline__ void store_rows(float *lds, const float4 (&r)[(ROWS * BK / 4 + kLargeThreads - 1) / kLargeThreads]) {
    constexpr int LPT = (ROWS * BK / 4 + kLargeThreads - 1) / kLargeThreads;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
        const int f = threadIdx.x + i * kLargeThreads;
        const int rr = f >> 3;
        const int kk = (f & 7) * 4;
        if (rr < ROWS) *reinterpret_cast<float4 *>(lds + rr * LDS_STRIDE + kk) = r[i];
    }
}

template <bool V4, bool PROX>
__global__ __launch_bounds__(kLargeThreads, 1) void wgrad_f32_large_kernel(
    int M, int Nn, int Kr, const float *__restrict__ A, int64_t lda, const float *__restrict__ Bt,
    int64_t ldb, float *__restrict__ C, int64_t ldc, prox_epi P) {
    constexpr int TM = LBM / LWM / 32, TN = LBN / LWN / 32;
    constexpr int LA = (LBM * BK / 4 + kLargeThreads - 1) / kLargeThreads;
    constexpr int LB = (LBN * BK / 4 + kLargeThreads - 1) / kLargeThreads;
    __shared__ __attribute__((aligned(16))) float As[2][LBM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) float Bs[2][LBN * LDS_STRIDE];
    const int m0 = blockIdx.y * LBM, n0 = blockIdx.x * LBN;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wm = (wave / LWN) * (LBM / LWM), wn = (wave % LWN) * (LBN / LWN);
    const int lr = lane & 31;
    const int lh = lane >> 5;

    floatx16 acc[TM][TN];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    const int nchunks = (Kr + BK - 1) / BK;
    float4 ra[LA], rb[LB];
    load_rows<V4, LBM>(A, lda, M, Kr, m0, 0, ra);
    load_rows<V4, LBN>(Bt, ldb, Nn, Kr, n0, 0, rb);
    store_rows<LBM>(As[0], ra);
    store_rows<LBN>(Bs[0], rb);
    __syncthreads();

    const int oa = (wm + lr) * LDS_STRIDE + lh * 16, ob = (wn + lr) * LDS_STRIDE + lh * 16;
    for (int c = 0; c < nchunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunks) {
            load_rows<V4, LBM>(A, lda, M, Kr, m0, (c + 1) * BK, ra);
            load_rows<V4, LBN>(Bt, ldb, Nn, Kr, n0, (c + 1) * BK, rb);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float av[TM][4], bv[TN][4];
#pragma unroll
            for (int a = 0; a < TM; ++a) {
                const float4 x = *reinterpret_cast<const float4 *>(As[buf] + oa + a * 32 * LDS_STRIDE + 4 * q);
                av[a][0] = x.x; av[a][1] = x.y; av[a][2] = x.z; av[a][3] = x.w;
            }
#pragma unroll
            for (int b = 0; b < TN; ++b) {
                const float4 x = *reinterpret_cast<const float4 *>(Bs[buf] + ob + b * 32 * LDS_STRIDE + 4 * q);
                bv[b][0] = x.x; bv[b][1] = x.y; bv[b][2] = x.z; bv[b][3] = x.w;
            }
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int a = 0; a < TM; ++a)
#pragma unroll
                    for (int b = 0; b < TN; ++b)
                        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[a][s], bv[b][s], acc[a][b], 0, 0, 0);
        }
        if (c + 1 < nchunks) {
            store_rows<LBM>(As[buf ^ 1], ra);
            store_rows<LBN>(Bs[buf ^ 1], rb);
        }
        __syncthreads();
    }
    if constexpr (PROX) {
        // the last chunk ended with a barrier: the operand buffers are free
        static_assert(TM == 2 && sizeof(As) >= sizeof(int2) * LBM * (LBN / 32), "staging space");
        int2 *stage = reinterpret_cast<int2 *>(&As[0][0]);
        prox_stage<LBM, LBN, kLargeThreads>(P, M, m0, n0, stage);
        // gather buffers of 2 MFMA tiles (8 KB) per wave: waves 0-5 in the A
        // buffers after the staged words, waves 6-11 in the B buffers
        constexpr int TPB = 2, GBF = 16 * TPB * kWave;  // floats per wave
        constexpr int kStageFloats = 2 * LBM * (LBN / 32);
        static_assert(sizeof(As) >= sizeof(float) * (kStageFloats + 6 * GBF) && sizeof(Bs) >= sizeof(float) * 6 * GBF &&
                      LWM * LWN == 12, "gather space");
        float *gbuf = wave < 6 ? &As[0][0] + kStageFloats + wave * GBF : &Bs[0][0] + (wave - 6) * GBF;
        prox_store<TN, LBN, TPB>(acc, M, Nn, m0, n0, wm, wn, stage, gbuf, C, ldc, P);
        return;
    }
    // D layout of the 32x32 MFMA (acc_row / acc_col for this wave grid)
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
            const int col = n0 + wn + b * 32 + lr;
            if (col >= Nn) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
                if (row < M) C[(int64_t)row * ldc + col] = acc[a][b][r];
            }
        }
}

// The 256x288 shape with its operand tiles brought in by direct global->LDS
// loads (no round trip through VGPRs, no LDS stores before each barrier).
// Rows are stored unpadded, 32 floats = eight 16-byte chunks, chunk c of tile
// row r at position c ^ f(r), f(r) = (r & 7) ^ ((r >> 3) & 1): the fragment
// reads (32 rows, one chunk each) then hit distinct banks in every group of 8
// lanes on 32 banks and of 16 lanes on 64 banks.  Each lane fetches the chunk
// that belongs at its position, so one load instruction fills 1 KB of LDS.
// Used when the reduction length is a multiple of 32 (no partial K-step to
// zero) and the operands are 16-byte aligned.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

typedef __attribute__((address_space(3))) void gemm_lds_void;

template <int ROWS>
__device__ __forceinline__ void dma_rows(const float *__restrict__ src, int64_t ld, int rows, int row0, int k0,
                                         float *dst) {
    constexpr int PIECES = ROWS * (BK / 4);  // 16-byte pieces of the tile
    static_assert(PIECES % kWave == 0, "whole waves");
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int q0 = 0; q0 < PIECES; q0 += kLargeThreads) {
        const int qw = q0 + wave * kWave;  // this wave's first piece
        if (qw < PIECES) {
            const int q = qw + lane;
            const int r = q >> 3, c = (q & 7) ^ swz(r);
            const int grow = row0 + r < rows ? row0 + r : rows - 1;  // rows past the matrix: never stored
            __builtin_amdgcn_global_load_lds((const void *)(src + (int64_t)grow * ld + k0 + 4 * c),
                                             (gemm_lds_void *)(dst + qw * 4), 16, 0, 0);
        }
    }
}

template <bool PROX>
__global__ __launch_bounds__(kLargeThreads, 1) void wgrad_f32_dma_kernel(
    int M, int Nn, int Kr, const float *__restrict__ A, int64_t lda, const float *__restrict__ Bt,
    int64_t ldb, float *__restrict__ C, int64_t ldc, prox_epi P) {
    constexpr int TM = LBM / LWM / 32, TN = LBN / LWN / 32;
    // the two buffers of each operand as separate arrays: the compiler can
    // then tell the reads of one from the loads into the other
    __shared__ __attribute__((aligned(16))) float A0[LBM * BK];
    __shared__ __attribute__((aligned(16))) float A1[LBM * BK];
    __shared__ __attribute__((aligned(16))) float B0[LBN * BK];
    __shared__ __attribute__((aligned(16))) float B1[LBN * BK];
    const int m0 = blockIdx.y * LBM, n0 = blockIdx.x * LBN;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wm = (wave / LWN) * (LBM / LWM), wn = (wave % LWN) * (LBN / LWN);
    const int lr = lane & 31;
    const int lh = lane >> 5;

    floatx16 acc[TM][TN];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    // fragment offsets: lane (lr, lh) reads chunk 4 lh + q of rows wm + 32a + lr
    // (A) and wn + 32b + lr (B); f of those rows is f(lr)
    int oa[4], ob[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int pos = (lh * 4 + q) ^ swz(lr);
        oa[q] = (wm + lr) * BK + 4 * pos;
        ob[q] = (wn + lr) * BK + 4 * pos;
    }
    const int nchunks = Kr / BK;
    auto step = [&](int c, const float *Ac, const float *Bc, float *An, float *Bn) {
        if (c + 1 < nchunks) {
            dma_rows<LBM>(A, lda, M, m0, (c + 1) * BK, An);
            dma_rows<LBN>(Bt, ldb, Nn, n0, (c + 1) * BK, Bn);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float av[TM][4], bv[TN][4];
#pragma unroll
            for (int a = 0; a < TM; ++a) {
                const float4 x = *reinterpret_cast<const float4 *>(Ac + oa[q] + a * 32 * BK);
                av[a][0] = x.x; av[a][1] = x.y; av[a][2] = x.z; av[a][3] = x.w;
            }
#pragma unroll
            for (int b = 0; b < TN; ++b) {
                const float4 x = *reinterpret_cast<const float4 *>(Bc + ob[q] + b * 32 * BK);
                bv[b][0] = x.x; bv[b][1] = x.y; bv[b][2] = x.z; bv[b][3] = x.w;
            }
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int a = 0; a < TM; ++a)
#pragma unroll
                    for (int b = 0; b < TN; ++b)
                        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[a][s], bv[b][s], acc[a][b], 0, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's loads of the next K-step landed
        __syncthreads();                     // ... and every wave's; this K-step's tiles are free
    };
    dma_rows<LBM>(A, lda, M, m0, 0, A0);
    dma_rows<LBN>(Bt, ldb, Nn, n0, 0, B0);
    __builtin_amdgcn_s_waitcnt(0x0f70);
    __syncthreads();
    for (int c = 0; c < nchunks; c += 2) {
        step(c, A0, B0, A1, B1);
        if (c + 1 < nchunks) step(c + 1, A1, B1, A0, B0);
    }
    if constexpr (PROX) {
        // the last K-step ended with a barrier: the operand buffers are free.
        // The staged index words in A0, then two gather buffers of one MFMA
        // tile each (8 KB) per wave: wave 0 after the words, waves 1-4 in A1,
        // 5-8 in B0, 9-11 in B1.
        constexpr int TPB = 1, GBF = 2 * 16 * TPB * kWave;  // floats per wave
        constexpr int kStageFloats = 2 * LBM * (LBN / 32);
        static_assert(TM == 2 && LWM * LWN == 12 && sizeof(A0) >= sizeof(float) * (kStageFloats + GBF) &&
                          sizeof(A1) >= sizeof(float) * 4 * GBF && sizeof(B0) >= sizeof(float) * 4 * GBF &&
                          sizeof(B1) >= sizeof(float) * 3 * GBF,
                      "staging and gather space");
        int2 *stage = reinterpret_cast<int2 *>(A0);
        prox_stage<LBM, LBN, kLargeThreads>(P, M, m0, n0, stage);
        float *gbuf = wave == 0 ? A0 + kStageFloats
                                : (wave < 5 ? A1 + (wave - 1) * GBF : (wave < 9 ? B0 + (wave - 5) * GBF : B1 + (wave - 9) * GBF));
        prox_store<TN, LBN, TPB, 2>(acc, M, Nn, m0, n0, wm, wn, stage, gbuf, C, ldc, P);
        return;
    }
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
            const int col = n0 + wn + b * 32 + lr;
            if (col >= Nn) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
                if (row < M) C[(int64_t)row * ldc + col] = acc[a][b][r];
            }
        }
}

// measured rates of the two shapes (whole chip, TFLOP/s) and the per-CU round
// model the host chooses by
constexpr int kCUs = 256;
constexpr double kSmallRate = 121.7, kLargeRate = 131.3;

double tile_model_us(int N, int K, int B, int bm, int bn, double rate) {
    const double tiles = (double)ceil_div(N, bm) * (double)ceil_div(K, bn);
    const double per_cu = std::ceil(tiles / kCUs);
    return per_cu * 2.0 * bm * bn * (double)(B > 0 ? B : 1) / (rate * 1e6 / kCUs);
}

// Split reduction for outputs too small to fill the chip (conv filter banks:
// a few 128 x 128 tiles, batch x positions in the tens of thousands): split s
// reduces batch indices [s*chunk, (s+1)*chunk) of every tile into its own
// partial P[s][M][Nn]; wgrad_reduce_kernel then adds the partials in split
// order, so the result is deterministic.
template <bool V4>
__global__ __launch_bounds__(kThreads, 2) void wgrad_split_kernel(
    int M, int Nn, int Kr, int chunk, const float *__restrict__ A, int64_t lda,
    const float *__restrict__ Bt, int64_t ldb, float *__restrict__ P) {
    __shared__ __attribute__((aligned(16))) tile_smem sm;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int k0 = blockIdx.z * chunk;
    const int kr = min(chunk, Kr - k0);
    floatx16 acc[2][2];
    mfma_tile<V4>(M, Nn, kr, A + k0, lda, Bt + k0, ldb, m0, n0, sm, acc);
    float *Ps = P + (int64_t)blockIdx.z * M * Nn;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int col = n0 + acc_col(b);
            if (col >= Nn) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + acc_row(a, r);
                if (row < M) Ps[(int64_t)row * Nn + col] = acc[a][b][r];
            }
        }
}

__global__ void wgrad_reduce_kernel(int M, int Nn, int S, const float *__restrict__ P,
                                    float *__restrict__ C, int64_t ldc) {
    const int64_t n = (int64_t)M * Nn;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        float acc = P[i];
        for (int s = 1; s < S; ++s) acc += P[(int64_t)s * n + i];
        const int64_t row = i / Nn;
        C[row * ldc + (i - row * Nn)] = acc;
    }
}

// the 256x288 shape where its modelled time is shorter
bool f32_large(int N, int K, int B) {
    return tile_model_us(N, K, B, LBM, LBN, kLargeRate) < tile_model_us(N, K, B, BM, BN, kSmallRate);
}

template <bool PROX>
hipError_t launch_f32_tiles(int N, int K, int B, const float *dY, int64_t ldy, const float *X, int64_t ldx,
                            float *C, int64_t ldc, bool v4, const prox_epi &P, hipStream_t s) {
    if (f32_large(N, K, B)) {
        dim3 grid((unsigned)ceil_div(K, LBN), (unsigned)ceil_div(N, LBM));
        if (v4 && B % BK == 0) {
            wgrad_f32_dma_kernel<PROX><<<grid, kLargeThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, C, ldc, P);
            return hipGetLastError();
        }
        if (v4)
            wgrad_f32_large_kernel<true, PROX><<<grid, kLargeThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, C, ldc, P);
        else
            wgrad_f32_large_kernel<false, PROX><<<grid, kLargeThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, C, ldc, P);
        return hipGetLastError();
    }
    dim3 grid((unsigned)ceil_div(K, BN), (unsigned)ceil_div(N, BM));
    if (v4)
        wgrad_f32_mfma_kernel<true, PROX><<<grid, kThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, C, ldc, P);
    else
        wgrad_f32_mfma_kernel<false, PROX><<<grid, kThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, C, ldc, P);
    return hipGetLastError();
}

}  // namespace

wgrad_split wgrad_plan(int N, int K, int B) {
    wgrad_split p{1, B};
    const int64_t tiles = ceil_div(N, BM) * ceil_div(K, BN);
    if (N == 0 || K == 0 || B == 0 || tiles >= 256) return p;
    int64_t s = ceil_div(512, tiles);                  // about 512 workgroups
    s = s < B / 256 ? s : B / 256;                      // at least 256 batch entries each
    s = s < 64 ? s : 64;
    if (s < 2) return p;
    const int64_t chunk = ceil_div(ceil_div(B, s), BK) * BK;  // whole K-steps, 16-byte aligned
    p.splits = (int)ceil_div(B, chunk);
    p.chunk = (int)chunk;
    return p;
}

size_t wgrad_workspace_bytes(int N, int K, int B) {
    const wgrad_split p = wgrad_plan(N, K, B);
    return p.splits > 1 ? sizeof(float) * (size_t)p.splits * N * K : 0;
}

hipError_t launch_wgrad_f32(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                            int64_t ldx, float *dW, int64_t ldw, void *ws, hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    const bool v4 = (ldy % 4 == 0) && (ldx % 4 == 0) && aligned16(dY) && aligned16(X);
    const wgrad_split p = wgrad_plan(N, K, B);
    if (ws != nullptr && p.splits > 1) {
        float *P = static_cast<float *>(ws);
        dim3 grid((unsigned)ceil_div(K, BN), (unsigned)ceil_div(N, BM), (unsigned)p.splits);
        if (v4)
            wgrad_split_kernel<true><<<grid, kThreads, 0, s>>>(N, K, B, p.chunk, dY, ldy, X, ldx, P);
        else
            wgrad_split_kernel<false><<<grid, kThreads, 0, s>>>(N, K, B, p.chunk, dY, ldy, X, ldx, P);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t n = (int64_t)N * K;
        const unsigned rgrid = (unsigned)(ceil_div(n, 256) < 4096 ? ceil_div(n, 256) : 4096);
        wgrad_reduce_kernel<<<rgrid, 256, 0, s>>>(N, K, p.splits, P, dW, ldw);
        return hipGetLastError();
    }
    return launch_f32_tiles<false>(N, K, B, dY, ldy, X, ldx, dW, ldw, v4, prox_epi{}, s);
}

int wgrad_f32_prox_slab(int N, int K, int B) {
    if (wgrad_plan(N, K, B).splits > 1) return 0;
    return f32_large(N, K, B) ? LBN / LWN : BN / 2;
}

hipError_t launch_wgrad_f32_prox(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                                 int64_t ldx, float *Z, int64_t ldz, const prox_epi &P, hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    const bool v4 = (ldy % 4 == 0) && (ldx % 4 == 0) && aligned16(dY) && aligned16(X);
    return launch_f32_tiles<true>(N, K, B, dY, ldy, X, ldx, Z, ldz, v4, P, s);
}

}  // namespace l1csr
