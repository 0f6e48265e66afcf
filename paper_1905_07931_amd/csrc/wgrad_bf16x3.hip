// Dense weight gradient dW[N][K] = dY[N][B] . X[K][B]^T on the bf16 matrix
// cores (v_mfma_f32_32x32x16_bf16) with each fp32 operand split into two bf16
// parts: hi = bf16(x), lo = bf16(x - hi) (x - hi is exact in fp32).  A product
// is taken as hi_a hi_b + hi_a lo_b + lo_a hi_b; every bf16 product is exact
// in fp32 and accumulated in fp32.  The dropped lo_a lo_b term and the parts'
// own rounding leave at most 3 (1 + 2^-7) 2^-16 |a b| per product, inside the
// fp32 contract of the l1-phase gradient, at about twice the fp32 matrix-core
// speed (the bf16 pipe is 16x the fp32 one; three products per pair).
//
// Tiling as in the fp32 kernel: a 256-thread workgroup owns a 128x128 tile of
// dW as 2x2 waves of 64x64, each wave 2x2 MFMA tiles of 32x32.  Reduction
// chunks of 32 (two MFMA steps of 16) are loaded as fp32, split while they are
// staged into LDS (hi and lo tiles, rows of 40 bf16 = 80 bytes, so the
// 16-byte fragment reads of 16 consecutive rows fall on distinct banks) and
// double buffered.  An MFMA step pairs the A and B elements at the same (lane
// half, position) of their fragments; both operands map the step's 16
// reduction indices to those slots the same way (lane half h, position j ->
// index 8h + j), so every product pairs matching batch indices.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDS_STRIDE = BK + 8;  // bf16 elements per LDS row
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

// hi = bf16(x) and lo = bf16(x - hi), both round to nearest even
__device__ __forceinline__ void store_split(__bf16 *hi, __bf16 *lo, const float4 (&r)[kLoadsPerThread]) {
#pragma unroll
    for (int i = 0; i < kLoadsPerThread; ++i) {
        const int f = threadIdx.x + i * kThreads;
        const int rr = f >> 3;
        const int kk = (f & 7) * 4;
        const float v[4] = {r[i].x, r[i].y, r[i].z, r[i].w};
        bf16x4 h, l;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            h[e] = (__bf16)v[e];
            l[e] = (__bf16)(v[e] - (float)h[e]);
        }
        *reinterpret_cast<bf16x4 *>(hi + rr * LDS_STRIDE + kk) = h;
        *reinterpret_cast<bf16x4 *>(lo + rr * LDS_STRIDE + kk) = l;
    }
}

__device__ __forceinline__ floatx16 mfma(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

template <bool V4>
__global__ __launch_bounds__(kThreads, 2) void wgrad_bf16x3_mfma_kernel(
    int M, int Nn, int Kr, const float *__restrict__ A, int64_t lda, const float *__restrict__ Bt,
    int64_t ldb, float *__restrict__ C, int64_t ldc) {
    __shared__ __attribute__((aligned(16))) __bf16 Ah[2][BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) __bf16 Al[2][BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) __bf16 Bh[2][BN * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) __bf16 Bl[2][BN * LDS_STRIDE];

    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
    const int lr = lane & 31;  // row inside a 32x32 tile (A) / column (B)
    const int lh = lane >> 5;  // lane half: reduction indices 8h .. 8h+7 of a step

    floatx16 acc[2][2];
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
    store_split(Ah[0], Al[0], ra);
    store_split(Bh[0], Bl[0], rb);
    __syncthreads();

    const int oa0 = (wm + lr) * LDS_STRIDE + lh * 8, oa1 = oa0 + 32 * LDS_STRIDE;
    const int ob0 = (wn + lr) * LDS_STRIDE + lh * 8, ob1 = ob0 + 32 * LDS_STRIDE;
    for (int c = 0; c < nchunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunks) {
            load_tile<V4>(A, lda, M, Kr, m0, (c + 1) * BK, ra);
            load_tile<V4>(Bt, ldb, Nn, Kr, n0, (c + 1) * BK, rb);
        }
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            const bf16x8 a0h = *reinterpret_cast<const bf16x8 *>(Ah[buf] + oa0 + 16 * s);
            const bf16x8 a1h = *reinterpret_cast<const bf16x8 *>(Ah[buf] + oa1 + 16 * s);
            const bf16x8 b0h = *reinterpret_cast<const bf16x8 *>(Bh[buf] + ob0 + 16 * s);
            const bf16x8 b1h = *reinterpret_cast<const bf16x8 *>(Bh[buf] + ob1 + 16 * s);
            const bf16x8 a0l = *reinterpret_cast<const bf16x8 *>(Al[buf] + oa0 + 16 * s);
            const bf16x8 a1l = *reinterpret_cast<const bf16x8 *>(Al[buf] + oa1 + 16 * s);
            const bf16x8 b0l = *reinterpret_cast<const bf16x8 *>(Bl[buf] + ob0 + 16 * s);
            const bf16x8 b1l = *reinterpret_cast<const bf16x8 *>(Bl[buf] + ob1 + 16 * s);
            // the two small terms first, then hi . hi
            acc[0][0] = mfma(a0l, b0h, acc[0][0]);
            acc[0][1] = mfma(a0l, b1h, acc[0][1]);
            acc[1][0] = mfma(a1l, b0h, acc[1][0]);
            acc[1][1] = mfma(a1l, b1h, acc[1][1]);
            acc[0][0] = mfma(a0h, b0l, acc[0][0]);
            acc[0][1] = mfma(a0h, b1l, acc[0][1]);
            acc[1][0] = mfma(a1h, b0l, acc[1][0]);
            acc[1][1] = mfma(a1h, b1l, acc[1][1]);
            acc[0][0] = mfma(a0h, b0h, acc[0][0]);
            acc[0][1] = mfma(a0h, b1h, acc[0][1]);
            acc[1][0] = mfma(a1h, b0h, acc[1][0]);
            acc[1][1] = mfma(a1h, b1h, acc[1][1]);
        }
        if (c + 1 < nchunks) {
            store_split(Ah[buf ^ 1], Al[buf ^ 1], ra);
            store_split(Bh[buf ^ 1], Bl[buf ^ 1], rb);
        }
        __syncthreads();
    }

    // D layout of the 32x32 MFMA: lane l, register r holds
    // row 8*(r/4) + 4*(l/32) + r%4, column l%32 of the 32x32 tile.
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int col = n0 + wn + b * 32 + lr;
            if (col >= Nn) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm + a * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
                if (row < M) C[(int64_t)row * ldc + col] = acc[a][b][r];
            }
        }
}

}  // namespace

hipError_t launch_wgrad_bf16x3(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                               int64_t ldx, float *dW, int64_t ldw, hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    dim3 grid((unsigned)ceil_div(K, BN), (unsigned)ceil_div(N, BM));
    const bool v4 = (ldy % 4 == 0) && (ldx % 4 == 0) && aligned16(dY) && aligned16(X);
    if (v4)
        wgrad_bf16x3_mfma_kernel<true><<<grid, kThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, dW, ldw);
    else
        wgrad_bf16x3_mfma_kernel<false><<<grid, kThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, dW, ldw);
    return hipGetLastError();
}

}  // namespace l1csr
