// Dense weight gradient dW[N][K] = dY[N][B] . X[K][B]^T with bf16 operands on
// the matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
// The operands stay fp32 in memory; each element is rounded to bf16 (round to
// nearest even, v_cvt_pk_bf16_f32) as its tile is staged into LDS.  A product
// of two bf16 values is exact in fp32, so the only differences from the fp32
// path are the input roundings (at most 2^-8 relative each: 8 significant
// bits, nearest even) and the fp32 summation.
//
// Same tiling as the fp32 kernel: a 256-thread workgroup owns a 128x128 tile
// of dW as 2x2 waves of 64x64, each wave 2x2 MFMA tiles of 32x32; reduction
// chunks of 64 (four MFMA steps of 16) are double buffered through LDS.  LDS
// rows are 72 bf16 (144 bytes): the 16-byte fragment reads of 16 consecutive
// rows then fall on distinct bank groups.  An MFMA step pairs the A and B
// elements that sit at the same (lane half, position) of their fragments;
// both operands use the same assignment of the chunk's 16 reduction indices
// to those slots (lane half h, position j -> index 8h + j), so the sum is the
// product's.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // bf16 elements per LDS row
constexpr int kThreads = 256;
constexpr int kLoadsPerThread = (BM * BK / 4) / kThreads;  // float4 loads per operand: 8

template <bool V4>
__device__ __forceinline__ void load_tile(const float *__restrict__ src, int64_t ld, int rows,
                                          int kred, int row0, int k0, float4 (&r)[kLoadsPerThread]) {
#pragma unroll
    for (int i = 0; i < kLoadsPerThread; ++i) {
        const int f = threadIdx.x + i * kThreads;  // float4 index inside the tile
        const int rr = f >> 4;                      // 16 float4 per tile row
        const int kk = (f & 15) * 4;
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

__device__ __forceinline__ void store_tile(__bf16 *lds, const float4 (&r)[kLoadsPerThread]) {
#pragma unroll
    for (int i = 0; i < kLoadsPerThread; ++i) {
        const int f = threadIdx.x + i * kThreads;
        const int rr = f >> 4;
        const int kk = (f & 15) * 4;
        bf16x4 h;
        h[0] = (__bf16)r[i].x;
        h[1] = (__bf16)r[i].y;
        h[2] = (__bf16)r[i].z;
        h[3] = (__bf16)r[i].w;
        *reinterpret_cast<bf16x4 *>(lds + rr * LDS_STRIDE + kk) = h;
    }
}

template <bool V4>
__global__ __launch_bounds__(kThreads, 2) void wgrad_bf16_mfma_kernel(
    int M, int Nn, int Kr, const float *__restrict__ A, int64_t lda, const float *__restrict__ Bt,
    int64_t ldb, float *__restrict__ C, int64_t ldc) {
    __shared__ __attribute__((aligned(16))) __bf16 As[2][BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) __bf16 Bs[2][BN * LDS_STRIDE];

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
    store_tile(As[0], ra);
    store_tile(Bs[0], rb);
    __syncthreads();

    for (int c = 0; c < nchunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunks) {
            load_tile<V4>(A, lda, M, Kr, m0, (c + 1) * BK, ra);
            load_tile<V4>(Bt, ldb, Nn, Kr, n0, (c + 1) * BK, rb);
        }
        const __bf16 *as0 = As[buf] + (wm + lr) * LDS_STRIDE + lh * 8;
        const __bf16 *as1 = as0 + 32 * LDS_STRIDE;
        const __bf16 *bs0 = Bs[buf] + (wn + lr) * LDS_STRIDE + lh * 8;
        const __bf16 *bs1 = bs0 + 32 * LDS_STRIDE;
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(as0 + 16 * s);
            const bf16x8 a1 = *reinterpret_cast<const bf16x8 *>(as1 + 16 * s);
            const bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(bs0 + 16 * s);
            const bf16x8 b1 = *reinterpret_cast<const bf16x8 *>(bs1 + 16 * s);
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        }
        if (c + 1 < nchunks) {
            store_tile(As[buf ^ 1], ra);
            store_tile(Bs[buf ^ 1], rb);
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

hipError_t launch_wgrad_bf16(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                             int64_t ldx, float *dW, int64_t ldw, hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    dim3 grid((unsigned)ceil_div(K, BN), (unsigned)ceil_div(N, BM));
    const bool v4 = (ldy % 4 == 0) && (ldx % 4 == 0) && aligned16(dY) && aligned16(X);
    if (v4)
        wgrad_bf16_mfma_kernel<true><<<grid, kThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, dW, ldw);
    else
        wgrad_bf16_mfma_kernel<false><<<grid, kThreads, 0, s>>>(N, K, B, dY, ldy, X, ldx, dW, ldw);
    return hipGetLastError();
}

}  // namespace l1csr
