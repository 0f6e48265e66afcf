// Dense weight gradient dW[N][K] = dY[N][B] . X[K][B]^T on the bf16 matrix
// cores (v_mfma_f32_32x32x16_bf16) with each fp32 operand split into two bf16
// parts: hi = bf16(x), lo = bf16(x - hi) (x - hi is exact in fp32).  A product
// is taken as hi_a hi_b + hi_a lo_b + lo_a hi_b; every bf16 product is exact
// in fp32 and accumulated in fp32.  The dropped lo_a lo_b term and the parts'
// own rounding leave at most 3 (1 + 2^-7) 2^-16 |a b| per product, inside the
// fp32 contract of the l1-phase gradient, at about twice the fp32 matrix-core
// speed (the bf16 pipe is 16x the fp32 one; three products per pair).
//
// Tiles: a workgroup of WM x WN waves owns a BM x BN tile of dW, each wave
// (BM/WM) x (BN/WN) as TM x TN MFMA tiles of 32x32.  Reduction chunks of BK
// are loaded as fp32, split while they are staged into LDS (hi and lo tiles,
// rows of BK + 8 bf16, so the 16-byte fragment reads of 16 consecutive rows
// fall on distinct banks) and double buffered.  An MFMA step pairs the A and
// B elements at the same (lane half, position) of their fragments; both
// operands map the step's 16 reduction indices to those slots the same way
// (lane half h, position j -> index 8h + j), so every product pairs matching
// batch indices.  Two shapes are built:
//   128 x 128, 2 x 2 waves of 64 x 64, BK 32, two workgroups per CU;
//   256 x 288, 4 x 3 waves of 64 x 96, BK 16, one workgroup of 12 waves per CU
//     (fewer LDS reads and staged bytes per MFMA; 4096 x 9216 is 512 tiles,
//     two whole rounds of the 256 CUs).
// The host picks the shape with the shorter modelled time: per CU, the tiles
// it runs (ceil(tiles / 256)) times the tile's time at the shape's measured
// rate.
#include <cmath>

#include "common.hpp"
#include "launch.hpp"
#include "prox_epilogue.hpp"

namespace l1csr {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kCUs = 256;

template <bool V4, int BK, int ROWS, int NT>
__device__ __forceinline__ void load_tile(const float *__restrict__ src, int64_t ld, int rows, int kred,
                                          int row0, int k0, float4 (&r)[(ROWS * BK / 4 + NT - 1) / NT]) {
    constexpr int LPT = (ROWS * BK / 4 + NT - 1) / NT;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
        const int f = threadIdx.x + i * NT;  // float4 index inside the tile
        const int rr = f / (BK / 4), kk = (f % (BK / 4)) * 4;
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

// hi = bf16(x) and lo = bf16(x - hi), both round to nearest even
template <int BK, int ROWS, int NT>
__device__ __forceinline__ void store_split(__bf16 *hi, __bf16 *lo, const float4 (&r)[(ROWS * BK / 4 + NT - 1) / NT]) {
    constexpr int LPT = (ROWS * BK / 4 + NT - 1) / NT, STR = BK + 8;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
        const int f = threadIdx.x + i * NT;
        const int rr = f / (BK / 4), kk = (f % (BK / 4)) * 4;
        if (rr >= ROWS) continue;
        const float v[4] = {r[i].x, r[i].y, r[i].z, r[i].w};
        bf16x4 h, l;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            h[e] = (__bf16)v[e];
            l[e] = (__bf16)(v[e] - (float)h[e]);
        }
        *reinterpret_cast<bf16x4 *>(hi + rr * STR + kk) = h;
        *reinterpret_cast<bf16x4 *>(lo + rr * STR + kk) = l;
    }
}

__device__ __forceinline__ floatx16 mfma(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// PROX: the epilogue writes Z = S_t(W - eta*dW) and the per-(row, slab)
// counts instead of dW (prox_epilogue.hpp)
template <bool V4, int BM, int BN, int WM, int WN, int BK, int MINB, bool PROX>
__global__ __launch_bounds__(64 * WM * WN, MINB) void wgrad_bf16x3_mfma_kernel(
    int M, int Nn, int Kr, const float *__restrict__ A, int64_t lda, const float *__restrict__ Bt,
    int64_t ldb, float *__restrict__ C, int64_t ldc, prox_epi P) {
    constexpr int NT = 64 * WM * WN, TM = BM / WM / 32, TN = BN / WN / 32, STR = BK + 8;
    constexpr int LA = (BM * BK / 4 + NT - 1) / NT, LB = (BN * BK / 4 + NT - 1) / NT;
    static_assert(TM * WM * 32 == BM && TN * WN * 32 == BN && BK % 16 == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) __bf16 Ah[2][BM * STR];
    __shared__ __attribute__((aligned(16))) __bf16 Al[2][BM * STR];
    __shared__ __attribute__((aligned(16))) __bf16 Bh[2][BN * STR];
    __shared__ __attribute__((aligned(16))) __bf16 Bl[2][BN * STR];

    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wm = (wave / WN) * (BM / WM), wn = (wave % WN) * (BN / WN);
    const int lr = lane & 31;  // row inside a 32x32 tile (A) / column (B)
    const int lh = lane >> 5;  // lane half: reduction indices 8h .. 8h+7 of a step

    floatx16 acc[TM][TN];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    const int nchunks = (Kr + BK - 1) / BK;
    float4 ra[LA], rb[LB];
    load_tile<V4, BK, BM, NT>(A, lda, M, Kr, m0, 0, ra);
    load_tile<V4, BK, BN, NT>(Bt, ldb, Nn, Kr, n0, 0, rb);
    store_split<BK, BM, NT>(Ah[0], Al[0], ra);
    store_split<BK, BN, NT>(Bh[0], Bl[0], rb);
    __syncthreads();

    const int oa = (wm + lr) * STR + lh * 8, ob = (wn + lr) * STR + lh * 8;
    for (int c = 0; c < nchunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunks) {
            load_tile<V4, BK, BM, NT>(A, lda, M, Kr, m0, (c + 1) * BK, ra);
            load_tile<V4, BK, BN, NT>(Bt, ldb, Nn, Kr, n0, (c + 1) * BK, rb);
        }
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            bf16x8 ah[TM], al[TM], bh[TN], bl[TN];
#pragma unroll
            for (int a = 0; a < TM; ++a) {
                ah[a] = *reinterpret_cast<const bf16x8 *>(Ah[buf] + oa + a * 32 * STR + 16 * s);
                al[a] = *reinterpret_cast<const bf16x8 *>(Al[buf] + oa + a * 32 * STR + 16 * s);
            }
#pragma unroll
            for (int b = 0; b < TN; ++b) {
                bh[b] = *reinterpret_cast<const bf16x8 *>(Bh[buf] + ob + b * 32 * STR + 16 * s);
                bl[b] = *reinterpret_cast<const bf16x8 *>(Bl[buf] + ob + b * 32 * STR + 16 * s);
            }
            // the two small terms first, then hi . hi
#pragma unroll
            for (int a = 0; a < TM; ++a)
#pragma unroll
                for (int b = 0; b < TN; ++b) acc[a][b] = mfma(al[a], bh[b], acc[a][b]);
#pragma unroll
            for (int a = 0; a < TM; ++a)
#pragma unroll
                for (int b = 0; b < TN; ++b) acc[a][b] = mfma(ah[a], bl[b], acc[a][b]);
#pragma unroll
            for (int a = 0; a < TM; ++a)
#pragma unroll
                for (int b = 0; b < TN; ++b) acc[a][b] = mfma(ah[a], bh[b], acc[a][b]);
        }
        if (c + 1 < nchunks) {
            store_split<BK, BM, NT>(Ah[buf ^ 1], Al[buf ^ 1], ra);
            store_split<BK, BN, NT>(Bh[buf ^ 1], Bl[buf ^ 1], rb);
        }
        __syncthreads();
    }

    if constexpr (PROX) {
        // the last chunk ended with a barrier: the operand buffers are free
        static_assert(TM == 2 && sizeof(Ah) >= sizeof(int2) * BM * (BN / 32), "staging space");
        int2 *stage = reinterpret_cast<int2 *>(&Ah[0][0]);
        prox_stage<BM, BN, NT>(P, M, m0, n0, stage);
        // gather buffers of one MFMA tile (4 KB) per wave: half the waves in
        // the bf16 hi tiles of B, half in the lo tiles
        constexpr int GBF = 16 * kWave;
        static_assert(sizeof(Bh) >= sizeof(float) * GBF * (NT / 128) && sizeof(Bl) >= sizeof(float) * GBF * (NT / 128),
                      "gather space");
        const int hw = wave % (NT / 128);
        float *gbuf = (wave < NT / 128 ? reinterpret_cast<float *>(&Bh[0][0]) : reinterpret_cast<float *>(&Bl[0][0])) +
                      hw * GBF;
        prox_store<TN, BN, 1>(acc, M, Nn, m0, n0, wm, wn, stage, gbuf, C, ldc, P);
        return;
    }
    // D layout of the 32x32 MFMA: lane l, register r holds
    // row 8*(r/4) + 4*(l/32) + r%4, column l%32 of the 32x32 tile.
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

// one built shape and its measured rate (fp32-equivalent TFLOP/s, whole chip)
template <int BM, int BN, int WM, int WN, int BK, int MINB>
struct x3_shape {
    static double model_us(int N, int K, int B, double rate_tflops) {
        const double tiles = (double)ceil_div(N, BM) * (double)ceil_div(K, BN);
        const double per_cu = std::ceil(tiles / kCUs);
        const double tile_flops = 2.0 * BM * BN * (double)(B > 0 ? B : 1);
        return per_cu * tile_flops / (rate_tflops * 1e6 / kCUs);
    }
    static constexpr int kSlab = 32 * (BN / WN / 32);  // a wave's columns
    template <bool PROX>
    static hipError_t launch(int N, int K, int B, const float *dY, int64_t ldy, const float *X, int64_t ldx,
                             float *dW, int64_t ldw, bool v4, const prox_epi &P, hipStream_t s) {
        dim3 grid((unsigned)ceil_div(K, BN), (unsigned)ceil_div(N, BM));
        if (v4)
            wgrad_bf16x3_mfma_kernel<true, BM, BN, WM, WN, BK, MINB, PROX><<<grid, 64 * WM * WN, 0, s>>>(
                N, K, B, dY, ldy, X, ldx, dW, ldw, P);
        else
            wgrad_bf16x3_mfma_kernel<false, BM, BN, WM, WN, BK, MINB, PROX><<<grid, 64 * WM * WN, 0, s>>>(
                N, K, B, dY, ldy, X, ldx, dW, ldw, P);
        return hipGetLastError();
    }
};
using x3_small = x3_shape<128, 128, 2, 2, 32, 2>;
using x3_large = x3_shape<256, 288, 4, 3, 16, 1>;
constexpr double kSmallRate = 283.0, kLargeRate = 355.0;

bool x3_large_shape(int N, int K, int B) {
    return x3_large::model_us(N, K, B, kLargeRate) < x3_small::model_us(N, K, B, kSmallRate);
}

}  // namespace

hipError_t launch_wgrad_bf16x3(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                               int64_t ldx, float *dW, int64_t ldw, hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    const bool v4 = (ldy % 4 == 0) && (ldx % 4 == 0) && aligned16(dY) && aligned16(X);
    if (x3_large_shape(N, K, B))
        return x3_large::launch<false>(N, K, B, dY, ldy, X, ldx, dW, ldw, v4, prox_epi{}, s);
    return x3_small::launch<false>(N, K, B, dY, ldy, X, ldx, dW, ldw, v4, prox_epi{}, s);
}

int wgrad_bf16x3_prox_slab(int N, int K, int B) {
    return x3_large_shape(N, K, B) ? x3_large::kSlab : x3_small::kSlab;
}

hipError_t launch_wgrad_bf16x3_prox(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                                    int64_t ldx, float *Z, int64_t ldz, const prox_epi &P, hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    const bool v4 = (ldy % 4 == 0) && (ldx % 4 == 0) && aligned16(dY) && aligned16(X);
    if (x3_large_shape(N, K, B)) return x3_large::launch<true>(N, K, B, dY, ldy, X, ldx, Z, ldz, v4, P, s);
    return x3_small::launch<true>(N, K, B, dY, ldy, X, ldx, Z, ldz, v4, P, s);
}

}  // namespace l1csr
