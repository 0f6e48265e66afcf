// CSR x dense products with the batch index contiguous (forward Y = W.X and,
// over the CSC copy, backward dX = W^T.dY).
//
// Mapping: one wave per (row, batch chunk).  Lanes run over the batch, so the
// X row of every nonzero is read as one coalesced 64*VEC-float segment and the
// nonzero's column and value are wave-uniform: the wave loads 64 (col, val)
// pairs with one coalesced load each and broadcasts them with readlane, so
// the index stream costs 8 bytes per nonzero instead of a dependent load per
// lane.  No cross-lane reduction is needed.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

template <int VEC>
struct vec_t;
template <>
struct vec_t<1> {
    using type = float;
};
template <>
struct vec_t<4> {
    using type = float4;
};

template <int VEC>
__device__ __forceinline__ void load_vec(const float *p, float (&x)[VEC]) {
    if constexpr (VEC == 4) {
        const float4 t = *reinterpret_cast<const float4 *>(p);
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    } else {
        x[0] = *p;
    }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float *p, const float (&x)[VEC]) {
    if constexpr (VEC == 4) {
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
    } else {
        *p = x[0];
    }
}

constexpr int kRowsPerBlock = 4;  // 4 waves per 256-thread block

// Y[row][b] = sum_p vals[perm? perm[p] : p] * X[idx[p]][b]
template <int VEC, bool PERM>
__global__ __launch_bounds__(256) void spmm_rows_kernel(
    int n_rows, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ vals, const int *__restrict__ perm, const float *__restrict__ X,
    int64_t ldx, int B, float *__restrict__ Y, int64_t ldy) {
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int b = (blockIdx.y * kWave + lane) * VEC;
    const bool active = b < B;
    const int start = uniform(ptr[row]);
    const int end = uniform(ptr[row + 1]);

    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;

    for (int base = start; base < end; base += kWave) {
        const int n = min(kWave, end - base);
        int c = 0;
        float v = 0.f;
        if (lane < n) {
            const int q = base + lane;
            c = idx[q];
            v = vals[PERM ? perm[q] : q];
        }
        int j = 0;
        for (; j + 4 <= n; j += 4) {
            const int c0 = lane_bcast(c, j), c1 = lane_bcast(c, j + 1);
            const int c2 = lane_bcast(c, j + 2), c3 = lane_bcast(c, j + 3);
            const float v0 = lane_bcast(v, j), v1 = lane_bcast(v, j + 1);
            const float v2 = lane_bcast(v, j + 2), v3 = lane_bcast(v, j + 3);
            if (active) {
                float x0[VEC], x1[VEC], x2[VEC], x3[VEC];
                load_vec<VEC>(X + (int64_t)c0 * ldx + b, x0);
                load_vec<VEC>(X + (int64_t)c1 * ldx + b, x1);
                load_vec<VEC>(X + (int64_t)c2 * ldx + b, x2);
                load_vec<VEC>(X + (int64_t)c3 * ldx + b, x3);
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    acc[e] = fmaf(v0, x0[e], acc[e]);
                    acc[e] = fmaf(v1, x1[e], acc[e]);
                    acc[e] = fmaf(v2, x2[e], acc[e]);
                    acc[e] = fmaf(v3, x3[e], acc[e]);
                }
            }
        }
        for (; j < n; ++j) {
            const int cj = lane_bcast(c, j);
            const float vj = lane_bcast(v, j);
            if (active) {
                float x0[VEC];
                load_vec<VEC>(X + (int64_t)cj * ldx + b, x0);
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc[e] = fmaf(vj, x0[e], acc[e]);
            }
        }
    }
    if (active) store_vec<VEC>(Y + (int64_t)row * ldy + b, acc);
}

// dX[idx[p]][b] += vals[p] * dY[row][b] with float atomics (order varies)
template <int VEC>
__global__ __launch_bounds__(256) void spmm_scatter_atomic_kernel(
    int n_rows, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ vals, const float *__restrict__ dY, int64_t ldy, int B,
    float *__restrict__ dX, int64_t ldx) {
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int b = (blockIdx.y * kWave + lane) * VEC;
    const bool active = b < B;
    const int start = uniform(ptr[row]);
    const int end = uniform(ptr[row + 1]);
    float y[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) y[e] = 0.f;
    if (active) load_vec<VEC>(dY + (int64_t)row * ldy + b, y);
    for (int base = start; base < end; base += kWave) {
        const int n = min(kWave, end - base);
        int c = 0;
        float v = 0.f;
        if (lane < n) {
            c = idx[base + lane];
            v = vals[base + lane];
        }
        for (int j = 0; j < n; ++j) {
            const int cj = lane_bcast(c, j);
            const float vj = lane_bcast(v, j);
            if (active) {
                float *d = dX + (int64_t)cj * ldx + b;
#pragma unroll
                for (int e = 0; e < VEC; ++e) unsafeAtomicAdd(d + e, vj * y[e]);
            }
        }
    }
}

}  // namespace

hipError_t launch_spmm_rows(int n_rows, int64_t nnz, const int *ptr, const int *idx,
                            const float *vals, const int *perm, const float *X, int64_t ldx,
                            int B, float *Y, int64_t ldy, hipStream_t s) {
    (void)nnz;
    if (n_rows == 0 || B == 0) return hipSuccess;
    const bool v4 = (B % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) && aligned16(Y);
    const int vec = v4 ? 4 : 1;
    dim3 grid((unsigned)ceil_div(n_rows, kRowsPerBlock), (unsigned)ceil_div(B, kWave * vec));
    if (v4) {
        if (perm)
            spmm_rows_kernel<4, true><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, perm, X, ldx, B, Y, ldy);
        else
            spmm_rows_kernel<4, false><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, perm, X, ldx, B, Y, ldy);
    } else {
        if (perm)
            spmm_rows_kernel<1, true><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, perm, X, ldx, B, Y, ldy);
        else
            spmm_rows_kernel<1, false><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, perm, X, ldx, B, Y, ldy);
    }
    return hipGetLastError();
}

hipError_t launch_spmm_scatter_atomic(int n_rows, int n_cols, const int *ptr, const int *idx,
                                      const float *vals, const float *dY, int64_t ldy, int B,
                                      float *dX, int64_t ldx, hipStream_t s) {
    hipError_t e = launch_fill_rows_f32(dX, n_cols, B, ldx, 0.f, s);
    if (e != hipSuccess || n_rows == 0 || B == 0) return e;
    const bool v4 = (B % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(dY) && aligned16(dX);
    const int vec = v4 ? 4 : 1;
    dim3 grid((unsigned)ceil_div(n_rows, kRowsPerBlock), (unsigned)ceil_div(B, kWave * vec));
    if (v4)
        spmm_scatter_atomic_kernel<4><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, dY, ldy, B, dX, ldx);
    else
        spmm_scatter_atomic_kernel<1><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, dY, ldy, B, dX, ldx);
    return hipGetLastError();
}

}  // namespace l1csr
