// Proximal soft-threshold step, Eq. (prox):  Z = S_t(W - eta*G), t = eta*lambda.
//
// Arithmetic in double (the precision of the paper's prox kernel): eta*g is
// exact in double, so z = w - eta*g rounds once; S_t(z) rounds once more to
// float.  S_t(z) = z - t for z > t, z + t for z < -t, +0 otherwise, which is
// sgn(z)*max(|z|-t, 0) written branch by branch.
//
// Dense mode: one 256-thread workgroup per row.  The row of W (CSR) is
// scattered into a zeroed LDS copy, then the row of G is streamed with 16-byte
// loads; Z is written and the nonzeros of the row are counted.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kProxThreads = 256;
constexpr int kProxTile = 8192;  // columns per LDS pass (32 KB)

__device__ __forceinline__ float soft_threshold(float w, float g, double eta, double t) {
    const double z = (double)w - eta * (double)g;
    const double s = z > t ? z - t : (z < -t ? z + t : 0.0);
    return (float)s;
}

template <bool V4>
__global__ __launch_bounds__(kProxThreads) void prox_dense_kernel(
    int n_rows, int n_cols, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ vals, const float *G, int64_t ldg, double eta, double t, float *Z,
    int64_t ldz, int *__restrict__ row_counts) {
    __shared__ float wrow[kProxTile];
    __shared__ int wave_cnt[kProxThreads / kWave];
    const int row = blockIdx.x;
    const int tid = threadIdx.x;
    const int s = ptr[row], e = ptr[row + 1];
    const float *g = G + (int64_t)row * ldg;
    float *z = Z + (int64_t)row * ldz;
    int cnt = 0;
    for (int k0 = 0; k0 < n_cols; k0 += kProxTile) {
        const int k1 = min(n_cols, k0 + kProxTile);
        for (int k = tid; k < k1 - k0; k += kProxThreads) wrow[k] = 0.f;
        __syncthreads();
        for (int p = s + tid; p < e; p += kProxThreads) {
            const int k = idx[p];
            if (k >= k0 && k < k1) wrow[k - k0] = vals[p];
        }
        __syncthreads();
        if (V4) {
            for (int k = k0 + tid * 4; k < k1; k += kProxThreads * 4) {
                if (k + 3 < k1) {
                    const float4 gv = *reinterpret_cast<const float4 *>(g + k);
                    float4 o;
                    o.x = soft_threshold(wrow[k - k0 + 0], gv.x, eta, t);
                    o.y = soft_threshold(wrow[k - k0 + 1], gv.y, eta, t);
                    o.z = soft_threshold(wrow[k - k0 + 2], gv.z, eta, t);
                    o.w = soft_threshold(wrow[k - k0 + 3], gv.w, eta, t);
                    *reinterpret_cast<float4 *>(z + k) = o;
                    cnt += (o.x != 0.f) + (o.y != 0.f) + (o.z != 0.f) + (o.w != 0.f);
                } else {
                    for (int kk = k; kk < k1; ++kk) {
                        const float o = soft_threshold(wrow[kk - k0], g[kk], eta, t);
                        z[kk] = o;
                        cnt += (o != 0.f);
                    }
                }
            }
        } else {
            for (int k = k0 + tid; k < k1; k += kProxThreads) {
                const float o = soft_threshold(wrow[k - k0], g[k], eta, t);
                z[k] = o;
                cnt += (o != 0.f);
            }
        }
        __syncthreads();
    }
    if (row_counts) {
        cnt = wave_sum_int(cnt);
        if ((tid & 63) == 0) wave_cnt[tid >> 6] = cnt;
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < kProxThreads / kWave; ++w) tot += wave_cnt[w];
            row_counts[row] = tot;
        }
    }
}

__global__ void prox_csr_kernel(int64_t nnz, float *__restrict__ vals, const float *__restrict__ g,
                                double eta, double t) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * blockDim.x)
        vals[p] = soft_threshold(vals[p], g[p], eta, t);
}

}  // namespace

hipError_t launch_prox_dense(int n_rows, int n_cols, const int *ptr, const int *idx,
                             const float *vals, const float *G, int64_t ldg, float eta, double t,
                             float *Z, int64_t ldz, int *row_counts, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    const bool v4 = (ldg % 4 == 0) && (ldz % 4 == 0) && aligned16(G) && aligned16(Z);
    if (v4)
        prox_dense_kernel<true><<<n_rows, kProxThreads, 0, s>>>(n_rows, n_cols, ptr, idx, vals, G, ldg,
                                                                (double)eta, t, Z, ldz, row_counts);
    else
        prox_dense_kernel<false><<<n_rows, kProxThreads, 0, s>>>(n_rows, n_cols, ptr, idx, vals, G, ldg,
                                                                 (double)eta, t, Z, ldz, row_counts);
    return hipGetLastError();
}

hipError_t launch_prox_csr(int64_t nnz, float *vals, const float *g, float eta, double t,
                           hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    int64_t grid = ceil_div(nnz, 256);
    if (grid > 65536) grid = 65536;
    prox_csr_kernel<<<(unsigned)grid, 256, 0, s>>>(nnz, vals, g, (double)eta, t);
    return hipGetLastError();
}

}  // namespace l1csr
