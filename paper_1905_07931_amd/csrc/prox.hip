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
#include "prox_epilogue.hpp"

namespace l1csr {

namespace {

constexpr int kProxThreads = 256;
constexpr int kProxTile = 8192;  // columns per LDS pass (32 KB)

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


// Fused prox + recompression, two passes over G without writing Z.  The work
// unit is a slab: kSlab consecutive columns of one row, one 256-thread
// workgroup each, so that many rows are in flight on a CU at once (a slab
// keeps an 8 KB LDS copy of its part of W's row and two 16-byte G loads per
// thread in registers).
//   COUNT: counts[slab] = number of nonzero S_t(w - eta*g) in the slab
//   FILL:  recompute the same values and compact them to off[slab] in the
//          output, in column order (a block-wide prefix per 1024-column
//          chunk: one ballot per column slot, wave totals through LDS).
// Slabs are numbered row-major, so the exclusive scan of the counts is
// exactly the CSR layout of the result, and row_ptr[row] = off[row * S].
// seg[row][j] (j = 0 .. S) = first entry of the row with column >= j * kSlab,
// so a slab reads only its own entries of W.
constexpr int kSlabShift = kProxSlabShift;
constexpr int kSlab = 1 << kSlabShift;
constexpr int kSlabChunks = kSlab / (kProxThreads * 4);

template <bool V4, bool FILL>
__global__ __launch_bounds__(kProxThreads) void prox_slab_kernel(
    int n_cols, int slabs, const int *__restrict__ seg, const int *__restrict__ idx,
    const float *__restrict__ vals, const float *__restrict__ G, int64_t ldg, double eta, double t,
    int *__restrict__ counts, const int *__restrict__ off, int *__restrict__ col_out,
    float *__restrict__ val_out, int64_t capacity, int *__restrict__ row_ptr,
    int *__restrict__ nnz_out) {
    __shared__ __attribute__((aligned(16))) float wrow[kSlab];
    __shared__ int wave_tot[kProxThreads / kWave];
    const int64_t blk = blockIdx.x;
    const int row = (int)(blk / slabs);
    const int sl = (int)(blk - (int64_t)row * slabs);
    const int k0 = sl * kSlab;
    const int k1 = min(n_cols, k0 + kSlab);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int *sr = seg + (int64_t)row * (slabs + 1) + sl;
    const int s = sr[0], e = sr[1];
    const float *g = G + (int64_t)row * ldg;
    // every G load of the slab and the first W entries of the row in flight at once
    float4 gq[kSlabChunks];
#pragma unroll
    for (int c = 0; c < kSlabChunks; ++c) {
        const int k = k0 + c * kProxThreads * 4 + tid * 4;
        if (V4 && k + 3 < k1) {
            gq[c] = *reinterpret_cast<const float4 *>(g + k);
        } else {
            gq[c].x = k + 0 < k1 ? g[k + 0] : 0.f;
            gq[c].y = k + 1 < k1 ? g[k + 1] : 0.f;
            gq[c].z = k + 2 < k1 ? g[k + 2] : 0.f;
            gq[c].w = k + 3 < k1 ? g[k + 3] : 0.f;
        }
    }
    int wi[4];
    float wv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int p = s + tid + u * kProxThreads;
        wi[u] = p < e ? idx[p] : -1;
        wv[u] = p < e ? vals[p] : 0.f;
    }
    for (int k = tid * 4; k < kSlab; k += kProxThreads * 4)
        *reinterpret_cast<float4 *>(wrow + k) = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u)
        if (wi[u] >= k0 && wi[u] < k1) wrow[wi[u] - k0] = wv[u];
    for (int p = s + tid + 4 * kProxThreads; p < e; p += kProxThreads) {
        const int k = idx[p];
        if (k >= k0 && k < k1) wrow[k - k0] = vals[p];
    }
    __syncthreads();
    int64_t out = FILL ? off[blk] : 0;
    if (FILL && threadIdx.x == 0) {
        // row pointers: a row starts where its first slab does; the last slab
        // also closes the last row
        if (sl == 0) row_ptr[row] = (int)out;
        if (blk == (int64_t)gridDim.x - 1) {
            const int total = off[blk + 1];
            row_ptr[row + 1] = total;
            if (nnz_out) *nnz_out = total;
        }
    }
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < kSlabChunks; ++c) {
        const int kb = k0 + c * kProxThreads * 4;
        if (kb >= k1) continue;  // uniform
        const int k = kb + tid * 4;
        const float4 w4 = *reinterpret_cast<const float4 *>(wrow + (k - k0));
        const float wv4[4] = {w4.x, w4.y, w4.z, w4.w};
        const float gv[4] = {gq[c].x, gq[c].y, gq[c].z, gq[c].w};
        float o[4];
        bool keep[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            o[j] = k + j < k1 ? soft_threshold(wv4[j], gv[j], eta, t) : 0.f;
            keep[j] = o[j] != 0.f;
            cnt += keep[j];
        }
        if (FILL) {
            uint64_t m[4];
            int below = 0, wcnt = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                m[j] = wave_ballot(keep[j]);
                below += popc_below(m[j]);
                wcnt += __popcll(m[j]);
            }
            if (lane == 0) wave_tot[wave] = wcnt;
            __syncthreads();
            int woff = 0, tot = 0;
#pragma unroll
            for (int w = 0; w < kProxThreads / kWave; ++w) {
                const int wc = wave_tot[w];
                woff += w < wave ? wc : 0;
                tot += wc;
            }
            int mine = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (keep[j]) {
                    const int64_t pos = out + woff + below + mine;
                    if (pos < capacity) {
                        col_out[pos] = k + j;
                        val_out[pos] = o[j];
                    }
                    ++mine;
                }
            }
            out += tot;
            __syncthreads();  // wave_tot is reused by the next chunk
        }
    }
    if (!FILL) {
        cnt = wave_sum_int(cnt);
        if (lane == 0) wave_tot[wave] = cnt;
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < kProxThreads / kWave; ++w) tot += wave_tot[w];
            counts[blk] = tot;
        }
    }
}

// row_ptr[r] = off[r * slabs] for r <= n_rows (off has n_rows * slabs + 1 entries)
__global__ void slab_row_ptr_kernel(int n_rows, int slabs, const int *__restrict__ off,
                                    int *__restrict__ row_ptr, int *__restrict__ nnz_out) {
    for (int r = blockIdx.x * blockDim.x + threadIdx.x; r <= n_rows; r += gridDim.x * blockDim.x) {
        const int v = off[(int64_t)r * slabs];
        row_ptr[r] = v;
        if (r == n_rows && nnz_out) *nnz_out = v;
    }
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

namespace l1csr {

int prox_slabs(int n_cols) { return n_cols > 0 ? (int)ceil_div(n_cols, kSlab) : 1; }

prox_ws prox_carve(int n_rows, int n_cols, void *ws) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t n = (size_t)n_rows * prox_slabs(n_cols);
    prox_ws w{};
    char *b = static_cast<char *>(ws);
    size_t o = 0;
    w.counts = reinterpret_cast<int *>(b + o);
    o = al(o + sizeof(int) * n);
    w.off = reinterpret_cast<int *>(b + o);
    o = al(o + sizeof(int) * (n + 1));
    w.seg = reinterpret_cast<int *>(b + o);
    o += sizeof(int) * (size_t)n_rows * (prox_slabs(n_cols) + 1);
    w.bytes = o;
    return w;
}

size_t prox_recompress_workspace_bytes(int n_rows, int n_cols) {
    return prox_carve(n_rows, n_cols, nullptr).bytes;
}

hipError_t launch_prox_count(int n_rows, int n_cols, const int *ptr, const int *idx,
                             const float *vals, const float *G, int64_t ldg, float eta, double t,
                             int *seg, int *counts, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    const bool v4 = (ldg % 4 == 0) && aligned16(G);
    const int slabs = prox_slabs(n_cols);
    hipError_t e = launch_seg(n_rows, slabs, kSlabShift, ptr, idx, seg, s);
    if (e != hipSuccess) return e;
    const unsigned grid = (unsigned)((int64_t)n_rows * slabs);
    if (v4)
        prox_slab_kernel<true, false><<<grid, kProxThreads, 0, s>>>(
            n_cols, slabs, seg, idx, vals, G, ldg, (double)eta, t, counts, nullptr, nullptr, nullptr, 0,
            nullptr, nullptr);
    else
        prox_slab_kernel<false, false><<<grid, kProxThreads, 0, s>>>(
            n_cols, slabs, seg, idx, vals, G, ldg, (double)eta, t, counts, nullptr, nullptr, nullptr, 0,
            nullptr, nullptr);
    return hipGetLastError();
}

hipError_t launch_prox_row_ptr(int n_rows, int n_cols, const int *off, int *row_ptr, int *nnz_out,
                               hipStream_t s) {
    const int slabs = prox_slabs(n_cols);
    const unsigned grid = (unsigned)(ceil_div((int64_t)n_rows + 1, 256) < 4096 ? ceil_div((int64_t)n_rows + 1, 256) : 4096);
    slab_row_ptr_kernel<<<grid, 256, 0, s>>>(n_rows, slabs, off, row_ptr, nnz_out);
    return hipGetLastError();
}

hipError_t launch_prox_fill(int n_rows, int n_cols, const int *seg, const int *idx,
                            const float *vals, const float *G, int64_t ldg, float eta, double t,
                            const int *off, int *col_out, float *val_out, int64_t capacity,
                            int *row_ptr, int *nnz_out, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    const bool v4 = (ldg % 4 == 0) && aligned16(G);
    const int slabs = prox_slabs(n_cols);
    const unsigned grid = (unsigned)((int64_t)n_rows * slabs);
    if (v4)
        prox_slab_kernel<true, true><<<grid, kProxThreads, 0, s>>>(
            n_cols, slabs, seg, idx, vals, G, ldg, (double)eta, t, nullptr, off, col_out, val_out,
            capacity, row_ptr, nnz_out);
    else
        prox_slab_kernel<false, true><<<grid, kProxThreads, 0, s>>>(
            n_cols, slabs, seg, idx, vals, G, ldg, (double)eta, t, nullptr, off, col_out, val_out,
            capacity, row_ptr, nnz_out);
    return hipGetLastError();
}

}  // namespace l1csr
