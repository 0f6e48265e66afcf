// Deterministic CSR -> CSC for the backward product: column pointers, the row
// of every entry, its CSR position (perm) and its value in CSC order.
//
// Rows are taken in chunks of 256 and columns in tiles of up to 512 (segment
// pointers per (row, tile) come from the same planning pass as the products).
// For one (chunk, tile) a workgroup builds in LDS a 256-bit mask per column
// (eight 32-bit words) whose bit r says "row r of the chunk has an entry in
// this column" (atomicOr, so the result does not depend on order).  An entry
// (row r of chunk c, column k) then goes to
//     col_ptr[k]                              entries of earlier columns
//   + sum_{c' < c} popcount(mask_{c'}[k])     same column, earlier chunks
//   + popcount(mask_c[k] & ((1 << r) - 1))    same column, earlier rows of c
// which orders every column by row (the canonical CSC) without sorting and
// without order-dependent atomics.  A chunk's entries of one column land in
// one run (~23 entries at 9% density), so the scattered 8-byte stores mostly
// fill whole cache lines.  (128 x 1024 measured 62 us for the scatter at
// 4096 x 9216, 256 x 512 54 us, 512 x 256 114 us.)
// Passes: segment pointers -> counts -> per-column chunk scan -> column
// pointer scan -> scatter (rebuilds the masks, bases staged in LDS).
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kChunkRows = 256;
constexpr int kMaskWords = kChunkRows / 32;
constexpr int kTileShift = 9;
constexpr int kTileCols = 1 << kTileShift;
constexpr int kCscThreads = 1024;

__device__ __forceinline__ void build_masks(int n_rows, const int *__restrict__ seg, int ntc,
                                            const int *__restrict__ idx, int chunk, int t, int k0,
                                            int ncols_tile, uint32_t (*M)[kTileCols]) {
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int nwaves = blockDim.x >> 6;
    constexpr int kRowsPerWave = kChunkRows / (kCscThreads / kWave);
    // bounds of this wave's rows, then their first entries, before any use
    int sb[kRowsPerWave], eb[kRowsPerWave], k1st[kRowsPerWave];
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u) {
        const int row = chunk * kChunkRows + wave + u * nwaves;
        sb[u] = eb[u] = 0;
        if (row < n_rows) {
            const int *sr = seg + (int64_t)row * (ntc + 1) + t;
            sb[u] = sr[0];
            eb[u] = sr[1];
        }
    }
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u) k1st[u] = sb[u] + lane < eb[u] ? idx[sb[u] + lane] - k0 : -1;
    for (int k = threadIdx.x; k < kMaskWords * kTileCols; k += blockDim.x) M[k / kTileCols][k % kTileCols] = 0u;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kRowsPerWave; ++u) {
        const int r = wave + u * nwaves;
        if (k1st[u] >= 0 && k1st[u] < ncols_tile) atomicOr(&M[r >> 5][k1st[u]], 1u << (r & 31));
        for (int p = sb[u] + kWave + lane; p < eb[u]; p += kWave) {
            const int k = idx[p] - k0;
            if (k >= 0 && k < ncols_tile) atomicOr(&M[r >> 5][k], 1u << (r & 31));
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(kCscThreads) void csc_count_kernel(int n_rows, int n_cols, int ntc,
                                                                const int *__restrict__ seg,
                                                                const int *__restrict__ idx,
                                                                int *__restrict__ cnt) {
    __shared__ uint32_t M[kMaskWords][kTileCols];
    const int chunk = blockIdx.x, t = blockIdx.y;
    const int k0 = t * kTileCols;
    const int nct = min(kTileCols, n_cols - k0);
    build_masks(n_rows, seg, ntc, idx, chunk, t, k0, nct, M);
    int *c = cnt + (int64_t)chunk * n_cols + k0;
    for (int k = threadIdx.x; k < nct; k += blockDim.x) {
        int n = 0;
#pragma unroll
        for (int w = 0; w < kMaskWords; ++w) n += __popc(M[w][k]);
        c[k] = n;
    }
}

// cnt[c][k] <- sum_{c' < c} cnt[c'][k];  tot[k] <- sum_c cnt[c][k]
__global__ __launch_bounds__(256) void csc_colscan_kernel(int n_chunks, int n_cols,
                                                          int *__restrict__ cnt,
                                                          int *__restrict__ tot) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n_cols) return;
    int run = 0;
    int c = 0;
    for (; c + 8 <= n_chunks; c += 8) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = cnt[(int64_t)(c + u) * n_cols + k];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            cnt[(int64_t)(c + u) * n_cols + k] = run;
            run += v[u];
        }
    }
    for (; c < n_chunks; ++c) {
        const int64_t o = (int64_t)c * n_cols + k;
        const int v = cnt[o];
        cnt[o] = run;
        run += v;
    }
    tot[k] = run;
}

// one scattered 8-byte store per entry, (row, CSR position), into a staging
// array; csc_finish_kernel then writes row_idx, perm and vals_t coalesced
__global__ __launch_bounds__(kCscThreads) void csc_scatter_kernel(
    int n_rows, int n_cols, int ntc, const int *__restrict__ seg, const int *__restrict__ idx,
    const int *__restrict__ cnt, const int *__restrict__ col_ptr, int2 *__restrict__ pairs) {
    __shared__ uint32_t M[kMaskWords][kTileCols];
    __shared__ int base[kTileCols];
    const int chunk = blockIdx.x, t = blockIdx.y;
    const int k0 = t * kTileCols;
    const int nct = min(kTileCols, n_cols - k0);
    const int *c = cnt + (int64_t)chunk * n_cols + k0;
    for (int k = threadIdx.x; k < nct; k += blockDim.x) base[k] = col_ptr[k0 + k] + c[k];
    build_masks(n_rows, seg, ntc, idx, chunk, t, k0, nct, M);  // ends with a barrier
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int nwaves = blockDim.x >> 6;
    for (int r = wave; r < kChunkRows; r += nwaves) {
        const int row = chunk * kChunkRows + r;
        if (row >= n_rows) break;
        const int *sr = seg + (int64_t)row * (ntc + 1) + t;
        const int s = sr[0], e = sr[1];
        const int rw = r >> 5;
        const uint32_t below = (1u << (r & 31)) - 1u;
        for (int p = s + lane; p < e; p += kWave) {
            const int k = idx[p] - k0;
            if (k >= 0 && k < nct) {
                int rank = __popc(M[rw][k] & below);
#pragma unroll
                for (int w = 0; w < kMaskWords; ++w) rank += w < rw ? __popc(M[w][k]) : 0;
                pairs[base[k] + rank] = make_int2(row, p);
            }
        }
    }
}

// row_idx[q], perm[q] from the staged pairs; vals_t[q] = vals[perm[q]]
__global__ __launch_bounds__(256) void csc_finish_kernel(int n_rows, int64_t nnz,
                                                         const int *__restrict__ ptr,
                                                         const int2 *__restrict__ pairs,
                                                         const float *__restrict__ vals,
                                                         int *__restrict__ row_idx,
                                                         int *__restrict__ perm,
                                                         float *__restrict__ vals_t) {
    const int64_t n = min(nnz, (int64_t)ptr[n_rows]);  // nnz may be a capacity bound
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int2 rp = pairs[q];
        row_idx[q] = rp.x;
        perm[q] = rp.y;
        vals_t[q] = vals[rp.y];
    }
}

__global__ void gather_vals_kernel(int n_cols, const int *__restrict__ col_ptr,
                                   const int *__restrict__ perm, const float *__restrict__ vals,
                                   float *__restrict__ vals_t) {
    const int64_t nnz = col_ptr[n_cols];
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x)
        vals_t[q] = vals[perm[q]];
}

struct csc_layout {
    int n_chunks, ntc;
    int64_t seg_ints, cnt_ints, tot_ints, pair_ints;  // pairs start 8-byte aligned
};

csc_layout layout(int n_rows, int n_cols, int64_t nnz) {
    csc_layout l;
    l.n_chunks = (int)ceil_div(n_rows, kChunkRows);
    l.ntc = (int)ceil_div(n_cols, kTileCols);
    l.seg_ints = (int64_t)n_rows * (l.ntc + 1);
    l.cnt_ints = (int64_t)l.n_chunks * n_cols;
    l.tot_ints = ((int64_t)n_cols + 2) & ~(int64_t)1;
    if ((l.seg_ints + l.cnt_ints) & 1) l.tot_ints += 1;
    l.pair_ints = 2 * nnz;
    return l;
}

}  // namespace

bool csc_grid_fits(int n_rows, int n_cols) {
    return ceil_div(n_rows, kChunkRows) <= INT32_MAX && ceil_div(n_cols, kTileCols) <= 65535;
}

size_t csc_workspace_bytes(int n_rows, int n_cols, int64_t nnz) {
    const csc_layout l = layout(n_rows, n_cols, nnz);
    return sizeof(int) * (size_t)(l.seg_ints + l.cnt_ints + l.tot_ints + l.pair_ints);
}

hipError_t launch_csc_build(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                            const float *vals, int *col_ptr, int *row_idx, int *perm,
                            float *vals_t, void *ws, hipStream_t s) {
    if (n_cols == 0) return launch_fill_i32(col_ptr, 1, 0, s);
    if (n_rows == 0) return launch_fill_i32(col_ptr, (int64_t)n_cols + 1, 0, s);
    const csc_layout l = layout(n_rows, n_cols, nnz);
    int *seg = static_cast<int *>(ws);
    int *cnt = seg + l.seg_ints;
    int *tot = cnt + l.cnt_ints;
    int2 *pairs = reinterpret_cast<int2 *>(tot + l.tot_ints);
    hipError_t e = launch_seg(n_rows, l.ntc, kTileShift, ptr, idx, seg, s);
    if (e != hipSuccess) return e;
    dim3 grid(l.n_chunks, l.ntc);
    csc_count_kernel<<<grid, kCscThreads, 0, s>>>(n_rows, n_cols, l.ntc, seg, idx, cnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    csc_colscan_kernel<<<(unsigned)ceil_div(n_cols, 256), 256, 0, s>>>(l.n_chunks, n_cols, cnt, tot);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_exclusive_scan(tot, col_ptr, n_cols, nullptr, s)) != hipSuccess) return e;
    csc_scatter_kernel<<<grid, kCscThreads, 0, s>>>(n_rows, n_cols, l.ntc, seg, idx, cnt, col_ptr, pairs);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (nnz == 0) return hipSuccess;
    int64_t g = ceil_div(nnz, 256);
    if (g > 65536) g = 65536;
    csc_finish_kernel<<<(unsigned)g, 256, 0, s>>>(n_rows, nnz, ptr, pairs, vals, row_idx, perm, vals_t);
    return hipGetLastError();
}

hipError_t launch_csc_gather_vals(int n_cols, int64_t nnz_bound, const int *col_ptr, const int *perm,
                                  const float *vals, float *vals_t, hipStream_t s) {
    if (nnz_bound == 0) return hipSuccess;
    int64_t g = ceil_div(nnz_bound, 256);
    if (g > 65536) g = 65536;
    gather_vals_kernel<<<(unsigned)g, 256, 0, s>>>(n_cols, col_ptr, perm, vals, vals_t);
    return hipGetLastError();
}

}  // namespace l1csr
