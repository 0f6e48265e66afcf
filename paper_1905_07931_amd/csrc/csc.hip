// Deterministic CSR -> CSC (structure only, plus the CSR position of every
// entry) for the backward product.
//
// Rows are taken in chunks of 32.  For one chunk and one tile of columns a
// workgroup builds, in LDS, a 32-bit mask per column whose bit r says "row r
// of the chunk has an entry in this column" (atomicOr: order independent).
// Then for an entry (row r of chunk c, column k):
//     position = col_ptr[k]                         (entries of earlier columns)
//              + sum_{c' < c} popcount(mask_{c'}[k]) (earlier chunks, same column)
//              + popcount(mask_c[k] & ((1<<r)-1))    (earlier rows of this chunk)
// which orders each column by row without sorting and without any
// order-dependent atomics.  Passes: count -> per-column chunk scan ->
// column-pointer scan -> scatter (the scatter rebuilds the masks).
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kChunkRows = 32;
constexpr int kMaxTileCols = 16384;  // 64 KB of masks
constexpr int kCscThreads = 512;

__device__ __forceinline__ void build_masks(int n_rows, const int *__restrict__ ptr,
                                            const int *__restrict__ idx, int chunk, int k0,
                                            int k1, uint32_t *M) {
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int nwaves = blockDim.x >> 6;
    for (int k = threadIdx.x; k < k1 - k0; k += blockDim.x) M[k] = 0u;
    __syncthreads();
    for (int r = wave; r < kChunkRows; r += nwaves) {
        const int row = chunk * kChunkRows + r;
        if (row >= n_rows) break;
        const int s = ptr[row], e = ptr[row + 1];
        for (int p = s + lane; p < e; p += kWave) {
            const int k = idx[p];
            if (k >= k0 && k < k1) atomicOr(&M[k - k0], 1u << r);
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(kCscThreads) void csc_count_kernel(int n_rows, int n_cols,
                                                                const int *__restrict__ ptr,
                                                                const int *__restrict__ idx,
                                                                int *__restrict__ cnt) {
    extern __shared__ uint32_t M[];
    const int chunk = blockIdx.x;
    const int k0 = blockIdx.y * kMaxTileCols;
    const int k1 = min(n_cols, k0 + kMaxTileCols);
    build_masks(n_rows, ptr, idx, chunk, k0, k1, M);
    for (int k = threadIdx.x; k < k1 - k0; k += blockDim.x)
        cnt[(int64_t)chunk * n_cols + k0 + k] = __popc(M[k]);
}

// cnt[c][k] <- sum_{c' < c} cnt[c'][k]; tot[k] <- sum_c cnt[c][k]
__global__ void csc_colscan_kernel(int n_chunks, int n_cols, int *__restrict__ cnt,
                                   int *__restrict__ tot) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n_cols) return;
    int run = 0;
    for (int c = 0; c < n_chunks; ++c) {
        const int64_t o = (int64_t)c * n_cols + k;
        const int t = cnt[o];
        cnt[o] = run;
        run += t;
    }
    tot[k] = run;
}

__global__ __launch_bounds__(kCscThreads) void csc_scatter_kernel(
    int n_rows, int n_cols, const int *__restrict__ ptr, const int *__restrict__ idx,
    const int *__restrict__ cnt, const int *__restrict__ col_ptr, int *__restrict__ row_idx,
    int *__restrict__ perm) {
    extern __shared__ uint32_t M[];
    const int chunk = blockIdx.x;
    const int k0 = blockIdx.y * kMaxTileCols;
    const int k1 = min(n_cols, k0 + kMaxTileCols);
    build_masks(n_rows, ptr, idx, chunk, k0, k1, M);
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int nwaves = blockDim.x >> 6;
    for (int r = wave; r < kChunkRows; r += nwaves) {
        const int row = chunk * kChunkRows + r;
        if (row >= n_rows) break;
        const int s = ptr[row], e = ptr[row + 1];
        const uint32_t below = (1u << r) - 1u;
        for (int p = s + lane; p < e; p += kWave) {
            const int k = idx[p];
            if (k >= k0 && k < k1) {
                const int pos = col_ptr[k] + cnt[(int64_t)chunk * n_cols + k] +
                                __popc(M[k - k0] & below);
                row_idx[pos] = row;
                perm[pos] = p;
            }
        }
    }
}

}  // namespace

size_t csc_workspace_bytes(int n_rows, int n_cols) {
    const int64_t n_chunks = ceil_div(n_rows, kChunkRows);
    return sizeof(int) * (size_t)(n_chunks * (int64_t)n_cols + n_cols + 1);
}

hipError_t launch_csc_build(int n_rows, int n_cols, const int *ptr, const int *idx, int *col_ptr,
                            int *row_idx, int *perm, void *ws, hipStream_t s) {
    if (n_cols == 0) return launch_fill_i32(col_ptr, 1, 0, s);
    const int n_chunks = (int)ceil_div(n_rows, kChunkRows);
    int *cnt = static_cast<int *>(ws);
    int *tot = cnt + (int64_t)n_chunks * n_cols;
    if (n_rows == 0) return launch_fill_i32(col_ptr, (int64_t)n_cols + 1, 0, s);
    const int tiles = (int)ceil_div(n_cols, kMaxTileCols);
    const int tile_cols = n_cols < kMaxTileCols ? n_cols : kMaxTileCols;
    const size_t lds = sizeof(uint32_t) * (size_t)tile_cols;
    dim3 grid(n_chunks, tiles);
    csc_count_kernel<<<grid, kCscThreads, lds, s>>>(n_rows, n_cols, ptr, idx, cnt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    csc_colscan_kernel<<<(unsigned)ceil_div(n_cols, 256), 256, 0, s>>>(n_chunks, n_cols, cnt, tot);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_exclusive_scan(tot, col_ptr, n_cols, nullptr, s);
    if (e != hipSuccess) return e;
    csc_scatter_kernel<<<grid, kCscThreads, lds, s>>>(n_rows, n_cols, ptr, idx, cnt, col_ptr, row_idx,
                                                      perm);
    return hipGetLastError();
}

}  // namespace l1csr
