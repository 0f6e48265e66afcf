// Dense -> CSR recompression and CSR compaction by wave ballots.
//
// One wave per row.  The wave streams the row with 16-byte loads (4 columns
// per lane, 256 columns per step), takes one ballot per column slot, and
// places each kept entry at
//     row_ptr[row] + (entries kept in earlier steps)
//                  + (entries kept by lower lanes in this step)
//                  + (entries kept by this lane's lower slots)
// which is column order, so the output is the canonical CSR.  Row pointers
// come from an exclusive scan of per-row counts.
#include "../../include/l1csr.h"
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kRowsPerBlock = 4;

template <bool V4>
__global__ __launch_bounds__(256) void count_rows_kernel(int n_rows, int n_cols,
                                                         const float *__restrict__ Z, int64_t ldz,
                                                         float t, int *__restrict__ counts) {
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const float *z = Z + (int64_t)row * ldz;
    int cnt = 0;
    if (V4) {
        for (int k = lane * 4; k < n_cols; k += kWave * 4) {
            if (k + 3 < n_cols) {
                const float4 v = *reinterpret_cast<const float4 *>(z + k);
                cnt += (fabsf(v.x) > t) + (fabsf(v.y) > t) + (fabsf(v.z) > t) + (fabsf(v.w) > t);
            } else {
                for (int kk = k; kk < n_cols; ++kk) cnt += (fabsf(z[kk]) > t);
            }
        }
    } else {
        for (int k = lane; k < n_cols; k += kWave) cnt += (fabsf(z[k]) > t);
    }
    cnt = wave_sum_int(cnt);
    if (lane == 0) counts[row] = cnt;
}

template <bool V4>
__global__ __launch_bounds__(256) void recompress_fill_kernel(
    int n_rows, int n_cols, const float *__restrict__ Z, int64_t ldz, float t,
    const int *__restrict__ row_ptr, int *__restrict__ col_idx, float *__restrict__ vals,
    int64_t capacity) {
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const float *z = Z + (int64_t)row * ldz;
    int64_t out = row_ptr[row];
    if (V4) {
        for (int kb = 0; kb < n_cols; kb += kWave * 4) {
            const int k = kb + lane * 4;
            float v[4];
            if (k + 3 < n_cols) {
                const float4 q = *reinterpret_cast<const float4 *>(z + k);
                v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) v[j] = k + j < n_cols ? z[k + j] : 0.f;
            }
            bool keep[4];
            uint64_t m[4];
            int below = 0, step = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                keep[j] = (k + j < n_cols) && fabsf(v[j]) > t;
                m[j] = wave_ballot(keep[j]);
                below += popc_below(m[j]);
                step += __popcll(m[j]);
            }
            int mine = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (keep[j]) {
                    const int64_t pos = out + below + mine;
                    if (pos < capacity) {
                        col_idx[pos] = k + j;
                        vals[pos] = v[j];
                    }
                    ++mine;
                }
            }
            out += step;
        }
    } else {
        for (int kb = 0; kb < n_cols; kb += kWave) {
            const int k = kb + lane;
            const float v = k < n_cols ? z[k] : 0.f;
            const bool keep = (k < n_cols) && fabsf(v) > t;
            const uint64_t m = wave_ballot(keep);
            if (keep) {
                const int64_t pos = out + popc_below(m);
                if (pos < capacity) {
                    col_idx[pos] = k;
                    vals[pos] = v;
                }
            }
            out += __popcll(m);
        }
    }
}

__global__ __launch_bounds__(256) void compact_count_kernel(int n_rows, const int *__restrict__ ptr,
                                                            const float *__restrict__ vals,
                                                            int *__restrict__ counts) {
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    int cnt = 0;
    for (int p = ptr[row] + lane; p < ptr[row + 1]; p += kWave) cnt += (vals[p] != 0.f);
    cnt = wave_sum_int(cnt);
    if (lane == 0) counts[row] = cnt;
}

__global__ __launch_bounds__(256) void compact_fill_kernel(
    int n_rows, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ vals, const int *__restrict__ ptr_out, int *__restrict__ idx_out,
    float *__restrict__ vals_out) {
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int s = uniform(ptr[row]), e = uniform(ptr[row + 1]);
    int out = ptr_out[row];
    for (int pb = s; pb < e; pb += kWave) {
        const int p = pb + lane;
        const bool in = p < e;
        const float v = in ? vals[p] : 0.f;
        const bool keep = in && v != 0.f;
        const uint64_t m = wave_ballot(keep);
        if (keep) {
            idx_out[out + popc_below(m)] = idx[p];
            vals_out[out + popc_below(m)] = v;
        }
        out += __popcll(m);
    }
}

bool v4_ok(int64_t ld, const void *p) { return (ld % 4 == 0) && aligned16(p); }

}  // namespace

hipError_t launch_count_rows(int n_rows, int n_cols, const float *Z, int64_t ldz, float t,
                             int *counts, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    const unsigned grid = (unsigned)ceil_div(n_rows, kRowsPerBlock);
    if (v4_ok(ldz, Z))
        count_rows_kernel<true><<<grid, 256, 0, s>>>(n_rows, n_cols, Z, ldz, t, counts);
    else
        count_rows_kernel<false><<<grid, 256, 0, s>>>(n_rows, n_cols, Z, ldz, t, counts);
    return hipGetLastError();
}

hipError_t launch_recompress_fill(int n_rows, int n_cols, const float *Z, int64_t ldz, float t,
                                  const int *row_ptr, int *col_idx, float *vals, int64_t capacity,
                                  hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    const unsigned grid = (unsigned)ceil_div(n_rows, kRowsPerBlock);
    if (v4_ok(ldz, Z))
        recompress_fill_kernel<true><<<grid, 256, 0, s>>>(n_rows, n_cols, Z, ldz, t, row_ptr, col_idx,
                                                          vals, capacity);
    else
        recompress_fill_kernel<false><<<grid, 256, 0, s>>>(n_rows, n_cols, Z, ldz, t, row_ptr, col_idx,
                                                           vals, capacity);
    return hipGetLastError();
}

hipError_t launch_compact_count(int n_rows, const int *ptr, const float *vals, int *counts,
                                hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    compact_count_kernel<<<(unsigned)ceil_div(n_rows, kRowsPerBlock), 256, 0, s>>>(n_rows, ptr, vals,
                                                                                  counts);
    return hipGetLastError();
}

namespace {

// One wave per row: pointer checks, then the row's columns in chunks of 64
// (range and strict increase against the previous entry).  Reads are kept
// inside row_ptr[0 .. n_rows] and col_idx[0 .. nnz) whatever they hold; a
// violating wave stores L1CSR_EBADCSR (all writers store the same value).
__global__ __launch_bounds__(256) void csr_validate_kernel(int n_rows, int n_cols, int64_t nnz,
                                                           const int *__restrict__ ptr,
                                                           const int *__restrict__ idx,
                                                           int *__restrict__ status) {
    const int lane = threadIdx.x & 63;
    if (n_rows == 0) {
        if (blockIdx.x == 0 && threadIdx.x == 0 && (ptr[0] != 0 || nnz != 0)) *status = L1CSR_EBADCSR;
        return;
    }
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= n_rows) return;
    const int s = ptr[row], e = ptr[row + 1];
    bool bad = (row == 0 && s != 0) || (row == n_rows - 1 && (int64_t)e != nnz) || s < 0 || e < s ||
               (int64_t)e > nnz;
    if (!bad) {
        for (int p = s + lane; p < e; p += kWave) {
            const int c = idx[p];
            bool b = c < 0 || c >= n_cols;
            if (p > s) b = b || idx[p - 1] >= c;
            bad = bad || b;
        }
    }
    if (wave_ballot(bad) != 0 && lane == 0) *status = L1CSR_EBADCSR;
}

}  // namespace

hipError_t launch_csr_validate(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                               int *status, hipStream_t s) {
    hipError_t e = launch_fill_i32(status, 1, L1CSR_OK, s);
    if (e != hipSuccess) return e;
    const unsigned grid = n_rows == 0 ? 1u : (unsigned)ceil_div(n_rows, 4);
    csr_validate_kernel<<<grid, 256, 0, s>>>(n_rows, n_cols, nnz, ptr, idx, status);
    return hipGetLastError();
}

hipError_t launch_compact_fill(int n_rows, const int *ptr, const int *idx, const float *vals,
                               const int *ptr_out, int *idx_out, float *vals_out, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    compact_fill_kernel<<<(unsigned)ceil_div(n_rows, kRowsPerBlock), 256, 0, s>>>(
        n_rows, ptr, idx, vals, ptr_out, idx_out, vals_out);
    return hipGetLastError();
}

}  // namespace l1csr
