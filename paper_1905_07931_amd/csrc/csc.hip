// Deterministic CSR -> CSC for the backward product: column pointers, the row
// of every entry, its CSR position (perm) and its value in CSC order.
//
// Built from the bitmap index of W (launch_bitmap, word-major: mask[w][row]
// has bit c set iff (row, 32w + c) is stored, pos[w][row] is the CSR position
// of the row's first entry at a column >= 32w).  A workgroup takes one
// 32-column word and a block of up to 1024 rows; its 4 waves take 256 rows
// each (one row per lane, four groups) and hold the rows' mask and pos words
// in registers.  For every column of the word a ballot of the column's bit
// ranks the stored rows, so the column's entries come out in row order (the
// canonical CSC) and are written as contiguous runs, with no sorting and no
// atomics.  The entry's CSR position is pos + popcount(mask &
// below(c)).  Passes: counts per (row block, column) -> per-column scan over
// the blocks -> column pointer scan -> emit.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kRowBlock = 1024;  // rows per workgroup (256 threads, 4 waves of 256 rows)
constexpr int kCscThreads = 256;

// Each of the 4 waves takes 256 consecutive rows of the block (four groups of
// 64, one row per lane) and evaluates all 32 columns of the word per mask
// read: 32 ballots per group, no dependent chain through LDS.
constexpr int kWaveRows = kRowBlock / (kCscThreads / kWave);  // 256

// cnt[rb][c] = stored entries of column c in row block rb
__global__ __launch_bounds__(kCscThreads) void csc_count_kernel(int n_rows, int n_cols,
                                                                const unsigned *__restrict__ mask,
                                                                int *__restrict__ cnt) {
    __shared__ int part[kCscThreads / kWave][32];
    const int w = blockIdx.x, rb = blockIdx.y;
    const int r0 = rb * kRowBlock, r1 = min(n_rows, r0 + kRowBlock);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t o = (int64_t)w * n_rows;
    unsigned m[kWaveRows / kWave];
#pragma unroll
    for (int g = 0; g < kWaveRows / kWave; ++g) {
        const int i = r0 + wave * kWaveRows + g * kWave + lane;
        m[g] = i < r1 ? mask[o + i] : 0u;
    }
    int mine = 0;  // lane c < 32: this wave's count of column 32w + c
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        int n = 0;
#pragma unroll
        for (int g = 0; g < kWaveRows / kWave; ++g) n += __popcll(__ballot((m[g] >> c) & 1u));
        mine = lane == c ? n : mine;
    }
    if (lane < 32) part[wave][lane] = mine;
    __syncthreads();
    if (threadIdx.x < 32) {
        const int c = 32 * w + threadIdx.x;
        int n = 0;
#pragma unroll
        for (int j = 0; j < kCscThreads / kWave; ++j) n += part[j][threadIdx.x];
        if (c < n_cols) cnt[(int64_t)rb * n_cols + c] = n;
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

// row_idx, perm and vals_t of every (column, row block): the column's entries
// of the block at col_ptr[c] + cnt[rb][c] onwards, in row order.  Wave j's
// rows of column c start after the column's entries in the block's earlier
// waves (per-wave counts exchanged through LDS); inside a 64-row group a
// ballot ranks them.  Columns are taken eight at a time: every entry goes to
// an LDS run of its column (the first kRunCap of the block's entries of that
// column; any further ones, only in very dense columns, are stored directly),
// and the eight runs are then written as one sequence, consecutive threads on
// consecutive positions, with all of a thread's value gathers issued before
// its stores.
//
// Work items are (row block, word) in row-block-major order, and the blocks
// are dealt to the 8 XCDs in contiguous ranges: one XCD takes neighbouring
// words of a row block, whose entries share the cache lines of W's values
// (a row's entries of consecutive words are consecutive in the CSR).
constexpr int kRunCols = 8;
constexpr int kRunCap = 256;
constexpr int kRunPer = kRunCols * kRunCap / kCscThreads;  // staged entries per thread per chunk

__global__ __launch_bounds__(kCscThreads) void csc_emit_kernel(int n_rows, int n_cols, int kw,
                                                               const unsigned *__restrict__ mask,
                                                               const int *__restrict__ pos,
                                                               const float *__restrict__ vals,
                                                               const int *__restrict__ cnt,
                                                               const int *__restrict__ col_ptr,
                                                               int *__restrict__ row_idx,
                                                               int *__restrict__ perm,
                                                               float *__restrict__ vals_t) {
    constexpr int NW = kCscThreads / kWave, G = kWaveRows / kWave;
    __shared__ int start[NW + 1][32];  // [j][c]: column c's entries of waves < j (row NW: block total)
    __shared__ int64_t dst0[32];       // first output position of column c's entries of this block
    __shared__ int run_row[kRunCols][kRunCap];
    __shared__ int run_p[kRunCols][kRunCap];
    int64_t item = blockIdx.x;
    {
        const int64_t total = (int64_t)gridDim.x, per = total / 8;
        if (item < per * 8) item = (item % 8) * per + item / 8;
    }
    const int rb = (int)(item / kw), w = (int)(item - (int64_t)rb * kw);
    const int r0 = rb * kRowBlock, r1 = min(n_rows, r0 + kRowBlock);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int nc = min(32, n_cols - 32 * w);
    const int64_t o = (int64_t)w * n_rows;
    if (threadIdx.x < nc)
        dst0[threadIdx.x] = (int64_t)col_ptr[32 * w + threadIdx.x] + cnt[(int64_t)rb * n_cols + 32 * w + threadIdx.x];
    unsigned m[G];
    int ps[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int i = r0 + wave * kWaveRows + g * kWave + lane;
        m[g] = i < r1 ? mask[o + i] : 0u;
        ps[g] = i < r1 ? pos[o + i] : 0;
    }
    int mine = 0;
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        int n = 0;
#pragma unroll
        for (int g = 0; g < G; ++g) n += __popcll(__ballot((m[g] >> c) & 1u));
        mine = lane == c ? n : mine;
    }
    if (lane < 32) start[wave][lane] = mine;
    __syncthreads();
    if (threadIdx.x < 32) {  // exclusive scan over the waves (relative to the block's run)
        int run = 0;
#pragma unroll
        for (int j = 0; j < NW; ++j) {
            const int v = start[j][threadIdx.x];
            start[j][threadIdx.x] = run;
            run += v;
        }
        start[NW][threadIdx.x] = run;
    }
    __syncthreads();
    for (int c0 = 0; c0 < nc; c0 += kRunCols) {
#pragma unroll
        for (int cc = 0; cc < kRunCols; ++cc) {
            const int c = c0 + cc;
            if (c >= nc) break;  // uniform
            const unsigned below = (1u << c) - 1u;
            int q0 = start[wave][c];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const bool set = (m[g] >> c) & 1u;
                const uint64_t b = __ballot(set);
                if (set) {
                    const int q = q0 + popc_below(b);
                    const int row = r0 + wave * kWaveRows + g * kWave + lane;
                    const int p = ps[g] + __popc(m[g] & below);
                    if (q < kRunCap) {
                        run_row[cc][q] = row;
                        run_p[cc][q] = p;
                    } else {  // beyond the staged run: straight to the output
                        const int64_t d = dst0[c] + q;
                        row_idx[d] = row;
                        perm[d] = p;
                        vals_t[d] = vals[p];
                    }
                }
                q0 += __popcll(b);
            }
        }
        __syncthreads();
        // the staged runs of the chunk's columns back to back: entry i of the
        // sequence is entry i - roff[cc] of column cc's run
        int roff[kRunCols + 1];
        roff[0] = 0;
#pragma unroll
        for (int cc = 0; cc < kRunCols; ++cc)
            roff[cc + 1] = roff[cc] + (c0 + cc < nc ? min(kRunCap, start[NW][c0 + cc]) : 0);
        int qc[kRunPer], pv[kRunPer];
        float vv[kRunPer];
#pragma unroll
        for (int u = 0; u < kRunPer; ++u) {
            const int i = threadIdx.x + u * kCscThreads;
            int cc = 0;
#pragma unroll
            for (int j = 1; j < kRunCols; ++j) cc += i >= roff[j] ? 1 : 0;
            qc[u] = i < roff[kRunCols] ? (cc << 16) | (i - roff[cc]) : -1;
            if (qc[u] >= 0) {
                pv[u] = run_p[cc][i - roff[cc]];
                vv[u] = vals[pv[u]];
            }
        }
#pragma unroll
        for (int u = 0; u < kRunPer; ++u) {
            if (qc[u] < 0) continue;
            const int cc = qc[u] >> 16, q = qc[u] & 0xffff;
            const int64_t d = dst0[c0 + cc] + q;
            row_idx[d] = run_row[cc][q];
            perm[d] = pv[u];
            vals_t[d] = vv[u];
        }
        __syncthreads();  // the runs are refilled by the next columns
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
    int n_blocks, kw;
    int64_t bm_ints, cnt_ints, tot_ints;
};

csc_layout layout(int n_rows, int n_cols) {
    csc_layout l;
    l.n_blocks = (int)ceil_div(n_rows, kRowBlock);
    l.kw = (int)ceil_div(n_cols, 32);
    l.bm_ints = (int64_t)n_rows * l.kw;
    l.cnt_ints = (int64_t)l.n_blocks * n_cols;
    l.tot_ints = (int64_t)n_cols + 1;
    return l;
}

}  // namespace

bool csc_grid_fits(int n_rows, int n_cols) {
    return ceil_div(n_cols, 32) * ceil_div(n_rows, kRowBlock) <= INT32_MAX && ceil_div(n_rows, kRowBlock) <= 65535;
}

size_t csc_workspace_bytes(int n_rows, int n_cols, int64_t nnz) {
    (void)nnz;
    const csc_layout l = layout(n_rows, n_cols);
    return sizeof(int) * (size_t)(2 * l.bm_ints + l.cnt_ints + l.tot_ints);
}

hipError_t launch_csc_build(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                            const float *vals, const unsigned *mask, const int *pos, int *col_ptr, int *row_idx,
                            int *perm, float *vals_t, void *ws, hipStream_t s) {
    if (n_cols == 0) return launch_fill_i32(col_ptr, 1, 0, s);
    if (n_rows == 0) return launch_fill_i32(col_ptr, (int64_t)n_cols + 1, 0, s);
    const csc_layout l = layout(n_rows, n_cols);
    int *bm = static_cast<int *>(ws);
    int *cnt = bm + 2 * l.bm_ints;
    int *tot = cnt + l.cnt_ints;
    hipError_t e;
    if (mask == nullptr) {  // no bitmap index from the caller: build it here
        unsigned *m = reinterpret_cast<unsigned *>(bm);
        int *p = bm + l.bm_ints;
        if ((e = launch_bitmap(n_rows, n_cols, ptr, idx, m, p, s)) != hipSuccess) return e;
        mask = m;
        pos = p;
    }
    dim3 grid(l.kw, l.n_blocks);
    csc_count_kernel<<<grid, kCscThreads, 0, s>>>(n_rows, n_cols, mask, cnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    csc_colscan_kernel<<<(unsigned)ceil_div(n_cols, 256), 256, 0, s>>>(l.n_blocks, n_cols, cnt, tot);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_exclusive_scan(tot, col_ptr, n_cols, nullptr, s)) != hipSuccess) return e;
    if (nnz == 0) return hipSuccess;
    csc_emit_kernel<<<(unsigned)((int64_t)l.kw * l.n_blocks), kCscThreads, 0, s>>>(
        n_rows, n_cols, l.kw, mask, pos, vals, cnt, col_ptr, row_idx, perm, vals_t);
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
