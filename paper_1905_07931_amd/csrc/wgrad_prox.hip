// The l1-phase weight update of Eq. (prox) from the layer's activations
// straight to the new CSR, reading the dense gradient's result once:
//
//   1. bitmap index of W (bitmap_kernel): per row and 32-column word, the
//      stored-column mask and the CSR position of the word's first entry;
//   2. the weight-gradient GEMM with the prox epilogue (prox_epilogue.hpp):
//      Z = S_t(W - eta * dY.X^T) and the nonzero count of every 32-column
//      word of every row;
//   3. row totals of the word counts and their totals per block of 16-64
//      rows (row_block_sums_kernel);
//   4. compaction of Z into col_idx', vals' (compact_kernel): a workgroup per
//      (row, 3072-column chunk) starts at row_ptr'[row] plus the counts of
//      the row's words before the chunk, so no second pass over the gradient.
//      row_ptr'[row] is the sum of the block totals before the row's block
//      and of the row totals before it in its block, added up by each
//      workgroup itself (at most 256 + 63 integers, cached); the first chunk
//      of a row writes it.  Where the caller's capacity is below n_rows *
//      n_cols the host needs nnz' first, and past 16384 rows (256 blocks of
//      64) the sums grow long: an exclusive scan of the row totals writes
//      row_ptr' instead and the compaction reads it.
//
// Shapes whose GEMM has no prox epilogue (bf16 operands, or an fp32 product
// that splits its reduction) write dW into Z first and run the same prox in
// place (prox_words_kernel); the rest is shared.  Every value is the one
// prox_l1_step would compute from dense_wgrad's dW, and every structure the
// canonical CSR, so the result equals dense_wgrad + prox_l1_recompress bit
// for bit.
#include "common.hpp"
#include "launch.hpp"
#include "prox_epilogue.hpp"

namespace l1csr {

namespace {

constexpr int kCompactCols = 3072;  // columns per compaction workgroup (whole 32-column words)
constexpr int kCompactThreads = 256;
constexpr int kCompactVecs = kCompactCols / (4 * kCompactThreads);  // float4 per thread: 3
// rows per block of the two-level row prefix: 16, 32 or 64 (a workgroup of
// that many rows / 4 waves), the smallest that keeps the blocks of N rows to
// kPrefixMaxBlocks, the block totals a compaction workgroup adds up at most
constexpr int kPrefixMinRows = 16, kPrefixMaxRows = 64;
constexpr int kPrefixMaxBlocks = 256;
static_assert(kPrefixMaxBlocks <= kCompactThreads && kPrefixMaxRows <= kCompactThreads, "one load per thread");
int prefix_rows(int N) {
    int r = kPrefixMinRows;
    while (r < kPrefixMaxRows && ceil_div(N, r) > kPrefixMaxBlocks) r *= 2;
    return r;
}

// mask[w][row] bit c: column 32w + c is stored; pos[w][row]: CSR position of
// the row's first entry with column >= 32w (row_ptr[row + 1] past the last).
// Word-major ([ceil(n_cols / 32)][n_rows]): a GEMM tile reads a run of rows of
// each of its words, and the CSC build walks all rows of one word.
// A wave takes kBitmapSpan consecutive entries of one row (grid: rows x
// spans; waves past their row's end only handle an empty row), 64 at a time.
// Entries of one word sit in consecutive positions (columns are sorted), so a
// segmented OR scan across the lanes, carried from one 64-entry chunk to the
// next and seeded with the up to 31 entries before the span, gives each word's
// mask in the lane of its last entry in the row, which alone writes it.  The
// first entry of a word writes its pos and the pos of the empty words before
// it; the wave holding the row's last entry writes the words after it.  Every
// word is written exactly once, by one lane; no atomics.
constexpr int kBitmapSpan = 512;

// The words of one row's span: entries [s + span * kBitmapSpan, ...) of the
// row's entries [s, e); word x of the row goes to mr[x * st], pr[x * st]
// (global memory or an LDS block of rows).  One wave.
template <typename MP, typename PP>
__device__ __forceinline__ void bitmap_span(int s, int e, int span, int kw, const int *__restrict__ idx, MP mr,
                                            PP pr, int st) {
    const int lane = threadIdx.x & 63;
    const int b0 = s + span * kBitmapSpan;
    if (s == e) {  // an empty row: every word empty, pos = the row's start
        if (span == 0)
            for (int x = lane; x < kw; x += kWave) {
                mr[x * st] = 0u;
                pr[x * st] = s;
            }
        return;
    }
    if (b0 >= e) return;
    const int b1 = min(e, b0 + kBitmapSpan);
    // the entry before the span and the bits its word already has
    int prevw = -1;
    unsigned carry = 0u;
    if (b0 > s) {
        const int q = b0 - 32 + (lane & 31);
        const int cq = q >= s ? idx[q] : -1;
        prevw = lane_bcast(cq, 31) >> 5;
        const bool same = lane < 32 && cq >= 0 && (cq >> 5) == prevw;
        unsigned bit = same ? 1u << (cq & 31) : 0u;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) bit |= __shfl_xor(bit, d, kWave);
        carry = bit;
    }
    // the span's entries, plus the entry after it (to tell a word's last entry)
    constexpr int U = kBitmapSpan / kWave;
    int cu[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int q = b0 + u * kWave + lane;
        cu[u] = q < b1 ? idx[q] : 0;
    }
    const int after = b1 < e ? idx[b1] >> 5 : 0x7fffffff;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int base = b0 + u * kWave;
        if (base >= b1) break;
        const int p = base + lane;
        const bool valid = p < b1;
        const int c = cu[u];
        const int w = valid ? c >> 5 : 0x7fffffff;
        unsigned v = valid ? 1u << (c & 31) : 0u;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const unsigned vu = __shfl_up(v, d, kWave);
            const int wu = __shfl_up(w, d, kWave);
            if (lane >= d && wu == w) v |= vu;
        }
        if (w == prevw) v |= carry;
        const int n = min(kWave, b1 - base);
        int wn = __shfl_down(w, 1, kWave);
        if (lane == n - 1) wn = base + n < b1 ? lane_bcast(cu[u + 1 < U ? u + 1 : u], 0) >> 5 : after;
        if (valid && wn != w) mr[w * st] = v;  // the word's last entry in the row
        int pw = __shfl_up(w, 1, kWave);
        if (lane == 0) pw = prevw;
        if (valid && w != pw) {
            for (int x = pw + 1; x < w; ++x) {  // empty words before this one
                mr[x * st] = 0u;
                pr[x * st] = p;
            }
            pr[w * st] = p;
        }
        prevw = lane_bcast(w, n - 1);
        carry = (unsigned)lane_bcast((int)v, n - 1);
    }
    if (b1 == e)
        for (int x = prevw + 1 + lane; x < kw; x += kWave) {  // words past the row's last entry
            mr[x * st] = 0u;
            pr[x * st] = e;
        }
}

// A wave per (row, span) item, written straight to the word-major arrays
// (rows with more words than the LDS block holds).
__global__ __launch_bounds__(256) void bitmap_kernel(int n_rows, int kw, int spans, const int *__restrict__ ptr,
                                                     const int *__restrict__ idx, unsigned *__restrict__ mask,
                                                     int *__restrict__ pos) {
    const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int row = (int)(item / spans), span = (int)(item - (int64_t)row * spans);
    if (row >= n_rows) return;
    bitmap_span(ptr[row], ptr[row + 1], span, kw, idx, mask + row, pos + row, n_rows);
}

// A workgroup per 16 consecutive rows: the (row, span) items of its rows are
// dealt to its 16 waves and written to an LDS block [word][16 rows], which then
// goes out 16 rows of a word at a time (64-byte segments instead of 4-byte
// writes down the columns).
constexpr int kBitmapRows = 16;
constexpr int kBitmapThreads = 1024;
constexpr int kBitmapMaxWords = 320;  // LDS block: 320 words x 16 rows x 8 bytes = 40 KB

__global__ __launch_bounds__(kBitmapThreads) void bitmap_block_kernel(int n_rows, int kw, const int *__restrict__ ptr,
                                                           const int *__restrict__ idx,
                                                           unsigned *__restrict__ mask, int *__restrict__ pos) {
    __shared__ unsigned lm[kBitmapMaxWords * kBitmapRows];
    __shared__ int lp[kBitmapMaxWords * kBitmapRows];
    __shared__ int first_item[kBitmapRows + 1];
    const int r0 = blockIdx.x * kBitmapRows;
    const int nr = min(kBitmapRows, n_rows - r0);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    if (wave == 0) {  // items per row (an empty row still writes its words), exclusive scan
        int n = 0;
        if (lane < nr) {
            const int len = ptr[r0 + lane + 1] - ptr[r0 + lane];
            n = len == 0 ? 1 : (len + kBitmapSpan - 1) / kBitmapSpan;
        }
        const int incl = wave_incl_scan(n);
        if (lane < kBitmapRows) first_item[lane] = incl - n;
        if (lane == kBitmapRows - 1) first_item[kBitmapRows] = incl;
    }
    __syncthreads();
    const int items = first_item[kBitmapRows];
    for (int it = wave; it < items; it += kBitmapThreads / kWave) {
        int j = 0;  // the row of item it: last j with first_item[j] <= it
#pragma unroll
        for (int d = kBitmapRows / 2; d > 0; d >>= 1)
            if (first_item[j + d] <= it) j += d;
        const int row = r0 + j;
        bitmap_span(ptr[row], ptr[row + 1], it - first_item[j], kw, idx, lm + j, lp + j, kBitmapRows);
    }
    __syncthreads();
    for (int i = tid; i < kw * kBitmapRows; i += kBitmapThreads) {
        const int x = i / kBitmapRows, j = i - x * kBitmapRows;
        if (j < nr) {
            mask[(int64_t)x * n_rows + r0 + j] = lm[i];
            pos[(int64_t)x * n_rows + r0 + j] = lp[i];
        }
    }
}

// Z <- S_t(W - eta * Z) in place (Z holds dW), counts per 32-column word:
// one wave per (row, pair of words), lane = column.
__global__ __launch_bounds__(256) void prox_words_kernel(int n_rows, int n_cols, prox_epi P,
                                                         float *__restrict__ Z, int64_t ldz) {
    const int pairs = (P.kw + 1) / 2;
    const int64_t total = (int64_t)n_rows * pairs;
    const int lane = threadIdx.x & 63;
    const unsigned below = (1u << (lane & 31)) - 1u;
    for (int64_t it = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); it < total; it += (int64_t)gridDim.x * 4) {
        const int row = (int)(it / pairs), pr = (int)(it - (int64_t)row * pairs);
        const int col = pr * 64 + lane;
        const bool valid = col < n_cols;
        float o = 0.f;
        if (valid) {
            const int64_t wo = (int64_t)(col >> 5) * n_rows + row;
            const unsigned m = P.mask[wo];
            const bool stored = (m >> (lane & 31)) & 1u;
            const float w = stored ? P.vals[P.pos[wo] + __popc(m & below)] : 0.f;
            float *z = Z + (int64_t)row * ldz + col;
            o = soft_threshold(w, *z, P.eta, P.t);
            *z = o;
        }
        const uint64_t k = __ballot(valid && o != 0.f);
        if (lane == 0) P.counts[(int64_t)row * P.kw + 2 * pr] = __popcll(k & 0xffffffffull);
        if (lane == 32 && 2 * pr + 1 < P.kw) P.counts[(int64_t)row * P.kw + 2 * pr + 1] = __popcll(k >> 32);
    }
}

// row_counts[row] = sum of the row's word counts; blk[b] = sum over rows
// [R b, R b + R), R = 4 x the waves of the workgroup.  A wave per 4 rows;
// each round issues 4 words of each of the 4 rows (16 loads) before adding.
__global__ __launch_bounds__(1024) void row_block_sums_kernel(int n_rows, int kw, const int *__restrict__ counts,
                                                              int *__restrict__ row_counts, int *__restrict__ blk) {
    __shared__ int part[1024 / kWave];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x / kWave;
    const int r0 = (blockIdx.x * nwaves + wave) * 4;
    int v[4] = {0, 0, 0, 0};
    for (int j0 = lane; j0 < kw; j0 += 4 * kWave) {
        int a[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int j = j0 + u * kWave;
                a[q][u] = r0 + q < n_rows && j < kw ? counts[(int64_t)(r0 + q) * kw + j] : 0;
            }
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] += a[q][0] + a[q][1] + a[q][2] + a[q][3];
    }
    int mine = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int tot = wave_sum_int(v[q]);
        if (r0 + q < n_rows) {
            if (lane == 0) row_counts[r0 + q] = tot;
            mine += tot;
        }
    }
    if (lane == 0) part[wave] = mine;
    __syncthreads();
    if (threadIdx.x == 0) {
        int b = 0;
        for (int w = 0; w < nwaves; ++w) b += part[w];
        blk[blockIdx.x] = b;
    }
}

// Z -> col_idx', vals' for columns [c0, c0 + 3072) of one row, nonzeros in
// column order.  With blk, the row's start is row_ptr'[row] = blk[0 .. b) +
// row_counts[R b .. row) (b = row / R, R = prows), and the row's first chunk writes it
// (the last row's also row_ptr'[n_rows] and *d_nnz); without, row_ptr holds
// it.  Thread t holds the float4s t, t + 256, t + 512 of the chunk;
// ranks come from four ballots per float4 slot and the wave totals of all
// three slots are exchanged through LDS in one barrier.  The chunk's output
// is assembled in LDS and then written with every store instruction covering
// 64 consecutive positions (scattered per-lane stores measured 1.5x slower).
template <bool V4>
__global__ __launch_bounds__(kCompactThreads) void compact_kernel(
    int n_rows, int n_cols, int chunks, const float *__restrict__ Z, int64_t ldz, int kw,
    const int *__restrict__ counts, const int *__restrict__ row_counts, const int *__restrict__ blk, int prows,
    int *__restrict__ row_ptr, int *__restrict__ d_nnz, int *__restrict__ col_out, float *__restrict__ val_out,
    int64_t capacity) {
    __shared__ int red[kCompactThreads / kWave];
    __shared__ int tot[kCompactVecs][kCompactThreads / kWave];
    const int row = blockIdx.x / chunks, ch = blockIdx.x - row * chunks;
    const int c0 = ch * kCompactCols;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float *z = Z + (int64_t)row * ldz;
    float v[kCompactVecs][4];
#pragma unroll
    for (int u = 0; u < kCompactVecs; ++u) {
        const int c = c0 + 4 * (tid + u * kCompactThreads);
        if (V4 && c + 3 < n_cols) {
            const float4 t = *reinterpret_cast<const float4 *>(z + c);
            v[u][0] = t.x; v[u][1] = t.y; v[u][2] = t.z; v[u][3] = t.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[u][e] = c + e < n_cols ? z[c + e] : 0.f;
        }
    }
    // the row's output before this chunk: row_ptr' plus the earlier words
    const int s0 = c0 / 32;
    int before = 0;
    for (int j = tid; j < s0; j += kCompactThreads) before += counts[(int64_t)row * kw + j];
    int prefix = 0;  // row_ptr'[row], when added up here
    if (blk) {
        const int b = row / prows, r0 = b * prows;
        if (tid < b) prefix += blk[tid];
        if (tid < row - r0) prefix += row_counts[r0 + tid];
    }
    before = wave_sum_int(before + prefix);
    if (lane == 0) red[wave] = before;
    int below_lane[kCompactVecs];
#pragma unroll
    for (int u = 0; u < kCompactVecs; ++u) {
        int sum = 0, mine = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint64_t b = __ballot(v[u][e] != 0.f);
            sum += __popcll(b);
            mine += popc_below(b);
        }
        below_lane[u] = mine;
        if (lane == 0) tot[u][wave] = sum;
    }
    __syncthreads();
    int64_t base = blk ? 0 : row_ptr[row];
#pragma unroll
    for (int w = 0; w < kCompactThreads / kWave; ++w) base += red[w];
    if (blk && ch == 0 && tid == 0) {  // base = row_ptr'[row] (no words before the first chunk)
        row_ptr[row] = (int)base;
        if (row == n_rows - 1) {
            const int nnz = (int)base + row_counts[row];
            row_ptr[n_rows] = nnz;
            if (d_nnz) *d_nnz = nnz;
        }
    }
    __shared__ int lcol[kCompactCols];
    __shared__ float lval[kCompactCols];
    int lo = 0;  // position inside the chunk's output
#pragma unroll
    for (int u = 0; u < kCompactVecs; ++u) {
        int o = lo + below_lane[u];
#pragma unroll
        for (int w = 0; w < kCompactThreads / kWave; ++w) o += w < wave ? tot[u][w] : 0;
        const int c = c0 + 4 * (tid + u * kCompactThreads);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (v[u][e] != 0.f) {
                lcol[o] = c + e;
                lval[o] = v[u][e];
                ++o;
            }
        }
#pragma unroll
        for (int w = 0; w < kCompactThreads / kWave; ++w) lo += tot[u][w];
    }
    __syncthreads();
    for (int i = tid; i < lo; i += kCompactThreads) {
        if (base + i < capacity) {
            col_out[base + i] = lcol[i];
            val_out[base + i] = lval[i];
        }
    }
}

}  // namespace

size_t word_counts_bytes(int N, int K) { return sizeof(int) * (size_t)N * (size_t)ceil_div(K, 32); }

hipError_t launch_bitmap(int n_rows, int n_cols, const int *ptr, const int *idx, unsigned *mask, int *pos,
                         hipStream_t s) {
    if (n_rows == 0 || n_cols == 0) return hipSuccess;
    const int kw = (int)ceil_div(n_cols, 32);
    if (kw <= kBitmapMaxWords) {
        bitmap_block_kernel<<<(unsigned)ceil_div(n_rows, kBitmapRows), kBitmapThreads, 0, s>>>(n_rows, kw, ptr, idx,
                                                                                               mask, pos);
        return hipGetLastError();
    }
    const int spans = (int)ceil_div(n_cols, kBitmapSpan);  // a row holds at most n_cols entries
    const int64_t blocks = ceil_div((int64_t)n_rows * spans, 4);
    if (blocks > INT32_MAX) return hipErrorInvalidConfiguration;
    bitmap_kernel<<<(unsigned)blocks, 256, 0, s>>>(n_rows, kw, spans, ptr, idx, mask, pos);
    return hipGetLastError();
}

size_t wgrad_prox_split_bytes(int N, int K, int B, int precision) {
    const bool fused = precision == kPrecF32 ? wgrad_f32_prox_slab(N, K, B) > 0 : precision == kPrecBF16X3;
    return fused || precision != kPrecF32 ? 0 : wgrad_workspace_bytes(N, K, B);
}

hipError_t launch_wgrad_prox(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                             int64_t ldx, int precision, const float *vals, const unsigned *mask, const int *pos,
                             float eta, double t, float *Z, int64_t ldz, int *counts, void *split_ws,
                             hipStream_t s) {
    if (N == 0 || K == 0) return hipSuccess;
    prox_epi P{};
    P.mask = mask;
    P.pos = pos;
    P.vals = vals;
    P.eta = (double)eta;
    P.t = t;
    P.kw = (int)ceil_div(K, 32);
    P.counts = counts;
    if (precision == kPrecF32 && wgrad_f32_prox_slab(N, K, B) > 0)
        return launch_wgrad_f32_prox(N, K, B, dY, ldy, X, ldx, Z, ldz, P, s);
    if (precision == kPrecBF16X3) return launch_wgrad_bf16x3_prox(N, K, B, dY, ldy, X, ldx, Z, ldz, P, s);
    // dW into Z, then the prox in place
    hipError_t e;
    if (precision == kPrecF32)
        e = launch_wgrad_f32(N, K, B, dY, ldy, X, ldx, Z, ldz, split_ws, s);
    else
        e = launch_wgrad_bf16(N, K, B, dY, ldy, X, ldx, Z, ldz, s);
    if (e != hipSuccess) return e;
    const int64_t items = (int64_t)N * ((P.kw + 1) / 2);
    const int64_t grid = ceil_div(items, 4) < 8192 ? ceil_div(items, 4) : 8192;
    prox_words_kernel<<<(unsigned)grid, 256, 0, s>>>(N, K, P, Z, ldz);
    return hipGetLastError();
}

size_t counted_ws_ints(int N) { return (size_t)N + 1 + (size_t)ceil_div(N, kPrefixMinRows); }

bool counted_prefix_in_compact(int N) { return ceil_div(N, kPrefixMaxRows) <= kPrefixMaxBlocks; }

hipError_t launch_counted_sums(int N, int K, const int *counts, int *ws, hipStream_t s) {
    if (N == 0) return hipSuccess;
    const int kw = (int)ceil_div(K, 32), r = prefix_rows(N);
    row_block_sums_kernel<<<(unsigned)ceil_div(N, r), 16 * r, 0, s>>>(N, kw, counts, ws, ws + N + 1);
    return hipGetLastError();
}

hipError_t launch_counted_row_ptr(int N, const int *ws, int *row_ptr_out, hipStream_t s) {
    return launch_exclusive_scan(ws, row_ptr_out, N, nullptr, s);  // row_ptr_out[N] = nnz'
}

hipError_t launch_counted_compact(int N, int K, const float *Z, int64_t ldz, const int *counts, const int *ws,
                                  bool prefix_here, int *row_ptr_out, int *col_out, float *val_out,
                                  int64_t capacity, int *d_nnz_out, hipStream_t s) {
    const int kw = (int)ceil_div(K, 32);
    const int chunks = (int)ceil_div(K, kCompactCols);
    const int64_t blocks = (int64_t)N * chunks;
    if (blocks > INT32_MAX) return hipErrorInvalidConfiguration;
    if (prefix_here && !counted_prefix_in_compact(N)) return hipErrorInvalidValue;
    const int *blk = prefix_here ? ws + N + 1 : nullptr;
    int *dn = prefix_here ? d_nnz_out : nullptr;
    hipError_t e = hipSuccess;
    if (blocks > 0) {
        const bool v4 = (ldz % 4 == 0) && aligned16(Z);
        if (v4)
            compact_kernel<true><<<(unsigned)blocks, kCompactThreads, 0, s>>>(
                N, K, chunks, Z, ldz, kw, counts, ws, blk, prefix_rows(N), row_ptr_out, dn, col_out, val_out,
                capacity);
        else
            compact_kernel<false><<<(unsigned)blocks, kCompactThreads, 0, s>>>(
                N, K, chunks, Z, ldz, kw, counts, ws, blk, prefix_rows(N), row_ptr_out, dn, col_out, val_out,
                capacity);
        e = hipGetLastError();
    }
    if (e == hipSuccess && d_nnz_out && !prefix_here) e = launch_copy_i32(row_ptr_out + N, d_nnz_out, s);
    return e;
}

}  // namespace l1csr
