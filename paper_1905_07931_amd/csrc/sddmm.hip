// Masked weight gradient of the debiasing phase:
//     gv[p] = sum_b dY[row(p)][b] * X[col(p)][b]
//
// Work items.  The batch is cut into ranges of NCH chunks (a chunk is 64 lanes
// x VEC floats) and the columns into ranges of 2^shift, sized so that one
// (batch range, column range) "unit" of X is about 2 MB.  Every row gets
// k = ceil(len / lsplit) pieces; piece j of a row takes the row's entries
// j, j + k, j + 2k, ... that fall inside the unit's column range.  An item is
// (unit, piece), and one wave handles one item: it keeps its batch range of
// the dY row in registers, reads the X rows of the piece's entries (coalesced,
// lanes over the batch), and multiplies.  Items are numbered unit-major; the
// units are split into one contiguous range per XCD, and each XCD's waves walk
// their range in order, so an XCD works on about one unit at a time, with that
// unit's 2 MB of X in its own 4 MB L2, and no X row is fetched by two XCDs.
//
// Reduction over the lanes.  Four entries are reduced together: two
// permlane32 swaps and one permlane16 swap turn four 64-lane partial vectors
// into one vector whose 16-lane row r holds 4 lanes' worth of entry r, and
// four DPP steps finish inside the rows.  The order of the additions is fixed,
// so the result does not depend on scheduling.  With several batch ranges the
// per-range sums go to scratch and a second pass adds them in range order.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kGatherThreads = 256;                 // 4 waves
constexpr int kGatherBlocks = 256 * 8;              // persistent grid: 8 blocks per CU
constexpr int64_t kUnitBytes = 2 << 20;             // X bytes per (batch range, column range)
constexpr int kTargetItems = 8192;                  // enough waves to fill the chip
constexpr int64_t kXcdL2Bytes = 4 << 20;            // one XCD's L2
constexpr int64_t kSplitEntries = 32;               // entries per item that pay for an XCD split

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}

// v_r = per-lane partials of entry r (r < 4).  Returns, in every lane of the
// 16-lane row r, the sum of v_r over all 64 lanes.
__device__ __forceinline__ float reduce4(float v0, float v1, float v2, float v3) {
    // permlane32_swap(a, b): a keeps lanes 0-31 and takes b's lanes 0-31 in its
    // lanes 32-63; b takes a's lanes 32-63 in its lanes 0-31.
    const auto s02 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0), __float_as_uint(v2), false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v1), __float_as_uint(v3), false, false);
    const float w0 = __uint_as_float(s02[0]) + __uint_as_float(s02[1]);  // lanes < 32: entry 0, else 2
    const float w1 = __uint_as_float(s13[0]) + __uint_as_float(s13[1]);  // lanes < 32: entry 1, else 3
    // permlane16_swap(a, b): odd 16-lane rows of a trade places with even rows of b
    const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(w0), __float_as_uint(w1), false, false);
    float x = __uint_as_float(s[0]) + __uint_as_float(s[1]);             // row r: entry r
    x += dpp<0x128>(x);  // row_ror:8
    x += dpp<0x124>(x);  // row_ror:4
    x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
    x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
    return x;
}

template <int VEC>
__device__ __forceinline__ void load_vec(const float *p, float (&v)[VEC]) {
    if constexpr (VEC == 4) {
        const float4 t = *reinterpret_cast<const float4 *>(p);
        v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
    } else {
        v[0] = *p;
    }
}

// Extra pieces (row, j), j = 1 .. k_row - 1 with k_row = ceil(len / lsplit),
// listed in row order; their number goes to *ext_n.  One workgroup walks the
// rows in tiles with a carried offset.
__global__ __launch_bounds__(1024) void sddmm_extra_kernel(int n_rows, const int *__restrict__ ptr,
                                                           int lsplit, int2 *__restrict__ ext,
                                                           int *__restrict__ ext_n) {
    __shared__ int wave_tot[16];
    __shared__ int carry_s;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    for (int base = 0; base < n_rows; base += 1024) {
        const int i = base + tid;
        int e = 0;
        if (i < n_rows) {
            const int len = ptr[i + 1] - ptr[i];
            e = len > lsplit ? (len + lsplit - 1) / lsplit - 1 : 0;
        }
        const int incl = wave_incl_scan(e);
        if (lane == 63) wave_tot[wave] = incl;
        __syncthreads();
        if (wave == 0) {
            const int t = lane < 16 ? wave_tot[lane] : 0;
            const int ti = wave_incl_scan(t);
            if (lane < 16) wave_tot[lane] = ti - t;
        }
        __syncthreads();
        const int carry = carry_s;
        const int off = carry + wave_tot[wave] + incl - e;
        for (int j = 0; j < e; ++j) ext[off + j] = make_int2(i, j + 1);
        __syncthreads();
        if (tid == 1023) carry_s = off + e;
        __syncthreads();
    }
    if (tid == 0) *ext_n = carry_s;
}

// The entries of one item in steps of G: loads of all G entries issued
// together, reduced four at a time; entry e's sum is collected in lane e of
// the returned vector (up to 64 entries per call).  FULL: the whole batch
// range lies inside B (no per-lane guard on the loads).
template <int VEC, int NCH, int G, bool FULL>
__device__ __forceinline__ float item_block(const float *__restrict__ X, int64_t ldx, int b_lane, int B,
                                            const float (&dy)[NCH][VEC], int colv, int m) {
    constexpr int CH = kWave * VEC;
    const int lane = threadIdx.x & 63;
    float res = 0.f;
    for (int g = 0; g < m; g += G) {
        float xv[G][NCH][VEC];
#pragma unroll
        for (int i = 0; i < G; ++i) {
            // past the end: repeat the last entry (its sum is not stored)
            const int ci = lane_bcast(colv, min(g + i, m - 1));
            const float *xr = X + (int64_t)ci * ldx + b_lane;
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (FULL || b_lane + c * CH < B) {
                    load_vec<VEC>(xr + c * CH, xv[i][c]);
                } else {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) xv[i][c][v] = 0.f;
                }
            }
        }
        float part[G];
#pragma unroll
        for (int i = 0; i < G; ++i) {
            float a = 0.f;
#pragma unroll
            for (int c = 0; c < NCH; ++c)
#pragma unroll
                for (int v = 0; v < VEC; ++v) a = fmaf(dy[c][v], xv[i][c][v], a);
            part[i] = a;
        }
#pragma unroll
        for (int s4 = 0; s4 < G; s4 += 4) {
            const float tot = reduce4(part[s4], part[s4 + 1], part[s4 + 2], part[s4 + 3]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float v = lane_bcast(tot, 16 * r);
                if (lane == g + s4 + r) res = v;
            }
        }
    }
    return res;
}

// One wave per item, persistent grid.  seg (R > 1) holds the column-range
// bounds of every row: seg[row][cr] = first entry with column >= cr << shift.
// With at least 8 units (and a grid of a multiple of 8 blocks) the units are
// split into 8 contiguous ranges and block b walks range b mod 8 only: blocks
// are dealt to the XCDs round-robin, so every unit is read by one XCD and its
// X rows are fetched into one L2 (the entries of different rows that share a
// column then hit there); otherwise all blocks walk all items.
template <int VEC, int NCH, int G>
__global__ __launch_bounds__(kGatherThreads) void sddmm_gather_kernel(
    int n_rows, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ dY, int64_t ldy, const float *__restrict__ X, int64_t ldx, int B,
    int R, int nbr, int lsplit, const int *__restrict__ seg, const int2 *__restrict__ ext,
    const int *__restrict__ ext_n, float *__restrict__ out, int64_t nnz) {
    constexpr int CH = kWave * VEC;   // batch entries per chunk
    constexpr int BRW = NCH * CH;     // batch entries per range
    constexpr int WPB = kGatherThreads / kWave;
    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int P = n_rows + (ext_n ? uniform(*ext_n) : 0);
    const int64_t units = (int64_t)R * nbr;
    const bool by_xcd = units >= 8 && gridDim.x % 8 == 0;
    int64_t u_lo = 0, u_hi = units, stride, t0;
    if (by_xcd) {
        const int x = blockIdx.x % 8;
        u_lo = units * x / 8;
        u_hi = units * (x + 1) / 8;
        stride = (int64_t)(gridDim.x / 8) * WPB;
        t0 = (int64_t)(blockIdx.x / 8) * WPB + wave;
    } else {
        stride = (int64_t)gridDim.x * WPB;
        t0 = (int64_t)blockIdx.x * WPB + wave;
    }
    const int64_t total = (u_hi - u_lo) * P;
    // item t = (u - u_lo) * P + q, stepped incrementally
    const int64_t du = stride / P;
    const int dq = (int)(stride - du * P);
    int64_t u = u_lo + t0 / P;
    int q = (int)(t0 % P);

    for (int64_t t = t0; t < total; t += stride) {
        const int br = (int)(u / R);
        const int cr = (int)(u - (int64_t)br * R);
        int row, j;
        if (q < n_rows) {
            row = q;
            j = 0;
        } else {
            const int2 e = ext[q - n_rows];
            row = uniform(e.x);
            j = uniform(e.y);
        }
        u += du;
        q += dq;
        if (q >= P) {
            q -= P;
            ++u;
        }
        const int rs = ptr[row], re = ptr[row + 1];
        const int len = re - rs;
        const int k = len > lsplit ? (len + lsplit - 1) / lsplit : 1;
        int lo = rs, hi = re;
        if (R > 1) {
            const int *sr = seg + (int64_t)row * (R + 1) + cr;
            lo = sr[0];
            hi = sr[1];
        }
        const int first = lo + j;
        if (first >= hi) continue;
        const int n = (hi - first + k - 1) / k;

        const int b_lane = br * BRW + lane * VEC;
        const bool full = (int64_t)(br + 1) * BRW <= B;
        float dy[NCH][VEC];
        const float *dyr = dY + (int64_t)row * ldy + b_lane;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (b_lane + c * CH < B) {
                load_vec<VEC>(dyr + c * CH, dy[c]);
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v) dy[c][v] = 0.f;
            }
        }
        float *o = out + (int64_t)br * nnz + first;
        for (int base = 0; base < n; base += kWave) {
            const int m = min(kWave, n - base);
            const int colv = lane < m ? idx[first + (int64_t)(base + lane) * k] : 0;
            const float res = full ? item_block<VEC, NCH, G, true>(X, ldx, b_lane, B, dy, colv, m)
                                   : item_block<VEC, NCH, G, false>(X, ldx, b_lane, B, dy, colv, m);
            if (lane < m) o[(int64_t)(base + lane) * k] = res;
        }
    }
}

// Dense patterns: one wave per (unit, block of kRB consecutive rows).  The
// wave keeps the dY batch range of its kRB rows in registers and walks the
// unit's columns in windows of 64.  Per window it marks in a 64-word LDS table
// of its own which of its rows store each column (bit i: row r0 + i; columns
// are strictly increasing in a row, so a row's next 64 entries cover the
// window), then loads the X row of every marked column once and forms the
// products of all kRB rows with it, storing those present.  An X row then
// serves every row of the block that stores its column, where the gather
// reads it once per entry.  The per-entry arithmetic (fmaf chain over the
// lane's batch slice, then reduce4) is the gather's, so the results are too.
constexpr int kRB = 8;

template <int VEC, int NCH, int G>
__global__ __launch_bounds__(kGatherThreads) void sddmm_block_kernel(
    int n_rows, int n_cols, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ dY, int64_t ldy, const float *__restrict__ X, int64_t ldx, int B,
    int R, int nbr, int shift, const int *__restrict__ seg, float *__restrict__ out, int64_t nnz) {
    constexpr int CH = kWave * VEC;
    constexpr int BRW = NCH * CH;
    constexpr int WPB = kGatherThreads / kWave;
    __shared__ unsigned flags_s[WPB][kWave];
    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    unsigned *flags = flags_s[wave];
    const int nb = (n_rows + kRB - 1) / kRB;
    const int64_t units = (int64_t)R * nbr;
    const bool by_xcd = units >= 8 && gridDim.x % 8 == 0;
    int64_t u_lo = 0, u_hi = units, stride, t0;
    if (by_xcd) {
        const int x = blockIdx.x % 8;
        u_lo = units * x / 8;
        u_hi = units * (x + 1) / 8;
        stride = (int64_t)(gridDim.x / 8) * WPB;
        t0 = (int64_t)(blockIdx.x / 8) * WPB + wave;
    } else {
        stride = (int64_t)gridDim.x * WPB;
        t0 = (int64_t)blockIdx.x * WPB + wave;
    }
    const int64_t total = (u_hi - u_lo) * nb;
    const int r16 = lane >> 4;
    const bool head = (lane & 15) == 0;

    for (int64_t t = t0; t < total; t += stride) {
        const int64_t u = u_lo + t / nb;
        const int r0 = (int)(t % nb) * kRB;
        const int br = (int)(u / R);
        const int cr = (int)(u - (int64_t)br * R);
        const int c0 = cr << shift;
        const int c1 = min(n_cols, c0 + (1 << shift));
        const int b_lane = br * BRW + lane * VEC;
        const bool full = (int64_t)(br + 1) * BRW <= B;
        int cur[kRB], hi[kRB];
        float dy[kRB][NCH][VEC];
#pragma unroll
        for (int i = 0; i < kRB; ++i) {
            const int row = r0 + i;
            cur[i] = hi[i] = 0;
            if (row < n_rows) {
                if (R > 1) {
                    const int *sr = seg + (int64_t)row * (R + 1) + cr;
                    cur[i] = uniform(sr[0]);
                    hi[i] = uniform(sr[1]);
                } else {
                    cur[i] = uniform(ptr[row]);
                    hi[i] = uniform(ptr[row + 1]);
                }
            }
            const float *dyr = dY + (int64_t)row * ldy + b_lane;
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (row < n_rows && b_lane + c * CH < B) {
                    load_vec<VEC>(dyr + c * CH, dy[i][c]);
                } else {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) dy[i][c][v] = 0.f;
                }
            }
        }
        float *o = out + (int64_t)br * nnz;
        for (int ws = c0; ws < c1; ws += kWave) {
            flags[lane] = 0u;
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int i = 0; i < kRB; ++i) {
                const int k = cur[i] + lane;
                if (k < hi[i]) {
                    const int c = idx[k];
                    if (c >= ws && c < ws + kWave) atomicOr(&flags[c - ws], 1u << i);
                }
            }
            __builtin_amdgcn_wave_barrier();
            const unsigned f = flags[lane];
            __builtin_amdgcn_wave_barrier();
            uint64_t cm[kRB];
#pragma unroll
            for (int i = 0; i < kRB; ++i) cm[i] = wave_ballot((f >> i) & 1u);
            // the row mask and first position of this lane's 16-lane group
            // (entry r16 of each reduce4: rows r16 and 4 + r16)
            const uint64_t mA = r16 == 0 ? cm[0] : r16 == 1 ? cm[1] : r16 == 2 ? cm[2] : cm[3];
            const uint64_t mB = r16 == 0 ? cm[4] : r16 == 1 ? cm[5] : r16 == 2 ? cm[6] : cm[7];
            const int pA = r16 == 0 ? cur[0] : r16 == 1 ? cur[1] : r16 == 2 ? cur[2] : cur[3];
            const int pB = r16 == 0 ? cur[4] : r16 == 1 ? cur[5] : r16 == 2 ? cur[6] : cur[7];
            uint64_t U = wave_ballot(f != 0u);
            while (U) {
                int oc[G];
                bool ok[G];
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    ok[g] = U != 0;
                    oc[g] = ok[g] ? (int)__builtin_ctzll(U) : oc[g > 0 ? g - 1 : 0];
                    U &= U - 1;
                }
                float xv[G][NCH][VEC];
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const float *xr = X + (int64_t)(ws + oc[g]) * ldx + b_lane;
#pragma unroll
                    for (int c = 0; c < NCH; ++c) {
                        if (full || b_lane + c * CH < B) {
                            load_vec<VEC>(xr + c * CH, xv[g][c]);
                        } else {
#pragma unroll
                            for (int v = 0; v < VEC; ++v) xv[g][c][v] = 0.f;
                        }
                    }
                }
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    // rows storing this column (wave-uniform): the others'
                    // products and an all-absent half's reduction are skipped
                    const unsigned fc = (unsigned)__builtin_amdgcn_readlane((int)f, oc[g]);
                    float part[kRB];
#pragma unroll
                    for (int i = 0; i < kRB; ++i) {
                        float a = 0.f;
                        if ((fc >> i) & 1u) {
#pragma unroll
                            for (int c = 0; c < NCH; ++c)
#pragma unroll
                                for (int v = 0; v < VEC; ++v) a = fmaf(dy[i][c][v], xv[g][c][v], a);
                        }
                        part[i] = a;
                    }
                    float tA = 0.f, tB = 0.f;
                    if (fc & 0xFu) tA = reduce4(part[0], part[1], part[2], part[3]);
                    if (fc & 0xF0u) tB = reduce4(part[4], part[5], part[6], part[7]);
                    const uint64_t below = (1ull << oc[g]) - 1ull;
                    if (ok[g] && head) {
                        if ((mA >> oc[g]) & 1ull) o[pA + __builtin_popcountll(mA & below)] = tA;
                        if ((mB >> oc[g]) & 1ull) o[pB + __builtin_popcountll(mB & below)] = tB;
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < kRB; ++i) cur[i] += __builtin_popcountll(cm[i]);
        }
    }
}

// gv[p] = sum of part[s][p] over the nseg batch ranges.  A workgroup owns 64
// entries; its four waves add contiguous quarters of the ranges in ascending
// order and the quarters are added in order, so the result is deterministic.
__global__ __launch_bounds__(256) void sddmm_reduce_kernel(int64_t nnz, int nseg,
                                                           const float *__restrict__ part,
                                                           float *__restrict__ gv) {
    __shared__ float red[3][kWave];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t p = (int64_t)blockIdx.x * kWave + lane;
    const int per = (nseg + 3) / 4;
    const int s0 = min(nseg, wave * per), s1 = min(nseg, s0 + per);
    float acc = 0.f;
    if (p < nnz) {
        int s = s0;
        for (; s + 8 <= s1; s += 8) {
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = part[(int64_t)(s + i) * nnz + p];
#pragma unroll
            for (int i = 0; i < 8; ++i) acc += v[i];
        }
        for (; s < s1; ++s) acc += part[(int64_t)s * nnz + p];
    }
    if (wave > 0) red[wave - 1][lane] = acc;
    __syncthreads();
    if (wave == 0 && p < nnz) gv[p] = ((acc + red[0][lane]) + red[1][lane]) + red[2][lane];
}

struct gplan {
    int vec, nch, nbr;
    int shift, R;
    int lsplit;
    bool block;         // dense pattern: sddmm_block_kernel over blocks of kRB rows
    bool extras;        // some row can be longer than lsplit
    int64_t ext_max;    // bound on the number of extra pieces
};

int64_t plan_items(int n_rows, int64_t nnz, int R, int nbr, int lsplit) {
    return (int64_t)nbr * R * (n_rows + nnz / lsplit);
}

gplan make_plan(int n_rows, int n_cols, int64_t nnz, int B, bool v4) {
    gplan pl;
    pl.vec = v4 ? 4 : 1;
    const int ch = kWave * pl.vec;
    const int64_t nchunks = ceil_div(B, ch);
    auto shape = [&](int nch) {
        pl.nch = nch;
        pl.nbr = (int)ceil_div(nchunks, nch);
        const int64_t col_bytes = 4 * (int64_t)(B < nch * ch ? B : nch * ch);
        int shift = 6;
        while (shift < 30 && ((int64_t)2 << shift) * col_bytes <= kUnitBytes) ++shift;
        pl.shift = shift;
        pl.R = (int)ceil_div(n_cols, (int64_t)1 << shift);
        if (pl.R < 1) pl.R = 1;
        // Fewer than 8 units while X does not fit one XCD's L2: every XCD
        // would fetch all of X.  Narrower column ranges give each XCD a slice
        // of its own, at the price of one more read of a dY row per extra
        // item, which pays where items keep many entries (4096 x 4096,
        // batch 512: 17 % faster at 20 % density, 30 % at 50 %, 8 % slower
        // at 1 %).
        while ((int64_t)pl.R * pl.nbr < 8 && pl.shift > 6 && 4 * (int64_t)n_cols * B > kXcdL2Bytes) {
            const int r2 = (int)ceil_div(n_cols, (int64_t)1 << (pl.shift - 1));
            if (nnz < kSplitEntries * n_rows * r2) break;
            --pl.shift;
            pl.R = r2;
        }
    };
    // longest batch range (fewest reductions) that still yields enough items,
    // then shorter pieces if needed
    const int nchs[3] = {4, 2, 1};
    int c0 = 0;
    while (c0 < 2 && nchs[c0] > nchunks) ++c0;
    bool done = false;
    for (int c = c0; c < 3 && !done; ++c) {
        shape(nchs[c]);
        pl.lsplit = 64 * pl.R;
        if (plan_items(n_rows, nnz, pl.R, pl.nbr, pl.lsplit) >= kTargetItems) done = true;
    }
    if (!done) {
        while (pl.lsplit > 8 * pl.R && plan_items(n_rows, nnz, pl.R, pl.nbr, pl.lsplit) < kTargetItems)
            pl.lsplit /= 2;
    }
    pl.extras = pl.lsplit < n_cols;
    pl.ext_max = pl.extras ? nnz / pl.lsplit + 1 : 0;
    // a third of the entries stored or more (vector loads): blocks of kRB
    // rows, each X row loaded once per block; no row pieces, and narrower
    // column ranges until there are enough items.  (4096 x 4096, batch 512:
    // 940 -> 395-402 us at 50 % density; at 20 % it ties the gather, whose
    // 286 us it keeps.)
    pl.block = v4 && 3 * nnz >= (int64_t)n_rows * n_cols;
    if (pl.block) {
        pl.extras = false;
        pl.ext_max = 0;
        const int64_t nb = ceil_div(n_rows, kRB);
        while ((int64_t)pl.nbr * pl.R * nb < kTargetItems && pl.shift > 6) {
            --pl.shift;
            pl.R = (int)ceil_div(n_cols, (int64_t)1 << pl.shift);
        }
    }
    return pl;
}

struct gwork {
    int *seg;
    int2 *ext;
    int *ext_n;
    float *part;
    size_t bytes;
};

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

gwork carve(const gplan &pl, int n_rows, int64_t nnz, void *ws) {
    gwork w{};
    char *p = static_cast<char *>(ws);
    size_t off = 0;
    auto take = [&](size_t bytes) -> char * {
        char *r = p ? p + off : nullptr;
        off += align256(bytes);
        return r;
    };
    if (pl.R > 1) w.seg = reinterpret_cast<int *>(take(sizeof(int) * (size_t)n_rows * (pl.R + 1)));
    if (pl.extras) {
        w.ext_n = reinterpret_cast<int *>(take(sizeof(int)));
        w.ext = reinterpret_cast<int2 *>(take(sizeof(int2) * (size_t)pl.ext_max));
    }
    if (pl.nbr > 1) w.part = reinterpret_cast<float *>(take(sizeof(float) * (size_t)pl.nbr * nnz));
    w.bytes = off;
    return w;
}

template <int VEC, int NCH>
void launch_gather(const gplan &pl, const gwork &w, int n_rows, int64_t nnz, const int *ptr,
                   const int *idx, const float *dY, int64_t ldy, const float *X, int64_t ldx, int B,
                   float *out, hipStream_t s) {
    constexpr int G = NCH == 1 ? 8 : 4;
    const int64_t items = plan_items(n_rows, nnz, pl.R, pl.nbr, pl.lsplit);
    int64_t blocks = ceil_div(items, kGatherThreads / kWave);
    if (blocks > kGatherBlocks) blocks = kGatherBlocks;
    blocks = ceil_div(blocks, 8) * 8;  // whole rounds of the 8 XCDs
    sddmm_gather_kernel<VEC, NCH, G><<<(unsigned)blocks, kGatherThreads, 0, s>>>(
        n_rows, ptr, idx, dY, ldy, X, ldx, B, pl.R, pl.nbr, pl.lsplit, w.seg, w.ext, w.ext_n, out, nnz);
}

template <int NCH>
void launch_block(const gplan &pl, const gwork &w, int n_rows, int n_cols, int64_t nnz, const int *ptr,
                  const int *idx, const float *dY, int64_t ldy, const float *X, int64_t ldx, int B,
                  float *out, hipStream_t s) {
    constexpr int G = NCH == 4 ? 2 : 4;
    const int64_t items = (int64_t)pl.nbr * pl.R * ceil_div(n_rows, kRB);
    int64_t blocks = ceil_div(items, kGatherThreads / kWave);
    if (blocks > kGatherBlocks) blocks = kGatherBlocks;
    blocks = ceil_div(blocks, 8) * 8;  // whole rounds of the 8 XCDs
    sddmm_block_kernel<4, NCH, G><<<(unsigned)blocks, kGatherThreads, 0, s>>>(
        n_rows, n_cols, ptr, idx, dY, ldy, X, ldx, B, pl.R, pl.nbr, pl.shift, w.seg, out, nnz);
}

}  // namespace

size_t sddmm_workspace_bytes(int n_rows, int n_cols, int64_t nnz, int B) {
    if (nnz == 0 || B == 0) return 0;
    // the larger of the vector and scalar plans
    const size_t a = carve(make_plan(n_rows, n_cols, nnz, B, true), n_rows, nnz, nullptr).bytes;
    const size_t b = carve(make_plan(n_rows, n_cols, nnz, B, false), n_rows, nnz, nullptr).bytes;
    return a > b ? a : b;
}

hipError_t launch_sddmm(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                        const float *dY, int64_t ldy, const float *X, int64_t ldx, int B, float *gv,
                        void *ws, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    if (B == 0) return launch_fill_f32(gv, nnz, 0.f, s);
    hipError_t e;
    const bool v4 = (B % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) && aligned16(dY);
    const gplan pl = make_plan(n_rows, n_cols, nnz, B, v4);
    const gwork w = carve(pl, n_rows, nnz, ws);
    if (pl.R > 1 && (e = launch_seg(n_rows, pl.R, pl.shift, ptr, idx, w.seg, s)) != hipSuccess) return e;
    if (pl.extras) {
        sddmm_extra_kernel<<<1, 1024, 0, s>>>(n_rows, ptr, pl.lsplit, w.ext, w.ext_n);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    float *out = pl.nbr > 1 ? w.part : gv;
    if (pl.block) {
        if (pl.nch == 4) launch_block<4>(pl, w, n_rows, n_cols, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
        else if (pl.nch == 2) launch_block<2>(pl, w, n_rows, n_cols, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
        else launch_block<1>(pl, w, n_rows, n_cols, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
    } else if (pl.vec == 4) {
        if (pl.nch == 4) launch_gather<4, 4>(pl, w, n_rows, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
        else if (pl.nch == 2) launch_gather<4, 2>(pl, w, n_rows, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
        else launch_gather<4, 1>(pl, w, n_rows, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
    } else {
        if (pl.nch == 4) launch_gather<1, 4>(pl, w, n_rows, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
        else if (pl.nch == 2) launch_gather<1, 2>(pl, w, n_rows, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
        else launch_gather<1, 1>(pl, w, n_rows, nnz, ptr, idx, dY, ldy, X, ldx, B, out, s);
    }
    if ((e = hipGetLastError()) != hipSuccess || pl.nbr == 1) return e;
    sddmm_reduce_kernel<<<(unsigned)ceil_div(nnz, kWave), 256, 0, s>>>(nnz, pl.nbr, w.part, gv);
    return hipGetLastError();
}

}  // namespace l1csr
