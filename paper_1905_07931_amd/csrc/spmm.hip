// CSR x dense products with the batch index contiguous (forward Y = W.X and,
// over the CSC copy, backward dX = W^T.dY).
//
// Streamed tiled kernel (the hot path).  One 1024-thread workgroup per CU owns
// a chunk of BB = 64*VEC batch columns (32*VEC with half-wave units) and a set
// of rows; every lane keeps VEC accumulators for each of the wave's row pieces.  The dense operand passes
// through LDS in 64 KB tiles of KT rows, double buffered: while the waves work
// on tile t, the direct global->LDS loads of tile t+1 are in flight.
//
// The nonzeros are not read from the CSR arrays inside the kernel.  A
// planning pass writes, for every wave and tile, a chunk of a "pair stream":
// a header with the pair count of each of the wave's pieces in the tile, then
// the pairs (byte offset of the X row inside the tile, value), each piece's
// run padded to an even count with a zero pair.  The wave's chunk of tile t+1
// is loaded into LDS together with X, so the inner loop reads two pairs with
// one broadcast LDS read and then two X rows, with no global latency and no
// per-segment bookkeeping.  A chunk longer than its LDS slot is finished from
// global memory.
//
// Load balance (power-law row lengths): a row longer than half the mean wave
// load is cut into k pieces, piece j taking every k-th nonzero of the row, so
// a piece of a dense row spreads evenly over the tiles (contiguous pieces
// would pile one wave's work into a few tiles and stall the workgroup at
// every tile barrier).  Pieces are sorted by length (bucketed) and dealt to
// the waves in snake order.  A split row's pieces write partial rows that a
// fix-up pass sums in piece order; every piece is summed by one wave in a
// fixed order, so the result does not depend on the schedule.  The grid maps
// blocks to XCDs so that the workgroups of one XCD share a batch chunk (the
// same slice of X in that XCD's L2).
//
// Rows kernel (small, narrow or very sparse operands): one wave per (row,
// batch chunk) reading X directly from the cache hierarchy.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

template <int VEC>
__device__ __forceinline__ void load_vec(const float *p, float (&x)[VEC]) {
    if constexpr (VEC == 4) {
        const float4 t = *reinterpret_cast<const float4 *>(p);
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    } else if constexpr (VEC == 2) {
        const float2 t = *reinterpret_cast<const float2 *>(p);
        x[0] = t.x; x[1] = t.y;
    } else {
        x[0] = *p;
    }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float *p, const float (&x)[VEC]) {
    if constexpr (VEC == 4) {
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
    } else if constexpr (VEC == 2) {
        *reinterpret_cast<float2 *>(p) = make_float2(x[0], x[1]);
    } else {
        *p = x[0];
    }
}

// ---------------------------------------------------------------------------
// planning: segment pointers, pieces, length order, pair stream
// ---------------------------------------------------------------------------

// seg[row][t] = first position p of the row with idx[p] >= t << shift
// (t = 0..ntiles), so seg[row][0] = ptr[row] and seg[row][ntiles] = ptr[row+1].
__global__ __launch_bounds__(256) void seg_kernel(int n_rows, int ntiles, int shift,
                                                  const int *__restrict__ ptr,
                                                  const int *__restrict__ idx,
                                                  int *__restrict__ seg) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int s = ptr[row], e = ptr[row + 1];
    int *sr = seg + (int64_t)row * (ntiles + 1);
    // one search per tile boundary (lanes over tiles): 8-ary steps (seven
    // probes loaded together) while the interval is long, then binary.  The
    // answer stays in [lo, hi] ⊆ [s, e], also for a malformed row.
    for (int t = lane; t <= ntiles; t += kWave) {
        int lo = s, hi = e;
        if (t == 0) {
            hi = s;
        } else if (t < ntiles) {
            const int key = t << shift;
            while (hi - lo >= 8) {
                const int step = (hi - lo) >> 3;
                int v[7];
#pragma unroll
                for (int u = 0; u < 7; ++u) v[u] = idx[lo + (u + 1) * step];
                int c = 0;
#pragma unroll
                for (int u = 0; u < 7; ++u) c += v[u] < key ? 1 : 0;
                // probes 1..c lie before the answer, probe c + 1 (if any) at or after it
                const int nlo = c > 0 ? lo + c * step + 1 : lo;
                hi = c < 7 ? lo + (c + 1) * step : hi;
                lo = nlo;
            }
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (idx[mid] < key) lo = mid + 1; else hi = mid;
            }
        } else {
            lo = e;
        }
        sr[t] = lo;
    }
}

// entries of a piece (row length len): positions j, j + k, ... < len
__device__ __forceinline__ int piece_len(int len, int j, int k) {
    return len > j ? (len - j + k - 1) / k : 0;
}

// 16 buckets per octave of the piece length, plus empty: fine enough that the
// lengths of one matrix spread over many buckets (the planner's bucket
// counters are LDS atomics, and pieces of equal key serialise on one address)
constexpr int kBucketBits = 4;
constexpr int kBuckets = 1 + 31 * (1 << kBucketBits);

__device__ __forceinline__ int length_key(int len) {
    if (len <= 0) return 0;
    const int b = 31 - __clz(len);
    const int sub = b >= kBucketBits ? (len >> (b - kBucketBits)) & ((1 << kBucketBits) - 1)
                                     : (len << (kBucketBits - b)) & ((1 << kBucketBits) - 1);
    return 1 + b * (1 << kBucketBits) + sub;
}

// The planner cuts rows into pieces and deals them to the waves:
//   pieces: a row of len > cap entries is cut into k = ceil(len / cap) pieces
//           (cap = max(64, ceil(nnz / (2 nw))), so there are at most
//           n_rows + 2 nw pieces), piece j taking every k-th entry from the
//           j-th; pbeg[row] = index of the row's first piece (pieces are
//           numbered row by row, which is the order the fix-up sums them in);
//   deal:   pieces by decreasing length bucket, the piece at sorted position
//           p going to slot i = p / nw of wave g = p mod nw, snake order over
//           rounds (odd rounds reversed).  The order inside a bucket only
//           decides which wave computes a piece, never how it is summed.
//   table:  slot i of wave g = (row, first strided position, k, entries), row
//           = -1 for an empty slot.
// Two launches over contiguous row blocks (a counting sort by bucket):
// plan_hist_kernel writes every block's bucket histogram and piece count;
// plan_deal_kernel derives its block's start in every bucket and its pieces'
// numbers from all blocks' counts, then deals its pieces with LDS cursors.
constexpr int kPlanThreads = 256;
constexpr int kPlanMaxBlocks = 64;

__device__ __forceinline__ int plan_cap(const int *__restrict__ ptr, int n_rows, int nw) {
    // pieces of at most half the mean load per wave (from the actual number of
    // entries, read on the device): with the snake deal the heaviest and
    // lightest waves then differ by a few percent even for power-law row
    // lengths (a cap of the full mean leaves ~30%)
    const int64_t nnz = ptr[n_rows] - ptr[0];
    const int64_t cap64 = (nnz + 2 * (int64_t)nw - 1) / (2 * (int64_t)nw);
    return (int)(cap64 < 64 ? 64 : (cap64 > INT32_MAX ? INT32_MAX : cap64));
}

// block-wide exclusive scan of one value per thread (all kPlanThreads threads
// call it); total = the block's sum
__device__ __forceinline__ int plan_excl_scan(int v, int *wave_tot, int &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int incl = wave_incl_scan(v);
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int before = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kPlanThreads / kWave; ++w) {
        const int t = wave_tot[w];
        before += w < wave ? t : 0;
        total += t;
    }
    __syncthreads();  // wave_tot is reused by the next call
    return before + incl - v;
}

// a row of len entries in k pieces: len % k pieces of ceil(len / k) entries,
// the rest of floor(len / k)
// wsize[g] is set to wbase = a bound on the bytes of wave g's stream that do
// not depend on its pieces' lengths (chunk headers, 16 bytes per slot and
// tile for padding); plan_deal_kernel adds 8 bytes per entry of every piece it
// deals to g, rounded up to 16, so every stream starts 16-byte aligned.
__global__ __launch_bounds__(kPlanThreads) void plan_hist_kernel(int n_rows, const int *__restrict__ ptr, int nw,
                                                                 int rpb, int *__restrict__ bh,
                                                                 int *__restrict__ bsum, int *__restrict__ wsize,
                                                                 int wbase) {
    __shared__ int hist[kBuckets];
    __shared__ int wave_tot[kPlanThreads / kWave];
    const int b = blockIdx.x, tid = threadIdx.x;
    for (int g = b * kPlanThreads + tid; g < nw; g += gridDim.x * kPlanThreads) wsize[g] = wbase;
    const int cap = plan_cap(ptr, n_rows, nw);
    for (int i = tid; i < kBuckets; i += kPlanThreads) hist[i] = 0;
    __syncthreads();
    const int r0 = b * rpb, r1 = min(n_rows, r0 + rpb);
    int mine = 0;
    for (int r = r0 + tid; r < r1; r += kPlanThreads) {
        const int len = ptr[r + 1] - ptr[r];
        const int k = len > cap ? (len + cap - 1) / cap : 1;
        const int big = len % k, lo = len / k;
        if (big) atomicAdd(&hist[length_key(lo + 1)], big);
        atomicAdd(&hist[length_key(lo)], k - big);
        mine += k;
    }
    int total;
    plan_excl_scan(mine, wave_tot, total);  // (ends with a barrier: hist is complete)
    for (int i = tid; i < kBuckets; i += kPlanThreads) bh[(int64_t)b * kBuckets + i] = hist[i];
    if (tid == 0) bsum[b] = total;
}

__global__ __launch_bounds__(kPlanThreads) void plan_deal_kernel(int n_rows, const int *__restrict__ ptr, int nw,
                                                                 int rw, int rpb, int nb,
                                                                 const int *__restrict__ bh,
                                                                 const int *__restrict__ bsum,
                                                                 int *__restrict__ pbeg,
                                                                 int4 *__restrict__ table,
                                                                 int *__restrict__ wsize) {
    constexpr int KPT = (kBuckets + kPlanThreads - 1) / kPlanThreads;  // buckets per thread
    __shared__ int cursor[kBuckets];
    __shared__ int wave_tot[kPlanThreads / kWave];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int cap = plan_cap(ptr, n_rows, nw);
    // this block's start in every bucket: all pieces of larger buckets, plus
    // the pieces of the same bucket in earlier blocks.  Thread t holds the
    // buckets at descending positions KPT*t .. KPT*t + KPT - 1.
    // (the blocks' counts are read 8 blocks at a time, all loads in flight)
    int all[KPT], before[KPT], sum = 0;
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
        const int key = kBuckets - 1 - (KPT * tid + q);
        all[q] = 0;
        before[q] = 0;
        if (key >= 0)
            for (int c0 = 0; c0 < nb; c0 += 8) {
                int h[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) h[u] = c0 + u < nb ? bh[(int64_t)(c0 + u) * kBuckets + key] : 0;
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    all[q] += h[u];
                    before[q] += c0 + u < b ? h[u] : 0;
                }
            }
        sum += all[q];
    }
    int total;
    int run = plan_excl_scan(sum, wave_tot, total);
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
        const int key = kBuckets - 1 - (KPT * tid + q);
        if (key >= 0) cursor[key] = run + before[q];
        run += all[q];
    }
    // pieces before this block, and the total
    int first_piece = 0, n_pieces = 0;
    for (int c0 = 0; c0 < nb; c0 += 8) {
        int h[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) h[u] = c0 + u < nb ? bsum[c0 + u] : 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            first_piece += c0 + u < b ? h[u] : 0;
            n_pieces += h[u];
        }
    }
    // pbeg of the block's rows: each thread takes a contiguous run of rows
    const int r0 = b * rpb, r1 = min(n_rows, r0 + rpb);
    const int per = (rpb + kPlanThreads - 1) / kPlanThreads;
    const int t0 = min(r1, r0 + tid * per), t1 = min(r1, t0 + per);
    int mine = 0;
    for (int r = t0; r < t1; ++r) {
        const int len = ptr[r + 1] - ptr[r];
        mine += len > cap ? (len + cap - 1) / cap : 1;
    }
    int blk_total;
    int v = first_piece + plan_excl_scan(mine, wave_tot, blk_total);  // (barrier: cursors visible)
    for (int r = t0; r < t1; ++r) {
        const int s = ptr[r], len = ptr[r + 1] - s;
        const int k = len > cap ? (len + cap - 1) / cap : 1;
        pbeg[r] = v;
        v += k;
        for (int j = 0; j < k; ++j) {
            const int plen = piece_len(len, j, k);
            const int pos = atomicAdd(&cursor[length_key(plen)], 1);
            const int i = pos / nw, gq = pos - i * nw;
            const int g = (i & 1) ? nw - 1 - gq : gq;
            if (i < rw) {
                table[(int64_t)g * rw + i] = make_int4(r, s + j, k, plen);
                atomicAdd(&wsize[g], 8 * (plen + (plen & 1)));  // 16-byte multiples; integer sum
            }
        }
    }
    if (b == nb - 1 && tid == 0) pbeg[n_rows] = n_pieces;
    // empty slots
    for (int64_t pos = n_pieces + (int64_t)b * kPlanThreads + tid; pos < (int64_t)nw * rw;
         pos += (int64_t)nb * kPlanThreads) {
        const int i = (int)(pos / nw), gq = (int)(pos - (int64_t)i * nw);
        const int g = (i & 1) ? nw - 1 - gq : gq;
        table[(int64_t)g * rw + i] = make_int4(-1, 0, 1, 0);
    }
}

constexpr int kNW = 16;             // waves per workgroup (1024 threads)
constexpr int kTileFloats = 16384;  // 64 KB of X per tile buffer
constexpr int kChunk = 1024;        // bytes of a wave's pair stream staged per tile

// VEC batch columns per lane; HALF: the two half-waves take the two pairs of a
// unit, each over the same 32*VEC columns (twice the tile height of a
// full-wave workgroup for the same 64 KB of LDS)
template <int VEC, bool HALF>
struct tiled_cfg {
    static constexpr int LANES = HALF ? kWave / 2 : kWave;  // lanes across the batch
    static constexpr int BB = LANES * VEC;                  // batch columns per workgroup
    static constexpr int KT = kTileFloats / BB;             // X rows per tile
    static constexpr int SHIFT = KT == 256 ? 8 : (KT == 128 ? 7 : 6);
    static constexpr int MAXRW = VEC == 2 ? 24 : 12;          // pieces per wave in registers
    static constexpr int HDR = ((2 * MAXRW + 15) / 16) * 16;  // chunk header: uint16 count per piece
    static_assert((1 << SHIFT) == KT, "tile height must be a power of two");
};

// strided position bound of a piece in a tile: the number of its entries
// (positions first + m*k, m = 0, 1, ...) that lie before position p
__device__ __forceinline__ int piece_before(int p, int first, int k, int plen) {
    const int d = p - first;
    if (d <= 0) return 0;
    const int m = k == 1 ? d : (d + k - 1) / k;
    return m < plen ? m : plen;
}

// per wave stream g (one wave each, lanes over tiles): the byte offset of every
// chunk inside the stream (header + padded pair runs, exclusive scan over the
// tiles) and the stream's total size
template <int VEC, bool HALF>
__global__ __launch_bounds__(256) void stream_size_kernel(int nw, int rw, int ntiles,
                                                          const int4 *__restrict__ table,
                                                          const int *__restrict__ seg,
                                                          int *__restrict__ coff,
                                                          int *__restrict__ wsize) {
    constexpr int MAXRW = tiled_cfg<VEC, HALF>::MAXRW, HDR = tiled_cfg<VEC, HALF>::HDR;
    const int g = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (g >= nw) return;
    const int lane = threadIdx.x & 63;
    // lane i holds slot i's piece
    int4 e = make_int4(-1, 0, 1, 0);
    if (lane < rw && lane < MAXRW) e = table[(int64_t)g * rw + lane];
    int carry = 0;
    for (int t0 = 0; t0 < ntiles; t0 += kWave) {
        const int t = t0 + lane;
        int bytes = 0;
        if (t < ntiles) {
            bytes = HDR;
            for (int i = 0; i < rw && i < MAXRW; ++i) {
                const int row = lane_bcast(e.x, i);
                if (row < 0) continue;
                const int first = lane_bcast(e.y, i), k = lane_bcast(e.z, i), plen = lane_bcast(e.w, i);
                const int *sr = seg + (int64_t)row * (ntiles + 1);
                const int n = piece_before(sr[t + 1], first, k, plen) - piece_before(sr[t], first, k, plen);
                bytes += 8 * (n + (n & 1));
            }
        }
        const int incl = wave_incl_scan(bytes);
        if (t < ntiles) coff[(int64_t)g * ntiles + t] = carry + incl - bytes;
        carry += lane_bcast(incl, kWave - 1);
    }
    if (lane == 0) wsize[g] = carry;
}

// writes the chunks of (wave g, tiles t0 .. t0 + 64/G - 1): lane group tau of
// G lanes handles tile t0 + tau, lane i of the group the piece in slot i
template <int VEC, bool HALF>
__global__ __launch_bounds__(256) void stream_fill_kernel(
    int nw, int rw, int ntiles, const int *__restrict__ idx, const float *__restrict__ vals,
    const int4 *__restrict__ table, const int *__restrict__ seg, const int *__restrict__ coff,
    const int *__restrict__ woff, char *__restrict__ stream) {
    constexpr int BB = tiled_cfg<VEC, HALF>::BB, KT = tiled_cfg<VEC, HALF>::KT;
    constexpr int MAXRW = tiled_cfg<VEC, HALF>::MAXRW, HDR = tiled_cfg<VEC, HALF>::HDR;
    constexpr int G = MAXRW <= 16 ? 16 : 32;  // lanes per tile (>= MAXRW and >= HDR / 2)
    constexpr int TPW = kWave / G;            // tiles per wave
    static_assert(G >= MAXRW && G >= HDR / 2, "a lane per slot and per header word");
    const int tiles_per_g = (ntiles + TPW - 1) / TPW;
    const int64_t id = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    // no early exit: the whole workgroup meets at the barrier below
    const bool wave_ok = id < (int64_t)nw * tiles_per_g;
    const int lane = threadIdx.x & 63;
    const int g = wave_ok ? (int)(id / tiles_per_g) : 0;
    const int t0 = wave_ok ? (int)(id - (int64_t)g * tiles_per_g) * TPW : ntiles;
    const int tau = lane / G, i = lane - tau * G;
    const int t = t0 + tau;
    const bool tile_ok = t < ntiles;
    // this lane's slot in its tile: strided entries [m0, m0 + n) of the piece
    int n = 0, pbase = 0, k = 1;
    if (tile_ok && i < rw) {
        const int4 e = table[(int64_t)g * rw + i];
        if (e.x >= 0) {
            const int *sr = seg + (int64_t)e.x * (ntiles + 1);
            const int m0 = piece_before(sr[t], e.y, e.z, e.w);
            n = piece_before(sr[t + 1], e.y, e.z, e.w) - m0;
            k = e.z;
            pbase = e.y + m0 * k;
        }
    }
    const int np = n + (n & 1);  // padded to whole units
    // prefix over the slots of the group: first pair of this slot inside the chunk
    int incl = np;
#pragma unroll
    for (int d = 1; d < G; d <<= 1) {
        const int u = __shfl_up(incl, d, G);
        if (i >= d) incl += u;
    }
    const int start = incl - np;
    char *chunk = stream + (tile_ok ? woff[g] + coff[(int64_t)g * ntiles + t] : 0);
    // header: uint16 padded count per slot (zero past rw)
    if (tile_ok && i < HDR / 2) reinterpret_cast<unsigned short *>(chunk)[i] = (unsigned short)(i < MAXRW ? np : 0);
    // slot table of the wave's tiles in LDS: run starts (plus the end), first
    // position, stride and entries
    __shared__ int s_start[4][TPW][MAXRW + 1], s_base[4][TPW][MAXRW], s_k[4][TPW][MAXRW],
        s_n[4][TPW][MAXRW];
    const int wl = threadIdx.x >> 6;
    if (i < MAXRW) {
        s_start[wl][tau][i] = i < rw ? start : incl;  // empty slots start at the end
        s_base[wl][tau][i] = pbase;
        s_k[wl][tau][i] = k;
        s_n[wl][tau][i] = n;
    }
    if (i == G - 1) s_start[wl][tau][MAXRW] = incl;
    __syncthreads();
    // copy: lane q of the wave takes the q-th pair of the chunk of every tile
    // of the wave at once (coalesced stores, the loads of all tiles in
    // flight); its slot is found by binary search over the run starts
    int total[TPW];
    int2 *pp[TPW];
    int maxtot = 0;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
        const int tg = t0 + tt;
        total[tt] = tg < ntiles ? s_start[wl][tt][MAXRW] : 0;  // pairs of tile tg (padded)
        pp[tt] = reinterpret_cast<int2 *>(stream + (tg < ntiles ? woff[g] + coff[(int64_t)g * ntiles + tg] : 0) + HDR);
        maxtot = max(maxtot, total[tt]);
    }
    for (int q0 = 0; q0 < maxtot; q0 += kWave) {
        const int q = q0 + lane;
        int2 v[TPW];
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) {
            v[tt] = make_int2(0, 0);  // the padding pair of an odd run
            if (q < total[tt]) {
                // last slot j with start[j] <= q (starts are non-decreasing)
                int lo = 0, hi = MAXRW - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (s_start[wl][tt][mid] <= q) lo = mid; else hi = mid - 1;
                }
                const int u = q - s_start[wl][tt][lo];
                if (u < s_n[wl][tt][lo]) {
                    const int p = s_base[wl][tt][lo] + u * s_k[wl][tt][lo];
                    v[tt] = make_int2((idx[p] - (t0 + tt) * KT) * (BB * 4), __float_as_int(vals[p]));
                }
            }
        }
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt)
            if (q < total[tt]) pp[tt][q] = v[tt];
    }
}

// The pair stream of wave g in one workgroup (used while the per-(slot, tile)
// tables fit in 64 KB of LDS; the launches above otherwise).  A piece's
// entries are sorted by column, so its entries in tile t form one contiguous
// run: with n[i][t] the count of slot i's entries in tile t and start[i][t]
// their prefix over the tiles, entry m of slot i in tile t is pair
// m - start[i][t] of its run.  Counts go into LDS (integer atomics, order-
// independent), then the run starts, the runs' offsets inside each chunk and
// the chunks' offsets inside the stream are prefix sums, and every entry, the
// chunk headers and the padding pairs of odd runs are written to their places:
// the same bytes as the launches above, without the per-(row, tile) bounds.
// The stream starts at woff[g], the exclusive scan of the per-wave bounds of
// plan_deal_kernel: with wsize given, each workgroup adds up the bounds before
// its stream itself and writes woff[g] (and woff[nw] at the last); without, a
// scan launch has written woff.  The main kernel finds each chunk from the
// one before.  At most 64 VGPRs (8 waves per SIMD), so that two workgroups
// share a CU.
constexpr int kBucketThreads = 1024;

template <int VEC, bool HALF>
__global__ __launch_bounds__(kBucketThreads, 8) void stream_bucket_kernel(int rw, int ntiles, const int *__restrict__ idx,
                                                            const float *__restrict__ vals,
                                                            const int4 *__restrict__ table,
                                                            const int *__restrict__ wsize, int *__restrict__ woff,
                                                            char *__restrict__ stream) {
    constexpr int BB = tiled_cfg<VEC, HALF>::BB, KT = tiled_cfg<VEC, HALF>::KT, SHIFT = tiled_cfg<VEC, HALF>::SHIFT;
    constexpr int MAXRW = tiled_cfg<VEC, HALF>::MAXRW, HDR = tiled_cfg<VEC, HALF>::HDR;
    extern __shared__ int bsm[];
    int *cnt = bsm;                     // [rw][ntiles]: counts, then run starts (prefix over the tiles)
    int *roff = cnt + rw * ntiles;      // [rw][ntiles]: pair offset of the run inside its chunk
    int *choff = roff + rw * ntiles;    // [ntiles + 1]: byte offset of each chunk inside the stream
    __shared__ int4 slot[MAXRW];
    __shared__ int pfx[MAXRW + 1];      // entries before each slot
    __shared__ int wave_tot[kBucketThreads / kWave];
    const int g = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nrw = rw < MAXRW ? rw : MAXRW;
    if (tid < nrw) {
        int4 e = table[(int64_t)g * rw + tid];
        if (e.x < 0) e.w = 0;
        slot[tid] = e;
    }
    for (int x = tid; x < nrw * ntiles; x += kBucketThreads) cnt[x] = 0;
    if (wsize) {  // this stream's offset = the bounds of the streams before it, added up here
        int sz = 0;
        for (int x = tid; x < g; x += kBucketThreads) sz += wsize[x];
        sz = wave_sum_int(sz);
        if (lane == 0) wave_tot[wave] = sz;
    }
    __syncthreads();
    int wo;
    if (wsize) {
        wo = 0;
#pragma unroll
        for (int w = 0; w < kBucketThreads / kWave; ++w) wo += wave_tot[w];
        if (tid == 0) {
            woff[g] = wo;  // for the product kernel
            if (g == (int)gridDim.x - 1) woff[g + 1] = wo + wsize[g];
        }
    } else {
        wo = woff[g];
    }
    if (tid == 0) {
        int run = 0;
        for (int i = 0; i < nrw; ++i) {
            pfx[i] = run;
            run += slot[i].w;
        }
        pfx[nrw] = run;
    }
    __syncthreads();
    const int total = pfx[nrw];
    auto find = [&](int e) {  // the slot of entry e: last i with pfx[i] <= e
        int i = 0;
        for (int d = 16; d > 0; d >>= 1)
            if (i + d < nrw && pfx[i + d] <= e) i += d;
        return i;
    };
    // Entries U at a time per thread, their loads in flight together; the
    // first round's entries (slot, column, position in the piece, value) stay
    // in registers for the write pass.  The 64 lanes of a wave hold 64
    // consecutive entries, so equal (slot, tile) keys come in runs (a piece's
    // columns are sorted): the first lane of each run adds the run's length,
    // one LDS atomic per run.  Every thread makes the same number of rounds,
    // so the whole wave takes part in the lane exchanges (lanes past the end
    // hold the key -1).
    constexpr int U = 8;
    auto count_runs = [&](const int (&kk)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int prev = __shfl_up(kk[u], 1, kWave);
            const bool head = lane == 0 || kk[u] != prev;
            const uint64_t heads = __ballot(head);
            const uint64_t above = heads & ~((2ull << lane) - 1ull);  // heads past this lane (none for lane 63)
            const int next = above ? __builtin_ctzll(above) : kWave;
            if (head && kk[u] >= 0) atomicAdd(&cnt[kk[u]], next - lane);
        }
    };
    int ki[U], kc[U], km[U];
    float kv[U];
    {
        int kk[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = tid + u * kBucketThreads;
            ki[u] = kk[u] = -1;
            kc[u] = km[u] = 0;
            kv[u] = 0.f;
            if (e < total) {
                const int i = find(e);
                const int4 sl = slot[i];
                const int p = sl.y + (e - pfx[i]) * sl.z;
                ki[u] = i;
                km[u] = e - pfx[i];
                kc[u] = idx[p];
                kv[u] = vals[p];
                kk[u] = i * ntiles + (kc[u] >> SHIFT);
            }
        }
        count_runs(kk);
    }
    for (int e0 = U * kBucketThreads; e0 < total; e0 += U * kBucketThreads) {
        int kk[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = e0 + tid + u * kBucketThreads;
            kk[u] = -1;
            if (e < total) {
                const int i = find(e);
                const int4 sl = slot[i];
                kk[u] = i * ntiles + (idx[sl.y + (e - pfx[i]) * sl.z] >> SHIFT);
            }
        }
        count_runs(kk);
    }
    __syncthreads();
    // run starts per slot (one wave per slot) and, per tile, the runs' offsets
    // inside the chunk (padded to whole pairs of pairs)
    for (int i = wave; i < nrw; i += kBucketThreads / kWave) {
        int carry = 0;
        for (int t0 = 0; t0 < ntiles; t0 += kWave) {
            const int t = t0 + lane;
            const int n = t < ntiles ? cnt[i * ntiles + t] : 0;
            const int incl = wave_incl_scan(n);
            if (t < ntiles) cnt[i * ntiles + t] = carry + incl - n;
            carry += lane_bcast(incl, kWave - 1);
        }
    }
    __syncthreads();
    int mine = 0;  // this thread's tiles' chunk bytes (tiles tid * per .. + per)
    const int per = (ntiles + kBucketThreads - 1) / kBucketThreads;
    const int ta = min(ntiles, tid * per), tb = min(ntiles, ta + per);
    for (int t = ta; t < tb; ++t) {
        int r = 0;
        for (int i = 0; i < nrw; ++i) {
            const int st = cnt[i * ntiles + t];
            const int n = (t + 1 < ntiles ? cnt[i * ntiles + t + 1] : slot[i].w) - st;
            roff[i * ntiles + t] = r;
            r += n + (n & 1);
        }
        mine += HDR + 8 * r;
    }
    {
        const int incl = wave_incl_scan(mine);
        if (lane == 63) wave_tot[wave] = incl;
        __syncthreads();
        int before = 0;
        for (int w = 0; w < wave; ++w) before += wave_tot[w];
        int c = before + incl - mine;
        for (int t = ta; t < tb; ++t) {
            choff[t] = c;
            int r = 0;
            for (int i = 0; i < nrw; ++i) {
                const int st = cnt[i * ntiles + t];
                const int n = (t + 1 < ntiles ? cnt[i * ntiles + t + 1] : slot[i].w) - st;
                r += n + (n & 1);
            }
            c += HDR + 8 * r;
        }
    }
    __syncthreads();
    char *base = stream + wo;
    // headers: uint16 padded count per slot (zero past rw); padding pairs of odd runs
    for (int x = tid; x < ntiles * (HDR / 2); x += kBucketThreads) {
        const int t = x / (HDR / 2), i = x - t * (HDR / 2);
        int np = 0;
        if (i < nrw) {
            const int st = cnt[i * ntiles + t];
            const int n = (t + 1 < ntiles ? cnt[i * ntiles + t + 1] : slot[i].w) - st;
            np = n + (n & 1);
            if (n & 1)
                *reinterpret_cast<int2 *>(base + choff[t] + HDR + 8 * (roff[i * ntiles + t] + n)) = make_int2(0, 0);
        }
        reinterpret_cast<unsigned short *>(base + choff[t])[i] = (unsigned short)np;
    }
    auto put = [&](int i, int c, int m, float v) {  // entry m of slot i, column c, into its place
        const int t = c >> SHIFT;
        const int q = roff[i * ntiles + t] + m - cnt[i * ntiles + t];
        *reinterpret_cast<int2 *>(base + choff[t] + HDR + 8 * q) = make_int2((c - t * KT) * (BB * 4), __float_as_int(v));
    };
#pragma unroll
    for (int u = 0; u < U; ++u)
        if (ki[u] >= 0) put(ki[u], kc[u], km[u], kv[u]);
    for (int e0 = U * kBucketThreads + tid; e0 < total; e0 += U * kBucketThreads) {
        int ii[U], mm[U], cc[U];
        float vv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = e0 + u * kBucketThreads;
            ii[u] = -1;
            if (e < total) {
                ii[u] = find(e);
                const int4 sl = slot[ii[u]];
                mm[u] = e - pfx[ii[u]];
                const int p = sl.y + mm[u] * sl.z;
                cc[u] = idx[p];
                vv[u] = vals[p];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ii[u] >= 0) put(ii[u], cc[u], mm[u], vv[u]);
    }
}

size_t bucket_lds_bytes(int rw, int ntiles) { return sizeof(int) * ((size_t)2 * rw * ntiles + ntiles + 1); }

// ---------------------------------------------------------------------------
// streamed tiled kernel
// ---------------------------------------------------------------------------

typedef __attribute__((address_space(3))) void lds_void;

// Blocks are handed to the 8 XCDs round-robin; give XCD x a contiguous range
// of the (chunk-major) work list so its resident workgroups share a chunk.
__device__ __forceinline__ void map_block(int bid, int nblocks, int nrb, int &rb, int &ch) {
    const int per = nblocks / 8;
    const int w = bid < per * 8 ? (bid % 8) * per + bid / 8 : bid;
    ch = w / nrb;
    rb = w - ch * nrb;
}

// A unit is two (byte offset, value) pairs.  Full wave: every lane takes both
// pairs; half waves: the lower half-wave takes pair 0, the upper pair 1.
template <bool HALF>
struct unit_t {
    using type = int4;
};
template <>
struct unit_t<true> {
    using type = int2;
};

template <bool HALF>
__device__ __forceinline__ typename unit_t<HALF>::type load_unit(const char *base, int p, int half) {
    using U = typename unit_t<HALF>::type;
    return *reinterpret_cast<const U *>(base + p + (HALF ? 8 * half : 0));
}

// acc += v * X[o] for the pair(s) of a unit this lane takes
template <int VEC, bool HALF>
__device__ __forceinline__ void fma_unit(const char *xb, typename unit_t<HALF>::type pr,
                                         float (&acc)[VEC]) {
    if constexpr (HALF) {
        float x0[VEC];
        load_vec<VEC>(reinterpret_cast<const float *>(xb + pr.x), x0);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = fmaf(__int_as_float(pr.y), x0[e], acc[e]);
    } else {
        float x0[VEC], x1[VEC];
        load_vec<VEC>(reinterpret_cast<const float *>(xb + pr.x), x0);
        load_vec<VEC>(reinterpret_cast<const float *>(xb + pr.z), x1);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            acc[e] = fmaf(__int_as_float(pr.y), x0[e], acc[e]);
            acc[e] = fmaf(__int_as_float(pr.w), x1[e], acc[e]);
        }
    }
}

template <int VEC, bool HALF>
__global__ __launch_bounds__(1024, 1) void spmm_stream_kernel(
    int rw, int n_cols, int ntiles, const int4 *__restrict__ table, const int *__restrict__ pbeg,
    const int *__restrict__ ptr, const char *__restrict__ stream,
    const int *__restrict__ woff, const float *__restrict__ X, int64_t ldx, int B,
    float *__restrict__ Y, int64_t ldy, float *__restrict__ part, int nrb) {
    constexpr int BB = tiled_cfg<VEC, HALF>::BB, KT = tiled_cfg<VEC, HALF>::KT;
    constexpr int MAXRW = tiled_cfg<VEC, HALF>::MAXRW, HDR = tiled_cfg<VEC, HALF>::HDR;
    constexpr int Q = BB / 4;  // 16-byte pieces of a tile row
    // two tile buffers and two stream buffers as separate arrays: the compiler
    // can then see that reads of one never alias the loads into the other
    __shared__ __attribute__((aligned(16))) float Xs0[kTileFloats];
    __shared__ __attribute__((aligned(16))) float Xs1[kTileFloats];
    __shared__ __attribute__((aligned(16))) char St0[kNW * kChunk];
    __shared__ __attribute__((aligned(16))) char St1[kNW * kChunk];

    int rb, ch;
    map_block(blockIdx.x, gridDim.x, nrb, rb, ch);
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int nw = nrb * kNW;
    const int g = rb * kNW + wave;
    const int b0 = ch * BB;
    int64_t off = woff[g];

    // async loads of tile t: X rows [t*KT, t*KT + KT) x columns [b0, b0 + BB)
    // (clamped into the matrix: rows or columns outside it are never read
    // back) and this wave's stream chunk.  Each thread's four source
    // addresses move by KT rows per tile; rows are clamped on the last tile only.
    constexpr int NU = kTileFloats / (4 * kNW * kWave);  // 16-byte loads per thread per tile
    const float *xsrc[NU];
    int xrow[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int q = u * (kNW * kWave) + threadIdx.x;
        const int r = q / Q, c4 = q - r * Q;
        int b = b0 + c4 * 4;
        b = b + 3 < B ? b : B - 4;
        xrow[u] = r;
        xsrc[u] = X + (int64_t)r * ldx + b;
    }
    const int64_t tile_stride = (int64_t)KT * ldx;
    auto issue = [&](int t, float *xd, char *sd, int64_t soff) {
        const int64_t step = (int64_t)t * tile_stride;
        if ((t + 1) * KT <= n_cols) {
#pragma unroll
            for (int u = 0; u < NU; ++u)
                __builtin_amdgcn_global_load_lds((const void *)(xsrc[u] + step),
                                                 (lds_void *)(xd + (u * (kNW * kWave) + wave * kWave) * 4),
                                                 16, 0, 0);
        } else {
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int k = t * KT + xrow[u];
                const int64_t back = k < n_cols ? 0 : (int64_t)(k - (n_cols - 1)) * ldx;
                __builtin_amdgcn_global_load_lds((const void *)(xsrc[u] + step - back),
                                                 (lds_void *)(xd + (u * (kNW * kWave) + wave * kWave) * 4),
                                                 16, 0, 0);
            }
        }
        __builtin_amdgcn_global_load_lds((const void *)(stream + soff + lane * 16),
                                         (lds_void *)(sd + wave * kChunk), 16, 0, 0);
    };

    float acc[MAXRW][VEC];
#pragma unroll
    for (int i = 0; i < MAXRW; ++i)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[i][e] = 0.f;

    constexpr int LANES = tiled_cfg<VEC, HALF>::LANES;
    const int half = HALF ? lane >> 5 : 0;
    const int lb = (lane & (LANES - 1)) * VEC * 4;  // byte offset of this lane's columns in a tile row
    auto tile = [&](int t, const float *xc, const char *scur, float *xn, char *snext) {
        __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this wave's loads of tile t landed
        __syncthreads();                     // ... and every wave's; tile t-1 fully consumed
        const char *sc = scur + wave * kChunk;
        int nlen[MAXRW];
        int tot = 0;
#pragma unroll
        for (int w = 0; w < MAXRW / 2; ++w) {
            const unsigned hw = (unsigned)uniform((int)reinterpret_cast<const unsigned *>(sc)[w]);
            nlen[2 * w] = (int)(hw & 0xffffu);
            nlen[2 * w + 1] = (int)(hw >> 16);
            tot += nlen[2 * w] + nlen[2 * w + 1];
        }
        const int64_t next = off + HDR + 8 * (int64_t)tot;
        if (t + 1 < ntiles) issue(t + 1, xn, snext, next);
        const char *xb = reinterpret_cast<const char *>(xc) + lb;
        int p = HDR;  // byte position of the next unit in the chunk
        if constexpr (HALF) {
            // half waves read the units one step ahead: qa, qb hold the units at
            // p and p + 16 (each read clamped inside the chunk; a clamped read is
            // never used, because a unit past the chunk is read from global
            // memory instead)
            using U = typename unit_t<HALF>::type;
            // (the position is made opaque before the clamp: otherwise the
            // compiler rewrites min(p + c, m) as min(p, m - c) + c, loses track of
            // which buffer the read touches and waits for the DMA into the other
            // stream buffer before it)
            auto ahead = [&](int pos) {
                asm volatile("" : "+s"(pos));
                return load_unit<HALF>(sc, pos < kChunk - 16 ? pos : kChunk - 16, half);
            };
            U qa = ahead(p), qb = ahead(p + 16);
#pragma unroll
            for (int i = 0; i < MAXRW; ++i) {
                if (i < rw) {  // (a guard, not a break: keeps every acc[i] statically indexed)
                    const int pe = p + 8 * nlen[i];
                    const int pl = pe < kChunk ? pe : kChunk;  // part of the run staged in LDS
                    for (; p + 64 <= pl; p += 64) {  // four units per step
                        const U c0 = qa, c1 = qb;
                        const U c2 = ahead(p + 32), c3 = ahead(p + 48);
                        qa = ahead(p + 64);
                        qb = ahead(p + 80);
                        fma_unit<VEC, HALF>(xb, c0, acc[i]);
                        fma_unit<VEC, HALF>(xb, c1, acc[i]);
                        fma_unit<VEC, HALF>(xb, c2, acc[i]);
                        fma_unit<VEC, HALF>(xb, c3, acc[i]);
                    }
                    if (p + 32 <= pl) {
                        const U c0 = qa, c1 = qb;
                        qa = ahead(p + 32);
                        qb = ahead(p + 48);
                        fma_unit<VEC, HALF>(xb, c0, acc[i]);
                        fma_unit<VEC, HALF>(xb, c1, acc[i]);
                        p += 32;
                    }
                    if (p < pl) {
                        const U c0 = qa;
                        qa = qb;
                        qb = ahead(p + 32);
                        fma_unit<VEC, HALF>(xb, c0, acc[i]);
                        p += 16;
                    }
                    if (p < pe) {  // beyond the staged chunk: the stream in global memory
                        const char *gs = stream + off;
                        for (; p < pe; p += 16) fma_unit<VEC, HALF>(xb, load_unit<HALF>(gs, p, half), acc[i]);
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < MAXRW; ++i) {
                if (i < rw) {  // (a guard, not a break: keeps every acc[i] statically indexed)
                    const int pe = p + 8 * nlen[i];
                    const int pl = pe < kChunk ? pe : kChunk;  // part of the run staged in LDS
                    for (; p + 32 <= pl; p += 32) {
                        fma_unit<VEC, HALF>(xb, load_unit<HALF>(sc, p, half), acc[i]);
                        fma_unit<VEC, HALF>(xb, load_unit<HALF>(sc, p + 16, half), acc[i]);
                    }
                    if (p < pl) {
                        fma_unit<VEC, HALF>(xb, load_unit<HALF>(sc, p, half), acc[i]);
                        p += 16;
                    }
                    if (p < pe) {  // beyond the staged chunk: the stream in global memory
                        const char *gs = stream + off;
                        for (; p < pe; p += 16) fma_unit<VEC, HALF>(xb, load_unit<HALF>(gs, p, half), acc[i]);
                    }
                }
            }
        }
        off = next;
    };

    issue(0, Xs0, St0, off);
    for (int t = 0; t < ntiles; t += 2) {
        tile(t, Xs0, St0, Xs1, St1);
        if (t + 1 < ntiles) tile(t + 1, Xs1, St1, Xs0, St0);
    }

    // half waves: the two halves hold partial sums of the same columns
    if constexpr (HALF) {
#pragma unroll
        for (int i = 0; i < MAXRW; ++i)
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[i][e] += __shfl_xor(acc[i][e], kWave / 2, kWave);
    }
    // a whole row goes to Y; a piece of a split row to its partial row
    const int b = b0 + (lane & (LANES - 1)) * VEC;
#pragma unroll
    for (int i = 0; i < MAXRW; ++i) {
        if (i >= rw || half) continue;
        const int4 e = table[(int64_t)g * rw + i];
        const int row = uniform(e.x);
        if (row < 0) continue;
        const bool split = uniform(e.z) > 1;
        // pieces of a row are numbered from pbeg[row]; this one is j = first - ptr[row]
        const int pv = split ? uniform(pbeg[row] + e.y - ptr[row]) : 0;
        float *dst = split ? part + (int64_t)pv * B + b : Y + (int64_t)row * ldy + b;
        if (b + VEC - 1 < B) {
            store_vec<VEC>(dst, acc[i]);
        } else {
#pragma unroll
            for (int q = 0; q < VEC; ++q)
                if (b + q < B) dst[q] = acc[i][q];
        }
    }
}

// Y[row] = sum of the partial rows of its pieces, in piece order (split rows
// only).  Block (row, batch chunk of kFixupCols); the loads of all pieces are
// issued before the sum.
constexpr int kFixupCols = 1024;

__global__ __launch_bounds__(256) void fixup_kernel(int n_rows, const int *__restrict__ pbeg,
                                                    const float *__restrict__ part, int B,
                                                    float *__restrict__ Y, int64_t ldy) {
    const int row = blockIdx.x;
    const int v0 = pbeg[row], v1 = pbeg[row + 1];
    if (v1 - v0 < 2) return;
    const int b1 = min(B, (int)(blockIdx.y + 1) * kFixupCols);
    for (int b = blockIdx.y * kFixupCols + threadIdx.x; b < b1; b += blockDim.x) {
        constexpr int U = 8;
        float a = 0.f;
        int v = v0;
        for (; v + U <= v1; v += U) {
            float t[U];
#pragma unroll
            for (int u = 0; u < U; ++u) t[u] = part[(int64_t)(v + u) * B + b];
#pragma unroll
            for (int u = 0; u < U; ++u) a += t[u];
        }
        for (; v < v1; ++v) a += part[(int64_t)v * B + b];
        Y[(int64_t)row * ldy + b] = a;
    }
}

// ---------------------------------------------------------------------------
// rows kernel: one wave per (row, batch chunk), X from the cache hierarchy
// ---------------------------------------------------------------------------

constexpr int kRowsPerBlock = 4;

template <int VEC>
__global__ __launch_bounds__(256) void spmm_rows_kernel(int n_rows, const int *__restrict__ ptr,
                                                        const int *__restrict__ idx,
                                                        const float *__restrict__ vals,
                                                        const float *__restrict__ X, int64_t ldx,
                                                        int B, float *__restrict__ Y, int64_t ldy,
                                                        int nrb) {
    // blocks of one XCD take a contiguous run of batch chunks, so the rows that
    // share an X row segment read it through the same L2
    int rb, ch;
    map_block(blockIdx.x, gridDim.x, nrb, rb, ch);
    const int row = uniform(rb * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int b = (ch * kWave + lane) * VEC;
    const bool active = b < B;
    const int start = uniform(ptr[row]);
    const int end = uniform(ptr[row + 1]);
    constexpr int U = 8;  // X row segments in flight per wave

    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;

    for (int base = start; base < end; base += kWave) {
        const int n = min(kWave, end - base);
        int c = 0;
        float v = 0.f;
        if (lane < n) {
            c = idx[base + lane];
            v = vals[base + lane];
        }
        int j = 0;
        for (; j + U <= n; j += U) {
            float x[U][VEC];
            if (active) {
#pragma unroll
                for (int u = 0; u < U; ++u) load_vec<VEC>(X + (int64_t)lane_bcast(c, j + u) * ldx + b, x[u]);
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const float vu = lane_bcast(v, j + u);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) acc[e] = fmaf(vu, x[u][e], acc[e]);
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

// which path a product takes, and the shape of the tiled launch
struct spmm_plan {
    bool tiled;
    bool half;   // half-wave units (twice the tile height)
    int vec;     // batch columns per lane
    int ntiles;  // X tiles
    int nch;     // batch chunks of 64 x vec columns
    int nrb;     // row groups (workgroups per chunk)
    int rw;      // pieces per wave
    int64_t max_pieces;
    int64_t stream_bytes;  // bound on the pair stream
};

// the launch shape for (vec, half): returns false if the tiled kernel does not suit
template <int VEC, bool HALF>
bool shape_plan(spmm_plan &p, int n_rows, int n_cols, int64_t nnz, int B) {
    using cfg = tiled_cfg<VEC, HALF>;
    p.vec = VEC;
    p.half = HALF;
    p.nch = (int)ceil_div(B, cfg::BB);
    // one workgroup per CU over the whole grid, each with at least one row per wave
    int64_t nrb = 256 / p.nch;
    if (nrb < 1) nrb = 1;
    const int64_t nrb_max = ceil_div(n_rows, kNW);
    if (nrb > nrb_max) nrb = nrb_max;
    // staging an X tile pays off when a workgroup's rows use each X element ~2x
    const double density = (double)nnz / ((double)n_rows * n_cols);
    if (density * (double)n_rows / (double)nrb < 2.0) return false;
    int64_t nw = nrb * kNW;
    // the planner cuts rows into pieces of at most max(64, nnz / (2 nw))
    // entries (nnz counted on the device), so there are at most n_rows + 2 nw
    // pieces; more waves if a wave would get more pieces than it has slots
    int64_t rw = ceil_div(n_rows + 2 * nw, nw);
    if (rw > cfg::MAXRW) {
        rw = cfg::MAXRW;
        nrb = ceil_div(n_rows, (int64_t)kNW * (cfg::MAXRW - 2));
        nw = nrb * kNW;
    }
    p.max_pieces = n_rows + 2 * nw;
    p.rw = (int)rw;
    p.nrb = (int)nrb;
    p.ntiles = (int)ceil_div(n_cols, cfg::KT);
    // stream: every pair, one padding pair per (piece, tile) and a header per
    // (wave, tile); too much padding means the operand is too sparse per tile
    const int64_t slot_tiles = nw * rw * (int64_t)p.ntiles;
    if (slot_tiles > 2 * nnz + 4096) return false;
    // (the bound the per-wave streams are placed by: 16 bytes per slot and
    // tile, entries rounded to pairs of pairs per piece)
    p.stream_bytes = 8 * (nnz + p.max_pieces) + 16 * slot_tiles + (int64_t)cfg::HDR * nw * p.ntiles + kChunk + 256;
    if (p.stream_bytes > INT32_MAX / 2 || (int64_t)nrb * p.nch > INT32_MAX) return false;
    return true;
}

spmm_plan make_plan(int n_rows, int n_cols, int64_t nnz, int B, bool x4) {
    spmm_plan p{};
    if (!x4 || B < 128 || n_rows < kNW || n_cols <= 0) return p;
    // The tiled path costs about 20 us of planning and then runs ~1e7
    // (entry, batch column) products per us; the rows kernel starts at once and
    // streams ~5e6 per us out of L2.  Below ~1.7e8 products the rows kernel
    // finishes first.
    if ((double)nnz * (double)B < 1.7e8) return p;
    if (B >= 256) {
        // half-wave units halve the number of tiles; they pay off while a
        // wave's chunk of a tile (about nnz / (waves * tiles) pairs) still
        // fits its 1 KB LDS slot
        spmm_plan h{};
        if (shape_plan<4, true>(h, n_rows, n_cols, nnz, B)) {
            const double per_chunk = (double)nnz / ((double)h.nrb * kNW * h.ntiles);
            if (per_chunk <= 0.75 * (kChunk - tiled_cfg<4, true>::HDR) / 8.0) {
                h.tiled = true;
                return h;
            }
        }
        p.tiled = shape_plan<4, false>(p, n_rows, n_cols, nnz, B);
    } else {
        p.tiled = shape_plan<2, false>(p, n_rows, n_cols, nnz, B);
    }
    return p;
}

struct spmm_ws {
    int *bh;      // [plan blocks][kBuckets]: the planner's bucket histograms
    int *bsum;    // [plan blocks]: pieces per plan block
    int *pbeg;    // [n_rows + 1]
    int *seg;     // [n_rows][ntiles + 1]
    int4 *table;  // [nw][rw]: slot table
    int *coff;    // [nw][ntiles]: chunk sizes, then offsets inside the wave's stream
    int *wsize;   // [nw]
    int *woff;    // [nw + 1]
    char *stream; // [stream_bytes]
    float *part;  // [max_pieces][B]
    size_t bytes;
};

// workspace layout (256-byte aligned parts); base may be 0 to size it
spmm_ws carve(const spmm_plan &pl, int n_rows, int B, uintptr_t base) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t nw = (size_t)pl.nrb * kNW;
    spmm_ws w{};
    size_t off = 0;
    w.bh = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * (size_t)kPlanMaxBlocks * kBuckets);
    w.bsum = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * (size_t)kPlanMaxBlocks);
    w.pbeg = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * ((size_t)n_rows + 1));
    w.seg = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * (size_t)n_rows * (pl.ntiles + 1));
    w.table = reinterpret_cast<int4 *>(base + off);
    off = al(off + sizeof(int4) * nw * (size_t)pl.rw);
    w.coff = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * nw * pl.ntiles);
    w.wsize = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * nw);
    w.woff = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * (nw + 1));
    w.stream = reinterpret_cast<char *>(base + off);
    off = al(off + (size_t)pl.stream_bytes);
    w.part = reinterpret_cast<float *>(base + off);
    off = al(off + sizeof(float) * (size_t)pl.max_pieces * B);
    w.bytes = off;
    return w;
}

// the planning launches of a tiled product: pieces and the deal, per-(row,
// tile) bounds, chunk sizes and offsets, the pair stream (with W's values)
template <int VEC, bool HALF>
hipError_t plan_tiled(const spmm_plan &pl, int n_rows, const int *ptr, const int *idx, const float *vals, int B,
                      void *ws, hipStream_t s) {
    const spmm_ws w = carve(pl, n_rows, B, reinterpret_cast<uintptr_t>(ws));
    const int nw = pl.nrb * kNW;
    hipError_t e;
    {
        const int nb = (int)std::min<int64_t>(kPlanMaxBlocks, ceil_div(n_rows, kPlanThreads));
        const int rpb = (int)ceil_div(n_rows, nb);
        const int wbase = pl.ntiles * (tiled_cfg<VEC, HALF>::HDR + 16 * pl.rw);
        plan_hist_kernel<<<nb, kPlanThreads, 0, s>>>(n_rows, ptr, nw, rpb, w.bh, w.bsum, w.wsize, wbase);
        plan_deal_kernel<<<nb, kPlanThreads, 0, s>>>(n_rows, ptr, nw, pl.rw, rpb, nb, w.bh, w.bsum, w.pbeg,
                                                      w.table, w.wsize);
    }
    const size_t blds = bucket_lds_bytes(pl.rw, pl.ntiles);
    if (pl.rw <= tiled_cfg<VEC, HALF>::MAXRW && blds <= 65536) {
        // each stream written by one workgroup at the exclusive scan of the
        // streams' bounds; up to 4 bounds per thread the workgroups add up
        // their own offsets, else a scan launch writes them first
        if ((e = hipGetLastError()) != hipSuccess) return e;
        const bool own = nw <= 4 * kBucketThreads;
        if (!own && (e = launch_exclusive_scan(w.wsize, w.woff, nw, nullptr, s)) != hipSuccess) return e;
        stream_bucket_kernel<VEC, HALF><<<(unsigned)nw, kBucketThreads, blds, s>>>(
            pl.rw, pl.ntiles, idx, vals, w.table, own ? w.wsize : nullptr, w.woff, w.stream);
        return hipGetLastError();
    }
    seg_kernel<<<(unsigned)ceil_div(n_rows, 4), 256, 0, s>>>(n_rows, pl.ntiles, tiled_cfg<VEC, HALF>::SHIFT,
                                                             ptr, idx, w.seg);
    stream_size_kernel<VEC, HALF><<<(unsigned)ceil_div(nw, 4), 256, 0, s>>>(nw, pl.rw, pl.ntiles, w.table, w.seg,
                                                                       w.coff, w.wsize);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_exclusive_scan(w.wsize, w.woff, nw, nullptr, s)) != hipSuccess) return e;
    constexpr int TPW = kWave / (tiled_cfg<VEC, HALF>::MAXRW <= 16 ? 16 : 32);
    const int64_t fill_waves = (int64_t)nw * ceil_div(pl.ntiles, TPW);
    stream_fill_kernel<VEC, HALF><<<(unsigned)ceil_div(fill_waves, 4), 256, 0, s>>>(
        nw, pl.rw, pl.ntiles, idx, vals, w.table, w.seg, w.coff, w.woff, w.stream);
    return hipGetLastError();
}

// the product from a plan: the streamed kernel, then the fix-up of split rows
template <int VEC, bool HALF>
hipError_t exec_tiled(const spmm_plan &pl, int n_rows, int n_cols, const int *ptr, const float *X, int64_t ldx, int B,
                      float *Y, int64_t ldy, const void *ws, hipStream_t s) {
    const spmm_ws w = carve(pl, n_rows, B, reinterpret_cast<uintptr_t>(ws));
    hipError_t e;
    const unsigned nblocks = (unsigned)((int64_t)pl.nrb * pl.nch);
    spmm_stream_kernel<VEC, HALF><<<nblocks, kNW * kWave, 0, s>>>(pl.rw, n_cols, pl.ntiles, w.table, w.pbeg,
                                                            ptr, w.stream, w.woff, X, ldx, B, Y,
                                                            ldy, w.part, pl.nrb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    fixup_kernel<<<dim3((unsigned)n_rows, (unsigned)ceil_div(B, kFixupCols)), 256, 0, s>>>(
        n_rows, w.pbeg, w.part, B, Y, ldy);
    return hipGetLastError();
}

hipError_t plan_any(const spmm_plan &pl, int n_rows, const int *ptr, const int *idx, const float *vals, int B,
                    void *ws, hipStream_t s) {
    if (pl.vec == 4 && pl.half) return plan_tiled<4, true>(pl, n_rows, ptr, idx, vals, B, ws, s);
    if (pl.vec == 4) return plan_tiled<4, false>(pl, n_rows, ptr, idx, vals, B, ws, s);
    return plan_tiled<2, false>(pl, n_rows, ptr, idx, vals, B, ws, s);
}

hipError_t exec_any(const spmm_plan &pl, int n_rows, int n_cols, const int *ptr, const float *X, int64_t ldx, int B,
                    float *Y, int64_t ldy, const void *ws, hipStream_t s) {
    if (pl.vec == 4 && pl.half) return exec_tiled<4, true>(pl, n_rows, n_cols, ptr, X, ldx, B, Y, ldy, ws, s);
    if (pl.vec == 4) return exec_tiled<4, false>(pl, n_rows, n_cols, ptr, X, ldx, B, Y, ldy, ws, s);
    return exec_tiled<2, false>(pl, n_rows, n_cols, ptr, X, ldx, B, Y, ldy, ws, s);
}

// the row-per-wave kernel (no workspace)
hipError_t launch_rows(int n_rows, const int *ptr, const int *idx, const float *vals, const float *X, int64_t ldx,
                       int B, float *Y, int64_t ldy, int vec, hipStream_t s) {
    const int64_t nrb = ceil_div(n_rows, kRowsPerBlock), nch = ceil_div(B, kWave * vec);
    if (nrb * nch > INT32_MAX) return hipErrorInvalidConfiguration;
    const unsigned grid = (unsigned)(nrb * nch);
    if (vec == 4)
        spmm_rows_kernel<4><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy, (int)nrb);
    else if (vec == 2)
        spmm_rows_kernel<2><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy, (int)nrb);
    else
        spmm_rows_kernel<1><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy, (int)nrb);
    return hipGetLastError();
}

bool spmm_v4(const float *X, int64_t ldx, int B, const float *Y, int64_t ldy) {
    return (B % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) && aligned16(Y);
}

int spmm_vec(const float *X, int64_t ldx, int B, const float *Y, int64_t ldy) {
    if (spmm_v4(X, ldx, B, Y, ldy)) return 4;
    const bool v2 = (B % 2 == 0) && (ldx % 2 == 0) && (ldy % 2 == 0) &&
                    ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(Y)) & 7u) == 0;
    return v2 ? 2 : 1;
}

}  // namespace

hipError_t launch_seg(int n_rows, int ntiles, int shift, const int *ptr, const int *idx, int *seg,
                      hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    seg_kernel<<<(unsigned)ceil_div(n_rows, 4), 256, 0, s>>>(n_rows, ntiles, shift, ptr, idx, seg);
    return hipGetLastError();
}

size_t spmm_workspace_bytes(int n_rows, int n_cols, int64_t nnz, int B) {
    const spmm_plan pl = make_plan(n_rows, n_cols, nnz, B, true);
    if (!pl.tiled) return 0;
    return carve(pl, n_rows, B, 0).bytes;
}

hipError_t launch_spmm(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                       const float *vals, const float *X, int64_t ldx, int B, float *Y,
                       int64_t ldy, void *ws, hipStream_t s) {
    if (n_rows == 0 || B == 0) return hipSuccess;
    const int vec = spmm_vec(X, ldx, B, Y, ldy);
    const spmm_plan pl = make_plan(n_rows, n_cols, nnz, B, ws != nullptr && vec == 4);
    if (pl.tiled) {
        hipError_t e = plan_any(pl, n_rows, ptr, idx, vals, B, ws, s);
        if (e != hipSuccess) return e;
        return exec_any(pl, n_rows, n_cols, ptr, X, ldx, B, Y, ldy, ws, s);
    }
    return launch_rows(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy, vec, s);
}

hipError_t launch_spmm_plan(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx, const float *vals,
                            int B, void *plan, hipStream_t s) {
    if (n_rows == 0 || B == 0) return hipSuccess;
    const spmm_plan pl = make_plan(n_rows, n_cols, nnz, B, plan != nullptr);
    return pl.tiled ? plan_any(pl, n_rows, ptr, idx, vals, B, plan, s) : hipSuccess;
}

hipError_t launch_spmm_planned(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                               const float *vals, const float *X, int64_t ldx, int B, float *Y, int64_t ldy,
                               const void *plan, hipStream_t s) {
    if (n_rows == 0 || B == 0) return hipSuccess;
    const int vec = spmm_vec(X, ldx, B, Y, ldy);
    const spmm_plan pl = make_plan(n_rows, n_cols, nnz, B, plan != nullptr && vec == 4);
    if (pl.tiled) return exec_any(pl, n_rows, n_cols, ptr, X, ldx, B, Y, ldy, plan, s);
    return launch_rows(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy, vec, s);
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
