// CSR x dense products with the batch index contiguous (forward Y = W.X and,
// over the CSC copy, backward dX = W^T.dY).
//
// Tiled kernel (the hot path).  A 1024-thread workgroup owns a chunk of
// 64*VEC batch columns and a set of rows; each wave keeps up to MAXRW rows x
// VEC accumulators per lane in registers.  The dense operand is staged
// through LDS in 64 KB tiles (KT rows x 64*VEC columns); for each tile every
// wave walks the tile's segment of each of its rows: the (column, value)
// pairs of a segment are loaded by the lanes (coalesced, the next row's pairs
// in flight while the current row computes), written to a per-wave LDS slot
// and read back as broadcasts, and each nonzero costs one LDS read of the X
// row (lanes over the batch, conflict-free) and VEC fused multiply-adds.
//
// Load balance (power-law row lengths): a row longer than the average wave
// load is cut into "pieces" of at most that length; pieces are sorted by
// length (bucketed) and dealt to the waves in snake order, so every wave gets
// about the same number of nonzeros.  A row's pieces are summed by a fix-up
// pass in piece order, and every piece is summed by one wave in CSR order,
// so the result does not depend on the schedule.  The grid is exactly two
// workgroups per CU, mapped so that the workgroups resident on one XCD share
// a batch chunk (the same slice of X in that XCD's L2).
//
// Rows kernel (small or very sparse operands, where a workgroup would use few
// of a staged tile's X rows): one wave per (row, batch chunk) reading X
// directly from the cache hierarchy.
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
// planning: segment pointers, pieces, length order
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
    // one binary search per tile boundary (lanes over tiles); the result stays
    // inside [s, e] even for a malformed row
    for (int t = lane; t <= ntiles; t += kWave) {
        int lo = s, hi = e;
        if (t == 0) {
            hi = s;
        } else if (t < ntiles) {
            const int key = t << shift;
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

// pieces of a row: ceil(len / cap), at least one (an empty row is one empty piece)
__global__ void piece_count_kernel(int n_rows, const int *__restrict__ ptr, int cap,
                                   int *__restrict__ cnt) {
    for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < n_rows; r += gridDim.x * blockDim.x) {
        const int len = ptr[r + 1] - ptr[r];
        cnt[r] = len > cap ? (len + cap - 1) / cap : 1;
    }
}

// piece descriptors (row, first position, end position, row is split)
__global__ void piece_fill_kernel(int n_rows, const int *__restrict__ ptr,
                                  const int *__restrict__ pbeg, int4 *__restrict__ piece) {
    for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < n_rows; r += gridDim.x * blockDim.x) {
        const int s = ptr[r], len = ptr[r + 1] - s;
        const int v0 = pbeg[r], k = pbeg[r + 1] - v0;
        for (int j = 0; j < k; ++j)
            piece[v0 + j] = make_int4(r, s + (int)((int64_t)len * j / k),
                                      s + (int)((int64_t)len * (j + 1) / k), k > 1);
    }
}

constexpr int kBuckets = 129;  // 4 buckets per octave of the piece length, plus empty

__device__ __forceinline__ int length_key(int len) {
    if (len <= 0) return 0;
    const int b = 31 - __clz(len);
    const int sub = b >= 2 ? (len >> (b - 2)) & 3 : (len << (2 - b)) & 3;
    return 1 + b * 4 + sub;
}

// order[] = pieces by decreasing length bucket (order inside a bucket is
// arbitrary: it only decides which wave computes a piece)
__global__ __launch_bounds__(1024) void order_kernel(const int *__restrict__ n_pieces_ptr,
                                                     const int4 *__restrict__ piece,
                                                     int *__restrict__ order) {
    __shared__ int hist[kBuckets];
    __shared__ int start[kBuckets];
    const int n = *n_pieces_ptr;
    const int tid = threadIdx.x;
    for (int k = tid; k < kBuckets; k += blockDim.x) hist[k] = 0;
    __syncthreads();
    for (int v = tid; v < n; v += blockDim.x) atomicAdd(&hist[length_key(piece[v].z - piece[v].y)], 1);
    __syncthreads();
    if (tid == 0) {
        int run = 0;
        for (int k = kBuckets - 1; k >= 0; --k) {
            start[k] = run;
            run += hist[k];
        }
    }
    __syncthreads();
    for (int v = tid; v < n; v += blockDim.x)
        order[atomicAdd(&start[length_key(piece[v].z - piece[v].y)], 1)] = v;
}

// ---------------------------------------------------------------------------
// tiled kernel
// ---------------------------------------------------------------------------

constexpr int kNW = 16;             // waves per workgroup (1024 threads)
constexpr int kTileFloats = 16384;  // 64 KB of X per tile: two workgroups per CU

template <int VEC>
struct tiled_cfg {
    static constexpr int BB = kWave * VEC;       // batch columns per workgroup
    static constexpr int KT = kTileFloats / BB;  // X rows per tile
    static constexpr int SHIFT = VEC == 1 ? 8 : (VEC == 2 ? 7 : 6);
    static constexpr int MAXRW = VEC == 1 ? 16 : (VEC == 2 ? 12 : 8);  // pieces per wave in registers
    static_assert((1 << SHIFT) == KT, "tile height must be a power of two");
};

// Blocks are handed to the 8 XCDs round-robin; give XCD x a contiguous range
// of the (chunk-major) work list so its resident workgroups share a chunk.
__device__ __forceinline__ void map_block(int bid, int nblocks, int nrb, int &rb, int &ch) {
    const int per = nblocks / 8;
    const int w = bid < per * 8 ? (bid % 8) * per + bid / 8 : bid;
    ch = w / nrb;
    rb = w - ch * nrb;
}

template <int VEC, bool XV4>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8, 8))) void
spmm_tiled_kernel(int rw, int n_cols, const int *__restrict__ idx, const float *__restrict__ vals,
                  const int *__restrict__ seg, const int4 *__restrict__ piece,
                  const int *__restrict__ order, const int *__restrict__ n_pieces_ptr,
                  const float *__restrict__ X, int64_t ldx, int B, float *__restrict__ Y,
                  int64_t ldy, float *__restrict__ part, int nrb) {
    constexpr int BB = tiled_cfg<VEC>::BB;
    constexpr int KT = tiled_cfg<VEC>::KT;
    constexpr int MAXRW = tiled_cfg<VEC>::MAXRW;
    constexpr int Q = BB / 4;                       // float4 per tile row
    constexpr int PER = (KT * Q) / (kNW * kWave);   // float4 per thread per tile
    __shared__ __attribute__((aligned(16))) float Xs[KT * BB];
    __shared__ int2 slot[kNW][kWave];  // per-wave broadcast slot: (X row offset, value bits)

    const int n_pieces = uniform(*n_pieces_ptr);
    const int ntiles = (n_cols + KT - 1) / KT;
    int rb, ch;
    map_block(blockIdx.x, gridDim.x, nrb, rb, ch);
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int nw = nrb * kNW;
    const int g = rb * kNW + wave;
    const int b0 = ch * BB;

    // pieces of this wave: sorted position i*nw + g, snake order over rounds;
    // lane i holds the descriptor of piece i
    int pc[MAXRW];
    int4 my = make_int4(0, 0, 0, 0);
    int my_piece = -1;
#pragma unroll
    for (int i = 0; i < MAXRW; ++i) {
        const int j = i * nw + ((i & 1) ? (nw - 1 - g) : g);
        pc[i] = uniform((i < rw && j < n_pieces) ? order[j] : -1);
        if (lane == i) my_piece = pc[i];
    }
    if (my_piece >= 0) my = piece[my_piece];
    const int *my_seg = seg + (int64_t)my.x * (ntiles + 1);

    float acc[MAXRW][VEC];
#pragma unroll
    for (int i = 0; i < MAXRW; ++i)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[i][e] = 0.f;

    const float *xl = Xs + lane * VEC;
    int2 *ms = slot[wave];
    for (int t = 0; t < ntiles; ++t) {
        const int k0 = t * KT;
        // X tile and this tile's segment of every piece (lane i: piece i)
        float4 xr[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int f = threadIdx.x + u * (kNW * kWave);
            const int rr = f / Q, q = f - rr * Q;
            const int k = k0 + rr, b = b0 + q * 4;
            const float *src = X + (int64_t)k * ldx + b;
            if (XV4 && k < n_cols && b + 3 < B) {
                xr[u] = *reinterpret_cast<const float4 *>(src);
            } else {
                const bool kv = k < n_cols;
                xr[u].x = (kv && b + 0 < B) ? src[0] : 0.f;
                xr[u].y = (kv && b + 1 < B) ? src[1] : 0.f;
                xr[u].z = (kv && b + 2 < B) ? src[2] : 0.f;
                xr[u].w = (kv && b + 3 < B) ? src[3] : 0.f;
            }
        }
        int sl = 0, nl = 0;
        if (my_piece >= 0) {
            sl = max(my_seg[t], my.y);
            nl = max(min(my_seg[t + 1], my.z) - sl, 0);
        }
        __syncthreads();  // every wave is done with the previous tile
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int f = threadIdx.x + u * (kNW * kWave);
            *reinterpret_cast<float4 *>(Xs + f * 4) = xr[u];
        }
        __syncthreads();

        // pairs of piece i+1 are loaded while piece i computes
        int sN = lane_bcast(sl, 0), nN = lane_bcast(nl, 0);
        int cN = 0;
        float vN = 0.f;
        if (lane < nN) {
            cN = (idx[sN + lane] - k0) * BB;
            vN = vals[sN + lane];
        }
#pragma unroll
        for (int i = 0; i < MAXRW; ++i) {
            if (i < rw) {  // (a guard, not a break: keeps every acc[i] statically indexed)
            const int s = sN, n_total = nN;
            int c = cN;
            float v = vN;
            if (i + 1 < MAXRW) {
                sN = lane_bcast(sl, i + 1);
                nN = lane_bcast(nl, i + 1);
                if (lane < nN) {
                    cN = (idx[sN + lane] - k0) * BB;
                    vN = vals[sN + lane];
                }
            }
            for (int base = 0; base < n_total; base += kWave) {
                const int n = min(kWave, n_total - base);
                if (base > 0 && lane < n) {  // segments longer than one wave
                    c = (idx[s + base + lane] - k0) * BB;
                    v = vals[s + base + lane];
                }
                // one wave writes and reads its own slot: LDS keeps the order
                if (lane < n) ms[lane] = make_int2(c, __float_as_int(v));
                int j = 0;
                for (; j + 4 <= n; j += 4) {
                    const int2 p0 = ms[j], p1 = ms[j + 1], p2 = ms[j + 2], p3 = ms[j + 3];
                    float x0[VEC], x1[VEC], x2[VEC], x3[VEC];
                    load_vec<VEC>(xl + p0.x, x0);
                    load_vec<VEC>(xl + p1.x, x1);
                    load_vec<VEC>(xl + p2.x, x2);
                    load_vec<VEC>(xl + p3.x, x3);
#pragma unroll
                    for (int q = 0; q < VEC; ++q) {
                        acc[i][q] = fmaf(__int_as_float(p0.y), x0[q], acc[i][q]);
                        acc[i][q] = fmaf(__int_as_float(p1.y), x1[q], acc[i][q]);
                        acc[i][q] = fmaf(__int_as_float(p2.y), x2[q], acc[i][q]);
                        acc[i][q] = fmaf(__int_as_float(p3.y), x3[q], acc[i][q]);
                    }
                }
                for (; j < n; ++j) {
                    const int2 p0 = ms[j];
                    float x0[VEC];
                    load_vec<VEC>(xl + p0.x, x0);
#pragma unroll
                    for (int q = 0; q < VEC; ++q)
                        acc[i][q] = fmaf(__int_as_float(p0.y), x0[q], acc[i][q]);
                }
            }
            }
        }
    }

    // a whole row goes to Y; a piece of a split row to its partial row
    const int b = b0 + lane * VEC;
#pragma unroll
    for (int i = 0; i < MAXRW; ++i) {
        if (pc[i] < 0) continue;
        const int row = lane_bcast(my.x, i);
        const int split = lane_bcast(my.w, i);
        float *dst = split ? part + (int64_t)pc[i] * B + b : Y + (int64_t)row * ldy + b;
        if (b + VEC - 1 < B) {
            store_vec<VEC>(dst, acc[i]);
        } else {
#pragma unroll
            for (int q = 0; q < VEC; ++q)
                if (b + q < B) dst[q] = acc[i][q];
        }
    }
}

// Y[row] = sum of the partial rows of its pieces, in piece order (split rows only)
__global__ __launch_bounds__(256) void fixup_kernel(int n_rows, const int *__restrict__ pbeg,
                                                    const float *__restrict__ part, int B,
                                                    float *__restrict__ Y, int64_t ldy) {
    const int row = blockIdx.x;
    const int v0 = pbeg[row], v1 = pbeg[row + 1];
    if (v1 - v0 < 2) return;
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        float a = 0.f;
        for (int v = v0; v < v1; ++v) a += part[(int64_t)v * B + b];
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
                                                        int B, float *__restrict__ Y, int64_t ldy) {
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
            c = idx[base + lane];
            v = vals[base + lane];
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

// which path a product takes, and the shape of the tiled launch
struct spmm_plan {
    bool tiled;
    int vec;     // batch columns per lane
    int ntiles;  // X tiles
    int nch;     // batch chunks of 64 x vec columns
    int nrb;     // row groups (workgroups per chunk)
    int rw;      // pieces per wave
    int cap;     // longest piece
    int64_t max_pieces;
};

spmm_plan make_plan(int n_rows, int n_cols, int64_t nnz, int B, bool x4) {
    spmm_plan p{};
    if (!x4 || B < 32 || n_rows < 16 || n_cols <= 0) return p;
    p.vec = B >= 128 ? 2 : 1;
    const int BB = kWave * p.vec;
    p.nch = (int)ceil_div(B, BB);
    // two workgroups per CU over the whole grid, each with at least one row per wave
    int64_t nrb = 512 / p.nch;
    if (nrb < 1) nrb = 1;
    const int64_t nrb_max = ceil_div(n_rows, kNW);
    if (nrb > nrb_max) nrb = nrb_max;
    // staging an X tile pays off when a workgroup's rows use each X element ~2x
    const double density = (double)nnz / ((double)n_rows * n_cols);
    if (density * (double)n_rows / (double)nrb < 2.0) return p;
    p.tiled = true;
    const int64_t nw = nrb * kNW;
    int64_t cap = ceil_div(nnz, nw);
    if (cap < 64) cap = 64;
    p.cap = (int)(cap > INT32_MAX ? INT32_MAX : cap);
    p.max_pieces = n_rows + ceil_div(nnz, p.cap);
    const int maxrw = p.vec == 1 ? 16 : (p.vec == 2 ? 12 : 8);
    int64_t rw = ceil_div(p.max_pieces, nw);
    if (rw > maxrw) {
        rw = maxrw;
        nrb = ceil_div(p.max_pieces, (int64_t)kNW * maxrw);
    }
    p.rw = (int)rw;
    p.nrb = (int)nrb;
    p.ntiles = (int)ceil_div(n_cols, kTileFloats / BB);
    return p;
}

struct spmm_ws {
    int *pbeg;    // [n_rows + 1]
    int4 *piece;  // [max_pieces]
    int *order;   // [max_pieces]
    int *seg;     // [n_rows][ntiles + 1]
    float *part;  // [max_pieces][B]
    size_t bytes;
};

// workspace layout (256-byte aligned parts); base may be 0 to size it
spmm_ws carve(const spmm_plan &pl, int n_rows, int B, uintptr_t base) {
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    spmm_ws w{};
    size_t off = 0;
    w.pbeg = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * ((size_t)n_rows + 1));
    w.piece = reinterpret_cast<int4 *>(base + off);
    off = al(off + sizeof(int4) * (size_t)pl.max_pieces);
    w.order = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * (size_t)pl.max_pieces);
    w.seg = reinterpret_cast<int *>(base + off);
    off = al(off + sizeof(int) * (size_t)n_rows * (pl.ntiles + 1));
    w.part = reinterpret_cast<float *>(base + off);
    off = al(off + sizeof(float) * (size_t)pl.max_pieces * B);
    w.bytes = off;
    return w;
}

template <int VEC>
hipError_t run_tiled(const spmm_plan &pl, int n_rows, int n_cols, const int *ptr, const int *idx,
                     const float *vals, const float *X, int64_t ldx, int B, float *Y, int64_t ldy,
                     void *ws, hipStream_t s) {
    const spmm_ws w = carve(pl, n_rows, B, reinterpret_cast<uintptr_t>(ws));
    const unsigned g = (unsigned)ceil_div(n_rows, 256) < 4096 ? (unsigned)ceil_div(n_rows, 256) : 4096;
    piece_count_kernel<<<g, 256, 0, s>>>(n_rows, ptr, pl.cap, w.order);  // counts in order[] scratch
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = launch_exclusive_scan(w.order, w.pbeg, n_rows, nullptr, s)) != hipSuccess) return e;
    piece_fill_kernel<<<g, 256, 0, s>>>(n_rows, ptr, w.pbeg, w.piece);
    order_kernel<<<1, 1024, 0, s>>>(w.pbeg + n_rows, w.piece, w.order);
    seg_kernel<<<(unsigned)ceil_div(n_rows, 4), 256, 0, s>>>(n_rows, pl.ntiles,
                                                             tiled_cfg<VEC>::SHIFT, ptr, idx, w.seg);
    const unsigned nblocks = (unsigned)((int64_t)pl.nrb * pl.nch);
    const bool xv4 = (ldx % 4 == 0) && aligned16(X);
    if (xv4)
        spmm_tiled_kernel<VEC, true><<<nblocks, kNW * kWave, 0, s>>>(
            pl.rw, n_cols, idx, vals, w.seg, w.piece, w.order, w.pbeg + n_rows, X, ldx, B, Y, ldy,
            w.part, pl.nrb);
    else
        spmm_tiled_kernel<VEC, false><<<nblocks, kNW * kWave, 0, s>>>(
            pl.rw, n_cols, idx, vals, w.seg, w.piece, w.order, w.pbeg + n_rows, X, ldx, B, Y, ldy,
            w.part, pl.nrb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    fixup_kernel<<<(unsigned)n_rows, 256, 0, s>>>(n_rows, w.pbeg, w.part, B, Y, ldy);
    return hipGetLastError();
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
    const bool v4 = (B % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) && aligned16(Y);
    const bool v2 = (B % 2 == 0) && (ldx % 2 == 0) && (ldy % 2 == 0) &&
                    ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(Y)) & 7u) == 0;
    const spmm_plan pl = make_plan(n_rows, n_cols, nnz, B, ws != nullptr && v4);
    if (pl.tiled) {
        if (pl.vec == 2) return run_tiled<2>(pl, n_rows, n_cols, ptr, idx, vals, X, ldx, B, Y, ldy, ws, s);
        return run_tiled<1>(pl, n_rows, n_cols, ptr, idx, vals, X, ldx, B, Y, ldy, ws, s);
    }
    const int vec = v4 ? 4 : (v2 ? 2 : 1);
    dim3 grid((unsigned)ceil_div(n_rows, kRowsPerBlock), (unsigned)ceil_div(B, kWave * vec));
    if (vec == 4)
        spmm_rows_kernel<4><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy);
    else if (vec == 2)
        spmm_rows_kernel<2><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy);
    else
        spmm_rows_kernel<1><<<grid, 256, 0, s>>>(n_rows, ptr, idx, vals, X, ldx, B, Y, ldy);
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
