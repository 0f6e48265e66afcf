// Adaptive proximal steps: Prox-RMSProp (Algorithm 1) and Prox-ADAM
// (Algorithm 2).  Both keep the prox of eta*lambda*||.||_1 of Eq. (prox) and
// replace the plain step eta*g by a preconditioned one:
//   v' = beta2*v + (1-beta2)*g*g                         (both)
//   m' = beta1*m + (1-beta1)*g                           (ADAM)
//   u  = g / (sqrt(v') + eps)                            (RMSProp)
//   u  = (m'/(1-beta1^t)) / (sqrt(v'/(1-beta2^t)) + eps) (ADAM, bias-corrected)
//   w' = S_{eta*lambda}(w - eta*u)
// Arithmetic in double, as for the plain prox: the two moment updates round
// once each (an fma whose product beta*state is exact in double) and are
// stored as float; u is computed from the stored floats; w - eta*u rounds
// once (fma) and S_t of it once more, to float.  Zero results are +0.0.
//
// The fused l1-phase update uses the row slabs of the plain prox (2048
// columns of one row per 256-thread workgroup, W's slab scattered into LDS),
// with two passes:
//   count pass: read g, m, v; write m', v' back; count the nonzero w' per slab
//   fill pass:  read m', v' (ADAM) or g, v' (RMSProp), recompute w' from the
//               stored state and compact it to the scanned slab offsets.
// The recomputation sees exactly the floats the count pass stored, so both
// passes agree bit for bit.  When the caller's capacity may be too small the
// count pass leaves the state alone and the fill pass updates it, so a call
// that returns a capacity error has changed nothing.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kThreads = 256;
constexpr int kSlab = 1 << kProxSlabShift;
constexpr int kChunks = kSlab / (kThreads * 4);

// where the step reads its moments from
enum { kFromGrad = 0,     // g, m, v -> m', v' computed here
       kFromState = 1 };  // m', v' already stored (ADAM reads m', v'; RMSProp g, v')

// what a slab pass produces
enum { kCount = 0,        // counts[slab]
       kFill = 1,         // compacted CSR entries at off[slab]
       kDense = 2 };      // Z[i][k] and row_counts[i] (atomic integer adds)

template <int SOLVER, int SRC>
__device__ __forceinline__ float adaptive_update(const adaptive_params &P, float w, float g,
                                                 float &m, float &v) {
    if (SRC == kFromGrad) {
        const double gd = (double)g;
        v = (float)fma(P.omb2, gd * gd, P.beta2 * (double)v);
        if (SOLVER == kSolverAdam) m = (float)fma(P.omb1, gd, P.beta1 * (double)m);
    }
    double u;
    if (SOLVER == kSolverAdam)
        u = ((double)m / P.bc1) / (sqrt((double)v / P.bc2) + P.eps);
    else
        u = (double)g / (sqrt((double)v) + P.eps);
    const double z = fma(-P.eta, u, (double)w);
    const double s = z > P.thr ? z - P.thr : (z < -P.thr ? z + P.thr : 0.0);
    return (float)s;
}

template <bool V4>
__device__ __forceinline__ float4 load4(const float *p, int k, int k1) {
    if (V4 && k + 3 < k1) return *reinterpret_cast<const float4 *>(p + k);
    float4 r;
    r.x = k + 0 < k1 ? p[k + 0] : 0.f;
    r.y = k + 1 < k1 ? p[k + 1] : 0.f;
    r.z = k + 2 < k1 ? p[k + 2] : 0.f;
    r.w = k + 3 < k1 ? p[k + 3] : 0.f;
    return r;
}

template <bool V4>
__device__ __forceinline__ void store4(float *p, int k, int k1, const float (&a)[4]) {
    if (V4 && k + 3 < k1) {
        *reinterpret_cast<float4 *>(p + k) = make_float4(a[0], a[1], a[2], a[3]);
        return;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (k + j < k1) p[k + j] = a[j];
}

struct slab_io {
    const int *seg;          // [n_rows][slabs + 1] entry bounds of W per slab
    const int *idx;          // W col_idx
    const float *vals;       // W vals
    const float *G;          // [n_rows][ldg]
    float *M, *V;            // [n_rows][lds] moments (M unused by RMSProp)
    int64_t ldg, lds;
    int *counts;             // kCount
    const int *off;          // kFill: exclusive scan of counts (n_slabs + 1)
    int *col_out;            // kFill
    float *val_out;          // kFill
    int64_t capacity;        // kFill
    int *row_ptr;            // kFill
    int *nnz_out;            // kFill (nullable)
    float *Z;                // kDense
    int64_t ldz;             // kDense
    int *row_counts;         // kDense (nullable; zeroed before the launch)
};

template <int SOLVER, int SRC, bool WRITE, int PASS, bool V4>
__global__ __launch_bounds__(kThreads) void adaptive_slab_kernel(int n_cols, int slabs, slab_io io,
                                                                 adaptive_params P) {
    __shared__ __attribute__((aligned(16))) float wrow[kSlab];
    __shared__ int wave_tot[kThreads / kWave];
    const int64_t blk = blockIdx.x;
    const int row = (int)(blk / slabs);
    const int sl = (int)(blk - (int64_t)row * slabs);
    const int k0 = sl * kSlab;
    const int k1 = min(n_cols, k0 + kSlab);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int *sr = io.seg + (int64_t)row * (slabs + 1) + sl;
    const int s = sr[0], e = sr[1];
    constexpr bool kNeedG = SRC == kFromGrad || SOLVER == kSolverRms;
    constexpr bool kNeedM = SOLVER == kSolverAdam;
    const float *g = io.G + (int64_t)row * io.ldg;
    float *mrow = kNeedM ? io.M + (int64_t)row * io.lds : nullptr;
    float *vrow = io.V + (int64_t)row * io.lds;

    // every operand load of the slab in flight before W is staged
    float4 gq[kChunks], mq[kChunks], vq[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
        const int k = k0 + c * kThreads * 4 + tid * 4;
        gq[c] = kNeedG ? load4<V4>(g, k, k1) : make_float4(0.f, 0.f, 0.f, 0.f);
        mq[c] = kNeedM ? load4<V4>(mrow, k, k1) : make_float4(0.f, 0.f, 0.f, 0.f);
        vq[c] = load4<V4>(vrow, k, k1);
    }
    for (int k = tid * 4; k < kSlab; k += kThreads * 4)
        *reinterpret_cast<float4 *>(wrow + k) = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();
    for (int p = s + tid; p < e; p += kThreads) {
        const int k = io.idx[p];
        if (k >= k0 && k < k1) wrow[k - k0] = io.vals[p];
    }
    __syncthreads();

    int64_t out = PASS == kFill ? io.off[blk] : 0;
    if (PASS == kFill && tid == 0) {
        if (sl == 0) io.row_ptr[row] = (int)out;
        if (blk == (int64_t)gridDim.x - 1) {
            const int total = io.off[blk + 1];
            io.row_ptr[row + 1] = total;
            if (io.nnz_out) *io.nnz_out = total;
        }
    }
    int cnt = 0;
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
        const int kb = k0 + c * kThreads * 4;
        if (kb >= k1) continue;  // uniform
        const int k = kb + tid * 4;
        const float4 w4 = *reinterpret_cast<const float4 *>(wrow + (k - k0));
        const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
        const float gv[4] = {gq[c].x, gq[c].y, gq[c].z, gq[c].w};
        float mv[4] = {mq[c].x, mq[c].y, mq[c].z, mq[c].w};
        float vv[4] = {vq[c].x, vq[c].y, vq[c].z, vq[c].w};
        float o[4];
        bool keep[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            o[j] = k + j < k1 ? adaptive_update<SOLVER, SRC>(P, wv[j], gv[j], mv[j], vv[j]) : 0.f;
            keep[j] = o[j] != 0.f;
            cnt += keep[j];
        }
        if (WRITE) {
            if (kNeedM) store4<V4>(mrow, k, k1, mv);
            store4<V4>(vrow, k, k1, vv);
        }
        if (PASS == kDense) store4<V4>(io.Z + (int64_t)row * io.ldz, k, k1, o);
        if (PASS == kFill) {
            uint64_t msk[4];
            int below = 0, wcnt = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                msk[j] = wave_ballot(keep[j]);
                below += popc_below(msk[j]);
                wcnt += __popcll(msk[j]);
            }
            if (lane == 0) wave_tot[wave] = wcnt;
            __syncthreads();
            int woff = 0, tot = 0;
#pragma unroll
            for (int w = 0; w < kThreads / kWave; ++w) {
                const int wc = wave_tot[w];
                woff += w < wave ? wc : 0;
                tot += wc;
            }
            int mine = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (keep[j]) {
                    const int64_t pos = out + woff + below + mine;
                    if (pos < io.capacity) {
                        io.col_out[pos] = k + j;
                        io.val_out[pos] = o[j];
                    }
                    ++mine;
                }
            }
            out += tot;
            __syncthreads();  // wave_tot is reused by the next chunk
        }
    }
    if (PASS == kCount || (PASS == kDense && io.row_counts != nullptr)) {
        cnt = wave_sum_int(cnt);
        if (lane == 0) wave_tot[wave] = cnt;
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < kThreads / kWave; ++w) tot += wave_tot[w];
            if (PASS == kCount)
                io.counts[blk] = tot;
            else if (tot != 0)
                atomicAdd(io.row_counts + row, tot);
        }
    }
}

// The stored-entry form (one state entry per stored weight): debiasing with an
// adaptive solver (lambda = 0) or a support-restricted prox.
template <int SOLVER>
__global__ void adaptive_csr_kernel(int64_t nnz, float *__restrict__ vals, const float *__restrict__ g,
                                    float *__restrict__ M, float *__restrict__ V, adaptive_params P) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * blockDim.x) {
        float m = SOLVER == kSolverAdam ? M[p] : 0.f;
        float v = V[p];
        vals[p] = adaptive_update<SOLVER, kFromGrad>(P, vals[p], g[p], m, v);
        if (SOLVER == kSolverAdam) M[p] = m;
        V[p] = v;
    }
}

template <int SOLVER, int SRC, bool WRITE, int PASS>
hipError_t run_slabs(int n_rows, int n_cols, const slab_io &io, const adaptive_params &P, bool v4,
                     hipStream_t s) {
    const int slabs = prox_slabs(n_cols);
    const unsigned grid = (unsigned)((int64_t)n_rows * slabs);
    if (v4)
        adaptive_slab_kernel<SOLVER, SRC, WRITE, PASS, true><<<grid, kThreads, 0, s>>>(n_cols, slabs, io, P);
    else
        adaptive_slab_kernel<SOLVER, SRC, WRITE, PASS, false><<<grid, kThreads, 0, s>>>(n_cols, slabs, io, P);
    return hipGetLastError();
}

template <int SOLVER>
hipError_t dispatch_pass(int stage, int n_rows, int n_cols, const slab_io &io, const adaptive_params &P,
                         bool v4, hipStream_t s) {
    switch (stage) {
        case kStageCountWrite: return run_slabs<SOLVER, kFromGrad, true, kCount>(n_rows, n_cols, io, P, v4, s);
        case kStageCountKeep: return run_slabs<SOLVER, kFromGrad, false, kCount>(n_rows, n_cols, io, P, v4, s);
        case kStageFillStored: return run_slabs<SOLVER, kFromState, false, kFill>(n_rows, n_cols, io, P, v4, s);
        case kStageFillWrite: return run_slabs<SOLVER, kFromGrad, true, kFill>(n_rows, n_cols, io, P, v4, s);
        case kStageDense: return run_slabs<SOLVER, kFromGrad, true, kDense>(n_rows, n_cols, io, P, v4, s);
        default: return hipErrorInvalidValue;
    }
}

bool vec_ok(const void *p, int64_t ld) { return p == nullptr || (aligned16(p) && ld % 4 == 0); }

}  // namespace

hipError_t launch_adaptive_slabs(int stage, int n_rows, int n_cols, const int *ptr, const int *idx,
                                 const float *vals, const float *G, int64_t ldg, float *M, float *V,
                                 int64_t lds, const adaptive_params &P, int *seg, int *counts,
                                 const int *off, int *col_out, float *val_out, int64_t capacity,
                                 int *row_ptr, int *nnz_out, float *Z, int64_t ldz, int *row_counts,
                                 hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    if (stage == kStageCountWrite || stage == kStageCountKeep || stage == kStageDense) {
        // per-(row, slab) entry bounds of W (the fill pass reuses them)
        hipError_t e = launch_seg(n_rows, prox_slabs(n_cols), kProxSlabShift, ptr, idx, seg, s);
        if (e != hipSuccess) return e;
    }
    if (stage == kStageDense && row_counts != nullptr) {
        hipError_t e = launch_fill_i32(row_counts, n_rows, 0, s);
        if (e != hipSuccess) return e;
    }
    slab_io io{};
    io.seg = seg;
    io.idx = idx;
    io.vals = vals;
    io.G = G;
    io.M = M;
    io.V = V;
    io.ldg = ldg;
    io.lds = lds;
    io.counts = counts;
    io.off = off;
    io.col_out = col_out;
    io.val_out = val_out;
    io.capacity = capacity;
    io.row_ptr = row_ptr;
    io.nnz_out = nnz_out;
    io.Z = Z;
    io.ldz = ldz;
    io.row_counts = row_counts;
    const bool v4 = vec_ok(G, ldg) && vec_ok(M, lds) && vec_ok(V, lds) &&
                    (stage != kStageDense || vec_ok(Z, ldz));
    if (P.solver == kSolverAdam) return dispatch_pass<kSolverAdam>(stage, n_rows, n_cols, io, P, v4, s);
    return dispatch_pass<kSolverRms>(stage, n_rows, n_cols, io, P, v4, s);
}

hipError_t launch_adaptive_csr(int64_t nnz, float *vals, const float *g, float *M, float *V,
                               const adaptive_params &P, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    int64_t grid = ceil_div(nnz, 256);
    if (grid > 65536) grid = 65536;
    if (P.solver == kSolverAdam)
        adaptive_csr_kernel<kSolverAdam><<<(unsigned)grid, 256, 0, s>>>(nnz, vals, g, M, V, P);
    else
        adaptive_csr_kernel<kSolverRms><<<(unsigned)grid, 256, 0, s>>>(nnz, vals, g, M, V, P);
    return hipGetLastError();
}

}  // namespace l1csr
