// Convolution layers with CSR filter banks, computed directly on the
// batch-contiguous maps (no lowered operand for the products):
//
//   forward     Y[(co,oh,ow)][b] = sum_{p in row co} w_p X[(ci, oh*SH-PH+kh, ow*SW-PW+kw)][b]
//   backward    dX[(ci,ih,iw)][b] = sum over CSC entries q of the columns (ci,kh,kw)
//               with ih = oh*SH-PH+kh, iw = ow*SW-PW+kw of w_q dY[(co_q,oh,ow)][b]
//   im2col      the lowered operand Xcol[(ci,kh,kw)][(oh*OW+ow)*B + b], used only
//               for the weight gradient (a dense contraction: matrix cores, or
//               the pattern-sampled product)
//   max pool    Y[(c,oh,ow)][b] = max of the KH x KW window
//
// A filter column is (ci*KH + kh)*KW + kw (Caffe's im2col row order).  Each
// output is summed by one thread in a fixed order (forward: CSR order;
// backward: kh, kw, then CSC order), so results are reproducible.  The input
// maps of LeNet-sized layers fit in L2, so the shifted re-reads of X by the
// direct products stay on chip; only the lowered operand of the weight
// gradient is streamed from HBM.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kThreads = 256;
constexpr int kStage = 2048;  // filter entries staged in LDS per pass
constexpr int kBatch = 8;     // entries whose loads are in flight together
constexpr int kMaxKK = 1024;  // filter positions KH*KW per channel (backward)

struct geom_t {
    int C, H, W, KH, KW, SH, SW, PH, PW, OH, OW;
};

geom_t to_geom(const conv_geom &g) {
    geom_t t;
    t.C = g.C; t.H = g.H; t.W = g.W; t.KH = g.KH; t.KW = g.KW;
    t.SH = g.SH; t.SW = g.SW; t.PH = g.PH; t.PW = g.PW;
    t.OH = (g.H + 2 * g.PH - g.KH) / g.SH + 1;
    t.OW = (g.W + 2 * g.PW - g.KW) / g.SW + 1;
    return t;
}

template <int VEC>
struct vec_t;
template <>
struct vec_t<1> {
    typedef float T;
    static __device__ __forceinline__ T load(const float *p) { return *p; }
    static __device__ __forceinline__ void store(float *p, T v) { *p = v; }
    static __device__ __forceinline__ void fma(T &a, float w, T x) { a = fmaf(w, x, a); }
    static __device__ __forceinline__ T zero() { return 0.f; }
    static __device__ __forceinline__ void vmax(T &a, T x) { a = x > a ? x : a; }
};
template <>
struct vec_t<4> {
    typedef float4 T;
    static __device__ __forceinline__ T load(const float *p) { return *reinterpret_cast<const float4 *>(p); }
    static __device__ __forceinline__ void store(float *p, T v) { *reinterpret_cast<float4 *>(p) = v; }
    static __device__ __forceinline__ void fma(T &a, float w, T x) {
        a.x = fmaf(w, x.x, a.x);
        a.y = fmaf(w, x.y, a.y);
        a.z = fmaf(w, x.z, a.z);
        a.w = fmaf(w, x.w, a.w);
    }
    static __device__ __forceinline__ T zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
    static __device__ __forceinline__ void vmax(T &a, T x) {
        a.x = x.x > a.x ? x.x : a.x;
        a.y = x.y > a.y ? x.y : a.y;
        a.z = x.z > a.z ? x.z : a.z;
        a.w = x.w > a.w ? x.w : a.w;
    }
};

// Forward.  Block (co, slice): the output block of channel co is the flattened
// [OH*OW][B] range f = pos*B + b; each thread takes VEC consecutive f of one
// position (B % VEC == 0).  Row co's entries are decoded into LDS once per
// pass: the input-row offset of output position (0, 0) and (kh, kw) for the
// range test.
template <int VEC>
__global__ __launch_bounds__(kThreads) void conv_fwd_kernel(geom_t g, int B, const int *__restrict__ ptr,
                                                            const int *__restrict__ idx,
                                                            const float *__restrict__ vals,
                                                            const float *__restrict__ X, int64_t ldx,
                                                            float *__restrict__ Y, int64_t ldy, int slices) {
    typedef vec_t<VEC> V;
    __shared__ int off_s[kStage];
    __shared__ int khw_s[kStage];
    __shared__ float w_s[kStage];
    const int co = blockIdx.x;
    const int64_t F = (int64_t)g.OH * g.OW * B;
    const int s = ptr[co], e = ptr[co + 1];
    auto stage = [&](int p0, int n) {
        __syncthreads();  // the previous entries are consumed
        for (int i = threadIdx.x; i < n; i += kThreads) {
            const int col = idx[p0 + i];
            const int ci = col / (g.KH * g.KW);
            const int r = col - ci * g.KH * g.KW;
            const int kh = r / g.KW, kw = r - kh * g.KW;
            off_s[i] = (ci * g.H + kh) * g.W + kw;
            khw_s[i] = (kh << 16) | kw;
            w_s[i] = vals[p0 + i];
        }
        __syncthreads();
    };
    const bool one_pass = e - s <= kStage;
    if (one_pass) stage(s, e - s);  // once for every slice of this block
    // the block walks slices blockIdx.y, blockIdx.y + gridDim.y, ... of channel co
    for (int slice = blockIdx.y; slice < slices; slice += gridDim.y) {
        const int64_t f = ((int64_t)slice * kThreads + threadIdx.x) * VEC;
        const bool active = f < F;
        const int pos = active ? (int)(f / B) : 0;
        const int b = active ? (int)(f - (int64_t)pos * B) : 0;
        const int oh = pos / g.OW, ow = pos - oh * g.OW;
        const int ih0 = oh * g.SH - g.PH, iw0 = ow * g.SW - g.PW;
        const int64_t base = (int64_t)(ih0 * g.W + iw0);
        typename V::T acc = V::zero();
        for (int p0 = s; p0 < e; p0 += kStage) {
            const int n = min(kStage, e - p0);
            if (!one_pass) stage(p0, n);
            if (!active) continue;
            // kBatch entries' loads in flight at a time; an entry whose input
            // position is outside the map loads row 0 instead and is skipped
            for (int i0 = 0; i0 < n; i0 += kBatch) {
                typename V::T x[kBatch];
                bool ok[kBatch];
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int i = i0 + u < n ? i0 + u : n - 1;
                    const int kh = khw_s[i] >> 16, kw = khw_s[i] & 0xffff;
                    const int ih = ih0 + kh, iw = iw0 + kw;
                    ok[u] = i0 + u < n && ih >= 0 && ih < g.H && iw >= 0 && iw < g.W;
                    x[u] = V::load(X + (ok[u] ? (base + off_s[i]) * ldx : 0) + b);
                }
#pragma unroll
                for (int u = 0; u < kBatch; ++u)
                    if (ok[u]) V::fma(acc, w_s[i0 + u], x[u]);
            }
        }
        if (active) V::store(Y + ((int64_t)co * g.OH * g.OW + pos) * ldy + b, acc);
    }
}

// Backward for the input maps.  Block (ci, slice) over the flattened
// [H*W][B] range of channel ci; the CSC columns (ci, kh, kw), kh, kw in order,
// are staged as (output-channel row offset, kh, kw, value).
template <int VEC>
__global__ __launch_bounds__(kThreads) void conv_bwd_kernel(geom_t g, int B, const int *__restrict__ col_ptr,
                                                            const int *__restrict__ row_idx,
                                                            const float *__restrict__ vals_t,
                                                            const float *__restrict__ dY, int64_t ldy,
                                                            float *__restrict__ dX, int64_t ldx, int slices) {
    typedef vec_t<VEC> V;
    __shared__ int co_s[kStage];
    __shared__ int khw_s[kStage];
    __shared__ float w_s[kStage];
    __shared__ int cp_s[kMaxKK + 1];
    const int ci = blockIdx.x;
    const int64_t F = (int64_t)g.H * g.W * B;
    const int kk = g.KH * g.KW;
    // the column pointers of this channel's KH*KW filter columns (kk <= kMaxKK)
    for (int c = threadIdx.x; c <= kk; c += kThreads) cp_s[c] = col_ptr[ci * kk + c];
    __syncthreads();
    const int s = cp_s[0], e = cp_s[kk];
    auto stage = [&](int q0, int n) {
        __syncthreads();
        for (int i = threadIdx.x; i < n; i += kThreads) {
            // the filter column of CSC entry q0 + i: last c with cp_s[c] <= q0 + i
            const int q = q0 + i;
            int lo = 0, hi = kk - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (cp_s[mid] <= q) lo = mid; else hi = mid - 1;
            }
            const int kh = lo / g.KW, kw = lo - kh * g.KW;
            co_s[i] = row_idx[q];
            khw_s[i] = (kh << 16) | kw;
            w_s[i] = vals_t[q];
        }
        __syncthreads();
    };
    const bool one_pass = e - s <= kStage;
    if (one_pass) stage(s, e - s);
    for (int slice = blockIdx.y; slice < slices; slice += gridDim.y) {
        const int64_t f = ((int64_t)slice * kThreads + threadIdx.x) * VEC;
        const bool active = f < F;
        const int pos = active ? (int)(f / B) : 0;
        const int b = active ? (int)(f - (int64_t)pos * B) : 0;
        const int ih = pos / g.W, iw = pos - ih * g.W;
        typename V::T acc = V::zero();
        for (int q0 = s; q0 < e; q0 += kStage) {
            const int n = min(kStage, e - q0);
            if (!one_pass) stage(q0, n);
            if (!active) continue;
            for (int i0 = 0; i0 < n; i0 += kBatch) {
                typename V::T y[kBatch];
                bool ok[kBatch];
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int i = i0 + u < n ? i0 + u : n - 1;
                    const int kh = khw_s[i] >> 16, kw = khw_s[i] & 0xffff;
                    const int th = ih + g.PH - kh, tw = iw + g.PW - kw;  // oh*SH, ow*SW
                    const int oh = th >= 0 ? th / g.SH : -1, ow = tw >= 0 ? tw / g.SW : -1;
                    ok[u] = i0 + u < n && oh >= 0 && ow >= 0 && oh * g.SH == th && ow * g.SW == tw &&
                            oh < g.OH && ow < g.OW;
                    const int64_t row = ok[u] ? (int64_t)(co_s[i] * g.OH + oh) * g.OW + ow : 0;
                    y[u] = V::load(dY + row * ldy + b);
                }
#pragma unroll
                for (int u = 0; u < kBatch; ++u)
                    if (ok[u]) V::fma(acc, w_s[i0 + u], y[u]);
            }
        }
        if (active) V::store(dX + ((int64_t)ci * g.H * g.W + pos) * ldx + b, acc);
    }
}

// im2col: row r = (ci, kh, kw) of the lowered operand, flattened columns
// f = pos*B + b; VEC consecutive f per thread (one position).
template <int VEC>
__global__ __launch_bounds__(kThreads) void im2col_kernel(geom_t g, int B, const float *__restrict__ X,
                                                          int64_t ldx, float *__restrict__ Xc, int64_t ldc,
                                                          int slices) {
    typedef vec_t<VEC> V;
    const int r = blockIdx.x / slices;
    const int slice = blockIdx.x - r * slices;
    const int64_t F = (int64_t)g.OH * g.OW * B;
    const int64_t f = ((int64_t)slice * kThreads + threadIdx.x) * VEC;
    if (f >= F) return;
    const int pos = (int)(f / B);
    const int b = (int)(f - (int64_t)pos * B);
    const int oh = pos / g.OW, ow = pos - oh * g.OW;
    const int ci = r / (g.KH * g.KW);
    const int kh = (r / g.KW) % g.KH, kw = r % g.KW;
    const int ih = oh * g.SH - g.PH + kh, iw = ow * g.SW - g.PW + kw;
    typename V::T v = V::zero();
    if (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W) v = V::load(X + ((int64_t)(ci * g.H + ih) * g.W + iw) * ldx + b);
    V::store(Xc + (int64_t)r * ldc + f, v);
}

template <int VEC>
__global__ __launch_bounds__(kThreads) void maxpool_kernel(geom_t g, int B, const float *__restrict__ X,
                                                           int64_t ldx, float *__restrict__ Y, int64_t ldy,
                                                           int slices) {
    typedef vec_t<VEC> V;
    const int c = blockIdx.x / slices;
    const int slice = blockIdx.x - c * slices;
    const int64_t F = (int64_t)g.OH * g.OW * B;
    const int64_t f = ((int64_t)slice * kThreads + threadIdx.x) * VEC;
    if (f >= F) return;
    const int pos = (int)(f / B);
    const int b = (int)(f - (int64_t)pos * B);
    const int oh = pos / g.OW, ow = pos - oh * g.OW;
    const float *x0 = X + ((int64_t)(c * g.H + oh * g.SH) * g.W + ow * g.SW) * ldx + b;
    typename V::T m = V::load(x0);
    for (int i = 0; i < g.KH; ++i)
        for (int j = 0; j < g.KW; ++j) V::vmax(m, V::load(x0 + ((int64_t)i * g.W + j) * ldx));
    V::store(Y + ((int64_t)(c * g.OH + oh) * g.OW + ow) * ldy + b, m);
}

bool vec4_ok(int B, int64_t lda, const void *a, int64_t ldb, const void *b) {
    return B % 4 == 0 && lda % 4 == 0 && ldb % 4 == 0 && aligned16(a) && aligned16(b);
}

int64_t slices_of(int64_t F, int vec) { return ceil_div(F, (int64_t)kThreads * vec); }

constexpr int64_t kMaxGridX = 0x7fffffff;
// blocks per channel: one per slice (many short blocks keep the most gathers in
// flight; fewer blocks walking several slices each measured slower), at most
// 65535, the rest walked by the blocks' slice loop
int64_t slice_blocks(int64_t slices, int64_t channels) {
    (void)channels;
    return slices < 65535 ? (slices < 1 ? 1 : slices) : 65535;
}

}  // namespace

bool conv_out_dims(const conv_geom &g, int *OH, int *OW) {
    if (g.C < 1 || g.H < 1 || g.W < 1 || g.KH < 1 || g.KW < 1 || g.SH < 1 || g.SW < 1 || g.PH < 0 || g.PW < 0)
        return false;
    if (g.KH > 0xffff || g.KW > 0xffff) return false;
    if ((int64_t)g.KH * g.KW > kMaxKK) return false;
    if (g.H + 2 * g.PH < g.KH || g.W + 2 * g.PW < g.KW) return false;
    const geom_t t = to_geom(g);
    *OH = t.OH;
    *OW = t.OW;
    return true;
}

hipError_t launch_conv_fwd(const conv_geom &cg, int N, int B, const int *ptr, const int *idx,
                           const float *vals, const float *X, int64_t ldx, float *Y, int64_t ldy,
                           hipStream_t s) {
    const geom_t g = to_geom(cg);
    const int64_t F = (int64_t)g.OH * g.OW * B;
    if (N == 0 || F == 0) return hipSuccess;
    const bool v4 = vec4_ok(B, ldx, X, ldy, Y);
    const int64_t sl = slices_of(F, v4 ? 4 : 1);
    if (sl > INT32_MAX || N > kMaxGridX) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)N, (unsigned)slice_blocks(sl, N));
    if (v4)
        conv_fwd_kernel<4><<<grid, kThreads, 0, s>>>(g, B, ptr, idx, vals, X, ldx, Y, ldy, (int)sl);
    else
        conv_fwd_kernel<1><<<grid, kThreads, 0, s>>>(g, B, ptr, idx, vals, X, ldx, Y, ldy, (int)sl);
    return hipGetLastError();
}

hipError_t launch_conv_bwd_data(const conv_geom &cg, int N, int B, const int *col_ptr, const int *row_idx,
                                const float *vals_t, const float *dY, int64_t ldy, float *dX, int64_t ldx,
                                hipStream_t s) {
    const geom_t g = to_geom(cg);
    const int64_t F = (int64_t)g.H * g.W * B;
    if (F == 0) return hipSuccess;
    (void)N;
    const bool v4 = vec4_ok(B, ldy, dY, ldx, dX);
    const int64_t sl = slices_of(F, v4 ? 4 : 1);
    if (sl > INT32_MAX || g.C > kMaxGridX) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)g.C, (unsigned)slice_blocks(sl, g.C));
    if (v4)
        conv_bwd_kernel<4><<<grid, kThreads, 0, s>>>(g, B, col_ptr, row_idx, vals_t, dY, ldy, dX, ldx, (int)sl);
    else
        conv_bwd_kernel<1><<<grid, kThreads, 0, s>>>(g, B, col_ptr, row_idx, vals_t, dY, ldy, dX, ldx, (int)sl);
    return hipGetLastError();
}

hipError_t launch_im2col(const conv_geom &cg, int B, const float *X, int64_t ldx, float *Xc, int64_t ldc,
                         hipStream_t s) {
    const geom_t g = to_geom(cg);
    const int64_t F = (int64_t)g.OH * g.OW * B;
    const int64_t R = (int64_t)g.C * g.KH * g.KW;
    if (F == 0 || R == 0) return hipSuccess;
    const bool v4 = vec4_ok(B, ldx, X, ldc, Xc);
    const int64_t sl = slices_of(F, v4 ? 4 : 1);
    if (sl * R > INT32_MAX) return hipErrorInvalidConfiguration;
    const unsigned grid = (unsigned)(sl * R);
    if (v4)
        im2col_kernel<4><<<grid, kThreads, 0, s>>>(g, B, X, ldx, Xc, ldc, (int)sl);
    else
        im2col_kernel<1><<<grid, kThreads, 0, s>>>(g, B, X, ldx, Xc, ldc, (int)sl);
    return hipGetLastError();
}

hipError_t launch_maxpool_fwd(const conv_geom &cg, int B, const float *X, int64_t ldx, float *Y, int64_t ldy,
                              hipStream_t s) {
    const geom_t g = to_geom(cg);
    const int64_t F = (int64_t)g.OH * g.OW * B;
    if (F == 0) return hipSuccess;
    const bool v4 = vec4_ok(B, ldx, X, ldy, Y);
    const int64_t sl = slices_of(F, v4 ? 4 : 1);
    if (sl * g.C > INT32_MAX) return hipErrorInvalidConfiguration;
    const unsigned grid = (unsigned)(sl * g.C);
    if (v4)
        maxpool_kernel<4><<<grid, kThreads, 0, s>>>(g, B, X, ldx, Y, ldy, (int)sl);
    else
        maxpool_kernel<1><<<grid, kThreads, 0, s>>>(g, B, X, ldx, Y, ldy, (int)sl);
    return hipGetLastError();
}

}  // namespace l1csr
