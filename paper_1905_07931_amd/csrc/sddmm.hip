// Masked weight gradient of the debiasing phase:
//     gv[p] = sum_b dY[row(p)][b] * X[col(p)][b]
// One wave per (row, batch segment).  The wave keeps its segment of the dY row
// in registers, and for every nonzero of the row reads the matching segment of
// the X row (coalesced, lanes over the batch), multiplies and reduces across
// the wave.  With several batch segments the per-segment partial sums go to
// scratch and a second pass adds them in segment order, so the result does not
// depend on scheduling.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kRowsPerBlock = 4;

// R float4 per lane: a segment covers 256*R batch entries (vector path) or
// 64*R entries (scalar path, VEC4 = false).
template <int R, bool VEC4>
__global__ __launch_bounds__(256) void sddmm_rows_kernel(
    int n_rows, const int *__restrict__ ptr, const int *__restrict__ idx,
    const float *__restrict__ dY, int64_t ldy, const float *__restrict__ X, int64_t ldx, int B,
    float *__restrict__ out, int64_t out_stride) {
    constexpr int W = VEC4 ? 4 : 1;
    constexpr int SEG = kWave * W * R;
    const int row = uniform(blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6));
    if (row >= n_rows) return;
    const int lane = threadIdx.x & 63;
    const int seg = blockIdx.y;
    const int start = uniform(ptr[row]);
    const int end = uniform(ptr[row + 1]);
    if (start == end) return;

    // batch index of (lane, r, w): seg*SEG + r*64*W + lane*W + w
    float y[R][W];
    const float *dyr = dY + (int64_t)row * ldy;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int b = seg * SEG + r * kWave * W + lane * W;
        if constexpr (VEC4) {
            if (b < B) {
                const float4 t = *reinterpret_cast<const float4 *>(dyr + b);
                y[r][0] = t.x; y[r][1] = t.y; y[r][2] = t.z; y[r][3] = t.w;
            } else {
#pragma unroll
                for (int w = 0; w < W; ++w) y[r][w] = 0.f;
            }
        } else {
            y[r][0] = b < B ? dyr[b] : 0.f;
        }
    }

    float *o = out + (int64_t)seg * out_stride;
    for (int base = start; base < end; base += kWave) {
        const int n = min(kWave, end - base);
        const int c = lane < n ? idx[base + lane] : 0;
        float mine = 0.f;
        for (int j = 0; j < n; ++j) {
            const int cj = lane_bcast(c, j);
            const float *xr = X + (int64_t)cj * ldx;
            float part = 0.f;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int b = seg * SEG + r * kWave * W + lane * W;
                if constexpr (VEC4) {
                    if (b < B) {
                        const float4 t = *reinterpret_cast<const float4 *>(xr + b);
                        part = fmaf(y[r][0], t.x, part);
                        part = fmaf(y[r][1], t.y, part);
                        part = fmaf(y[r][2], t.z, part);
                        part = fmaf(y[r][3], t.w, part);
                    }
                } else {
                    if (b < B) part = fmaf(y[r][0], xr[b], part);
                }
            }
            const float tot = wave_sum(part);
            if (lane == j) mine = tot;
        }
        if (lane < n) o[base + lane] = mine;
    }
}

// gv[p] = sum_{s < nseg} part[s][p], s ascending
__global__ void sddmm_reduce_kernel(int64_t nnz, int nseg, const float *__restrict__ part,
                                    float *__restrict__ gv) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * blockDim.x) {
        float acc = 0.f;
        for (int s = 0; s < nseg; ++s) acc += part[(int64_t)s * nnz + p];
        gv[p] = acc;
    }
}

struct plan {
    int R;
    bool v4;
    int seg;
    int nseg;
};

plan make_plan(int n_rows, int B, bool v4) {
    plan pl;
    pl.v4 = v4;
    const int W = v4 ? 4 : 1;
    // longest segments that still give enough waves to fill the chip
    pl.R = 4;
    if ((int64_t)n_rows * ceil_div(B, kWave * W * 4) < 4096) pl.R = 1;
    pl.seg = kWave * W * pl.R;
    pl.nseg = (int)ceil_div(B, pl.seg);
    if (pl.nseg < 1) pl.nseg = 1;
    return pl;
}

}  // namespace

size_t sddmm_workspace_bytes(int64_t nnz, int B) {
    // worst case over the plans: scalar path with R = 1 (64 entries per segment)
    const int64_t nseg = ceil_div(B, kWave);
    return nseg > 1 ? sizeof(float) * (size_t)(nseg * nnz) : 0;
}

hipError_t launch_sddmm(int n_rows, int64_t nnz, const int *ptr, const int *idx, const float *dY,
                        int64_t ldy, const float *X, int64_t ldx, int B, float *gv, void *ws,
                        hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    if (B == 0) return launch_fill_f32(gv, nnz, 0.f, s);
    const bool v4 = (B % 4 == 0) && (ldx % 4 == 0) && (ldy % 4 == 0) && aligned16(X) && aligned16(dY);
    const plan pl = make_plan(n_rows, B, v4);
    float *out = pl.nseg > 1 ? static_cast<float *>(ws) : gv;
    dim3 grid((unsigned)ceil_div(n_rows, kRowsPerBlock), (unsigned)pl.nseg);
    if (pl.v4) {
        if (pl.R == 4)
            sddmm_rows_kernel<4, true><<<grid, 256, 0, s>>>(n_rows, ptr, idx, dY, ldy, X, ldx, B, out, nnz);
        else
            sddmm_rows_kernel<1, true><<<grid, 256, 0, s>>>(n_rows, ptr, idx, dY, ldy, X, ldx, B, out, nnz);
    } else {
        if (pl.R == 4)
            sddmm_rows_kernel<4, false><<<grid, 256, 0, s>>>(n_rows, ptr, idx, dY, ldy, X, ldx, B, out, nnz);
        else
            sddmm_rows_kernel<1, false><<<grid, 256, 0, s>>>(n_rows, ptr, idx, dY, ldy, X, ldx, B, out, nnz);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || pl.nseg == 1) return e;
    int64_t g = ceil_div(nnz, 256);
    if (g > 65536) g = 65536;
    sddmm_reduce_kernel<<<(unsigned)g, 256, 0, s>>>(nnz, pl.nseg, out, gv);
    return hipGetLastError();
}

}  // namespace l1csr
