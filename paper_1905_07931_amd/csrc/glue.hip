// Layer glue of the fully connected ReLU networks: ReLU forward/backward and
// the mean softmax cross-entropy over batch columns (logits [C][B], batch
// contiguous).  The loss is reduced per workgroup and then summed in
// workgroup order by one thread, so it does not depend on scheduling.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

unsigned grid_for(int64_t n) {
    int64_t g = ceil_div(n, 256);
    if (g > 65536) g = 65536;
    if (g < 1) g = 1;
    return (unsigned)g;
}

__global__ void relu_fwd_kernel(int64_t n, const float *__restrict__ x, float *__restrict__ y) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const float v = x[i];
        y[i] = v > 0.f ? v : 0.f;
    }
}

__global__ void relu_bwd_kernel(int64_t n, const float *__restrict__ x, const float *__restrict__ dy,
                                float *__restrict__ dx) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        dx[i] = x[i] > 0.f ? dy[i] : 0.f;
}

constexpr int kSmThreads = 256;

__global__ __launch_bounds__(kSmThreads) void softmax_xent_kernel(
    int C, int B, const float *__restrict__ z, int64_t ld, const int *__restrict__ labels,
    float *__restrict__ dz, float *__restrict__ partial) {
    __shared__ float wsum[kSmThreads / kWave];
    const int b = blockIdx.x * kSmThreads + threadIdx.x;
    float loss = 0.f;
    if (b < B) {
        const int lab = labels[b];
        if (lab >= 0 && lab < C) {
            float m = z[b];
            for (int c = 1; c < C; ++c) m = fmaxf(m, z[(int64_t)c * ld + b]);
            float s = 0.f;
            for (int c = 0; c < C; ++c) s += expf(z[(int64_t)c * ld + b] - m);
            const float inv_s = 1.f / s;
            const float inv_b = 1.f / (float)B;
            for (int c = 0; c < C; ++c) {
                const float p = expf(z[(int64_t)c * ld + b] - m) * inv_s;
                dz[(int64_t)c * ld + b] = (p - (c == lab ? 1.f : 0.f)) * inv_b;
            }
            loss = logf(s) + m - z[(int64_t)lab * ld + b];
        } else {
            for (int c = 0; c < C; ++c) dz[(int64_t)c * ld + b] = 0.f;
        }
    }
    loss = wave_sum(loss);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = loss;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int w = 0; w < kSmThreads / kWave; ++w) t += wsum[w];
        partial[blockIdx.x] = t;
    }
}

__global__ void sum_partials_kernel(int n, const float *__restrict__ partial, float scale,
                                    float *__restrict__ out) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        float t = 0.f;
        for (int i = 0; i < n; ++i) t += partial[i];
        *out = t * scale;
    }
}

}  // namespace

hipError_t launch_relu_fwd(int64_t n, const float *x, float *y, hipStream_t s) {
    if (n == 0) return hipSuccess;
    relu_fwd_kernel<<<grid_for(n), 256, 0, s>>>(n, x, y);
    return hipGetLastError();
}

hipError_t launch_relu_bwd(int64_t n, const float *x, const float *dy, float *dx, hipStream_t s) {
    if (n == 0) return hipSuccess;
    relu_bwd_kernel<<<grid_for(n), 256, 0, s>>>(n, x, dy, dx);
    return hipGetLastError();
}

hipError_t launch_softmax_xent(int C, int B, const float *z, int64_t ld, const int *labels,
                               float *dz, float *loss, float *ws, hipStream_t s) {
    if (B == 0) return launch_fill_f32(loss, 1, 0.f, s);
    const int nblk = (int)ceil_div(B, kSmThreads);
    softmax_xent_kernel<<<nblk, kSmThreads, 0, s>>>(C, B, z, ld, labels, dz, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    sum_partials_kernel<<<1, 64, 0, s>>>(nblk, ws, 1.f / (float)B, loss);
    return hipGetLastError();
}

}  // namespace l1csr
