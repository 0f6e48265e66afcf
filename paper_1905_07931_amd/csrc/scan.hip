// Exclusive prefix sum of int32 counts (row or column pointers) and fills.
//
// The counts scanned here have one entry per matrix row, column or slab (a few
// thousand to a few hundred thousand), so a single 1024-thread workgroup walks
// the array in tiles of 4096 with a carried running total (the next tile's
// loads are issued before the current tile is scanned); every wave scans its
// lanes' sums with shuffles and the 16 wave totals are scanned through LDS.
#include "common.hpp"
#include "launch.hpp"

namespace l1csr {

namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanPerThread = 4;
constexpr int kScanTile = kScanThreads * kScanPerThread;

__global__ __launch_bounds__(kScanThreads) void exclusive_scan_kernel(const int *__restrict__ in,
                                                                      int *__restrict__ out, int n,
                                                                      int *__restrict__ total_out) {
    __shared__ int wave_tot[kScanThreads / kWave];
    __shared__ int carry_s;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    int nv[kScanPerThread];
    auto load = [&](int base) {
#pragma unroll
        for (int e = 0; e < kScanPerThread; ++e) {
            const int j = base + tid * kScanPerThread + e;
            nv[e] = j < n ? in[j] : 0;
        }
    };
    load(0);
    for (int base = 0; base < n; base += kScanTile) {
        int v[kScanPerThread];
        int local = 0;
#pragma unroll
        for (int e = 0; e < kScanPerThread; ++e) {
            v[e] = nv[e];
            local += v[e];
        }
        if (base + kScanTile < n) load(base + kScanTile);
        const int incl = wave_incl_scan(local);
        if (lane == 63) wave_tot[wave] = incl;
        __syncthreads();
        if (wave == 0) {
            const int t = lane < kScanThreads / kWave ? wave_tot[lane] : 0;
            const int ti = wave_incl_scan(t);
            if (lane < kScanThreads / kWave) wave_tot[lane] = ti - t;  // exclusive
        }
        __syncthreads();
        const int carry = carry_s;
        int run = carry + wave_tot[wave] + incl - local;
#pragma unroll
        for (int e = 0; e < kScanPerThread; ++e) {
            const int j = base + tid * kScanPerThread + e;
            run += v[e];
            if (j < n) out[j + 1] = run;  // inclusive value at j is exclusive at j+1
        }
        __syncthreads();
        if (tid == kScanThreads - 1) carry_s = run;
        __syncthreads();
    }
    if (tid == 0) {
        out[0] = 0;
        if (total_out) *total_out = carry_s;
    }
}

__global__ void fill_i32_kernel(int *p, int64_t n, int v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void fill_f32_kernel(float *p, int64_t n, float v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void fill_rows_f32_kernel(float *p, int64_t rows, int64_t cols, int64_t ld, float v) {
    const int64_t total = rows * cols;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / cols, c = i - r * cols;
        p[r * ld + c] = v;
    }
}

__global__ void copy_i32_kernel(const int *src, int *dst) {
    if (threadIdx.x == 0) *dst = *src;
}

unsigned fill_grid(int64_t n) {
    int64_t g = ceil_div(n, 256);
    if (g > 65536) g = 65536;
    if (g < 1) g = 1;
    return (unsigned)g;
}

}  // namespace

hipError_t launch_exclusive_scan(const int *in, int *out, int n, int *total_out, hipStream_t s) {
    exclusive_scan_kernel<<<1, kScanThreads, 0, s>>>(in, out, n, total_out);
    return hipGetLastError();
}

hipError_t launch_fill_i32(int *p, int64_t n, int v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_i32_kernel<<<fill_grid(n), 256, 0, s>>>(p, n, v);
    return hipGetLastError();
}

hipError_t launch_copy_i32(const int *src, int *dst, hipStream_t s) {
    copy_i32_kernel<<<1, 64, 0, s>>>(src, dst);
    return hipGetLastError();
}

hipError_t launch_fill_f32(float *p, int64_t n, float v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_f32_kernel<<<fill_grid(n), 256, 0, s>>>(p, n, v);
    return hipGetLastError();
}

hipError_t launch_fill_rows_f32(float *p, int64_t rows, int64_t cols, int64_t ld, float v,
                                hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    fill_rows_f32_kernel<<<fill_grid(rows * cols), 256, 0, s>>>(p, rows, cols, ld, v);
    return hipGetLastError();
}

}  // namespace l1csr
