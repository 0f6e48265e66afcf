// C ABI of the l1csr library: host-side validation, workspace sizing and
// dispatch to the gfx950 kernels.  Every entry point validates all of its
// arguments before launching anything and only enqueues work on the caller's
// stream (csr_recompress with a short capacity is the one documented wait).
#include <math.h>

#include <mutex>

#include "../../include/l1csr.h"
#include "common.hpp"
#include "launch.hpp"

using namespace l1csr;

namespace {

constexpr int64_t kMaxGridY = 65535;

int hip_status(hipError_t e) { return e == hipSuccess ? L1CSR_OK : L1CSR_EHIP; }

bool finite_f(float x) { return isfinite(x) != 0; }

size_t round_up(size_t x) { return (x + 255) & ~(size_t)255; }

// a [rows][ld] matrix with rows > 0 and cols > 0 needs a pointer and ld >= cols
bool bad_dense(const void *p, int64_t rows, int64_t cols, int64_t ld) {
    if (ld < cols || ld < 0) return true;
    if (rows > 0 && cols > 0 && p == nullptr) return true;
    return false;
}

bool bad_csr(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
             const int32_t *col_idx, const void *vals, bool need_vals) {
    if (n_rows < 0 || n_cols < 0 || nnz < 0) return true;
    if (nnz > (int64_t)n_rows * (int64_t)n_cols) return true;
    if (nnz > INT32_MAX) return true;
    if (n_rows > 0 && row_ptr == nullptr) return true;
    if (nnz > 0 && (col_idx == nullptr || (need_vals && vals == nullptr))) return true;
    return false;
}

// [rows][ld] float matrices p (cols wide) and q: do their byte ranges overlap?
bool overlap(const float *p, int64_t ldp, const float *q, int64_t ldq, int64_t rows, int64_t cols) {
    if (p == nullptr || q == nullptr || rows <= 0 || cols <= 0) return false;
    const char *p0 = reinterpret_cast<const char *>(p);
    const char *p1 = p0 + sizeof(float) * ((rows - 1) * ldp + cols);
    const char *q0 = reinterpret_cast<const char *>(q);
    const char *q1 = q0 + sizeof(float) * ((rows - 1) * ldq + cols);
    return p0 < q1 && q0 < p1;
}

// byte ranges [a, a + na) and [b, b + nb) intersect (null or empty never does)
bool bytes_overlap(const void *a, size_t na, const void *b, size_t nb) {
    if (a == nullptr || b == nullptr || na == 0 || nb == 0) return false;
    const char *a0 = static_cast<const char *>(a), *b0 = static_cast<const char *>(b);
    return a0 < b0 + nb && b0 < a0 + na;
}

// extent in bytes of a [rows][ld] float matrix with `cols` columns used
size_t dense_bytes(int64_t rows, int64_t cols, int64_t ld) {
    return rows > 0 && cols > 0 ? sizeof(float) * (size_t)((rows - 1) * ld + cols) : 0;
}

// The output CSR of an out-of-place update (row_ptr_out [n_rows + 1],
// col_idx_out / vals_out [capacity]) must not share memory with any input the
// kernels still read while it is written (W's arrays, the gradient, states).
bool outputs_overlap(int32_t n_rows, int64_t nnz, const int32_t *row_ptr, const int32_t *col_idx,
                     const float *vals, const int32_t *row_ptr_out, const int32_t *col_idx_out,
                     const float *vals_out, int64_t capacity, const void *const *dense_in,
                     const size_t *dense_in_bytes, int n_dense) {
    const size_t rp = sizeof(int32_t) * ((size_t)n_rows + 1);
    const size_t cap = sizeof(int32_t) * (size_t)capacity;  // int32 and float alike
    const size_t in = sizeof(int32_t) * (size_t)nnz;
    const void *outs[3] = {row_ptr_out, col_idx_out, vals_out};
    const size_t out_b[3] = {rp, cap, cap};
    const void *ins[3] = {row_ptr, col_idx, vals};
    const size_t in_b[3] = {rp, in, in};
    for (int o = 0; o < 3; ++o) {
        for (int q = o + 1; q < 3; ++q)
            if (bytes_overlap(outs[o], out_b[o], outs[q], out_b[q])) return true;
        for (int i = 0; i < 3; ++i)
            if (bytes_overlap(outs[o], out_b[o], ins[i], in_b[i])) return true;
        for (int d = 0; d < n_dense; ++d)
            if (bytes_overlap(outs[o], out_b[o], dense_in[d], dense_in_bytes[d])) return true;
    }
    return false;
}

// Prox-RMSProp / Prox-ADAM hyper-parameters -> the kernels' double constants;
// false if any is out of range (Algorithms 1-2: eta > 0, eps > 0, decay rates
// in [0, 1), t >= 1 for ADAM's bias corrections; lambda >= 0).
bool make_adaptive(int solver, float eta, float lambda, float eps, float beta1, float beta2,
                   int64_t t, adaptive_params *P) {
    if (solver != L1CSR_SOLVER_RMSPROP && solver != L1CSR_SOLVER_ADAM) return false;
    if (!finite_f(eta) || !finite_f(lambda) || !finite_f(eps)) return false;
    if (!(eta > 0.f) || !(lambda >= 0.f) || !(eps > 0.f)) return false;
    if (!(beta2 >= 0.f && beta2 < 1.f)) return false;
    const bool adam = solver == L1CSR_SOLVER_ADAM;
    if (adam && (!(beta1 >= 0.f && beta1 < 1.f) || t < 1)) return false;
    P->solver = adam ? kSolverAdam : kSolverRms;
    P->eta = (double)eta;
    P->thr = (double)eta * (double)lambda;  // exact in double
    P->eps = (double)eps;
    P->beta1 = adam ? (double)beta1 : 0.0;
    P->beta2 = (double)beta2;
    P->omb1 = 1.0 - P->beta1;
    P->omb2 = 1.0 - P->beta2;
    P->bc1 = adam ? 1.0 - pow((double)beta1, (double)t) : 1.0;
    P->bc2 = adam ? 1.0 - pow((double)beta2, (double)t) : 1.0;
    return true;
}

// the geometry array of the conv calls: C, H, W, KH, KW, SH, SW, PH, PW (host)
bool read_geom(const int32_t *geom, conv_geom *g, int *OH, int *OW) {
    if (geom == nullptr) return false;
    g->C = geom[0]; g->H = geom[1]; g->W = geom[2]; g->KH = geom[3]; g->KW = geom[4];
    g->SH = geom[5]; g->SW = geom[6]; g->PH = geom[7]; g->PW = geom[8];
    if (!conv_out_dims(*g, OH, OW)) return false;
    // every flattened map and filter index fits int32
    const int64_t in = (int64_t)g->C * g->H * g->W, kk = (int64_t)g->C * g->KH * g->KW;
    return in <= INT32_MAX && kk <= INT32_MAX && (int64_t)*OH * *OW <= INT32_MAX;
}

// argument checks of prox_l1_recompress (every one but the workspace)
int prox_recompress_check(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                          const int32_t *col_idx, const float *vals, const float *G, int64_t ldg,
                          float eta, float lambda, const int32_t *row_ptr_out, const int32_t *col_idx_out,
                          const float *vals_out, int64_t capacity) {
    if (!finite_f(eta) || !finite_f(lambda) || eta <= 0.f || lambda < 0.f) return L1CSR_EINVAL;
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if (bad_dense(G, n_rows, n_cols, ldg) || row_ptr_out == nullptr || capacity < 0)
        return L1CSR_EINVAL;
    const int64_t total = (int64_t)n_rows * (int64_t)n_cols;
    if (total > INT32_MAX) return L1CSR_EUNSUPPORTED;  // int32 row pointers
    if (capacity > 0 && (col_idx_out == nullptr || vals_out == nullptr)) return L1CSR_EINVAL;
    if ((int64_t)n_rows * prox_slabs(n_cols) > INT32_MAX) return L1CSR_EUNSUPPORTED;
    // out of place: no output array may share memory with W or G
    const void *din[1] = {G};
    const size_t dinb[1] = {dense_bytes(n_rows, n_cols, ldg)};
    if (outputs_overlap(n_rows, nnz, row_ptr, col_idx, vals, row_ptr_out, col_idx_out, vals_out, capacity,
                        din, dinb, 1))
        return L1CSR_EINVAL;
    return L1CSR_OK;
}

// the launches of prox_l1_recompress on checked arguments, with ws holding
// prox_recompress_workspace_bytes(n_rows, n_cols) bytes
int prox_recompress_run(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                        const int32_t *col_idx, const float *vals, const float *G, int64_t ldg,
                        float eta, float lambda, int32_t *row_ptr_out, int32_t *col_idx_out,
                        float *vals_out, int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                        void *ws, hipStream_t stream) {
    (void)nnz;
    const int64_t total = (int64_t)n_rows * (int64_t)n_cols;
    if (n_rows == 0) {
        hipError_t e = launch_fill_i32(row_ptr_out, 1, 0, stream);
        if (e == hipSuccess && d_nnz_out) e = launch_fill_i32(d_nnz_out, 1, 0, stream);
        if (h_nnz_required) *h_nnz_required = capacity < total ? 0 : -1;
        return hip_status(e);
    }
    const double t = (double)eta * (double)lambda;     // exact in double
    // scratch: per-slab entry bounds and counts, then the counts' exclusive
    // scan (the output layout)
    const int64_t n_slabs = (int64_t)n_rows * prox_slabs(n_cols);
    const prox_ws pw = prox_carve(n_rows, n_cols, ws);
    hipError_t e = launch_prox_count(n_rows, n_cols, row_ptr, col_idx, vals, G, ldg, eta, t, pw.seg,
                                     pw.counts, stream);
    if (e == hipSuccess) e = launch_exclusive_scan(pw.counts, pw.off, (int)n_slabs, nullptr, stream);
    if (e != hipSuccess) return L1CSR_EHIP;
    if (capacity < total) {
        // the host needs the output size before the fill: row pointers now
        e = launch_prox_row_ptr(n_rows, n_cols, pw.off, row_ptr_out, d_nnz_out, stream);
        if (e != hipSuccess) return L1CSR_EHIP;
        int32_t h = 0;
        e = hipMemcpyAsync(&h, row_ptr_out + n_rows, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return L1CSR_EHIP;
        if (h_nnz_required) *h_nnz_required = h;
        if (h > capacity) return L1CSR_ECAPACITY;
    } else if (h_nnz_required) {
        *h_nnz_required = -1;
    }
    return hip_status(launch_prox_fill(n_rows, n_cols, pw.seg, col_idx, vals, G, ldg, eta, t, pw.off,
                                       col_idx_out, vals_out, capacity, row_ptr_out, d_nnz_out, stream));
}

// Static scratch of the entry points that allocate nothing (callers that
// cannot call hipMalloc: graph capture, serving loops).  Each GPU the library
// runs on holds its own copy until the process ends; every such call on one
// GPU shares it, so calls that overlap on one GPU race.  Host code never
// passes the array's name to a kernel: the name is a host-side stand-in, and
// the device address is looked up once per device (scratch_ptr).
constexpr size_t kScratchBytes = L1CSR_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_dev[kMaxDevices] = {};

// device address of `scratch` on the device `stream` belongs to (the current
// device for the null stream), looked up with that device current on first use
hipError_t scratch_ptr(hipStream_t stream, void **out) {
    int dev = 0;
    hipError_t e = stream != nullptr ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dev[dev] == nullptr) {
        int cur = 0;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        const hipError_t e2 = cur != dev ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess) return e;
        if (e2 != hipSuccess) return e2;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {


const char *l1csr_status_str(int status) {
    switch (status) {
        case L1CSR_OK: return "ok";
        case L1CSR_EINVAL: return "invalid argument";
        case L1CSR_ECAPACITY: return "output capacity too small";
        case L1CSR_EBADCSR: return "malformed CSR";
        case L1CSR_EHIP: return "HIP runtime or launch error";
        case L1CSR_EUNSUPPORTED: return "unsupported size or combination";
        case L1CSR_ESCRATCH: return "needs more scratch than the library's static buffer holds";
        default: return "unknown status";
    }
}

int l1csr_host_alloc_mapped(size_t bytes, void **host, void **dev) {
    if (bytes == 0 || host == nullptr || dev == nullptr) return L1CSR_EINVAL;
    void *h = nullptr;
    if (hipHostMalloc(&h, bytes, hipHostMallocMapped | hipHostMallocPortable | hipHostMallocCoherent) != hipSuccess)
        return L1CSR_EHIP;
    void *d = nullptr;
    if (hipHostGetDevicePointer(&d, h, 0) != hipSuccess || d == nullptr) {
        (void)hipHostFree(h);
        return L1CSR_EHIP;
    }
    *host = h;
    *dev = d;
    return L1CSR_OK;
}

int l1csr_host_free_mapped(void *host) {
    if (host == nullptr) return L1CSR_EINVAL;
    return hipHostFree(host) == hipSuccess ? L1CSR_OK : L1CSR_EHIP;
}

size_t l1csr_workspace_bytes(int op, int32_t n_rows, int32_t n_cols, int64_t nnz, int32_t B) {
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || B < 0) return 0;
    switch (op) {
        case L1CSR_OP_CSC_BUILD: return round_up(csc_workspace_bytes(n_rows, n_cols, nnz));
        case L1CSR_OP_RECOMPRESS: return round_up(sizeof(int) * counted_ws_ints(n_rows));
        case L1CSR_OP_SDDMM: return round_up(sddmm_workspace_bytes(n_rows, n_cols, nnz, B));
        case L1CSR_OP_SPMM: return round_up(spmm_workspace_bytes(n_rows, n_cols, nnz, B));
        case L1CSR_OP_COMPACT: return round_up(sizeof(int) * ((size_t)n_rows + 1));
        case L1CSR_OP_PROX_RECOMPRESS: return round_up(prox_recompress_workspace_bytes(n_rows, n_cols));
        case L1CSR_OP_DENSE_WGRAD: return round_up(wgrad_workspace_bytes(n_rows, n_cols, B));
        case L1CSR_OP_WGRAD_PROX: return round_up(wgrad_prox_split_bytes(n_rows, n_cols, B, L1CSR_F32));
        case L1CSR_OP_SOFTMAX_XENT: return round_up(sizeof(float) * (size_t)(ceil_div(B, 256) + 1));
        default: return 0;
    }
}

int csr_spmm_fwd(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                 const int32_t *col_idx, const float *vals, const float *X, int64_t ldx, int32_t B,
                 float *Y, int64_t ldy, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true) || B < 0) return L1CSR_EINVAL;
    if (bad_dense(X, n_cols, B, ldx) || bad_dense(Y, n_rows, B, ldy)) return L1CSR_EINVAL;
    if (ws != nullptr && ws_bytes < spmm_workspace_bytes(n_rows, n_cols, nnz, B)) return L1CSR_EINVAL;
    if (ceil_div(B, kWave) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    return hip_status(launch_spmm(n_rows, n_cols, nnz, row_ptr, col_idx, vals, X, ldx, B, Y, ldy, ws,
                                  stream));
}

int csr_spmm_plan(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr, const int32_t *col_idx,
                  const float *vals, int32_t B, void *plan, size_t plan_bytes, hipStream_t stream) {
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true) || B < 0) return L1CSR_EINVAL;
    const size_t need = spmm_workspace_bytes(n_rows, n_cols, nnz, B);
    if (need > 0 && (plan == nullptr || plan_bytes < need)) return L1CSR_EINVAL;
    if (ceil_div(B, kWave) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    return hip_status(launch_spmm_plan(n_rows, n_cols, nnz, row_ptr, col_idx, vals, B, need > 0 ? plan : nullptr,
                                       stream));
}

int csr_spmm_planned(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr, const int32_t *col_idx,
                     const float *vals, const float *X, int64_t ldx, int32_t B, float *Y, int64_t ldy,
                     const void *plan, size_t plan_bytes, hipStream_t stream) {
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true) || B < 0) return L1CSR_EINVAL;
    if (bad_dense(X, n_cols, B, ldx) || bad_dense(Y, n_rows, B, ldy)) return L1CSR_EINVAL;
    const size_t need = spmm_workspace_bytes(n_rows, n_cols, nnz, B);
    if (need > 0 && (plan == nullptr || plan_bytes < need)) return L1CSR_EINVAL;
    if (ceil_div(B, kWave) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    if (need > 0 && bytes_overlap(Y, dense_bytes(n_rows, B, ldy), plan, need)) return L1CSR_EINVAL;
    return hip_status(launch_spmm_planned(n_rows, n_cols, nnz, row_ptr, col_idx, vals, X, ldx, B, Y, ldy,
                                          need > 0 ? plan : nullptr, stream));
}

int csc_build(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
              const int32_t *col_idx, const float *vals, const uint32_t *mask, const int32_t *pos,
              int32_t *col_ptr, int32_t *row_idx, int32_t *perm, float *vals_t, void *ws, size_t ws_bytes,
              hipStream_t stream) {
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if (col_ptr == nullptr) return L1CSR_EINVAL;
    if ((mask == nullptr) != (pos == nullptr)) return L1CSR_EINVAL;  // both or neither
    if (nnz > 0 && (row_idx == nullptr || perm == nullptr || vals_t == nullptr)) return L1CSR_EINVAL;
    if (n_rows > 0 && n_cols > 0 &&
        (ws == nullptr || ws_bytes < csc_workspace_bytes(n_rows, n_cols, nnz)))
        return L1CSR_EINVAL;
    if (!csc_grid_fits(n_rows, n_cols)) return L1CSR_EUNSUPPORTED;
    return hip_status(launch_csc_build(n_rows, n_cols, nnz, row_ptr, col_idx, vals,
                                       reinterpret_cast<const unsigned *>(mask), pos, col_ptr, row_idx, perm,
                                       vals_t, ws, stream));
}

int csc_update_vals(int32_t n_cols, int64_t nnz, const int32_t *col_ptr, const int32_t *perm,
                    const float *vals, float *vals_t, hipStream_t stream) {
    if (n_cols < 0 || nnz < 0 || nnz > INT32_MAX || col_ptr == nullptr) return L1CSR_EINVAL;
    if (nnz > 0 && (perm == nullptr || vals == nullptr || vals_t == nullptr)) return L1CSR_EINVAL;
    return hip_status(launch_csc_gather_vals(n_cols, nnz, col_ptr, perm, vals, vals_t, stream));
}

int csr_spmm_bwd_t(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                   const int32_t *col_idx, const float *vals, const int32_t *col_ptr,
                   const int32_t *row_idx, const float *vals_t, const float *dY, int64_t ldy,
                   int32_t B, float *dX, int64_t ldx, void *ws, size_t ws_bytes,
                   hipStream_t stream) {
    // CSC path: col_ptr given (row_idx and vals_t too unless nnz == 0); atomic path: all NULL
    const bool use_csc = col_ptr != nullptr;
    if (!use_csc && (row_idx != nullptr || vals_t != nullptr)) return L1CSR_EINVAL;
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || B < 0) return L1CSR_EINVAL;
    if (nnz > (int64_t)n_rows * (int64_t)n_cols || nnz > INT32_MAX) return L1CSR_EINVAL;
    if (use_csc) {
        if (nnz > 0 && (row_idx == nullptr || vals_t == nullptr)) return L1CSR_EINVAL;
        if (ws != nullptr && ws_bytes < spmm_workspace_bytes(n_cols, n_rows, nnz, B)) return L1CSR_EINVAL;
    } else if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true)) {
        return L1CSR_EINVAL;
    }
    if (bad_dense(dY, n_rows, B, ldy) || bad_dense(dX, n_cols, B, ldx)) return L1CSR_EINVAL;
    if (ceil_div(B, kWave) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    if (use_csc)  // the forward product of the transposed matrix
        return hip_status(launch_spmm(n_cols, n_rows, nnz, col_ptr, row_idx, vals_t, dY, ldy, B, dX,
                                      ldx, ws, stream));
    return hip_status(launch_spmm_scatter_atomic(n_rows, n_cols, row_ptr, col_idx, vals, dY, ldy, B,
                                                 dX, ldx, stream));
}

int dense_wgrad(int32_t N, int32_t K, int32_t B, const float *dY, int64_t ldy, const float *X,
                int64_t ldx, float *dW, int64_t ldw, int precision, void *ws, size_t ws_bytes,
                hipStream_t stream) {
    if (N < 0 || K < 0 || B < 0) return L1CSR_EINVAL;
    if (precision != L1CSR_F32 && precision != L1CSR_BF16 && precision != L1CSR_BF16X3)
        return L1CSR_EINVAL;
    if (bad_dense(dY, N, B, ldy) || bad_dense(X, K, B, ldx) || bad_dense(dW, N, K, ldw))
        return L1CSR_EINVAL;
    if (ws != nullptr && ws_bytes < wgrad_workspace_bytes(N, K, B)) return L1CSR_EINVAL;
    if (ceil_div(N, 128) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    if (precision == L1CSR_BF16)
        return hip_status(launch_wgrad_bf16(N, K, B, dY, ldy, X, ldx, dW, ldw, stream));
    if (precision == L1CSR_BF16X3)
        return hip_status(launch_wgrad_bf16x3(N, K, B, dY, ldy, X, ldx, dW, ldw, stream));
    return hip_status(launch_wgrad_f32(N, K, B, dY, ldy, X, ldx, dW, ldw, ws, stream));
}

int sddmm_masked_wgrad(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                       const int32_t *col_idx, const float *dY, int64_t ldy, const float *X,
                       int64_t ldx, int32_t B, float *gv, void *ws, size_t ws_bytes,
                       hipStream_t stream) {
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, nullptr, false) || B < 0)
        return L1CSR_EINVAL;
    if (nnz > 0 && gv == nullptr) return L1CSR_EINVAL;
    if (bad_dense(dY, n_rows, B, ldy) || bad_dense(X, n_cols, B, ldx)) return L1CSR_EINVAL;
    const size_t need = sddmm_workspace_bytes(n_rows, n_cols, nnz, B);
    if (need > 0 && (ws == nullptr || ws_bytes < need)) return L1CSR_EINVAL;
    if (ceil_div(B, kWave) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    return hip_status(
        launch_sddmm(n_rows, n_cols, nnz, row_ptr, col_idx, dY, ldy, X, ldx, B, gv, ws, stream));
}

int prox_l1_step(int mode, int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                 const int32_t *col_idx, float *vals, const float *G, int64_t ldg, float eta,
                 float lambda, float *Z, int64_t ldz, int32_t *row_counts, hipStream_t stream) {
    if (!finite_f(eta) || !finite_f(lambda) || eta <= 0.f || lambda < 0.f) return L1CSR_EINVAL;
    const double t = (double)eta * (double)lambda;  // exact in double
    if (mode == L1CSR_PROX_CSR) {
        if (nnz < 0 || (nnz > 0 && (vals == nullptr || G == nullptr))) return L1CSR_EINVAL;
        return hip_status(launch_prox_csr(nnz, vals, G, eta, t, stream));
    }
    if (mode != L1CSR_PROX_DENSE) return L1CSR_EINVAL;
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if (bad_dense(G, n_rows, n_cols, ldg) || bad_dense(Z, n_rows, n_cols, ldz)) return L1CSR_EINVAL;
    if (n_rows > 0 && n_cols > 0 && Z != G) {
        // distinct buffers must not overlap; the same buffer needs the same ld
        const char *g0 = reinterpret_cast<const char *>(G);
        const char *g1 = g0 + sizeof(float) * ((n_rows - 1) * ldg + n_cols);
        const char *z0 = reinterpret_cast<const char *>(Z);
        const char *z1 = z0 + sizeof(float) * ((n_rows - 1) * ldz + n_cols);
        if (z0 < g1 && g0 < z1) return L1CSR_EINVAL;
    }
    if (Z == G && ldz != ldg) return L1CSR_EINVAL;
    return hip_status(launch_prox_dense(n_rows, n_cols, row_ptr, col_idx, vals, G, ldg, eta, t, Z, ldz,
                                        row_counts, stream));
}

int csr_recompress(int32_t n_rows, int32_t n_cols, const float *Z, int64_t ldz, float t,
                   const int32_t *row_counts, int32_t *row_ptr_out, int32_t *col_idx_out,
                   float *vals_out, int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                   void *ws, size_t ws_bytes, hipStream_t stream) {
    if (n_rows < 0 || n_cols < 0 || capacity < 0 || !finite_f(t)) return L1CSR_EINVAL;
    const int64_t total = (int64_t)n_rows * (int64_t)n_cols;
    if (total > INT32_MAX) return L1CSR_EUNSUPPORTED;  // int32 row pointers
    if (bad_dense(Z, n_rows, n_cols, ldz) || row_ptr_out == nullptr) return L1CSR_EINVAL;
    if (capacity > 0 && (col_idx_out == nullptr || vals_out == nullptr)) return L1CSR_EINVAL;
    int *counts = const_cast<int *>(row_counts);
    if (counts == nullptr && n_rows > 0) {
        if (ws == nullptr || ws_bytes < sizeof(int) * (size_t)n_rows) return L1CSR_EINVAL;
        counts = static_cast<int *>(ws);
    }
    hipError_t e = hipSuccess;
    if (row_counts == nullptr) e = launch_count_rows(n_rows, n_cols, Z, ldz, t, counts, stream);
    if (e != hipSuccess) return L1CSR_EHIP;
    e = launch_exclusive_scan(counts, row_ptr_out, n_rows, d_nnz_out, stream);
    if (e != hipSuccess) return L1CSR_EHIP;
    if (capacity < total) {
        int32_t h = 0;
        e = hipMemcpyAsync(&h, row_ptr_out + n_rows, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return L1CSR_EHIP;
        if (h_nnz_required) *h_nnz_required = h;
        if (h > capacity) return L1CSR_ECAPACITY;
    } else if (h_nnz_required) {
        *h_nnz_required = -1;  // unknown on the host (no wait)
    }
    return hip_status(launch_recompress_fill(n_rows, n_cols, Z, ldz, t, row_ptr_out, col_idx_out,
                                             vals_out, capacity, stream));
}

int prox_l1_recompress(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                       const int32_t *col_idx, const float *vals, const float *G, int64_t ldg,
                       float eta, float lambda, int32_t *row_ptr_out, int32_t *col_idx_out,
                       float *vals_out, int64_t capacity, int32_t *d_nnz_out,
                       int64_t *h_nnz_required, void *ws, size_t ws_bytes, hipStream_t stream) {
    const int v = prox_recompress_check(n_rows, n_cols, nnz, row_ptr, col_idx, vals, G, ldg, eta, lambda,
                                        row_ptr_out, col_idx_out, vals_out, capacity);
    if (v != L1CSR_OK) return v;
    if (n_rows > 0 && (ws == nullptr || ws_bytes < prox_recompress_workspace_bytes(n_rows, n_cols)))
        return L1CSR_EINVAL;
    return prox_recompress_run(n_rows, n_cols, nnz, row_ptr, col_idx, vals, G, ldg, eta, lambda,
                               row_ptr_out, col_idx_out, vals_out, capacity, d_nnz_out, h_nnz_required, ws,
                               stream);
}

int prox_l1_recompress_noalloc(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                               const int32_t *col_idx, const float *vals, const float *G, int64_t ldg,
                               float eta, float lambda, int32_t *row_ptr_out, int32_t *col_idx_out,
                               float *vals_out, int64_t capacity, int32_t *d_nnz_out,
                               int64_t *h_nnz_required, hipStream_t stream) {
    const int v = prox_recompress_check(n_rows, n_cols, nnz, row_ptr, col_idx, vals, G, ldg, eta, lambda,
                                        row_ptr_out, col_idx_out, vals_out, capacity);
    if (v != L1CSR_OK) return v;
    if (n_rows > 0 && prox_recompress_workspace_bytes(n_rows, n_cols) > kScratchBytes)
        return L1CSR_ESCRATCH;
    void *ws = nullptr;
    if (n_rows > 0 && scratch_ptr(stream, &ws) != hipSuccess) return L1CSR_EHIP;
    return prox_recompress_run(n_rows, n_cols, nnz, row_ptr, col_idx, vals, G, ldg, eta, lambda,
                               row_ptr_out, col_idx_out, vals_out, capacity, d_nnz_out, h_nnz_required, ws,
                               stream);
}

int dense_wgrad_prox(int32_t N, int32_t K, int32_t B, const float *dY, int64_t ldy, const float *X, int64_t ldx,
                     int precision, int64_t nnz, const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                     const uint32_t *mask, const int32_t *pos, float eta, float lambda, float *Z, int64_t ldz,
                     int32_t *word_counts, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (N < 0 || K < 0 || B < 0) return L1CSR_EINVAL;
    if (precision != L1CSR_F32 && precision != L1CSR_BF16 && precision != L1CSR_BF16X3) return L1CSR_EINVAL;
    if (!finite_f(eta) || !finite_f(lambda) || eta <= 0.f || lambda < 0.f) return L1CSR_EINVAL;
    if (bad_csr(N, K, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if (bad_dense(dY, N, B, ldy) || bad_dense(X, K, B, ldx) || bad_dense(Z, N, K, ldz)) return L1CSR_EINVAL;
    if ((int64_t)N * K > 0 && (mask == nullptr || pos == nullptr || word_counts == nullptr)) return L1CSR_EINVAL;
    if ((int64_t)N * K > INT32_MAX) return L1CSR_EUNSUPPORTED;  // int32 positions in the bitmap index
    if (ceil_div(N, 128) > kMaxGridY) return L1CSR_EUNSUPPORTED;
    const size_t split = wgrad_prox_split_bytes(N, K, B, precision);
    if (split > 0 && (ws == nullptr || ws_bytes < split)) return L1CSR_EINVAL;
    {  // the outputs Z and word_counts apart from each other and from every input
        const size_t wc = word_counts_bytes(N, K), in = sizeof(int32_t) * (size_t)nnz;
        const void *outs[2] = {Z, word_counts};
        const size_t ob[2] = {dense_bytes(N, K, ldz), wc};
        const void *ins[7] = {dY, X, row_ptr, col_idx, vals, mask, pos};
        const size_t ib[7] = {dense_bytes(N, B, ldy), dense_bytes(K, B, ldx), sizeof(int32_t) * ((size_t)N + 1), in,
                              in, wc, wc};
        if (bytes_overlap(outs[0], ob[0], outs[1], ob[1])) return L1CSR_EINVAL;
        for (int o = 0; o < 2; ++o)
            for (int i = 0; i < 7; ++i)
                if (bytes_overlap(outs[o], ob[o], ins[i], ib[i])) return L1CSR_EINVAL;
    }
    const double t = (double)eta * (double)lambda;  // exact in double
    return hip_status(launch_wgrad_prox(N, K, B, dY, ldy, X, ldx, precision, vals,
                                        reinterpret_cast<const unsigned *>(mask), pos, eta, t, Z, ldz, word_counts,
                                        split > 0 ? ws : nullptr, stream));
}

int csr_recompress_counted(int32_t n_rows, int32_t n_cols, const float *Z, int64_t ldz,
                           const int32_t *word_counts, int32_t *row_ptr_out, int32_t *col_idx_out,
                           float *vals_out, int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                           void *ws, size_t ws_bytes, hipStream_t stream) {
    if (n_rows < 0 || n_cols < 0 || capacity < 0) return L1CSR_EINVAL;
    const int64_t total = (int64_t)n_rows * (int64_t)n_cols;
    if (total > INT32_MAX) return L1CSR_EUNSUPPORTED;  // int32 row pointers
    if (bad_dense(Z, n_rows, n_cols, ldz) || row_ptr_out == nullptr) return L1CSR_EINVAL;
    if (total > 0 && word_counts == nullptr) return L1CSR_EINVAL;
    if (capacity > 0 && (col_idx_out == nullptr || vals_out == nullptr)) return L1CSR_EINVAL;
    const size_t wsn = sizeof(int) * counted_ws_ints(n_rows);
    if (n_rows > 0 && (ws == nullptr || ws_bytes < wsn)) return L1CSR_EINVAL;
    {  // outputs apart from each other and from Z and the counts
        const size_t cap = sizeof(int32_t) * (size_t)capacity, rp = sizeof(int32_t) * ((size_t)n_rows + 1);
        const void *outs[3] = {row_ptr_out, col_idx_out, vals_out};
        const size_t ob[3] = {rp, cap, cap};
        const void *ins[3] = {Z, word_counts, ws};
        const size_t ib[3] = {dense_bytes(n_rows, n_cols, ldz), word_counts_bytes(n_rows, n_cols), wsn};
        for (int o = 0; o < 3; ++o) {
            for (int q = o + 1; q < 3; ++q)
                if (bytes_overlap(outs[o], ob[o], outs[q], ob[q])) return L1CSR_EINVAL;
            for (int i = 0; i < 3; ++i)
                if (bytes_overlap(outs[o], ob[o], ins[i], ib[i])) return L1CSR_EINVAL;
        }
    }
    hipError_t e;
    if (total == 0) {  // no weights: an empty CSR
        e = launch_fill_i32(row_ptr_out, (int64_t)n_rows + 1, 0, stream);
        if (e == hipSuccess && d_nnz_out) e = launch_fill_i32(d_nnz_out, 1, 0, stream);
        if (h_nnz_required) *h_nnz_required = capacity < total ? 0 : -1;
        return hip_status(e);
    }
    int *sums = static_cast<int *>(ws);
    e = launch_counted_sums(n_rows, n_cols, word_counts, sums, stream);
    if (e != hipSuccess) return L1CSR_EHIP;
    // row_ptr' added up inside the compaction unless the host needs nnz' first
    const bool prefix_here = capacity >= total && counted_prefix_in_compact(n_rows);
    if (!prefix_here) {
        e = launch_counted_row_ptr(n_rows, sums, row_ptr_out, stream);
        if (e != hipSuccess) return L1CSR_EHIP;
    }
    if (capacity < total) {
        int32_t h = 0;
        e = hipMemcpyAsync(&h, row_ptr_out + n_rows, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return L1CSR_EHIP;
        if (h_nnz_required) *h_nnz_required = h;
        if (h > capacity) {
            if (d_nnz_out) launch_copy_i32(row_ptr_out + n_rows, d_nnz_out, stream);
            return L1CSR_ECAPACITY;
        }
    } else if (h_nnz_required) {
        *h_nnz_required = -1;
    }
    return hip_status(launch_counted_compact(n_rows, n_cols, Z, ldz, word_counts, sums, prefix_here, row_ptr_out,
                                             col_idx_out, vals_out, capacity, d_nnz_out, stream));
}

int csr_bitmap_build(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                     const int32_t *col_idx, uint32_t *mask, int32_t *pos, hipStream_t stream) {
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, nullptr, false)) return L1CSR_EINVAL;
    if ((int64_t)n_rows * n_cols > 0 && (mask == nullptr || pos == nullptr)) return L1CSR_EINVAL;
    const size_t bm = sizeof(int32_t) * (size_t)n_rows * (size_t)ceil_div(n_cols, 32);
    if (bytes_overlap(mask, bm, pos, bm)) return L1CSR_EINVAL;
    return hip_status(launch_bitmap(n_rows, n_cols, row_ptr, col_idx, reinterpret_cast<unsigned *>(mask), pos,
                                    stream));
}

int prox_adaptive_step(int mode, int solver, int32_t n_rows, int32_t n_cols, int64_t nnz,
                       const int32_t *row_ptr, const int32_t *col_idx, float *vals, const float *G,
                       int64_t ldg, float *m, float *v, int64_t lds, float eta, float lambda,
                       float eps, float beta1, float beta2, int64_t t, float *Z, int64_t ldz,
                       int32_t *row_counts, void *ws, size_t ws_bytes, hipStream_t stream) {
    adaptive_params P;
    if (!make_adaptive(solver, eta, lambda, eps, beta1, beta2, t, &P)) return L1CSR_EINVAL;
    const bool adam = solver == L1CSR_SOLVER_ADAM;
    if (mode == L1CSR_PROX_CSR) {
        if (nnz < 0 || nnz > INT32_MAX) return L1CSR_EINVAL;
        if (nnz > 0 && (vals == nullptr || G == nullptr || v == nullptr || (adam && m == nullptr)))
            return L1CSR_EINVAL;
        // state and gradient arrays are distinct, one entry per stored weight
        if (overlap(G, nnz, v, nnz, 1, nnz) || overlap(vals, nnz, v, nnz, 1, nnz) ||
            (adam && (overlap(m, nnz, v, nnz, 1, nnz) || overlap(m, nnz, G, nnz, 1, nnz) ||
                      overlap(m, nnz, vals, nnz, 1, nnz))))
            return L1CSR_EINVAL;
        return hip_status(launch_adaptive_csr(nnz, vals, G, adam ? m : nullptr, v, P, stream));
    }
    if (mode != L1CSR_PROX_DENSE) return L1CSR_EINVAL;
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if (bad_dense(G, n_rows, n_cols, ldg) || bad_dense(Z, n_rows, n_cols, ldz) ||
        bad_dense(v, n_rows, n_cols, lds) || (adam && bad_dense(m, n_rows, n_cols, lds)))
        return L1CSR_EINVAL;
    if (Z == G ? ldz != ldg : overlap(Z, ldz, G, ldg, n_rows, n_cols)) return L1CSR_EINVAL;
    if (overlap(v, lds, G, ldg, n_rows, n_cols) || overlap(v, lds, Z, ldz, n_rows, n_cols))
        return L1CSR_EINVAL;
    if (adam && (overlap(m, lds, G, ldg, n_rows, n_cols) || overlap(m, lds, Z, ldz, n_rows, n_cols) ||
                 overlap(m, lds, v, lds, n_rows, n_cols)))
        return L1CSR_EINVAL;
    if (n_rows > 0 && (ws == nullptr || ws_bytes < prox_recompress_workspace_bytes(n_rows, n_cols)))
        return L1CSR_EINVAL;
    const int64_t n_slabs = (int64_t)n_rows * prox_slabs(n_cols);
    if (n_slabs > INT32_MAX) return L1CSR_EUNSUPPORTED;
    if (n_rows == 0) return L1CSR_OK;
    if (n_cols == 0)
        return hip_status(row_counts ? launch_fill_i32(row_counts, n_rows, 0, stream) : hipSuccess);
    const prox_ws pw = prox_carve(n_rows, n_cols, ws);
    return hip_status(launch_adaptive_slabs(kStageDense, n_rows, n_cols, row_ptr, col_idx, vals, G,
                                            ldg, adam ? m : nullptr, v, lds, P, pw.seg, nullptr,
                                            nullptr, nullptr, nullptr, 0, nullptr, nullptr, Z, ldz,
                                            row_counts, stream));
}

int prox_adaptive_recompress(int solver, int32_t n_rows, int32_t n_cols, int64_t nnz,
                             const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                             const float *G, int64_t ldg, float *m, float *v, int64_t lds,
                             float eta, float lambda, float eps, float beta1, float beta2, int64_t t,
                             int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                             int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                             void *ws, size_t ws_bytes, hipStream_t stream) {
    adaptive_params P;
    if (!make_adaptive(solver, eta, lambda, eps, beta1, beta2, t, &P)) return L1CSR_EINVAL;
    const bool adam = solver == L1CSR_SOLVER_ADAM;
    if (bad_csr(n_rows, n_cols, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if (bad_dense(G, n_rows, n_cols, ldg) || bad_dense(v, n_rows, n_cols, lds) ||
        (adam && bad_dense(m, n_rows, n_cols, lds)) || row_ptr_out == nullptr || capacity < 0)
        return L1CSR_EINVAL;
    if (overlap(v, lds, G, ldg, n_rows, n_cols) ||
        (adam && (overlap(m, lds, G, ldg, n_rows, n_cols) || overlap(m, lds, v, lds, n_rows, n_cols))))
        return L1CSR_EINVAL;
    const int64_t total = (int64_t)n_rows * (int64_t)n_cols;
    if (total > INT32_MAX) return L1CSR_EUNSUPPORTED;  // int32 row pointers
    if (capacity > 0 && (col_idx_out == nullptr || vals_out == nullptr)) return L1CSR_EINVAL;
    if (n_rows > 0 && (ws == nullptr || ws_bytes < prox_recompress_workspace_bytes(n_rows, n_cols)))
        return L1CSR_EINVAL;
    {  // out of place: no output array may share memory with W, G or the states
        const void *din[3] = {G, v, adam ? m : nullptr};
        const size_t dinb[3] = {dense_bytes(n_rows, n_cols, ldg), dense_bytes(n_rows, n_cols, lds),
                                adam ? dense_bytes(n_rows, n_cols, lds) : 0};
        if (outputs_overlap(n_rows, nnz, row_ptr, col_idx, vals, row_ptr_out, col_idx_out, vals_out,
                            capacity, din, dinb, 3))
            return L1CSR_EINVAL;
    }
    if (n_rows == 0) {
        hipError_t e = launch_fill_i32(row_ptr_out, 1, 0, stream);
        if (e == hipSuccess && d_nnz_out) e = launch_fill_i32(d_nnz_out, 1, 0, stream);
        if (h_nnz_required) *h_nnz_required = capacity < total ? 0 : -1;
        return hip_status(e);
    }
    const int64_t n_slabs = (int64_t)n_rows * prox_slabs(n_cols);
    if (n_slabs > INT32_MAX) return L1CSR_EUNSUPPORTED;
    float *M = adam ? m : nullptr;
    const prox_ws pw = prox_carve(n_rows, n_cols, ws);
    // with room for every weight the count pass stores the new moments and the
    // fill pass recomputes from them; otherwise the state is only written once
    // the output is known to fit
    const bool roomy = capacity >= total;
    hipError_t e = launch_adaptive_slabs(roomy ? kStageCountWrite : kStageCountKeep, n_rows, n_cols,
                                         row_ptr, col_idx, vals, G, ldg, M, v, lds, P, pw.seg,
                                         pw.counts, nullptr, nullptr, nullptr, 0, nullptr, nullptr,
                                         nullptr, 0, nullptr, stream);
    if (e == hipSuccess) e = launch_exclusive_scan(pw.counts, pw.off, (int)n_slabs, nullptr, stream);
    if (e != hipSuccess) return L1CSR_EHIP;
    if (!roomy) {
        e = launch_prox_row_ptr(n_rows, n_cols, pw.off, row_ptr_out, d_nnz_out, stream);
        if (e != hipSuccess) return L1CSR_EHIP;
        int32_t h = 0;
        e = hipMemcpyAsync(&h, row_ptr_out + n_rows, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) return L1CSR_EHIP;
        if (h_nnz_required) *h_nnz_required = h;
        if (h > capacity) return L1CSR_ECAPACITY;
    } else if (h_nnz_required) {
        *h_nnz_required = -1;
    }
    return hip_status(launch_adaptive_slabs(roomy ? kStageFillStored : kStageFillWrite, n_rows, n_cols,
                                            row_ptr, col_idx, vals, G, ldg, M, v, lds, P, pw.seg,
                                            nullptr, pw.off, col_idx_out, vals_out, capacity,
                                            row_ptr_out, d_nnz_out, nullptr, 0, nullptr, stream));
}

int csr_compact(int32_t n_rows, int64_t nnz, const int32_t *row_ptr, const int32_t *col_idx,
                const float *vals, int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                int32_t *d_nnz_out, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (n_rows < 0 || nnz < 0 || nnz > INT32_MAX) return L1CSR_EINVAL;
    if (n_rows > 0 && (row_ptr == nullptr || row_ptr_out == nullptr)) return L1CSR_EINVAL;
    if (nnz > 0 && (col_idx == nullptr || vals == nullptr || col_idx_out == nullptr ||
                    vals_out == nullptr))
        return L1CSR_EINVAL;
    if (n_rows > 0 && (ws == nullptr || ws_bytes < sizeof(int) * (size_t)n_rows)) return L1CSR_EINVAL;
    if (n_rows == 0) {
        if (row_ptr_out == nullptr) return L1CSR_EINVAL;
        hipError_t e = launch_fill_i32(row_ptr_out, 1, 0, stream);
        if (e == hipSuccess && d_nnz_out) e = launch_fill_i32(d_nnz_out, 1, 0, stream);
        return hip_status(e);
    }
    int *counts = static_cast<int *>(ws);
    hipError_t e = launch_compact_count(n_rows, row_ptr, vals, counts, stream);
    if (e == hipSuccess) e = launch_exclusive_scan(counts, row_ptr_out, n_rows, d_nnz_out, stream);
    if (e == hipSuccess)
        e = launch_compact_fill(n_rows, row_ptr, col_idx, vals, row_ptr_out, col_idx_out, vals_out,
                                stream);
    return hip_status(e);
}

int csr_validate(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                 const int32_t *col_idx, int32_t *d_status, hipStream_t stream) {
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || nnz > INT32_MAX) return L1CSR_EINVAL;
    if (row_ptr == nullptr || d_status == nullptr || (nnz > 0 && col_idx == nullptr))
        return L1CSR_EINVAL;
    return hip_status(launch_csr_validate(n_rows, n_cols, nnz, row_ptr, col_idx, d_status, stream));
}

int csr_conv_fwd(const int32_t *geom, int32_t n_out, int64_t nnz, const int32_t *row_ptr,
                 const int32_t *col_idx, const float *vals, const float *X, int64_t ldx, int32_t B,
                 float *Y, int64_t ldy, hipStream_t stream) {
    conv_geom g;
    int OH, OW;
    if (!read_geom(geom, &g, &OH, &OW) || B < 0) return L1CSR_EINVAL;
    const int64_t K = (int64_t)g.C * g.KH * g.KW;
    if (bad_csr(n_out, (int32_t)K, nnz, row_ptr, col_idx, vals, true)) return L1CSR_EINVAL;
    if ((int64_t)n_out * OH * OW > INT32_MAX) return L1CSR_EUNSUPPORTED;
    if (bad_dense(X, (int64_t)g.C * g.H * g.W, B, ldx) || bad_dense(Y, (int64_t)n_out * OH * OW, B, ldy))
        return L1CSR_EINVAL;
    return hip_status(launch_conv_fwd(g, n_out, B, row_ptr, col_idx, vals, X, ldx, Y, ldy, stream));
}

int csr_conv_bwd_data(const int32_t *geom, int32_t n_out, int64_t nnz, const int32_t *col_ptr,
                      const int32_t *row_idx, const float *vals_t, const float *dY, int64_t ldy, int32_t B,
                      float *dX, int64_t ldx, hipStream_t stream) {
    conv_geom g;
    int OH, OW;
    if (!read_geom(geom, &g, &OH, &OW) || B < 0 || n_out < 0 || nnz < 0) return L1CSR_EINVAL;
    const int64_t K = (int64_t)g.C * g.KH * g.KW;
    if (nnz > (int64_t)n_out * K || nnz > INT32_MAX || col_ptr == nullptr) return L1CSR_EINVAL;
    if (nnz > 0 && (row_idx == nullptr || vals_t == nullptr)) return L1CSR_EINVAL;
    if ((int64_t)n_out * OH * OW > INT32_MAX) return L1CSR_EUNSUPPORTED;
    if (bad_dense(dY, (int64_t)n_out * OH * OW, B, ldy) || bad_dense(dX, (int64_t)g.C * g.H * g.W, B, ldx))
        return L1CSR_EINVAL;
    return hip_status(launch_conv_bwd_data(g, n_out, B, col_ptr, row_idx, vals_t, dY, ldy, dX, ldx, stream));
}

int conv_im2col(const int32_t *geom, const float *X, int64_t ldx, int32_t B, float *Xcol, int64_t ldc,
                hipStream_t stream) {
    conv_geom g;
    int OH, OW;
    if (!read_geom(geom, &g, &OH, &OW) || B < 0) return L1CSR_EINVAL;
    const int64_t cols = (int64_t)OH * OW * B;
    if (bad_dense(X, (int64_t)g.C * g.H * g.W, B, ldx) || bad_dense(Xcol, (int64_t)g.C * g.KH * g.KW, cols, ldc))
        return L1CSR_EINVAL;
    return hip_status(launch_im2col(g, B, X, ldx, Xcol, ldc, stream));
}

int l1csr_maxpool_fwd(const int32_t *geom, const float *X, int64_t ldx, int32_t B, float *Y, int64_t ldy,
                      hipStream_t stream) {
    conv_geom g;
    int OH, OW;
    if (!read_geom(geom, &g, &OH, &OW) || B < 0) return L1CSR_EINVAL;
    if (g.PH != 0 || g.PW != 0) return L1CSR_EUNSUPPORTED;
    if (bad_dense(X, (int64_t)g.C * g.H * g.W, B, ldx) || bad_dense(Y, (int64_t)g.C * OH * OW, B, ldy))
        return L1CSR_EINVAL;
    return hip_status(launch_maxpool_fwd(g, B, X, ldx, Y, ldy, stream));
}

int l1csr_relu_fwd(int64_t n, const float *x, float *y, hipStream_t stream) {
    if (n < 0 || (n > 0 && (x == nullptr || y == nullptr))) return L1CSR_EINVAL;
    return hip_status(launch_relu_fwd(n, x, y, stream));
}

int l1csr_relu_bwd(int64_t n, const float *x, const float *dy, float *dx, hipStream_t stream) {
    if (n < 0 || (n > 0 && (x == nullptr || dy == nullptr || dx == nullptr))) return L1CSR_EINVAL;
    return hip_status(launch_relu_bwd(n, x, dy, dx, stream));
}

int l1csr_softmax_xent(int32_t C, int32_t B, const float *logits, int64_t ld,
                       const int32_t *labels, float *dlogits, float *loss, void *ws,
                       size_t ws_bytes, hipStream_t stream) {
    if (C <= 0 || B < 0 || loss == nullptr) return L1CSR_EINVAL;
    if (bad_dense(logits, C, B, ld) || bad_dense(dlogits, C, B, ld)) return L1CSR_EINVAL;
    if (B > 0 && labels == nullptr) return L1CSR_EINVAL;
    if (B > 0 && (ws == nullptr || ws_bytes < sizeof(float) * (size_t)ceil_div(B, 256)))
        return L1CSR_EINVAL;
    return hip_status(
        launch_softmax_xent(C, B, logits, ld, labels, dlogits, loss, static_cast<float *>(ws), stream));
}

}  // extern "C"
