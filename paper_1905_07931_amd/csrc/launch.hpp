// Internal launchers: one per kernel family, called by the C ABI after the
// arguments have been validated on the host.  Each returns hipSuccess or the
// launch error.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace l1csr {

// spmm.hip -----------------------------------------------------------------
// Y = A.X for a CSR operand A (n_rows x n_cols); ws (nullable) holds the plan
// and partial rows of the tiled kernel, spmm_workspace_bytes(n_rows, n_cols,
// nnz, B) bytes (0: the tiled kernel is not used for these sizes).
size_t spmm_workspace_bytes(int n_rows, int n_cols, int64_t nnz, int B);
hipError_t launch_spmm(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                       const float *vals, const float *X, int64_t ldx, int B, float *Y,
                       int64_t ldy, void *ws, hipStream_t s);
// the tiled product in two parts: its planning launches (depend on W and B
// only) into plan, then the product from that plan
hipError_t launch_spmm_plan(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx, const float *vals,
                            int B, void *plan, hipStream_t s);
hipError_t launch_spmm_planned(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                               const float *vals, const float *X, int64_t ldx, int B, float *Y, int64_t ldy,
                               const void *plan, hipStream_t s);
hipError_t launch_spmm_scatter_atomic(int n_rows, int n_cols, const int *ptr, const int *idx,
                                      const float *vals, const float *dY, int64_t ldy, int B,
                                      float *dX, int64_t ldx, hipStream_t s);
// seg[row][t] = first position of the row with column >= t << shift, t = 0..ntiles
hipError_t launch_seg(int n_rows, int ntiles, int shift, const int *ptr, const int *idx, int *seg,
                      hipStream_t s);

// csc.hip ------------------------------------------------------------------
size_t csc_workspace_bytes(int n_rows, int n_cols, int64_t nnz);
// the (row chunk, column tile) grid of the build fits the launch limits
bool csc_grid_fits(int n_rows, int n_cols);
hipError_t launch_csc_build(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                            const float *vals, const unsigned *mask, const int *pos, int *col_ptr, int *row_idx,
                            int *perm, float *vals_t, void *ws, hipStream_t s);
// vals_t[q] = vals[perm[q]] for q < col_ptr[n_cols] (read on the device)
hipError_t launch_csc_gather_vals(int n_cols, int64_t nnz_bound, const int *col_ptr, const int *perm,
                                  const float *vals, float *vals_t, hipStream_t s);

// scan.hip -----------------------------------------------------------------
// out[0] = 0, out[j+1] = in[0] + ... + in[j] for j < n (out has n+1 entries);
// optionally also writes the total to *total_out.
hipError_t launch_exclusive_scan(const int *in, int *out, int n, int *total_out, hipStream_t s);
hipError_t launch_fill_i32(int *p, int64_t n, int v, hipStream_t s);
// *dst = *src in stream order (one device int; capture-safe, no memcpy node)
hipError_t launch_copy_i32(const int *src, int *dst, hipStream_t s);
hipError_t launch_fill_f32(float *p, int64_t n, float v, hipStream_t s);
hipError_t launch_fill_rows_f32(float *p, int64_t rows, int64_t cols, int64_t ld, float v,
                                hipStream_t s);

// gemm.hip -----------------------------------------------------------------
// dense dW with the batch reduction split over `splits` ranges of `chunk`
// (partials in ws, added in split order) when the output has few tiles
struct wgrad_split {
    int splits, chunk;
};
wgrad_split wgrad_plan(int N, int K, int B);
size_t wgrad_workspace_bytes(int N, int K, int B);
// ws (nullable) holds wgrad_workspace_bytes(); without it no split is made
hipError_t launch_wgrad_f32(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                            int64_t ldx, float *dW, int64_t ldw, void *ws, hipStream_t s);
// the same with operands rounded to bf16 (wgrad_bf16.hip)
hipError_t launch_wgrad_bf16(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                             int64_t ldx, float *dW, int64_t ldw, hipStream_t s);
// the same with operands split into bf16 hi + lo, three products (wgrad_bf16x3.hip)
hipError_t launch_wgrad_bf16x3(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                               int64_t ldx, float *dW, int64_t ldw, hipStream_t s);

// wgrad_prox.hip / the GEMMs' prox epilogue (prox_epilogue.hpp) ------------
struct prox_epi;
// columns per counted slab of the fp32 / split-bf16 GEMM with the prox
// epilogue at this shape (0: the fp32 product would split its reduction,
// which has no such epilogue)
int wgrad_f32_prox_slab(int N, int K, int B);
int wgrad_bf16x3_prox_slab(int N, int K, int B);
// dense_wgrad precision codes (the ABI's l1csr_precision)
constexpr int kPrecF32 = 0, kPrecBF16 = 1, kPrecBF16X3 = 2;
// Z = S_t(W - eta * dY.X^T) and P.counts, in one GEMM launch
hipError_t launch_wgrad_f32_prox(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                                 int64_t ldx, float *Z, int64_t ldz, const prox_epi &P, hipStream_t s);
hipError_t launch_wgrad_bf16x3_prox(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                                    int64_t ldx, float *Z, int64_t ldz, const prox_epi &P, hipStream_t s);
// the l1 update in two calls (wgrad_prox.hip):
//   launch_wgrad_prox: Z and the per-(row, 32-column word) nonzero counts
//     (counts [N][ceil(K / 32)]) from W's bitmap index (mask / pos); split_ws
//     holds wgrad_prox_split_bytes() (fp32 products that split their batch);
//   launch_counted_sums: the row totals of the counts and their totals per
//     block of 16-64 rows into ws (counted_ws_ints(N) ints);
//   launch_counted_row_ptr: row_ptr_out (row_ptr_out[N] = nnz') by a scan of
//     the row totals;
//   launch_counted_compact: col_out / val_out (< capacity), nnz' to d_nnz_out;
//     prefix_here (only where counted_prefix_in_compact(N)): the workgroups
//     add up each row's start from the totals and write row_ptr_out
//     themselves, else they read it (launch_counted_row_ptr first).
size_t word_counts_bytes(int N, int K);
size_t wgrad_prox_split_bytes(int N, int K, int B, int precision);
hipError_t launch_wgrad_prox(int N, int K, int B, const float *dY, int64_t ldy, const float *X,
                             int64_t ldx, int precision, const float *vals, const unsigned *mask, const int *pos,
                             float eta, double t, float *Z, int64_t ldz, int *counts, void *split_ws,
                             hipStream_t s);
size_t counted_ws_ints(int N);
bool counted_prefix_in_compact(int N);
hipError_t launch_counted_sums(int N, int K, const int *counts, int *ws, hipStream_t s);
hipError_t launch_counted_row_ptr(int N, const int *ws, int *row_ptr_out, hipStream_t s);
hipError_t launch_counted_compact(int N, int K, const float *Z, int64_t ldz, const int *counts, const int *ws,
                                  bool prefix_here, int *row_ptr_out, int *col_out, float *val_out,
                                  int64_t capacity, int *d_nnz_out, hipStream_t s);
// bitmap index of a CSR pattern: mask / pos [n_rows][ceil(n_cols / 32)]
hipError_t launch_bitmap(int n_rows, int n_cols, const int *ptr, const int *idx, unsigned *mask, int *pos,
                         hipStream_t s);
// sddmm.hip ----------------------------------------------------------------
// gv[p] = sum_b dY[row(p)][b] X[col(p)][b]; ws holds sddmm_workspace_bytes()
size_t sddmm_workspace_bytes(int n_rows, int n_cols, int64_t nnz, int B);
hipError_t launch_sddmm(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                        const float *dY, int64_t ldy, const float *X, int64_t ldx, int B, float *gv,
                        void *ws, hipStream_t s);

// prox.hip -----------------------------------------------------------------
// the fused prox kernels work on slabs of 1 << kProxSlabShift columns of a row
constexpr int kProxSlabShift = 11;
hipError_t launch_prox_dense(int n_rows, int n_cols, const int *ptr, const int *idx,
                             const float *vals, const float *G, int64_t ldg, float eta, double t,
                             float *Z, int64_t ldz, int *row_counts, hipStream_t s);
hipError_t launch_prox_csr(int64_t nnz, float *vals, const float *g, float eta, double t,
                           hipStream_t s);
// fused prox + recompression over row slabs (prox_slabs(n_cols) per row,
// numbered row-major): per-(row, slab) entry bounds of W, counts per slab;
// their exclusive scan off[] (n_rows * slabs + 1 entries) is the output
// layout; row_ptr[r] = off[r * slabs]; then the compacted output.  Scratch:
// prox_carve() splits prox_recompress_workspace_bytes() into counts, off and
// the bounds (256-byte aligned parts).
int prox_slabs(int n_cols);
struct prox_ws {
    int *counts, *off, *seg;
    size_t bytes;
};
prox_ws prox_carve(int n_rows, int n_cols, void *ws);
size_t prox_recompress_workspace_bytes(int n_rows, int n_cols);
hipError_t launch_prox_count(int n_rows, int n_cols, const int *ptr, const int *idx,
                             const float *vals, const float *G, int64_t ldg, float eta, double t,
                             int *seg, int *counts, hipStream_t s);
hipError_t launch_prox_row_ptr(int n_rows, int n_cols, const int *off, int *row_ptr, int *nnz_out,
                               hipStream_t s);
// (also writes row_ptr and *nnz_out, nullable, from off[])
hipError_t launch_prox_fill(int n_rows, int n_cols, const int *seg, const int *idx,
                            const float *vals, const float *G, int64_t ldg, float eta, double t,
                            const int *off, int *col_out, float *val_out, int64_t capacity,
                            int *row_ptr, int *nnz_out, hipStream_t s);

// prox_adaptive.hip --------------------------------------------------------
// Prox-RMSProp / Prox-ADAM parameters, prepared on the host in double
constexpr int kSolverRms = 1;
constexpr int kSolverAdam = 2;
struct adaptive_params {
    int solver;
    double eta, thr, eps;       // step, threshold eta*lambda, safeguard
    double beta1, beta2;        // decay rates (RMSProp: beta2 is its beta)
    double omb1, omb2;          // 1 - beta1, 1 - beta2
    double bc1, bc2;            // ADAM: 1 - beta^t; RMSProp: unused
};
// slab passes of the adaptive step (stages of one call)
enum {
    kStageCountWrite = 0,   // count the new weights per slab, store m', v'
    kStageCountKeep = 1,    // count only (state untouched)
    kStageFillStored = 2,   // compact, recomputing from the stored m', v'
    kStageFillWrite = 3,    // compact and store m', v'
    kStageDense = 4         // write Z and row counts, store m', v'
};
// seg and counts are the prox_carve() parts; the count and dense stages also
// compute seg.  Arguments a stage does not use may be null.
hipError_t launch_adaptive_slabs(int stage, int n_rows, int n_cols, const int *ptr, const int *idx,
                                 const float *vals, const float *G, int64_t ldg, float *M, float *V,
                                 int64_t lds, const adaptive_params &P, int *seg, int *counts,
                                 const int *off, int *col_out, float *val_out, int64_t capacity,
                                 int *row_ptr, int *nnz_out, float *Z, int64_t ldz, int *row_counts,
                                 hipStream_t s);
hipError_t launch_adaptive_csr(int64_t nnz, float *vals, const float *g, float *M, float *V,
                               const adaptive_params &P, hipStream_t s);

// recompress.hip -----------------------------------------------------------
hipError_t launch_count_rows(int n_rows, int n_cols, const float *Z, int64_t ldz, float t,
                             int *counts, hipStream_t s);
hipError_t launch_recompress_fill(int n_rows, int n_cols, const float *Z, int64_t ldz, float t,
                                  const int *row_ptr, int *col_idx, float *vals, int64_t capacity,
                                  hipStream_t s);
hipError_t launch_compact_count(int n_rows, const int *ptr, const float *vals, int *counts,
                                hipStream_t s);
// *status = L1CSR_OK or L1CSR_EBADCSR (canonical CSR check)
hipError_t launch_csr_validate(int n_rows, int n_cols, int64_t nnz, const int *ptr, const int *idx,
                               int *status, hipStream_t s);
hipError_t launch_compact_fill(int n_rows, const int *ptr, const int *idx, const float *vals,
                               const int *ptr_out, int *idx_out, float *vals_out, hipStream_t s);

// conv.hip -----------------------------------------------------------------
// convolution geometry: input channels C, map H x W, filter KH x KW, stride
// SH x SW, zero padding PH x PW
struct conv_geom {
    int C, H, W, KH, KW, SH, SW, PH, PW;
};
// output map size (floor); false if the geometry is invalid
bool conv_out_dims(const conv_geom &g, int *OH, int *OW);
hipError_t launch_conv_fwd(const conv_geom &g, int N, int B, const int *ptr, const int *idx,
                           const float *vals, const float *X, int64_t ldx, float *Y, int64_t ldy,
                           hipStream_t s);
hipError_t launch_conv_bwd_data(const conv_geom &g, int N, int B, const int *col_ptr, const int *row_idx,
                                const float *vals_t, const float *dY, int64_t ldy, float *dX, int64_t ldx,
                                hipStream_t s);
hipError_t launch_im2col(const conv_geom &g, int B, const float *X, int64_t ldx, float *Xc, int64_t ldc,
                         hipStream_t s);
hipError_t launch_maxpool_fwd(const conv_geom &g, int B, const float *X, int64_t ldx, float *Y, int64_t ldy,
                              hipStream_t s);

// glue.hip -----------------------------------------------------------------
hipError_t launch_relu_fwd(int64_t n, const float *x, float *y, hipStream_t s);
hipError_t launch_relu_bwd(int64_t n, const float *x, const float *dy, float *dx, hipStream_t s);
hipError_t launch_softmax_xent(int C, int B, const float *z, int64_t ld, const int *labels,
                               float *dz, float *loss, float *ws, hipStream_t s);

}  // namespace l1csr
