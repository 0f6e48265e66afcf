/*
 * l1csr — the data-parallel hot path of l1-regularised compressed learning
 * (S. Lee and J. Lee, "Compressed Learning of Deep Neural Networks for
 * OpenCL-Capable Embedded Systems", Appl. Sci. 9(8), 2019) on AMD Instinct
 * MI355X (gfx950).
 *
 * One training step of a layer whose N x K weight matrix W is kept in CSR:
 *   forward            Y  = W . X                 csr_spmm_fwd
 *   backward (data)    dX = W^T . dY              csr_spmm_bwd_t (+ csc_build)
 *   weight gradient    dW = dY . X^T  (l1 phase)  dense_wgrad
 *                      gv = (dY . X^T) on W's pattern (debiasing)  sddmm_masked_wgrad
 *   proximal step      Z  = S_t(W - eta*dW), t = eta*lambda        prox_l1_step
 *   recompression      Z -> CSR                   csr_recompress
 *   adaptive solvers   Prox-RMSProp / Prox-ADAM   prox_adaptive_step, prox_adaptive_recompress
 *   conv layers        direct sparse convolution  csr_conv_fwd, csr_conv_bwd_data, conv_im2col
 *
 * Conventions shared by every call
 *   - CSR: row_ptr[n_rows+1] (row_ptr[0] = 0, non-decreasing), col_idx[nnz]
 *     strictly increasing inside each row, vals[nnz]; int32 indices, float32
 *     values (Section 3.1 and Fig. 1(iii): ptr / indices / data).
 *   - Dense activations keep the batch index contiguous: X[K][B], Y[N][B],
 *     dY[N][B], dX[K][B], each with a leading dimension ld >= B (the paper's
 *     "internal_cols" of the row-major Dmat / result, Figs. 2-3).  Y = W.X is
 *     the transpose of the paper's X_T = X_B.W' (Section 3.2), the same numbers.
 *   - dW, Z are [N][K] row-major with leading dimension >= K.
 *   - Every pointer argument is DEVICE memory unless its comment says "host".
 *     All device buffers are owned and allocated by the caller; no call
 *     allocates or frees memory.  Scratch space is passed in as (ws, ws_bytes),
 *     sized by l1csr_workspace_bytes().
 *   - Every call only enqueues work on `stream` and returns without waiting,
 *     except csr_recompress with capacity < n_rows*n_cols (documented there).
 *   - Arguments are validated on the host before anything is launched:
 *     a null pointer, a negative size, ld < row length, a non-finite or
 *     negative eta/lambda, or a workspace that is too small returns
 *     L1CSR_EINVAL and launches nothing.  CSR well-formedness is a
 *     precondition, not checked by the hot calls.  A HIP launch error
 *     returns L1CSR_EHIP.  Values must be finite (precondition).
 *   - Calls on the same stream are ordered; calls that share output buffers on
 *     different streams race.
 */
#ifndef L1CSR_H
#define L1CSR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum l1csr_status {
    L1CSR_OK = 0,
    L1CSR_EINVAL = -1,       /* bad argument; nothing launched */
    L1CSR_ECAPACITY = -2,    /* output capacity too small (csr_recompress) */
    L1CSR_EBADCSR = -3,      /* malformed CSR (csr_validate, via its device status) */
    L1CSR_EHIP = -4,         /* a HIP runtime or launch error */
    L1CSR_EUNSUPPORTED = -5, /* valid but unsupported combination */
    L1CSR_ESCRATCH = -6      /* a no-allocation call needs more than its static scratch */
};

/* dense_wgrad operand precision */
enum l1csr_precision {
    L1CSR_F32 = 0,           /* fp32 operands, fp32 matrix cores: the 1e-4 contract */
    L1CSR_BF16 = 1,          /* operands rounded to bf16 (nearest even), exact products, fp32 sums */
    L1CSR_BF16X3 = 2         /* operands split into bf16 hi + lo, three exact products, fp32 sums */
};

/* prox_l1_step modes */
enum l1csr_prox_mode {
    L1CSR_PROX_DENSE = 0,    /* every one of the N*K weights, dense gradient */
    L1CSR_PROX_CSR = 1       /* W's stored entries only, gradient per entry  */
};

/* adaptive solvers of prox_adaptive_step / prox_adaptive_recompress */
enum l1csr_solver {
    L1CSR_SOLVER_RMSPROP = 1,  /* Prox-RMSProp, Algorithm 1 */
    L1CSR_SOLVER_ADAM = 2      /* Prox-ADAM, Algorithm 2    */
};

/* workspace queries (l1csr_workspace_bytes) */
enum l1csr_op {
    L1CSR_OP_CSC_BUILD = 1,
    L1CSR_OP_RECOMPRESS = 2,
    L1CSR_OP_SDDMM = 3,
    L1CSR_OP_SPMM = 4,
    L1CSR_OP_COMPACT = 5,
    L1CSR_OP_SOFTMAX_XENT = 6,
    L1CSR_OP_PROX_RECOMPRESS = 7,
    L1CSR_OP_DENSE_WGRAD = 8,
    L1CSR_OP_WGRAD_PROX = 9    /* dense_wgrad_prox, fp32 (other precisions need none) */
};

/* Human-readable name of a status code (static string, never NULL). */
const char *l1csr_status_str(int status);

/* Bytes of scratch that `op` needs for the given sizes (0 if none).  nnz is an
 * upper bound on the number of stored entries; B the batch size. */
size_t l1csr_workspace_bytes(int op, int32_t n_rows, int32_t n_cols, int64_t nnz, int32_t B);

/*
 * Pinned host memory that kernels can write directly, for small results the
 * host reads after the call (a d_nnz_out below, say), so that no copy has to
 * be queued behind the call: `bytes` bytes from hipHostMalloc (mapped, portable,
 * coherent); *host receives the host address, *dev the address kernels use.
 * The caller owns the memory and frees it with l1csr_host_free_mapped once
 * no queued work can still write it.  L1CSR_EINVAL for bytes == 0 or a NULL
 * out-pointer; L1CSR_EHIP if the runtime refuses (nothing allocated then).
 */
int l1csr_host_alloc_mapped(size_t bytes, void **host, void **dev);
int l1csr_host_free_mapped(void *host);

/*
 * Forward product, Section 3.2 "Forward: X_T <- X_B W'" (dense x compressed'),
 * in batch-contiguous layout:
 *     Y[i][b] = sum_{p = row_ptr[i]}^{row_ptr[i+1]-1} vals[p] * X[col_idx[p]][b]
 * for 0 <= i < n_rows, 0 <= b < B.  X is [n_cols][ldx], Y is [n_rows][ldy];
 * every Y[i][0..B) is written (an empty row gives zeros).  nnz is the number
 * of stored entries (row_ptr[n_rows]) or an upper bound on it (it only picks
 * the kernel).  ws (nullable) enables the LDS-tiled kernel and must then hold
 * l1csr_workspace_bytes(L1CSR_OP_SPMM, n_rows, n_cols, nnz, B) bytes; without
 * it a row-per-wave kernel runs.  Summation order (fp32 fused multiply-adds):
 * the row-per-wave kernel sums each Y entry in ascending p order; the tiled
 * kernel sums a row in ascending p order too unless it cuts the row into k
 * strided pieces (long rows: piece j takes p = row_ptr[i] + j, + j + k, ...),
 * each summed in ascending p order and the k partial sums then added in piece
 * order.  Either order is fixed by the operands alone, so results are
 * reproducible run to run and under any schedule.
 */
int csr_spmm_fwd(int32_t n_rows, int32_t n_cols, int64_t nnz,
                 const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                 const float *X, int64_t ldx, int32_t B,
                 float *Y, int64_t ldy, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * csr_spmm_fwd in two parts, for callers that can plan a product before its
 * dense operand exists (Section 3.2's products; the plan depends on W and B
 * only).  csr_spmm_plan enqueues the planning launches of the tiled kernel
 * (row pieces, their deal to the waves, the pair stream holding W's column
 * offsets and values) into the caller's buffer plan; csr_spmm_planned then
 * computes Y = W . X from it, the same bits as csr_spmm_fwd with the same
 * arguments.  Arguments as for csr_spmm_fwd; plan must hold
 * l1csr_workspace_bytes(L1CSR_OP_SPMM, n_rows, n_cols, nnz, B) bytes (0: the
 * product does not take the tiled path, plan may be NULL and csr_spmm_plan
 * enqueues nothing).  Preconditions: both calls get the same n_rows, n_cols,
 * nnz, row_ptr, col_idx, vals and B; W and plan are not modified in between;
 * csr_spmm_planned runs after csr_spmm_plan (same stream, or ordered by the
 * caller).  If X or Y is not 16-byte aligned with ldx, ldy and B multiples of
 * 4, csr_spmm_planned runs the row-per-wave kernel and does not read the plan.
 * A Y overlapping the plan is L1CSR_EINVAL.  For the backward product over a
 * CSC copy pass (n_cols, n_rows, nnz, col_ptr, row_idx, vals_t) as the CSR and
 * dY, dX as X, Y.
 */
int csr_spmm_plan(int32_t n_rows, int32_t n_cols, int64_t nnz,
                  const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                  int32_t B, void *plan, size_t plan_bytes, hipStream_t stream);
int csr_spmm_planned(int32_t n_rows, int32_t n_cols, int64_t nnz,
                     const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                     const float *X, int64_t ldx, int32_t B, float *Y, int64_t ldy,
                     const void *plan, size_t plan_bytes, hipStream_t stream);

/*
 * Column-major copy of W (CSC) for the backward product.  Section 3.2 notes
 * that the dense x compressed product reads W by columns and cannot be
 * coalesced unless such a column-wise copy is stored; this builds it:
 *     col_ptr[n_cols+1], row_idx[nnz], perm[nnz], vals_t[nnz]
 * with row_idx strictly increasing inside each column (the unique canonical
 * CSC), perm[q] = the CSR position of CSC entry q and vals_t[q] = vals[perm[q]].
 * It is built from W's bitmap index (csr_bitmap_build): mask / pos given by
 * the caller (both, e.g. shared with dense_wgrad_prox), or both NULL and the
 * call builds them in ws.  nnz is row_ptr[n_rows] or an upper bound on it.
 * Deterministic.  ws must hold
 * l1csr_workspace_bytes(L1CSR_OP_CSC_BUILD, n_rows, n_cols, nnz, 0) bytes.
 */
int csc_build(int32_t n_rows, int32_t n_cols, int64_t nnz,
              const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
              const uint32_t *mask, const int32_t *pos,
              int32_t *col_ptr, int32_t *row_idx, int32_t *perm, float *vals_t,
              void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Refresh the CSC values after an update of W's values only (debiasing keeps
 * the pattern, Section 2.4): vals_t[q] = vals[perm[q]] for 0 <= q < nnz', where
 * nnz' = col_ptr[n_cols] is read on the device and nnz is an upper bound on it
 * (it sizes the launch).
 */
int csc_update_vals(int32_t n_cols, int64_t nnz, const int32_t *col_ptr, const int32_t *perm,
                    const float *vals, float *vals_t, hipStream_t stream);

/*
 * Backward product for the data gradient, Section 3.2 "Backward:
 * dLoss/dX_B <- dLoss/dX_T W" (dense x compressed), batch-contiguous:
 *     dX[k][b] = sum_{p : col_idx[p] = k} vals[p] * dY[row(p)][b]
 * for 0 <= k < n_cols.  With a CSC copy (col_ptr, row_idx, vals_t from
 * csc_build, all non-NULL) this is the forward product of W^T: a gather in
 * ascending row order, reproducible; ws (nullable) as for csr_spmm_fwd with
 * the dimensions swapped, l1csr_workspace_bytes(L1CSR_OP_SPMM, n_cols, n_rows,
 * nnz, B).  With all three NULL the call scatters W's CSR with float atomics
 * instead (the summation order, and so the low bits, vary from run to run);
 * dX is zeroed first by the call.  dY is [n_rows][ldy], dX is [n_cols][ldx].
 */
int csr_spmm_bwd_t(int32_t n_rows, int32_t n_cols, int64_t nnz,
                   const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                   const int32_t *col_ptr, const int32_t *row_idx, const float *vals_t,
                   const float *dY, int64_t ldy, int32_t B,
                   float *dX, int64_t ldx, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Dense weight gradient of the l1 phase (the minibatch gradient that enters
 * the proximal step, Eq. (prox)):
 *     dW[i][k] = sum_{b < B} dY[i][b] * X[k][b]      (dW = dY . X^T)
 * dY [N][ldy], X [K][ldx], dW [N][ldw], ldw >= K.  No 1/B factor: dY carries
 * the loss scaling.  Inputs are fp32 in memory either way.
 * precision L1CSR_F32: fp32 matrix-core products and sums.
 * precision L1CSR_BF16: every dY and X element is rounded to bf16 (round to
 *   nearest even) before it is multiplied; products are exact and summed in
 *   fp32: each operand rounds by at most 2^-8 relative, so |dW - exact| <=
 *   (2^-7 + 2^-16) sum_b |dY X| plus the fp32 summation error:
 *   outside the fp32 accuracy contract, reported separately.
 * precision L1CSR_BF16X3: every dY and X element x is split into
 *   hi = bf16(x) and lo = bf16(x - hi) (nearest even; x - hi is exact), and
 *   each product is taken as hi_a hi_b + hi_a lo_b + lo_a hi_b on the bf16
 *   matrix cores, all exact, summed in fp32.  Per product the error is at most
 *   3 (1 + 2^-7) 2^-16 |ab| < 4.7e-5 |ab| (the dropped lo_a lo_b and the
 *   parts' rounding), so |dW - exact| <= 4.7e-5 sum_b |dY X| plus the fp32
 *   summation error: inside the 1e-4 contract, at about twice the speed of
 *   L1CSR_F32.
 * Any other precision value returns L1CSR_EINVAL.
 * ws (nullable) with l1csr_workspace_bytes(L1CSR_OP_DENSE_WGRAD, N, K, 0, B)
 * bytes lets an fp32 product with few 128 x 128 output tiles and a long batch
 * (conv filter banks over batch x positions) split its reduction into ranges
 * whose partial sums are added in a fixed order afterwards; the size is 0
 * when no split is planned.  Results are reproducible either way.
 */
int dense_wgrad(int32_t N, int32_t K, int32_t B,
                const float *dY, int64_t ldy, const float *X, int64_t ldx,
                float *dW, int64_t ldw, int precision, void *ws, size_t ws_bytes,
                hipStream_t stream);

/*
 * Weight gradient of the debiasing phase (Section 2.4: retrain without the
 * regulariser with the zero weights excluded), i.e. the dense gradient sampled
 * on W's pattern:
 *     gv[p] = sum_{b < B} dY[row(p)][b] * X[col_idx[p]][b],  0 <= p < nnz.
 * gv has nnz entries (host nnz = row_ptr[n_rows]).  ws must hold
 * l1csr_workspace_bytes(L1CSR_OP_SDDMM, n_rows, n_cols, nnz, B) bytes.
 */
int sddmm_masked_wgrad(int32_t n_rows, int32_t n_cols, int64_t nnz,
                       const int32_t *row_ptr, const int32_t *col_idx,
                       const float *dY, int64_t ldy, const float *X, int64_t ldx, int32_t B,
                       float *gv, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Minibatch proximal gradient step, Eq. (prox), with the soft-threshold
 * closed form of Section 2.2 and the elementwise kernel of Fig. 4:
 *     S_t(z) = sgn(z) * max(|z| - t, 0),   t = eta * lambda,
 *     z = w - eta * g.
 * The arithmetic is done in double (the precision of the paper's kernels):
 * eta*g and eta*lambda are exact in double, z rounds once, S_t(z) rounds once
 * more to float.  Zero results are +0.0.
 *
 * mode L1CSR_PROX_DENSE: g = G[i][k] ([n_rows][ldg], ldg >= n_cols), w = the
 *   CSR value at (i, k) or 0 where W has no entry (all N*K weights take part,
 *   so zero weights can become nonzero).  Writes Z[i][k] ([n_rows][ldz]; Z may
 *   be the same buffer as G with ldz == ldg) and, if row_counts is not NULL,
 *   row_counts[i] = number of nonzero Z[i][.].  vals is read only.
 * mode L1CSR_PROX_CSR: g = G[p] (one gradient per stored entry, as produced by
 *   sddmm_masked_wgrad), vals[p] <- S_t(vals[p] - eta*G[p]) in place for
 *   0 <= p < nnz; the pattern is unchanged (entries that become 0 stay stored;
 *   csr_compact drops them).  lambda = 0 is plain SGD (debiasing).  Z,
 *   row_counts, ldg, ldz are ignored.
 */
int prox_l1_step(int mode, int32_t n_rows, int32_t n_cols, int64_t nnz,
                 const int32_t *row_ptr, const int32_t *col_idx, float *vals,
                 const float *G, int64_t ldg, float eta, float lambda,
                 float *Z, int64_t ldz, int32_t *row_counts, hipStream_t stream);

/*
 * Dense -> CSR (Section 3.1: store only the nonzero weights).  Keeps the
 * entries with |Z[i][k]| > t in row-major order (t = 0 after prox_l1_step) and
 * writes the canonical CSR: row_ptr_out[n_rows+1], col_idx_out[nnz'],
 * vals_out[nnz'].  row_counts (nullable) are the per-row counts prox_l1_step
 * produced for the same Z and t = 0; when NULL they are recomputed.
 * d_nnz_out (nullable; device memory or l1csr_host_alloc_mapped's *dev)
 * receives nnz' from the call's kernels, in both capacity modes below (so a
 * mapped word is written in stream order even when *h_nnz_required already
 * gives the count on the host).
 *   capacity >= n_rows*n_cols: never overflows and never waits (hot path).
 *   capacity <  n_rows*n_cols: the call counts first, waits for the stream,
 *     and returns L1CSR_ECAPACITY with *h_nnz_required (host, nullable) = nnz'
 *     if nnz' > capacity (row_ptr_out is then valid, col/vals untouched);
 *     otherwise it fills and sets *h_nnz_required = nnz'.
 * ws must hold l1csr_workspace_bytes(L1CSR_OP_RECOMPRESS, n_rows, n_cols, 0, 0).
 */
int csr_recompress(int32_t n_rows, int32_t n_cols, const float *Z, int64_t ldz, float t,
                   const int32_t *row_counts,
                   int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                   int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                   void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * prox_l1_step (dense mode) followed by csr_recompress (t = 0) in one call,
 * without materialising Z: the l1-phase weight update of Eq. (prox) from the
 * CSR weights W and the dense gradient G straight to the new CSR W'.  The
 * output is bit-identical to the two calls.  G is read twice (a counting pass
 * and a filling pass); row_ptr_out, col_idx_out, vals_out, capacity,
 * d_nnz_out and h_nnz_required behave as in csr_recompress.  The output arrays
 * must not overlap W's arrays, G or one another (L1CSR_EINVAL).  ws as
 * l1csr_workspace_bytes(L1CSR_OP_PROX_RECOMPRESS, n_rows, n_cols, nnz, 0).
 */
int prox_l1_recompress(int32_t n_rows, int32_t n_cols, int64_t nnz,
                       const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                       const float *G, int64_t ldg, float eta, float lambda,
                       int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                       int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                       void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * The l1-phase weight update of Eq. (prox) with the layer's minibatch
 * gradient, without storing the gradient:
 *     dW = dY . X^T                      (as dense_wgrad with `precision`)
 *     Z  = S_t(W - eta * dW),  t = eta * lambda   (as prox_l1_step, dense mode)
 * The GEMM's epilogue applies the soft threshold to its own result, reading W
 * through its bitmap index (csr_bitmap_build: mask, pos), and also writes
 * word_counts[i][w] = the number of nonzero Z[i][32w .. 32w + 32), the input
 * of csr_recompress_counted (so the recompression reads Z once and never W).
 * Z is bit-identical to dense_wgrad + prox_l1_step.
 * dY [N][ldy], X [K][ldx], W (N x K CSR with nnz entries), mask / pos
 * [ceil(K/32)][N] (read), Z [N][ldz] (ldz >= K) and word_counts
 * [N][ceil(K/32)] (written); the outputs must be disjoint from each other
 * and from every input (L1CSR_EINVAL).  ws as
 * l1csr_workspace_bytes(L1CSR_OP_WGRAD_PROX, N, K, nnz, B) for fp32 (0 unless
 * the product splits its reduction: few output tiles, a long batch).
 */
int dense_wgrad_prox(int32_t N, int32_t K, int32_t B,
                     const float *dY, int64_t ldy, const float *X, int64_t ldx, int precision,
                     int64_t nnz, const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                     const uint32_t *mask, const int32_t *pos, float eta, float lambda,
                     float *Z, int64_t ldz, int32_t *word_counts, void *ws, size_t ws_bytes,
                     hipStream_t stream);

/*
 * Dense -> CSR (Section 3.1) from the per-word nonzero counts that
 * dense_wgrad_prox wrote with Z: keeps the nonzero Z entries (|Z| > 0) in
 * row-major order, bit-identical to csr_recompress(Z, t = 0).  Row pointers
 * come from the counts (row sums, then their prefix sums), so Z is read once:
 * with capacity >= n_rows * n_cols and n_rows <= 16384 the compaction adds up
 * each row's start itself from per-row and per-block (16-64 rows) totals (two launches,
 * no host synchronisation); otherwise a scan writes row_ptr_out first.
 * row_ptr_out [n_rows+1], col_idx_out / vals_out [capacity]; capacity,
 * d_nnz_out and h_nnz_required behave as in csr_recompress.  The outputs
 * must not overlap each other, Z, the counts or ws.  ws holds
 * l1csr_workspace_bytes(L1CSR_OP_RECOMPRESS, n_rows, n_cols, 0, 0) bytes.
 */
int csr_recompress_counted(int32_t n_rows, int32_t n_cols, const float *Z, int64_t ldz,
                           const int32_t *word_counts, int32_t *row_ptr_out, int32_t *col_idx_out,
                           float *vals_out, int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                           void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Bitmap index of W's pattern (the CSR of Section 3.1 seen by 32-column
 * words), read by dense_wgrad_prox to find w_ik for every (i, k):
 *     mask[w][i] bit c = 1 iff W stores (i, 32w + c)
 *     pos[w][i]  = CSR position of row i's first entry with column >= 32w
 *                  (row_ptr[i + 1] if there is none)
 * for 0 <= w < ceil(n_cols / 32), word-major: both
 * [ceil(n_cols / 32)][n_rows], caller-owned, disjoint.  Deterministic; depends
 * only on the pattern (also the input of csc_build).
 */
int csr_bitmap_build(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                     const int32_t *col_idx, uint32_t *mask, int32_t *pos, hipStream_t stream);

/*
 * prox_l1_recompress for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments without (ws, ws_bytes), the same kernels and bit-identical
 * results.  Its scratch (per-slab entry bounds, counts and offsets,
 * l1csr_workspace_bytes(L1CSR_OP_PROX_RECOMPRESS, n_rows, n_cols, nnz, 0)
 * bytes) lives in a static device array of L1CSR_NOALLOC_SCRATCH_BYTES
 * (16 MiB) that each GPU the library runs on holds until the process ends;
 * a larger need returns L1CSR_ESCRATCH before anything is launched.  The
 * call allocates and frees nothing.  Every call of this entry point on one
 * GPU shares that GPU's array (the last call's contents stay in it; nothing
 * in it needs to start at zero), so such calls that overlap in time on one
 * GPU, on different streams or from different threads, race: the caller
 * orders them.  The first call on a device looks up the array's device
 * address (a runtime call that does not enqueue work).
 */
#define L1CSR_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int prox_l1_recompress_noalloc(int32_t n_rows, int32_t n_cols, int64_t nnz,
                               const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                               const float *G, int64_t ldg, float eta, float lambda,
                               int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                               int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                               hipStream_t stream);

/*
 * Adaptive proximal steps: Prox-RMSProp (Algorithm 1) and Prox-ADAM
 * (Algorithm 2), Section 2.3.  Both keep the prox of eta*lambda*||.||_1 of
 * Eq. (prox) and precondition the minibatch gradient g with per-weight state:
 *     v' = beta2*v + (1 - beta2)*g*g                     (both; RMSProp's beta)
 *     m' = beta1*m + (1 - beta1)*g                       (ADAM only)
 *     u  = g / (sqrt(v') + eps)                                      (RMSProp)
 *     u  = (m'/(1 - beta1^t)) / (sqrt(v'/(1 - beta2^t)) + eps)       (ADAM)
 *     w' = S_t(w - eta*u),   t_thr = eta*lambda,  S_t as in prox_l1_step.
 * Arithmetic in double: each moment update is one fma rounded to float and
 * stored; u is computed from the stored floats; w - eta*u rounds once (fma)
 * and S_t once more to float; zero results are +0.0.  beta^t is pow() in
 * double on the host.  Hyper-parameters: eta > 0, lambda >= 0, eps > 0 (all
 * finite), 0 <= beta2 < 1; ADAM also needs 0 <= beta1 < 1 and t >= 1 (the
 * step number, counted from 1); RMSProp ignores beta1, t and m (may be NULL).
 * A value out of range returns L1CSR_EINVAL.  The state arrays start at zero
 * (Algorithms 1-2 initialise m and v to 0) and are owned by the caller.
 *
 * prox_adaptive_step, mode L1CSR_PROX_DENSE: every one of the N*K weights
 *   (w = W's value or 0 where W has no entry), g = G[i][k] ([n_rows][ldg]);
 *   the states m, v are [n_rows][lds] (lds >= n_cols) and are updated in
 *   place; writes Z[i][k] ([n_rows][ldz]; Z may be G itself with ldz == ldg,
 *   but must not overlap m or v) and, if row_counts is not NULL, row_counts[i]
 *   = number of nonzero Z[i][.].  ws must hold
 *   l1csr_workspace_bytes(L1CSR_OP_PROX_RECOMPRESS, n_rows, n_cols, nnz, 0).
 * prox_adaptive_step, mode L1CSR_PROX_CSR: W's stored entries only, with one
 *   gradient G[p] and one state entry m[p], v[p] per stored weight;
 *   vals[p] is updated in place for 0 <= p < nnz and the pattern is kept
 *   (lambda = 0: the debiasing phase of Section 2.4 with an adaptive solver).
 *   ldg, lds, Z, ldz, row_counts and ws are ignored.
 * G, m and v must not overlap one another in either mode.
 */
int prox_adaptive_step(int mode, int solver, int32_t n_rows, int32_t n_cols, int64_t nnz,
                       const int32_t *row_ptr, const int32_t *col_idx, float *vals,
                       const float *G, int64_t ldg, float *m, float *v, int64_t lds,
                       float eta, float lambda, float eps, float beta1, float beta2, int64_t t,
                       float *Z, int64_t ldz, int32_t *row_counts,
                       void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * prox_adaptive_step (dense mode) followed by csr_recompress (t = 0) in one
 * call, without materialising Z: the l1-phase update of Algorithm 1 or 2 from
 * the CSR weights W, the dense gradient G and the dense states m, v straight
 * to the new CSR W'.  m and v are updated in place exactly as by
 * prox_adaptive_step; the output is bit-identical to the two calls.
 * row_ptr_out, col_idx_out, vals_out, capacity, d_nnz_out and h_nnz_required
 * behave as in prox_l1_recompress; when the call returns L1CSR_ECAPACITY it
 * has left m and v unchanged.  With capacity >= n_rows*n_cols (no wait) G and
 * the states are read in a counting pass that stores m', v', and m', v' (ADAM)
 * or G, v' (RMSProp) are read again by the filling pass.  The output arrays
 * must not overlap W's arrays, G, m, v or one another (L1CSR_EINVAL).  ws as
 * l1csr_workspace_bytes(L1CSR_OP_PROX_RECOMPRESS, n_rows, n_cols, nnz, 0).
 */
int prox_adaptive_recompress(int solver, int32_t n_rows, int32_t n_cols, int64_t nnz,
                             const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                             const float *G, int64_t ldg, float *m, float *v, int64_t lds,
                             float eta, float lambda, float eps, float beta1, float beta2, int64_t t,
                             int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                             int64_t capacity, int32_t *d_nnz_out, int64_t *h_nnz_required,
                             void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * CSR -> CSR without its stored zeros (after a support-restricted prox step in
 * CSR mode).  Out of place: the output arrays must not overlap the input ones
 * and hold at least nnz entries.  d_nnz_out (nullable, device) receives the new
 * count.  ws as l1csr_workspace_bytes(L1CSR_OP_COMPACT, n_rows, 0, nnz, 0).
 */
int csr_compact(int32_t n_rows, int64_t nnz,
                const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out,
                int32_t *d_nnz_out, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * CSR well-formedness check (the canonical form of Section 3.1 / Fig. 1 that
 * every other call assumes): row_ptr[0] = 0, row_ptr non-decreasing,
 * row_ptr[n_rows] = nnz, 0 <= col_idx < n_cols and strictly increasing inside
 * each row.  Writes L1CSR_OK or L1CSR_EBADCSR to *d_status (one device int32)
 * in stream order; the host return value only reports argument or launch
 * errors.  Reads only row_ptr[0 .. n_rows] and col_idx[0 .. nnz), whatever
 * they hold.  Not used by the hot calls.
 */
int csr_validate(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *row_ptr,
                 const int32_t *col_idx, int32_t *d_status, hipStream_t stream);

/*
 * Convolution layers with CSR filter banks (the conv rows of Tables A1-A4; in
 * Caffe, which the method is built on, a convolution is the product of
 * Section 3.2 with the im2col-lowered input).  Shared conventions:
 *   - geom (HOST memory, 9 int32): C, H, W, KH, KW, SH, SW, PH, PW = input
 *     channels, map height and width, filter height and width, stride, zero
 *     padding.  Output maps OH = (H + 2 PH - KH)/SH + 1, OW likewise (floor).
 *     An invalid geometry (a size < 1, negative padding, a filter larger than
 *     the padded map, more than 1024 filter positions KH*KW) returns
 *     L1CSR_EINVAL.
 *   - Maps are batch-contiguous matrices like every other activation here:
 *     X[(c*H + h)*W + w][b] with leading dimension ldx >= B; outputs
 *     Y[(co*OH + oh)*OW + ow][b].
 *   - The filter bank is an n_out x (C*KH*KW) CSR matrix, column
 *     (ci*KH + kh)*KW + kw (Caffe's im2col row order); cross-correlation, no
 *     flip.
 *
 * csr_conv_fwd: the forward product computed directly on the maps,
 *     Y[(co,oh,ow)][b] = sum_{p in row co} vals[p] * X[(ci, oh*SH-PH+kh, ow*SW-PW+kw)][b]
 *   over the entries whose input position lies inside the map (padding
 *   contributes zero), summed in CSR order by one thread per output element.
 *   Equal to csr_spmm_fwd on conv_im2col(X) without forming the lowered
 *   operand.
 * csr_conv_bwd_data: the backward product for the input maps (the adjoint of
 *   csr_conv_fwd), from the CSC copy of the filter bank (csc_build with
 *   n_rows = n_out, n_cols = C*KH*KW):
 *     dX[(ci,ih,iw)][b] = sum over the entries (co; ci,kh,kw) and the output
 *     positions with oh*SH-PH+kh = ih, ow*SW-PW+kw = iw of w * dY[(co,oh,ow)][b],
 *   summed by one thread per element in (kh, kw, CSC) order, reproducible.
 * conv_im2col: the lowered input, Xcol[(ci*KH + kh)*KW + kw][(oh*OW + ow)*B + b]
 *   (0 in the padding), Xcol [C*KH*KW][ldc], ldc >= OH*OW*B.  With dY
 *   stored with ldy == B, dY is the [n_out][OH*OW*B] matrix of the lowered
 *   product, so dense_wgrad(dY, Xcol) and sddmm_masked_wgrad(W, dY, Xcol) give
 *   the filter gradient of the l1 and the debiasing phase.
 * l1csr_maxpool_fwd: max over KH x KW windows with stride SH x SW (the
 *   subsampling layers of LeNet-5), Y[(c,oh,ow)][b]; geom's padding must be 0
 *   (else L1CSR_EUNSUPPORTED).  Values must be finite.
 */
int csr_conv_fwd(const int32_t *geom, int32_t n_out, int64_t nnz,
                 const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                 const float *X, int64_t ldx, int32_t B, float *Y, int64_t ldy, hipStream_t stream);
int csr_conv_bwd_data(const int32_t *geom, int32_t n_out, int64_t nnz,
                      const int32_t *col_ptr, const int32_t *row_idx, const float *vals_t,
                      const float *dY, int64_t ldy, int32_t B, float *dX, int64_t ldx,
                      hipStream_t stream);
int conv_im2col(const int32_t *geom, const float *X, int64_t ldx, int32_t B,
                float *Xcol, int64_t ldc, hipStream_t stream);
int l1csr_maxpool_fwd(const int32_t *geom, const float *X, int64_t ldx, int32_t B,
                      float *Y, int64_t ldy, hipStream_t stream);

/*
 * Layer glue of the fully connected ReLU networks the method trains (their
 * He initialisation, Section 4, targets ReLU units).  n elements, any layout.
 *   relu_fwd: y = x > 0 ? x : +0
 *   relu_bwd: dx = x > 0 ? dy : +0      (x is the pre-activation)
 */
int l1csr_relu_fwd(int64_t n, const float *x, float *y, hipStream_t stream);
int l1csr_relu_bwd(int64_t n, const float *x, const float *dy, float *dx, hipStream_t stream);

/*
 * Mean softmax cross-entropy over the batch for logits[C][ld] (class-major,
 * batch contiguous) and labels[B] in [0, C) (device int32):
 *   loss = (1/B) sum_b ( log sum_c exp(z_cb) - z_{label_b, b} )   -> *loss (device)
 *   dlogits[c][b] = (softmax(z_.b)_c - [c == label_b]) / B        ([C][ld])
 * A label outside [0, C) is a precondition violation (its column is zeroed).
 * ws as l1csr_workspace_bytes(L1CSR_OP_SOFTMAX_XENT, C, 0, 0, B).
 */
int l1csr_softmax_xent(int32_t C, int32_t B, const float *logits, int64_t ld,
                       const int32_t *labels, float *dlogits, float *loss,
                       void *ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* L1CSR_H */
