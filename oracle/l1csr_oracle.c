/*
 * l1csr oracle — plain CPU definitions of every operation on the hot path of
 * l1-regularised compressed learning (Lee & Lee, "Compressed Learning of Deep
 * Neural Networks for OpenCL-Capable Embedded Systems", Appl. Sci. 2019).
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load this library.
 * It shares no code, header or table with the HIP implementation.
 *
 * Conventions (the same ones the library's public header documents):
 *   - W is an N x K matrix in CSR: row_ptr[N+1], col_idx[nnz] (strictly
 *     increasing inside a row), vals[nnz]; indices are int32.
 *   - Dense operands keep the batch index contiguous: X[K][B], Y[N][B],
 *     dY[N][B], dX[K][B] with leading dimensions ld* >= B; dW, Z are [N][K].
 *     Y = W.X is the transpose of the paper's X_T = X_B.W' (Section 3.2).
 *   - Every reduction accumulates in double, in the order stated next to it,
 *     and rounds once to float at the end.
 *   - Built with -ffp-contract=off so that no product is fused silently.
 *
 * Return value of every int function: 0 on success, negative on bad
 * arguments (-1) or insufficient output capacity (-2).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ECAPACITY (-2)

int orc_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------
 * Forward product (Section 3.2, "Forward: X_T <- X_B W'", dense x compressed').
 * In batch-contiguous layout:  Y[i][b] = sum_{p in row i} vals[p] * X[col[p]][b].
 * Summation order: p ascending.
 * ---------------------------------------------------------------------- */
int orc_spmm_fwd(int32_t N, int32_t K, int32_t B,
                 const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                 const float *X, int64_t ldx, float *Y, int64_t ldy) {
    if (N < 0 || K < 0 || B < 0 || ldx < B || ldy < B) return ORC_EINVAL;
    #pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)(B > 0 ? B : 1));
        #pragma omp for schedule(dynamic, 16)
        for (int32_t i = 0; i < N; ++i) {
            for (int32_t b = 0; b < B; ++b) acc[b] = 0.0;
            for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
                const double w = (double)vals[p];
                const float *xr = X + (int64_t)col_idx[p] * ldx;
                for (int32_t b = 0; b < B; ++b) acc[b] += w * (double)xr[b];
            }
            for (int32_t b = 0; b < B; ++b) Y[(int64_t)i * ldy + b] = (float)acc[b];
        }
        free(acc);
    }
    (void)K;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Backward product for the data gradient (Section 3.2, "Backward:
 * dLoss/dX_B <- dLoss/dX_T W", dense x compressed).  In batch-contiguous layout:
 *   dX[k][b] = sum_{p : col[p] = k} vals[p] * dY[row(p)][b].
 * Written as the scatter over W's nonzeros in CSR order (row ascending, then
 * p ascending), which is the definition read directly off the CSR arrays.
 * Threads split the batch index only, so every sum keeps that order.
 * ---------------------------------------------------------------------- */
int orc_spmm_bwd_t(int32_t N, int32_t K, int32_t B,
                   const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                   const float *dY, int64_t ldy, float *dX, int64_t ldx) {
    if (N < 0 || K < 0 || B < 0 || ldx < B || ldy < B) return ORC_EINVAL;
    const int32_t CH = 32; /* batch columns per task */
    const int32_t nchunks = (B + CH - 1) / CH;
    #pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * ((size_t)K * CH + 1));
        #pragma omp for schedule(dynamic, 1)
        for (int32_t c = 0; c < nchunks; ++c) {
            const int32_t b0 = c * CH;
            const int32_t nb = (B - b0) < CH ? (B - b0) : CH;
            memset(acc, 0, sizeof(double) * (size_t)K * CH);
            for (int32_t i = 0; i < N; ++i)
                for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
                    const double w = (double)vals[p];
                    const float *dyr = dY + (int64_t)i * ldy + b0;
                    double *a = acc + (size_t)col_idx[p] * CH;
                    for (int32_t j = 0; j < nb; ++j) a[j] += w * (double)dyr[j];
                }
            for (int32_t k = 0; k < K; ++k)
                for (int32_t j = 0; j < nb; ++j)
                    dX[(int64_t)k * ldx + b0 + j] = (float)acc[(size_t)k * CH + j];
        }
        free(acc);
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Dense weight gradient of the l1 phase (the gradient that enters the
 * minibatch proximal step, Eq. (prox); the paper leaves its computation to
 * the dense framework):  dW[i][k] = sum_b dY[i][b] * X[k][b], b ascending.
 * No 1/|B| factor: the caller's dY already carries the loss scaling.
 * ---------------------------------------------------------------------- */
int orc_dense_wgrad(int32_t N, int32_t K, int32_t B,
                    const float *dY, int64_t ldy, const float *X, int64_t ldx,
                    float *dW, int64_t ldw) {
    if (N < 0 || K < 0 || B < 0 || ldx < B || ldy < B || ldw < K) return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 4)
    for (int32_t i = 0; i < N; ++i) {
        const float *dyr = dY + (int64_t)i * ldy;
        for (int32_t k = 0; k < K; ++k) {
            const float *xr = X + (int64_t)k * ldx;
            double acc = 0.0;
            for (int32_t b = 0; b < B; ++b) acc += (double)dyr[b] * (double)xr[b];
            dW[(int64_t)i * ldw + k] = (float)acc;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * bf16 rounding, written from its definition: keep 8 significant bits
 * (1 implicit + 7 stored), round to nearest, ties to even.  frexp gives
 * x = m 2^e with 0.5 <= |m| < 1, so m 2^8 holds the 8 kept bits in its integer
 * part; nearbyint rounds it in the default (nearest-even) mode.  Finite inputs
 * whose exponent is in the normal range of float (every input here).
 * ---------------------------------------------------------------------- */
float orc_bf16_round(float x) {
    if (x == 0.0f) return x;
    int e;
    const double m = frexp((double)x, &e);
    return (float)ldexp(nearbyint(ldexp(m, 8)), e - 8);
}

/* Dense weight gradient with bf16 operands (the reduced-precision variant of
 * the l1-phase gradient): every element of dY and X is rounded to bf16 first,
 * then dW[i][k] = sum_b bf16(dY[i][b]) * bf16(X[k][b]) in double, b ascending. */
int orc_dense_wgrad_bf16(int32_t N, int32_t K, int32_t B,
                         const float *dY, int64_t ldy, const float *X, int64_t ldx,
                         float *dW, int64_t ldw) {
    if (N < 0 || K < 0 || B < 0 || ldx < B || ldy < B || ldw < K) return ORC_EINVAL;
    float *ry = (float *)malloc(sizeof(float) * ((size_t)N * B + 1));
    float *rx = (float *)malloc(sizeof(float) * ((size_t)K * B + 1));
    if (!ry || !rx) {
        free(ry);
        free(rx);
        return ORC_EINVAL;
    }
    for (int32_t i = 0; i < N; ++i)
        for (int32_t b = 0; b < B; ++b) ry[(int64_t)i * B + b] = orc_bf16_round(dY[(int64_t)i * ldy + b]);
    for (int32_t k = 0; k < K; ++k)
        for (int32_t b = 0; b < B; ++b) rx[(int64_t)k * B + b] = orc_bf16_round(X[(int64_t)k * ldx + b]);
    const int rc = orc_dense_wgrad(N, K, B, ry, B, rx, B, dW, ldw);
    free(ry);
    free(rx);
    return rc;
}

/* Dense weight gradient with each operand split into two bf16 parts:
 * hi = bf16(x), lo = bf16(x - hi) (x - hi is exact in float), and each product
 * taken as hi_a hi_b + hi_a lo_b + lo_a hi_b (the lo_a lo_b term is dropped);
 * every product is exact, the three are added in that order and summed over
 * b ascending in double. */
int orc_dense_wgrad_bf16x3(int32_t N, int32_t K, int32_t B,
                           const float *dY, int64_t ldy, const float *X, int64_t ldx,
                           float *dW, int64_t ldw) {
    if (N < 0 || K < 0 || B < 0 || ldx < B || ldy < B || ldw < K) return ORC_EINVAL;
    const size_t ny = (size_t)N * B + 1, nx = (size_t)K * B + 1;
    float *hy = (float *)malloc(sizeof(float) * ny), *ly = (float *)malloc(sizeof(float) * ny);
    float *hx = (float *)malloc(sizeof(float) * nx), *lx = (float *)malloc(sizeof(float) * nx);
    if (!hy || !ly || !hx || !lx) {
        free(hy);
        free(ly);
        free(hx);
        free(lx);
        return ORC_EINVAL;
    }
    for (int32_t i = 0; i < N; ++i)
        for (int32_t b = 0; b < B; ++b) {
            const float v = dY[(int64_t)i * ldy + b];
            hy[(int64_t)i * B + b] = orc_bf16_round(v);
            ly[(int64_t)i * B + b] = orc_bf16_round(v - hy[(int64_t)i * B + b]);
        }
    for (int32_t k = 0; k < K; ++k)
        for (int32_t b = 0; b < B; ++b) {
            const float v = X[(int64_t)k * ldx + b];
            hx[(int64_t)k * B + b] = orc_bf16_round(v);
            lx[(int64_t)k * B + b] = orc_bf16_round(v - hx[(int64_t)k * B + b]);
        }
    for (int32_t i = 0; i < N; ++i)
        for (int32_t k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int32_t b = 0; b < B; ++b) {
                const double ha = hy[(int64_t)i * B + b], la = ly[(int64_t)i * B + b];
                const double hb = hx[(int64_t)k * B + b], lb = lx[(int64_t)k * B + b];
                acc += ha * hb + ha * lb + la * hb;
            }
            dW[(int64_t)i * ldw + k] = (float)acc;
        }
    free(hy);
    free(ly);
    free(hx);
    free(lx);
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Weight gradient of the debiasing phase (Section 2.4: retraining without the
 * regulariser, zero-valued weights excluded from training).  The gradient is
 * the dense one sampled on W's pattern:
 *   gv[p] = sum_b dY[row(p)][b] * X[col[p]][b], b ascending.
 * ---------------------------------------------------------------------- */
int orc_sddmm(int32_t N, int32_t K, int32_t B,
              const int32_t *row_ptr, const int32_t *col_idx,
              const float *dY, int64_t ldy, const float *X, int64_t ldx, float *gv) {
    if (N < 0 || K < 0 || B < 0 || ldx < B || ldy < B) return ORC_EINVAL;
    #pragma omp parallel for schedule(dynamic, 4)
    for (int32_t i = 0; i < N; ++i) {
        const float *dyr = dY + (int64_t)i * ldy;
        for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            const float *xr = X + (int64_t)col_idx[p] * ldx;
            double acc = 0.0;
            for (int32_t b = 0; b < B; ++b) acc += (double)dyr[b] * (double)xr[b];
            gv[p] = (float)acc;
        }
    }
    (void)K;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Soft-thresholding operator: the closed form of prox of t*||.||_1
 * (Section 2.2):  [prox(z)]_i = sgn(z_i) * max(|z_i| - t, 0).
 * Evaluated in double, the precision of the paper's prox kernel (Fig. 4).
 * The "+ 0.0" turns the -0.0 that sgn(z) * 0 gives for negative z into the
 * canonical +0.0; it does not change any nonzero result.
 * ---------------------------------------------------------------------- */
static double sgn(double z) { return (double)((z > 0.0) - (z < 0.0)); }

double orc_soft_threshold(double z, double t) {
    return sgn(z) * fmax(fabs(z) - t, 0.0) + 0.0;
}

/* The prox step's threshold: eta * lambda (Eq. (prox): prox of eta*Psi with
 * Psi = lambda*||w||_1; Fig. 4 uses lambda*learning_rate).  The product of two
 * floats is exact in double. */
double orc_threshold(float eta, float lambda) { return (double)eta * (double)lambda; }

/* The prox step's argument A = w - eta*g (Eq. (prox); Fig. 4's caption says A
 * holds w^k - eta G(w^k)).  eta*g is exact in double, so this rounds once. */
double orc_prox_arg(float w, float g, float eta) { return (double)w - (double)eta * (double)g; }

/* ------------------------------------------------------------------------
 * Minibatch proximal gradient step on the dense A of Fig. 4 (Eq. (prox)):
 *   Z[i][k] = float( S_t( w_ik - eta * G[i][k] ) ),  t = eta * lambda,
 * with w_ik = 0 where W has no entry (every one of the N*K weights takes part,
 * so a zero weight may become nonzero again).  row_counts[i] (optional)
 * receives the number of nonzero Z[i][k].
 * ---------------------------------------------------------------------- */
int orc_prox_dense(int32_t N, int32_t K,
                   const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                   const float *G, int64_t ldg, float eta, float lambda,
                   float *Z, int64_t ldz, int32_t *row_counts) {
    if (N < 0 || K < 0 || ldg < K || ldz < K) return ORC_EINVAL;
    const double t = orc_threshold(eta, lambda);
    #pragma omp parallel
    {
        float *wrow = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
        #pragma omp for schedule(dynamic, 8)
        for (int32_t i = 0; i < N; ++i) {
            for (int32_t k = 0; k < K; ++k) wrow[k] = 0.0f;
            for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) wrow[col_idx[p]] = vals[p];
            int32_t cnt = 0;
            for (int32_t k = 0; k < K; ++k) {
                const double z = orc_prox_arg(wrow[k], G[(int64_t)i * ldg + k], eta);
                const float s = (float)orc_soft_threshold(z, t);
                Z[(int64_t)i * ldz + k] = s;
                cnt += (s != 0.0f);
            }
            if (row_counts) row_counts[i] = cnt;
        }
        free(wrow);
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * The same step restricted to W's stored entries (debiasing with lambda = 0
 * is plain SGD on the fixed pattern, Section 2.4; lambda > 0 gives the
 * support-restricted prox):  vals_out[p] = float( S_t(vals[p] - eta*gv[p]) ).
 * vals_out may alias vals.
 * ---------------------------------------------------------------------- */
int orc_prox_csr(int32_t nnz, const float *vals, const float *gv,
                 float eta, float lambda, float *vals_out) {
    if (nnz < 0) return ORC_EINVAL;
    const double t = orc_threshold(eta, lambda);
    for (int32_t p = 0; p < nnz; ++p)
        vals_out[p] = (float)orc_soft_threshold(orc_prox_arg(vals[p], gv[p], eta), t);
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Adaptive proximal steps: Prox-RMSProp (Algorithm 1) and Prox-ADAM
 * (Algorithm 2).  Both replace the plain step -eta*g of Eq. (prox) by a
 * preconditioned one and keep the same prox of eta*lambda*||.||_1.
 *
 * The algorithms state the mathematics, not the arithmetic.  Readings:
 *   - each weight's state (v; and m for ADAM) is kept in float, and a step
 *     reads the stored values;
 *   - the arithmetic is double, as for the plain prox (Fig. 4 computes in
 *     double);
 *   - a moment update  s <- beta*s + (1-beta)*x  is one rounding of that
 *     expression (beta*s is a product of two floats, exact in double; the
 *     fma rounds once), then one rounding to float for storage;
 *   - ADAM's bias corrections divide by 1 - pow(beta, t), in double;
 *   - the step argument z = w - eta*u rounds once (fma), and the new weight
 *     is float(S_{eta*lambda}(z)), as in the plain prox step;
 *   - RMSProp's beta is its squared-gradient decay; it plays beta2's role.
 * Solver codes: 1 = Prox-RMSProp, 2 = Prox-ADAM.
 * ---------------------------------------------------------------------- */
#define ORC_RMSPROP 1
#define ORC_ADAM 2

typedef struct {
    int solver;
    double eta, thr, eps;
    double beta1, beta2;
    double bc1, bc2;  /* 1 - pow(beta1, t), 1 - pow(beta2, t) (ADAM only) */
} orc_adaptive;

static int orc_adaptive_setup(int32_t solver, float eta, float lambda, float eps,
                              float beta1, float beta2, int64_t t, orc_adaptive *a) {
    if (solver != ORC_RMSPROP && solver != ORC_ADAM) return ORC_EINVAL;
    if (!(eta > 0.0f) || !(lambda >= 0.0f) || !(eps > 0.0f) || !isfinite(eta) ||
        !isfinite(lambda) || !isfinite(eps))
        return ORC_EINVAL;
    if (!(beta2 >= 0.0f && beta2 < 1.0f)) return ORC_EINVAL;
    if (solver == ORC_ADAM && (!(beta1 >= 0.0f && beta1 < 1.0f) || t < 1)) return ORC_EINVAL;
    a->solver = solver;
    a->eta = (double)eta;
    a->thr = orc_threshold(eta, lambda);
    a->eps = (double)eps;
    a->beta1 = (double)beta1;
    a->beta2 = (double)beta2;
    a->bc1 = solver == ORC_ADAM ? 1.0 - pow((double)beta1, (double)t) : 1.0;
    a->bc2 = solver == ORC_ADAM ? 1.0 - pow((double)beta2, (double)t) : 1.0;
    return ORC_OK;
}

/* One weight: updates *m (ADAM) and *v in place, returns the new weight. */
static float orc_adaptive_elem(const orc_adaptive *a, float w, float g, float *m, float *v) {
    const double gd = (double)g;
    double u;
    /* second moment (both algorithms): v_t = beta2*v_{t-1} + (1-beta2)*g_t.g_t */
    *v = (float)fma(1.0 - a->beta2, gd * gd, a->beta2 * (double)*v);
    if (a->solver == ORC_ADAM) {
        /* first moment: m_t = beta1*m_{t-1} + (1-beta1)*g_t */
        *m = (float)fma(1.0 - a->beta1, gd, a->beta1 * (double)*m);
        /* bias corrections, then the step m^_t / (sqrt(v^_t) + eps) */
        const double mhat = (double)*m / a->bc1;
        const double vhat = (double)*v / a->bc2;
        u = mhat / (sqrt(vhat) + a->eps);
    } else {
        /* RMSProp: g_t / (sqrt(v_t) + eps) */
        u = gd / (sqrt((double)*v) + a->eps);
    }
    const double z = fma(-a->eta, u, (double)w);
    return (float)orc_soft_threshold(z, a->thr);
}

/* Dense (l1-phase) form over all N*K weights, like orc_prox_dense: w_ik = 0
 * where W has no entry.  m (ADAM only; ignored for RMSProp) and v are [N][lds]
 * and are updated in place; Z[i][k] gets the new weight and row_counts[i]
 * (optional) the number of nonzero Z[i][.]. */
int orc_prox_adaptive_dense(int32_t solver, int32_t N, int32_t K,
                            const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                            const float *G, int64_t ldg, float *m, float *v, int64_t lds,
                            float eta, float lambda, float eps, float beta1, float beta2,
                            int64_t t, float *Z, int64_t ldz, int32_t *row_counts) {
    orc_adaptive a;
    if (N < 0 || K < 0 || ldg < K || ldz < K || lds < K) return ORC_EINVAL;
    if (orc_adaptive_setup(solver, eta, lambda, eps, beta1, beta2, t, &a) != ORC_OK)
        return ORC_EINVAL;
    #pragma omp parallel
    {
        float *wrow = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
        float m_unused = 0.0f;
        #pragma omp for schedule(dynamic, 8)
        for (int32_t i = 0; i < N; ++i) {
            for (int32_t k = 0; k < K; ++k) wrow[k] = 0.0f;
            for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) wrow[col_idx[p]] = vals[p];
            int32_t cnt = 0;
            for (int32_t k = 0; k < K; ++k) {
                const int64_t s = (int64_t)i * lds + k;
                float *mp = solver == ORC_ADAM ? &m[s] : &m_unused;
                const float o = orc_adaptive_elem(&a, wrow[k], G[(int64_t)i * ldg + k], mp, &v[s]);
                Z[(int64_t)i * ldz + k] = o;
                cnt += (o != 0.0f);
            }
            if (row_counts) row_counts[i] = cnt;
        }
        free(wrow);
    }
    return ORC_OK;
}

/* The same step on W's stored entries only, with one state entry per stored
 * weight (m[nnz] for ADAM, v[nnz]); lambda = 0 trains the fixed pattern
 * (debiasing, Section 2.4).  vals_out may alias vals. */
int orc_prox_adaptive_csr(int32_t solver, int32_t nnz, const float *vals, const float *gv,
                          float *m, float *v, float eta, float lambda, float eps,
                          float beta1, float beta2, int64_t t, float *vals_out) {
    orc_adaptive a;
    if (nnz < 0) return ORC_EINVAL;
    if (orc_adaptive_setup(solver, eta, lambda, eps, beta1, beta2, t, &a) != ORC_OK)
        return ORC_EINVAL;
    float m_unused = 0.0f;
    for (int32_t p = 0; p < nnz; ++p) {
        float *mp = solver == ORC_ADAM ? &m[p] : &m_unused;
        vals_out[p] = orc_adaptive_elem(&a, vals[p], gv[p], mp, &v[p]);
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Convolution layers with CSR filters (the conv rows of Tables A1-A4; Caffe,
 * which the paper builds on, lowers a convolution to the products of
 * Section 3.2 through im2col).  Layout, as for the fully connected layers:
 * maps are [C][H][W] rows of a batch-contiguous matrix, X[(c*H + h)*Wd + w][b];
 * the filter bank is a CSR matrix with one row per output channel and column
 * index (ci*KH + kh)*KW + kw.  Cross-correlation (no filter flip), stride
 * SH x SW, zero padding PH x PW, output OH = (H + 2 PH - KH)/SH + 1 (floor),
 * OW likewise.  The output maps are [(co*OH + oh)*OW + ow][b].
 * ---------------------------------------------------------------------- */
typedef struct {
    int32_t C, H, Wd, KH, KW, SH, SW, PH, PW, OH, OW;
} orc_conv_geom;

static int orc_conv_setup(int32_t C, int32_t H, int32_t Wd, int32_t KH, int32_t KW, int32_t SH,
                          int32_t SW, int32_t PH, int32_t PW, orc_conv_geom *g) {
    if (C < 1 || H < 1 || Wd < 1 || KH < 1 || KW < 1 || SH < 1 || SW < 1 || PH < 0 || PW < 0)
        return ORC_EINVAL;
    if (H + 2 * PH < KH || Wd + 2 * PW < KW) return ORC_EINVAL;
    g->C = C; g->H = H; g->Wd = Wd; g->KH = KH; g->KW = KW;
    g->SH = SH; g->SW = SW; g->PH = PH; g->PW = PW;
    g->OH = (H + 2 * PH - KH) / SH + 1;
    g->OW = (Wd + 2 * PW - KW) / SW + 1;
    return ORC_OK;
}

/* Forward: Y[(co,oh,ow)][b] = sum_{p in row co} vals[p] * X[(ci, oh*SH-PH+kh, ow*SW-PW+kw)][b]
 * over the entries whose input position lies inside the map (p ascending). */
int orc_conv_fwd(int32_t N, int32_t C, int32_t H, int32_t Wd, int32_t KH, int32_t KW, int32_t SH,
                 int32_t SW, int32_t PH, int32_t PW, int32_t B, const int32_t *row_ptr,
                 const int32_t *col_idx, const float *vals, const float *X, int64_t ldx, float *Y,
                 int64_t ldy) {
    orc_conv_geom g;
    if (N < 0 || B < 0 || ldx < B || ldy < B) return ORC_EINVAL;
    if (orc_conv_setup(C, H, Wd, KH, KW, SH, SW, PH, PW, &g) != ORC_OK) return ORC_EINVAL;
    #pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)(B > 0 ? B : 1));
        #pragma omp for schedule(dynamic, 4)
        for (int32_t co = 0; co < N; ++co) {
            for (int32_t oh = 0; oh < g.OH; ++oh)
                for (int32_t ow = 0; ow < g.OW; ++ow) {
                    for (int32_t b = 0; b < B; ++b) acc[b] = 0.0;
                    for (int32_t p = row_ptr[co]; p < row_ptr[co + 1]; ++p) {
                        const int32_t ci = col_idx[p] / (KH * KW);
                        const int32_t kh = (col_idx[p] / KW) % KH;
                        const int32_t kw = col_idx[p] % KW;
                        const int32_t ih = oh * SH - PH + kh, iw = ow * SW - PW + kw;
                        if (ih < 0 || ih >= H || iw < 0 || iw >= Wd) continue;
                        const double w = (double)vals[p];
                        const float *xr = X + ((int64_t)(ci * H + ih) * Wd + iw) * ldx;
                        for (int32_t b = 0; b < B; ++b) acc[b] += w * (double)xr[b];
                    }
                    float *yr = Y + ((int64_t)(co * g.OH + oh) * g.OW + ow) * ldy;
                    for (int32_t b = 0; b < B; ++b) yr[b] = (float)acc[b];
                }
        }
        free(acc);
    }
    return ORC_OK;
}

/* Backward for the input maps, the adjoint of orc_conv_fwd:
 *   dX[(ci,ih,iw)][b] = sum over entries p = (co; ci,kh,kw) and output positions
 *   (oh, ow) with oh*SH-PH+kh = ih, ow*SW-PW+kw = iw of vals[p] * dY[(co,oh,ow)][b].
 * Accumulated in double over (co, p, oh, ow) in that order, rounded once. */
int orc_conv_bwd_data(int32_t N, int32_t C, int32_t H, int32_t Wd, int32_t KH, int32_t KW,
                      int32_t SH, int32_t SW, int32_t PH, int32_t PW, int32_t B,
                      const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                      const float *dY, int64_t ldy, float *dX, int64_t ldx) {
    orc_conv_geom g;
    if (N < 0 || B < 0 || ldx < B || ldy < B) return ORC_EINVAL;
    if (orc_conv_setup(C, H, Wd, KH, KW, SH, SW, PH, PW, &g) != ORC_OK) return ORC_EINVAL;
    const int64_t rows = (int64_t)C * H * Wd;
    double *acc = (double *)calloc((size_t)(rows * B > 0 ? rows * B : 1), sizeof(double));
    if (!acc) return ORC_EINVAL;
    /* parallel over input channels: every entry p writes only into its own ci */
    #pragma omp parallel for schedule(dynamic, 1)
    for (int32_t cc = 0; cc < C; ++cc)
        for (int32_t co = 0; co < N; ++co)
            for (int32_t p = row_ptr[co]; p < row_ptr[co + 1]; ++p) {
                const int32_t ci = col_idx[p] / (KH * KW);
                if (ci != cc) continue;
                const int32_t kh = (col_idx[p] / KW) % KH;
                const int32_t kw = col_idx[p] % KW;
                const double w = (double)vals[p];
                for (int32_t oh = 0; oh < g.OH; ++oh)
                    for (int32_t ow = 0; ow < g.OW; ++ow) {
                        const int32_t ih = oh * SH - PH + kh, iw = ow * SW - PW + kw;
                        if (ih < 0 || ih >= H || iw < 0 || iw >= Wd) continue;
                        const float *dyr = dY + ((int64_t)(co * g.OH + oh) * g.OW + ow) * ldy;
                        double *ar = acc + ((int64_t)(ci * H + ih) * Wd + iw) * B;
                        for (int32_t b = 0; b < B; ++b) ar[b] += w * (double)dyr[b];
                    }
            }
    for (int64_t r = 0; r < rows; ++r)
        for (int32_t b = 0; b < B; ++b) dX[r * ldx + b] = (float)acc[r * B + b];
    free(acc);
    return ORC_OK;
}

/* im2col (Caffe's lowering): the matrix whose product with the filter bank is
 * the convolution,
 *   Xcol[(ci*KH + kh)*KW + kw][(oh*OW + ow)*B + b] = X[(ci, oh*SH-PH+kh, ow*SW-PW+kw)][b]
 * (0 where the position falls in the padding); Xcol is [C*KH*KW][ldc],
 * ldc >= OH*OW*B.  The product W . Xcol is then [N][OH*OW*B], the output maps
 * in the batch-contiguous layout. */
int orc_im2col(int32_t C, int32_t H, int32_t Wd, int32_t KH, int32_t KW, int32_t SH, int32_t SW,
               int32_t PH, int32_t PW, int32_t B, const float *X, int64_t ldx, float *Xcol,
               int64_t ldc) {
    orc_conv_geom g;
    if (B < 0 || ldx < B) return ORC_EINVAL;
    if (orc_conv_setup(C, H, Wd, KH, KW, SH, SW, PH, PW, &g) != ORC_OK) return ORC_EINVAL;
    if (ldc < (int64_t)g.OH * g.OW * B) return ORC_EINVAL;
    #pragma omp parallel for schedule(static)
    for (int32_t r = 0; r < C * KH * KW; ++r) {
        const int32_t ci = r / (KH * KW), kh = (r / KW) % KH, kw = r % KW;
        for (int32_t oh = 0; oh < g.OH; ++oh)
            for (int32_t ow = 0; ow < g.OW; ++ow) {
                const int32_t ih = oh * SH - PH + kh, iw = ow * SW - PW + kw;
                float *dst = Xcol + (int64_t)r * ldc + ((int64_t)oh * g.OW + ow) * B;
                const int inside = ih >= 0 && ih < H && iw >= 0 && iw < Wd;
                const float *src = inside ? X + ((int64_t)(ci * H + ih) * Wd + iw) * ldx : NULL;
                for (int32_t b = 0; b < B; ++b) dst[b] = inside ? src[b] : 0.0f;
            }
    }
    return ORC_OK;
}

/* Max pooling over KH x KW windows with stride SH x SW, no padding (the
 * subsampling layers of LeNet-5): Y[(c,oh,ow)][b] = max over the window of
 * X[(c, oh*SH+i, ow*SW+j)][b]; OH = (H - KH)/SH + 1 (floor). */
int orc_maxpool_fwd(int32_t C, int32_t H, int32_t Wd, int32_t KH, int32_t KW, int32_t SH, int32_t SW,
                    int32_t B, const float *X, int64_t ldx, float *Y, int64_t ldy) {
    orc_conv_geom g;
    if (B < 0 || ldx < B || ldy < B) return ORC_EINVAL;
    if (orc_conv_setup(C, H, Wd, KH, KW, SH, SW, 0, 0, &g) != ORC_OK) return ORC_EINVAL;
    #pragma omp parallel for schedule(static)
    for (int32_t c = 0; c < C; ++c)
        for (int32_t oh = 0; oh < g.OH; ++oh)
            for (int32_t ow = 0; ow < g.OW; ++ow) {
                float *yr = Y + ((int64_t)(c * g.OH + oh) * g.OW + ow) * ldy;
                for (int32_t b = 0; b < B; ++b) {
                    float m = -INFINITY;
                    for (int32_t i = 0; i < KH; ++i)
                        for (int32_t j = 0; j < KW; ++j) {
                            const float v = X[((int64_t)(c * H + oh * SH + i) * Wd + ow * SW + j) * ldx + b];
                            if (v > m) m = v;
                        }
                    yr[b] = m;
                }
            }
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Dense -> CSR (Section 3.1: store only the nonzero values; Fig. 1(iii)).
 * Keeps the entries with |Z[i][k]| > t (t = 0 after a prox step) in row-major
 * order.  Writes row_ptr[N+1] and, when nnz <= capacity, col_idx/vals.
 * *nnz_out always receives the required nnz; returns -2 when it exceeds
 * capacity (row_ptr is still written).
 * ---------------------------------------------------------------------- */
int orc_recompress(int32_t N, int32_t K, const float *Z, int64_t ldz, float t,
                   int32_t *row_ptr, int32_t *col_idx, float *vals,
                   int64_t capacity, int64_t *nnz_out) {
    if (N < 0 || K < 0 || ldz < K || capacity < 0) return ORC_EINVAL;
    int64_t nnz = 0;
    row_ptr[0] = 0;
    for (int32_t i = 0; i < N; ++i) {
        for (int32_t k = 0; k < K; ++k) {
            const float z = Z[(int64_t)i * ldz + k];
            if (fabsf(z) > t) {
                if (nnz < capacity) { col_idx[nnz] = k; vals[nnz] = z; }
                ++nnz;
            }
        }
        row_ptr[i + 1] = (int32_t)nnz;
    }
    *nnz_out = nnz;
    return nnz <= capacity ? ORC_OK : ORC_ECAPACITY;
}

/* ------------------------------------------------------------------------
 * CSR -> CSC, the column-wise copy of W that the backward product reads
 * (Section 3.2, "Backward": it needs W by columns).  The canonical CSC: the
 * entries of a column in ascending row order.  col_ptr[K+1], row_idx[nnz],
 * perm[nnz] (the CSR position of each CSC entry) and, if vals and vals_t are
 * both given, vals_t[q] = vals[perm[q]].  Counts per column, their prefix
 * sums, then the entries placed row by row.
 * ---------------------------------------------------------------------- */
int orc_csc(int32_t N, int32_t K, const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
            int32_t *col_ptr, int32_t *row_idx, int32_t *perm, float *vals_t) {
    if (N < 0 || K < 0) return ORC_EINVAL;
    for (int32_t k = 0; k <= K; ++k) col_ptr[k] = 0;
    for (int32_t i = 0; i < N; ++i)
        for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            if (col_idx[p] < 0 || col_idx[p] >= K) return ORC_EINVAL;
            ++col_ptr[col_idx[p] + 1];
        }
    for (int32_t k = 0; k < K; ++k) col_ptr[k + 1] += col_ptr[k];
    int32_t *next = (int32_t *)malloc(sizeof(int32_t) * (size_t)(K > 0 ? K : 1));
    if (!next) return ORC_EINVAL;
    for (int32_t k = 0; k < K; ++k) next[k] = col_ptr[k];
    for (int32_t i = 0; i < N; ++i)
        for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
            const int32_t q = next[col_idx[p]]++;
            row_idx[q] = i;
            perm[q] = p;
            if (vals && vals_t) vals_t[q] = vals[p];
        }
    free(next);
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * CSR -> CSR without its explicit zeros (after a support-restricted prox).
 * Out-of-place: the output arrays must not alias the input ones.
 * ---------------------------------------------------------------------- */
int orc_compact(int32_t N, const int32_t *row_ptr, const int32_t *col_idx, const float *vals,
                int32_t *row_ptr_out, int32_t *col_idx_out, float *vals_out, int64_t *nnz_out) {
    if (N < 0) return ORC_EINVAL;
    int64_t nnz = 0;
    row_ptr_out[0] = 0;
    for (int32_t i = 0; i < N; ++i) {
        for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
            if (vals[p] != 0.0f) { col_idx_out[nnz] = col_idx[p]; vals_out[nnz] = vals[p]; ++nnz; }
        row_ptr_out[i + 1] = (int32_t)nnz;
    }
    *nnz_out = nnz;
    return ORC_OK;
}

/* ------------------------------------------------------------------------
 * Layer glue of the fully connected networks the method trains (the paper
 * trains ReLU networks with a softmax cross-entropy loss; its He
 * initialisation targets ReLU units).  These follow the textbook definitions.
 * ---------------------------------------------------------------------- */

/* ReLU(x) = max(x, 0), with +0.0 for x <= 0. */
int orc_relu_fwd(int64_t n, const float *x, float *y) {
    for (int64_t j = 0; j < n; ++j) y[j] = x[j] > 0.0f ? x[j] : 0.0f;
    return ORC_OK;
}

/* d/dx ReLU = 1 for x > 0, 0 otherwise (0 at x = 0). */
int orc_relu_bwd(int64_t n, const float *x, const float *dy, float *dx) {
    for (int64_t j = 0; j < n; ++j) dx[j] = x[j] > 0.0f ? dy[j] : 0.0f;
    return ORC_OK;
}

/* Mean softmax cross-entropy over the batch.  logits[C][B] (class-major,
 * batch contiguous, leading dimension ld), labels[B] in [0, C).
 * loss = (1/B) sum_b ( log sum_c exp(z_cb) - z_{label_b, b} ),
 * dlogits[c][b] = (softmax(z_.b)_c - [c == label_b]) / B.
 * The column maximum is subtracted before exp (exact in real arithmetic). */
int orc_softmax_xent(int32_t C, int32_t B, const float *logits, int64_t ld,
                     const int32_t *labels, float *dlogits, double *loss) {
    if (C <= 0 || B < 0 || ld < B) return ORC_EINVAL;
    double total = 0.0;
    for (int32_t b = 0; b < B; ++b) {
        if (labels[b] < 0 || labels[b] >= C) return ORC_EINVAL;
        double m = (double)logits[b];
        for (int32_t c = 1; c < C; ++c) m = fmax(m, (double)logits[(int64_t)c * ld + b]);
        double s = 0.0;
        for (int32_t c = 0; c < C; ++c) s += exp((double)logits[(int64_t)c * ld + b] - m);
        total += log(s) + m - (double)logits[(int64_t)labels[b] * ld + b];
        for (int32_t c = 0; c < C; ++c) {
            const double pc = exp((double)logits[(int64_t)c * ld + b] - m) / s;
            dlogits[(int64_t)c * ld + b] = (float)((pc - (c == labels[b] ? 1.0 : 0.0)) / (double)B);
        }
    }
    *loss = B > 0 ? total / (double)B : 0.0;
    return ORC_OK;
}
