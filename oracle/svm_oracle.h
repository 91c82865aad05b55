/*
 * svm_oracle.h -- plain, slow, fp64 CPU oracle for the kernel-SVM dual solve.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this code; only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark use it.  It shares no code, header, table or
 * constant with the HIP path.
 *
 * What it computes (Wang et al., "Rgtsvm", arXiv 1706.05544):
 *   - the general dual of Eq. 2:  min_a  1/2 a^T Q a + p^T a
 *       s.t.  y^T a = 0,  0 <= a_t <= C,
 *     with Q_ts = y_t y_s K(x_smp(t), x_smp(s)) (Section 3, text after Eq. 1);
 *   - C-SVC: one variable per sample, p_t = -1 (Eq. 2 with the "all-one"
 *     linear term taken with the sign that makes Eq. 2 a minimisation, as
 *     in LIBSVM);
 *   - eps-SVR: two copies per sample (Section 3, "positive and negative
 *     copy"), copy (i,+) has y = +1 and p = eps - z_i, copy (i,-) has
 *     y = -1 and p = eps + z_i (Eq. 1 substituted into Eq. 2; the only
 *     assignment under which a free positive copy lies on f(x) = z - eps);
 *   - the four kernels of Section 3's feature list, in the e1071 (LIBSVM)
 *     parameterisation the paper's interface follows (the paper names them
 *     without formulas):
 *       linear      K(a,b) = a.b
 *       polynomial  K(a,b) = (gamma a.b + coef0)^degree
 *       RBF         K(a,b) = exp(-gamma * sum_k (a_k - b_k)^2)
 *       sigmoid     K(a,b) = tanh(gamma a.b + coef0)
 *
 * Solver: maximal-violating-pair SMO (Chang & Lin 2011, cited in Section 1
 * and Section 3 for Eq. 1), no shrinking, kernel values from the direct
 * definition in fp64, stop when m - M <= tol (Section 3: iterate "until
 * convergence", read as the KKT gap of LIBSVM).
 *
 * Notation used throughout (identical in the tests):
 *   F_i   = sum_t y_t a_t K(x_i, x_smp(t))      ("responses", Section 3)
 *   r_t   = -y_t p_t                            (SVC: y_t; SVR: z -/+ eps)
 *   v_t   = -y_t G_t = r_t - F_smp(t)           (violation key)
 *   I_up  = {y=+1, a<C} u {y=-1, a>0};  I_low = {y=+1, a>0} u {y=-1, a<C}
 *   m = max_{I_up} v,  M = min_{I_low} v,  gap = m - M
 */
#ifndef SVM_ORACLE_H
#define SVM_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A feature matrix: dense row-major fp32 (csr = 0) or CSR fp32 (csr = 1). */
typedef struct {
    int64_t n, d;
    int32_t csr;
    const float *val;        /* dense: n*ld values; CSR: nnz values */
    int64_t ld;              /* dense leading dimension (>= d) */
    const int64_t *row_ptr;  /* CSR: n+1 offsets */
    const int32_t *col;      /* CSR: column of each value, sorted per row */
} orc_mat;

enum { ORC_C_SVC = 0, ORC_EPS_SVR = 1 };
enum { ORC_LINEAR = 0, ORC_POLY = 1, ORC_RBF = 2, ORC_SIGMOID = 3 };
enum { ORC_OK = 0, ORC_MAX_ITER = 1, ORC_EINVAL = -1 };

typedef struct {
    int32_t type;       /* ORC_C_SVC or ORC_EPS_SVR */
    double C, eps, gamma, tol;
    int64_t max_iter;   /* <= 0: max(1e7, 100*N) */
    int32_t threads;    /* OpenMP threads for kernel rows (<=0: default) */
    int32_t kernel;     /* ORC_LINEAR, ORC_POLY, ORC_RBF or ORC_SIGMOID */
    int32_t degree;     /* polynomial degree (>= 1) */
    double coef0;       /* polynomial and sigmoid offset */
} orc_params;

typedef struct {
    int64_t iters;      /* SMO steps taken by this call */
    double gap;         /* m - M at exit */
    double m, M;
    double b;           /* bias: mean v over free variables, else (m+M)/2 */
    double obj;         /* dual objective f(a) */
    int64_t n_sv;       /* samples with non-zero coefficient */
    int64_t n_free;     /* variables with 0 < a < C */
    int32_t status;     /* ORC_OK or ORC_MAX_ITER */
} orc_result;

/* out[i*B->n + j] = K(a_i, b_j) for all pairs (kernel, gamma, degree and
 * coef0 of p). */
int orc_kernel(const orc_mat *A, const orc_mat *B, const orc_params *p,
               double *out);

/* out[j*X->n + r] = K(x_idx[j], x_r): q kernel rows against the whole set. */
int orc_kernel_rows(const orc_mat *X, const orc_params *p, const int64_t *idx,
                    int64_t q, int32_t threads, double *out);

/* Number of dual variables: n (C-SVC) or 2n (eps-SVR). */
int64_t orc_num_vars(int32_t type, int64_t n);

/* Run maximal-violating-pair SMO from the state (alpha[N], F[n]) until the
 * gap is <= tol or max_steps steps were taken (max_steps <= 0: p->max_iter).
 * alpha and F are updated in place; res receives gap, bias and objective. */
int orc_solve(const orc_mat *X, const float *y, const orc_params *p,
              int64_t max_steps, double *alpha, double *F, orc_result *res);

/* orc_solve from alpha = 0, F = 0. */
int orc_train(const orc_mat *X, const float *y, const orc_params *p,
              double *alpha, double *F, orc_result *res);

/* Gap, m, M, bias, objective and SV counts of a state (no solving). */
int orc_state_summary(int64_t n, const float *y, const orc_params *p,
                      const double *alpha, const double *F, orc_result *res);

/* F_i = sum_t y_t a_t K(x_i, x_smp(t)) recomputed from scratch. */
int orc_responses(const orc_mat *X, const float *y, const orc_params *p,
                  const double *alpha, double *F);

/* Working set of size <= q (q even): interleave the q/2 largest keys of I_up
 * with the q/2 smallest keys of I_low, ties to the lowest variable index,
 * dropping repeats (Section 3: the working set is chosen by the largest
 * partial derivatives under the constraints).  Returns |B| in *nB, m, M. */
int orc_select(int64_t n, const float *y, const orc_params *p,
               const double *alpha, const double *F, int32_t q,
               int32_t *B, int32_t *nB, double *m, double *M);

/* Subproblem on B (Section 3: the working set is optimised from the local
 * gradient): maximal-violating-pair steps restricted to B,
 * starting from keys v_B = r_B - F_smp(B), using the kernel block KBB
 * (nB x nB, KBB[a*nB+b] = K(x_smp(B_a), x_smp(B_b))).  Stops when the local
 * gap <= inner_tol or after max_inner steps.  Writes the new alpha_B. */
int orc_subproblem(int64_t n, const float *y, const orc_params *p,
                   int32_t nB, const int32_t *B, const double *alpha,
                   const double *F, const double *KBB, double inner_tol,
                   int32_t max_inner, double *alpha_B_new, int32_t *steps);

/* Decision values D(x) = sum_i coef_i K(sv_i, x) + b, summed in fp64. */
int orc_decision(const orc_mat *SV, const double *coef, double b,
                 const orc_mat *Xt, const orc_params *p, int32_t threads,
                 double *out);

#ifdef __cplusplus
}
#endif
#endif
