/*
 * svm_oracle.c -- plain fp64 CPU oracle for the kernel-SVM dual solve.
 *
 * TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the CPU
 * baseline leg of the benchmark, never by the product library.
 *
 * Every function follows the paper's statement of the problem (Wang et al.,
 * arXiv 1706.05544, Section 3, Eq. 1 and Eq. 2) and the maximal-violating-
 * pair decomposition of LIBSVM (Chang & Lin 2011, the solver the paper
 * extends).  No blocking, fusion or reordering: kernel values come from the
 * direct definitions in fp64 (RBF: exp(-gamma * sum (a_k - b_k)^2); the
 * others from the dot product sum a_k b_k), one pair of
 * variables is optimised per step, and the responses F are updated with two
 * full kernel rows per step.  OpenMP parallelism is only over independent
 * rows (each output element is computed by one thread in a fixed order), so
 * the result bits do not depend on the thread count.
 *
 * Parity pinned by: tests/test_oracle_closed_form.py (2- and 3-point
 * closed forms), tests/test_oracle_bruteforce.py (exact QP optimum by
 * active-set enumeration), tests/test_oracle_invariants.py (constraints, KKT,
 * monotone objective), tests/test_oracle_vs_libsvm.py (scikit-learn's LIBSVM
 * endpoint).  The subproblem and working-set helpers are pinned by
 * tests/test_oracle_select.py, the tie-break to the lowest index among
 * equal keys included (the alpha = 0 state, where all keys of a side tie).
 * The bias rule (mean key over the free variables, else the midpoint of m
 * and M) is pinned by tests/test_oracle_bias.py on hand-worked states where
 * the two differ.  The linear, polynomial and sigmoid kernels
 * are pinned by tests/test_oracle_kernels.py (scikit-learn's pairwise
 * kernels, worked numbers, the 2-point closed form and its single step,
 * the exact QP optimum, LIBSVM's endpoint).  tests/test_sanitizers.py
 * runs every function under AddressSanitizer and UndefinedBehaviorSanitizer.
 */
#include "svm_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define TAU 1e-12 /* curvature floor for a pair of coincident points (the
                     * paper is silent; LIBSVM uses the same floor) */

/* ---------------------------------------------------------------------- */
/* kernel                                                                 */
/* ---------------------------------------------------------------------- */

/* Squared Euclidean distance between row i of A and row j of B.  Rows are
 * walked in increasing column order; a dense row lists every column. */
static double sqdist(const orc_mat *A, int64_t i, const orc_mat *B, int64_t j)
{
    double sum = 0.0;
    if (!A->csr && !B->csr) {
        const float *a = A->val + i * A->ld;
        const float *b = B->val + j * B->ld;
        for (int64_t k = 0; k < A->d; ++k) {
            double diff = (double)a[k] - (double)b[k];
            sum += diff * diff;
        }
        return sum;
    }
    /* generic merge of two sorted (column, value) sequences */
    int64_t pa = 0, ea, pb = 0, eb;
    if (A->csr) { pa = A->row_ptr[i]; ea = A->row_ptr[i + 1]; } else { ea = A->d; }
    if (B->csr) { pb = B->row_ptr[j]; eb = B->row_ptr[j + 1]; } else { eb = B->d; }
    while (pa < ea || pb < eb) {
        int64_t ca = INT64_MAX, cb = INT64_MAX;
        double va = 0.0, vb = 0.0;
        if (pa < ea) {
            ca = A->csr ? A->col[pa] : pa;
            va = A->csr ? (double)A->val[pa] : (double)A->val[i * A->ld + pa];
        }
        if (pb < eb) {
            cb = B->csr ? B->col[pb] : pb;
            vb = B->csr ? (double)B->val[pb] : (double)B->val[j * B->ld + pb];
        }
        double diff;
        if (ca == cb) { diff = va - vb; ++pa; ++pb; }
        else if (ca < cb) { diff = va; ++pa; }
        else { diff = -vb; ++pb; }
        sum += diff * diff;
    }
    return sum;
}

/* Dot product of row i of A and row j of B, over the columns in increasing
 * order (the products of columns only one row holds are zero). */
static double dotp(const orc_mat *A, int64_t i, const orc_mat *B, int64_t j)
{
    double sum = 0.0;
    if (!A->csr && !B->csr) {
        const float *a = A->val + i * A->ld;
        const float *b = B->val + j * B->ld;
        for (int64_t k = 0; k < A->d; ++k) sum += (double)a[k] * (double)b[k];
        return sum;
    }
    int64_t pa = 0, ea, pb = 0, eb;
    if (A->csr) { pa = A->row_ptr[i]; ea = A->row_ptr[i + 1]; } else { ea = A->d; }
    if (B->csr) { pb = B->row_ptr[j]; eb = B->row_ptr[j + 1]; } else { eb = B->d; }
    while (pa < ea && pb < eb) {
        const int64_t ca = A->csr ? A->col[pa] : pa;
        const int64_t cb = B->csr ? B->col[pb] : pb;
        if (ca == cb) {
            const double va = A->csr ? (double)A->val[pa]
                                     : (double)A->val[i * A->ld + pa];
            const double vb = B->csr ? (double)B->val[pb]
                                     : (double)B->val[j * B->ld + pb];
            sum += va * vb;
            ++pa;
            ++pb;
        } else if (ca < cb) {
            ++pa;
        } else {
            ++pb;
        }
    }
    return sum;
}

/* The kernel of p, e1071/LIBSVM parameterisation (Section 3, kernel list). */
static double kval(const orc_params *p, const orc_mat *A, int64_t i,
                   const orc_mat *B, int64_t j)
{
    switch (p->kernel) {
    case ORC_LINEAR:
        return dotp(A, i, B, j);
    case ORC_POLY:
        return pow(p->gamma * dotp(A, i, B, j) + p->coef0, (double)p->degree);
    case ORC_SIGMOID:
        return tanh(p->gamma * dotp(A, i, B, j) + p->coef0);
    default:
        return exp(-p->gamma * sqdist(A, i, B, j));
    }
}

static int check_kernel(const orc_params *p)
{
    if (!p || p->kernel < ORC_LINEAR || p->kernel > ORC_SIGMOID) return 0;
    if (p->kernel != ORC_LINEAR && !(p->gamma > 0)) return 0;
    if (p->kernel == ORC_POLY && p->degree < 1) return 0;
    if (!isfinite(p->coef0)) return 0;
    return 1;
}

static void set_threads(int32_t threads)
{
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#else
    (void)threads;
#endif
}

int orc_kernel(const orc_mat *A, const orc_mat *B, const orc_params *p,
               double *out)
{
    if (!A || !B || !out || A->d != B->d || !check_kernel(p)) return ORC_EINVAL;
    for (int64_t i = 0; i < A->n; ++i)
        for (int64_t j = 0; j < B->n; ++j)
            out[i * B->n + j] = kval(p, A, i, B, j);
    return ORC_OK;
}

int orc_kernel_rows(const orc_mat *X, const orc_params *p, const int64_t *idx,
                    int64_t q, int32_t threads, double *out)
{
    if (!X || !idx || !out || !check_kernel(p)) return ORC_EINVAL;
    set_threads(threads);
    for (int64_t j = 0; j < q; ++j) {
        int64_t s = idx[j];
        double *row = out + j * X->n;
#pragma omp parallel for schedule(static)
        for (int64_t r = 0; r < X->n; ++r) row[r] = kval(p, X, s, X, r);
    }
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* the dual variables (Section 3, Eq. 1 / Eq. 2)                          */
/* ---------------------------------------------------------------------- */

int64_t orc_num_vars(int32_t type, int64_t n)
{
    return type == ORC_EPS_SVR ? 2 * n : n;
}

/* sample of variable t */
static int64_t smp(int32_t type, int64_t n, int64_t t)
{
    return (type == ORC_EPS_SVR && t >= n) ? t - n : t;
}

/* label y_t of variable t: the class label for C-SVC; +1 for the positive
 * copy and -1 for the negative copy for eps-SVR (Eq. 1, vector y). */
static double yv(int32_t type, int64_t n, const float *y, int64_t t)
{
    if (type == ORC_EPS_SVR) return t < n ? 1.0 : -1.0;
    return y[t] > 0.0f ? 1.0 : -1.0;
}

/* linear term p_t of Eq. 2: -1 for C-SVC (the paper's "all-one" vector with
 * the sign that makes Eq. 2 a minimisation, as in LIBSVM); eps - z_i for the
 * positive copy and eps + z_i for the negative copy (Eq. 1 substituted). */
static double pv(int32_t type, int64_t n, const float *y, double eps, int64_t t)
{
    if (type == ORC_EPS_SVR) {
        double z = (double)y[smp(type, n, t)];
        return t < n ? eps - z : eps + z;
    }
    return -1.0;
}

/* violation key v_t = -y_t G_t with G_t = y_t F_smp(t) + p_t */
static double key(int32_t type, int64_t n, const float *y, double eps,
                  const double *F, int64_t t)
{
    double yt = yv(type, n, y, t);
    double G = yt * F[smp(type, n, t)] + pv(type, n, y, eps, t);
    return -yt * G;
}

static int in_up(double yt, double a, double C)
{
    return (yt > 0 && a < C) || (yt < 0 && a > 0);
}

static int in_low(double yt, double a, double C)
{
    return (yt > 0 && a > 0) || (yt < 0 && a < C);
}

/* (k1,i1) precedes (k2,i2) in "largest key first, lowest index on ties" */
static int before_desc(double k1, int64_t i1, double k2, int64_t i2)
{
    return k1 > k2 || (k1 == k2 && i1 < i2);
}

static int before_asc(double k1, int64_t i1, double k2, int64_t i2)
{
    return k1 < k2 || (k1 == k2 && i1 < i2);
}

/* Maximal violating pair: i = argmax_{I_up} v, j = argmin_{I_low} v. */
static void mvp(int64_t n, const float *y, const orc_params *p,
                const double *alpha, const double *F, int64_t *oi,
                int64_t *oj, double *om, double *oM)
{
    int64_t N = orc_num_vars(p->type, n);
    int64_t bi = -1, bj = -1;
    double m = -INFINITY, M = INFINITY;
    for (int64_t t = 0; t < N; ++t) {
        double yt = yv(p->type, n, y, t);
        double v = key(p->type, n, y, p->eps, F, t);
        if (in_up(yt, alpha[t], p->C) && (bi < 0 || before_desc(v, t, m, bi))) {
            bi = t; m = v;
        }
        if (in_low(yt, alpha[t], p->C) && (bj < 0 || before_asc(v, t, M, bj))) {
            bj = t; M = v;
        }
    }
    *oi = bi; *oj = bj; *om = m; *oM = M;
}

int orc_state_summary(int64_t n, const float *y, const orc_params *p,
                      const double *alpha, const double *F, orc_result *res)
{
    int64_t N = orc_num_vars(p->type, n);
    int64_t i, j;
    double m, M;
    mvp(n, y, p, alpha, F, &i, &j, &m, &M);
    res->m = m;
    res->M = M;
    res->gap = (i < 0 || j < 0) ? 0.0 : m - M;

    /* bias (not defined in the paper): mean key over free variables, else
     * the midpoint of m and M, as in LIBSVM */
    double sum = 0.0;
    int64_t nfree = 0;
    for (int64_t t = 0; t < N; ++t) {
        if (alpha[t] > 0.0 && alpha[t] < p->C) {
            sum += key(p->type, n, y, p->eps, F, t);
            ++nfree;
        }
    }
    res->n_free = nfree;
    if (nfree > 0) res->b = sum / (double)nfree;
    else if (i >= 0 && j >= 0) res->b = 0.5 * (m + M);
    else res->b = 0.0;

    /* f(a) = 1/2 a^T Q a + p^T a, with (Q a)_t = y_t F_smp(t) */
    double quad = 0.0, lin = 0.0;
    for (int64_t t = 0; t < N; ++t) {
        double yt = yv(p->type, n, y, t);
        quad += alpha[t] * yt * F[smp(p->type, n, t)];
        lin += pv(p->type, n, y, p->eps, t) * alpha[t];
    }
    res->obj = 0.5 * quad + lin;

    /* support vectors: samples with non-zero coefficient */
    int64_t nsv = 0;
    for (int64_t s = 0; s < n; ++s) {
        double c;
        if (p->type == ORC_EPS_SVR) c = alpha[s] - alpha[s + n];
        else c = alpha[s];
        if (c != 0.0) ++nsv;
    }
    res->n_sv = nsv;
    return ORC_OK;
}

static int check_params(const orc_mat *X, const float *y, const orc_params *p)
{
    if (!X || !y || !p || X->n < 1 || X->d < 1) return ORC_EINVAL;
    if (!(p->C > 0) || !(p->tol > 0) || !(p->eps >= 0) || !check_kernel(p))
        return ORC_EINVAL;
    if (p->type != ORC_C_SVC && p->type != ORC_EPS_SVR) return ORC_EINVAL;
    return ORC_OK;
}

int orc_solve(const orc_mat *X, const float *y, const orc_params *p,
              int64_t max_steps, double *alpha, double *F, orc_result *res)
{
    if (check_params(X, y, p) != ORC_OK || !alpha || !F || !res)
        return ORC_EINVAL;
    const int64_t n = X->n;
    const int64_t N = orc_num_vars(p->type, n);
    const double C = p->C;
    int64_t cap = p->max_iter > 0 ? p->max_iter
                                  : (100 * N > 10000000 ? 100 * N : 10000000);
    if (max_steps > 0) cap = max_steps;
    set_threads(p->threads);

    double *Ki = (double *)malloc(sizeof(double) * (size_t)n);
    double *Kj = (double *)malloc(sizeof(double) * (size_t)n);
    if (!Ki || !Kj) { free(Ki); free(Kj); return ORC_EINVAL; }

    int64_t steps = 0;
    int32_t status = ORC_OK;
    for (;;) {
        int64_t i, j;
        double m, M;
        mvp(n, y, p, alpha, F, &i, &j, &m, &M);
        if (i < 0 || j < 0 || m - M <= p->tol) break;
        if (steps >= cap) { status = ORC_MAX_ITER; break; }

        const int64_t si = smp(p->type, n, i), sj = smp(p->type, n, j);
        const double yi = yv(p->type, n, y, i), yj = yv(p->type, n, y, j);
        /* second derivative along the pair direction, K_ii + K_jj - 2 K_ij
         * (0 for the two copies of one sample) */
        double a = 0.0;
        if (si != sj)
            a = kval(p, X, si, X, si) + kval(p, X, sj, X, sj) -
                2.0 * kval(p, X, si, X, sj);
        if (a <= 0.0) a = TAU;
        double s = (m - M) / a;
        /* largest feasible move of each variable */
        double Ui = yi > 0 ? C - alpha[i] : alpha[i];
        double Lj = yj > 0 ? alpha[j] : C - alpha[j];
        int clip_i = 0, clip_j = 0;
        if (Ui <= s) { s = Ui; clip_i = 1; }
        if (Lj <= s) { s = Lj; clip_j = 1; clip_i = (Ui == s); }
        alpha[i] += yi * s;
        alpha[j] -= yj * s;
        if (clip_i) alpha[i] = yi > 0 ? C : 0.0;
        if (clip_j) alpha[j] = yj > 0 ? 0.0 : C;

        /* responses: F_r += y_i da_i K(r,si) + y_j da_j K(r,sj) = s (Ki - Kj) */
        if (si != sj) {
#pragma omp parallel for schedule(static)
            for (int64_t r = 0; r < n; ++r) {
                Ki[r] = kval(p, X, si, X, r);
                Kj[r] = kval(p, X, sj, X, r);
            }
            for (int64_t r = 0; r < n; ++r) F[r] += s * (Ki[r] - Kj[r]);
        }
        ++steps;
    }
    free(Ki);
    free(Kj);
    orc_state_summary(n, y, p, alpha, F, res);
    res->iters = steps;
    res->status = status;
    return status;
}

int orc_train(const orc_mat *X, const float *y, const orc_params *p,
              double *alpha, double *F, orc_result *res)
{
    if (check_params(X, y, p) != ORC_OK || !alpha || !F || !res)
        return ORC_EINVAL;
    int64_t N = orc_num_vars(p->type, X->n);
    memset(alpha, 0, sizeof(double) * (size_t)N);
    memset(F, 0, sizeof(double) * (size_t)X->n);
    return orc_solve(X, y, p, 0, alpha, F, res);
}

int orc_responses(const orc_mat *X, const float *y, const orc_params *p,
                  const double *alpha, double *F)
{
    if (check_params(X, y, p) != ORC_OK || !alpha || !F) return ORC_EINVAL;
    const int64_t n = X->n;
    const int64_t N = orc_num_vars(p->type, n);
    set_threads(p->threads);
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < n; ++r) {
        double acc = 0.0;
        for (int64_t t = 0; t < N; ++t) {
            if (alpha[t] == 0.0) continue;
            acc += yv(p->type, n, y, t) * alpha[t] *
                   kval(p, X, r, X, smp(p->type, n, t));
        }
        F[r] = acc;
    }
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* working set of q variables and its subproblem (Section 3)              */
/* ---------------------------------------------------------------------- */

typedef struct { double k; int64_t t; } kv;

static int cmp_desc(const void *a, const void *b)
{
    const kv *x = (const kv *)a, *z = (const kv *)b;
    if (before_desc(x->k, x->t, z->k, z->t)) return -1;
    if (before_desc(z->k, z->t, x->k, x->t)) return 1;
    return 0;
}

static int cmp_asc(const void *a, const void *b)
{
    const kv *x = (const kv *)a, *z = (const kv *)b;
    if (before_asc(x->k, x->t, z->k, z->t)) return -1;
    if (before_asc(z->k, z->t, x->k, x->t)) return 1;
    return 0;
}

int orc_select(int64_t n, const float *y, const orc_params *p,
               const double *alpha, const double *F, int32_t q, int32_t *B,
               int32_t *nB, double *m, double *M)
{
    if (!y || !p || !alpha || !F || !B || !nB || q < 2 || (q & 1))
        return ORC_EINVAL;
    const int64_t N = orc_num_vars(p->type, n);
    kv *up = (kv *)malloc(sizeof(kv) * (size_t)N);
    kv *lo = (kv *)malloc(sizeof(kv) * (size_t)N);
    if (!up || !lo) { free(up); free(lo); return ORC_EINVAL; }
    int64_t nu = 0, nl = 0;
    for (int64_t t = 0; t < N; ++t) {
        double yt = yv(p->type, n, y, t);
        double v = key(p->type, n, y, p->eps, F, t);
        if (in_up(yt, alpha[t], p->C)) { up[nu].k = v; up[nu].t = t; ++nu; }
        if (in_low(yt, alpha[t], p->C)) { lo[nl].k = v; lo[nl].t = t; ++nl; }
    }
    qsort(up, (size_t)nu, sizeof(kv), cmp_desc);
    qsort(lo, (size_t)nl, sizeof(kv), cmp_asc);
    *m = nu ? up[0].k : -INFINITY;
    *M = nl ? lo[0].k : INFINITY;
    int32_t h = q / 2, cnt = 0;
    for (int32_t r = 0; r < h; ++r) {
        for (int side = 0; side < 2; ++side) {
            const kv *lst = side ? lo : up;
            int64_t len = side ? nl : nu;
            if (r >= len) continue;
            int64_t t = lst[r].t;
            int dup = 0;
            for (int32_t c = 0; c < cnt; ++c) dup |= (B[c] == (int32_t)t);
            if (!dup) B[cnt++] = (int32_t)t;
        }
    }
    *nB = cnt;
    free(up);
    free(lo);
    return ORC_OK;
}

int orc_subproblem(int64_t n, const float *y, const orc_params *p,
                   int32_t nB, const int32_t *B, const double *alpha,
                   const double *F, const double *KBB, double inner_tol,
                   int32_t max_inner, double *alpha_B_new, int32_t *steps)
{
    if (!y || !p || !B || !alpha || !F || !KBB || !alpha_B_new || nB < 1)
        return ORC_EINVAL;
    const double C = p->C;
    double *v = (double *)malloc(sizeof(double) * (size_t)nB);
    double *yb = (double *)malloc(sizeof(double) * (size_t)nB);
    if (!v || !yb) { free(v); free(yb); return ORC_EINVAL; }
    for (int32_t a = 0; a < nB; ++a) {
        alpha_B_new[a] = alpha[B[a]];
        v[a] = key(p->type, n, y, p->eps, F, B[a]);
        yb[a] = yv(p->type, n, y, B[a]);
    }
    int32_t k = 0;
    while (k < max_inner) {
        int32_t bi = -1, bj = -1;
        for (int32_t a = 0; a < nB; ++a) {
            if (in_up(yb[a], alpha_B_new[a], C) &&
                (bi < 0 || before_desc(v[a], B[a], v[bi], B[bi])))
                bi = a;
            if (in_low(yb[a], alpha_B_new[a], C) &&
                (bj < 0 || before_asc(v[a], B[a], v[bj], B[bj])))
                bj = a;
        }
        if (bi < 0 || bj < 0 || v[bi] - v[bj] <= inner_tol) break;
        double a2 = KBB[bi * nB + bi] + KBB[bj * nB + bj] - 2.0 * KBB[bi * nB + bj];
        if (a2 <= 0.0) a2 = TAU;
        double s = (v[bi] - v[bj]) / a2;
        double Ui = yb[bi] > 0 ? C - alpha_B_new[bi] : alpha_B_new[bi];
        double Lj = yb[bj] > 0 ? alpha_B_new[bj] : C - alpha_B_new[bj];
        int clip_i = 0, clip_j = 0;
        if (Ui <= s) { s = Ui; clip_i = 1; }
        if (Lj <= s) { s = Lj; clip_j = 1; clip_i = (Ui == s); }
        alpha_B_new[bi] += yb[bi] * s;
        alpha_B_new[bj] -= yb[bj] * s;
        if (clip_i) alpha_B_new[bi] = yb[bi] > 0 ? C : 0.0;
        if (clip_j) alpha_B_new[bj] = yb[bj] > 0 ? 0.0 : C;
        /* keys inside B move by -s (K(t,i) - K(t,j)) */
        for (int32_t a = 0; a < nB; ++a)
            v[a] -= s * (KBB[a * nB + bi] - KBB[a * nB + bj]);
        ++k;
    }
    if (steps) *steps = k;
    free(v);
    free(yb);
    return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* decision function                                                      */
/* ---------------------------------------------------------------------- */

int orc_decision(const orc_mat *SV, const double *coef, double b,
                 const orc_mat *Xt, const orc_params *p, int32_t threads,
                 double *out)
{
    if (!SV || !coef || !Xt || !out || SV->d != Xt->d || !check_kernel(p))
        return ORC_EINVAL;
    set_threads(threads);
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < Xt->n; ++r) {
        double acc = 0.0;
        for (int64_t s = 0; s < SV->n; ++s)
            acc += coef[s] * kval(p, SV, s, Xt, r);
        out[r] = acc + b;
    }
    return ORC_OK;
}
