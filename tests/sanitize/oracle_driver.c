/*
 * Drives every function of the fp64 oracle on small dense and CSR inputs,
 * and its argument checks, in a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (a CPU test: no GPU is involved).  Exits 0 when
 * every call returned what it should; a sanitizer report aborts the run.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "svm_oracle.h"

static int failures = 0;
#define EXPECT(c)                                                        \
    do {                                                                 \
        if (!(c)) {                                                      \
            fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #c); \
            ++failures;                                                  \
        }                                                                \
    } while (0)

static unsigned long long rng = 88172645463325252ULL;
static double unif(void)
{
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0;
}
static double gauss(void)
{
    double u = unif(), v = unif();
    if (u < 1e-300) u = 1e-300;
    return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

/* n x d dense rows with about a third of the entries zero, and the same
 * matrix in CSR form (columns increasing). */
typedef struct {
    int64_t n, d, nnz;
    float *dense;
    int64_t *rp;
    int32_t *ci;
    float *cv;
} data;

static data make_data(int64_t n, int64_t d)
{
    data D;
    D.n = n;
    D.d = d;
    D.dense = calloc((size_t)(n * d), sizeof(float));
    D.rp = calloc((size_t)(n + 1), sizeof(int64_t));
    D.ci = calloc((size_t)(n * d), sizeof(int32_t));
    D.cv = calloc((size_t)(n * d), sizeof(float));
    int64_t k = 0;
    for (int64_t i = 0; i < n; ++i) {
        D.rp[i] = k;
        for (int64_t j = 0; j < d; ++j) {
            if (unif() < 0.33) continue;
            const float v = (float)gauss();
            D.dense[i * d + j] = v;
            D.ci[k] = (int32_t)j;
            D.cv[k] = v;
            ++k;
        }
    }
    D.rp[n] = k;
    D.nnz = k;
    return D;
}

static void free_data(data* D)
{
    free(D->dense);
    free(D->rp);
    free(D->ci);
    free(D->cv);
}

static orc_mat dense_of(const data* D)
{
    orc_mat m = {D->n, D->d, 0, D->dense, D->d, NULL, NULL};
    return m;
}

static orc_mat csr_of(const data* D)
{
    orc_mat m = {D->n, D->d, 1, D->cv, 0, D->rp, D->ci};
    return m;
}

static orc_params params(int32_t type, int32_t kernel)
{
    orc_params p;
    memset(&p, 0, sizeof p);
    p.type = type;
    p.C = 1.0;
    p.eps = 0.1;
    p.gamma = 0.2;
    p.tol = 1e-3;
    p.max_iter = 0;
    p.threads = 2;
    p.kernel = kernel;
    p.degree = 3;
    p.coef0 = 0.5;
    return p;
}

static void run(int32_t type, int32_t kernel, int csr)
{
    const int64_t n = 60, d = 7, nt = 9;
    data D = make_data(n, d), T = make_data(nt, d);
    const orc_mat X = csr ? csr_of(&D) : dense_of(&D);
    const orc_mat Xd = dense_of(&D);
    const orc_mat Xt = csr ? csr_of(&T) : dense_of(&T);
    orc_params p = params(type, kernel);
    if (kernel == ORC_SIGMOID) p.gamma = 0.05;
    float* y = malloc((size_t)n * sizeof(float));
    for (int64_t i = 0; i < n; ++i)
        y[i] = type == ORC_C_SVC
                   ? (D.dense[i * d] + 0.3 * gauss() > 0 ? 1.0f : -1.0f)
                   : (float)(D.dense[i * d] + 0.1 * gauss());
    if (type == ORC_C_SVC) { y[0] = 1.0f; y[1] = -1.0f; }

    /* kernel matrices: CSR and dense inputs agree */
    double* K = malloc((size_t)(n * n) * sizeof(double));
    double* Kd = malloc((size_t)(n * n) * sizeof(double));
    EXPECT(orc_kernel(&X, &X, &p, K) == ORC_OK);
    EXPECT(orc_kernel(&Xd, &Xd, &p, Kd) == ORC_OK);
    for (int64_t i = 0; i < n * n; ++i)
        EXPECT(fabs(K[i] - Kd[i]) <= 1e-12 * (1.0 + fabs(Kd[i])));
    int64_t idx[3] = {0, 17, n - 1};
    double* R = malloc((size_t)(3 * n) * sizeof(double));
    EXPECT(orc_kernel_rows(&X, &p, idx, 3, 2, R) == ORC_OK);
    for (int j = 0; j < 3; ++j)
        for (int64_t r = 0; r < n; ++r)
            EXPECT(R[j * n + r] == K[idx[j] * n + r]);

    /* training to tol, then the state recomputed and summarised */
    const int64_t N = orc_num_vars(type, n);
    EXPECT(N == (type == ORC_C_SVC ? n : 2 * n));
    double* alpha = calloc((size_t)N, sizeof(double));
    double* F = calloc((size_t)n, sizeof(double));
    double* F2 = calloc((size_t)n, sizeof(double));
    orc_result res, s;
    EXPECT(orc_train(&X, y, &p, alpha, F, &res) == ORC_OK);
    EXPECT(res.status == ORC_OK && res.gap <= p.tol);
    EXPECT(orc_responses(&X, y, &p, alpha, F2) == ORC_OK);
    for (int64_t i = 0; i < n; ++i)
        EXPECT(fabs(F[i] - F2[i]) <= 1e-9 * (1.0 + fabs(F2[i])));
    EXPECT(orc_state_summary(n, y, &p, alpha, F2, &s) == ORC_OK);
    EXPECT(fabs(s.obj - res.obj) <= 1e-9 * (1.0 + fabs(res.obj)));

    /* selection and the subproblem from a state a few steps in */
    double* a2 = calloc((size_t)N, sizeof(double));
    double* F3 = calloc((size_t)n, sizeof(double));
    EXPECT(orc_solve(&X, y, &p, 5, a2, F3, &res) == ORC_MAX_ITER);
    EXPECT(res.iters == 5);
    const int32_t qs[3] = {2, 6, 16};
    for (int t = 0; t < 3; ++t) {
        int32_t B[16], nB = -1;
        double m = 0, M = 0;
        EXPECT(orc_select(n, y, &p, a2, F3, qs[t], B, &nB, &m, &M) == ORC_OK);
        EXPECT(nB >= 2 && nB <= qs[t]);
        double KBB[256], aB[16];
        for (int i = 0; i < nB; ++i) {
            EXPECT(B[i] >= 0 && B[i] < N);
            for (int j = 0; j < nB; ++j)
                KBB[i * nB + j] = K[(B[i] % n) * n + (B[j] % n)];
        }
        int32_t steps = -1;
        EXPECT(orc_subproblem(n, y, &p, nB, B, a2, F3, KBB, 1e-6, 100, aB,
                              &steps) == ORC_OK);
        EXPECT(steps >= 0 && steps <= 100);
        for (int i = 0; i < nB; ++i) EXPECT(aB[i] >= 0.0 && aB[i] <= p.C);
    }

    /* decision values of the trained model on test rows */
    double* coef = malloc((size_t)n * sizeof(double));
    for (int64_t i = 0; i < n; ++i) {
        coef[i] = type == ORC_C_SVC ? y[i] * alpha[i] : alpha[i] - alpha[n + i];
    }
    double* out = malloc((size_t)nt * sizeof(double));
    EXPECT(orc_decision(&X, coef, 0.25, &Xt, &p, 2, out) == ORC_OK);
    for (int64_t i = 0; i < nt; ++i) EXPECT(isfinite(out[i]));

    free(out); free(coef); free(a2); free(F3); free(F2); free(F); free(alpha);
    free(R); free(Kd); free(K); free(y);
    free_data(&D);
    free_data(&T);
}

static void argument_checks(void)
{
    data D = make_data(10, 3);
    const orc_mat X = dense_of(&D);
    orc_params p = params(ORC_C_SVC, ORC_RBF);
    float y[10];
    for (int i = 0; i < 10; ++i) y[i] = i & 1 ? 1.0f : -1.0f;
    double a[10] = {0}, F[10] = {0}, out[100];
    orc_result r;
    EXPECT(orc_kernel(NULL, &X, &p, out) == ORC_EINVAL);
    EXPECT(orc_kernel(&X, &X, &p, NULL) == ORC_EINVAL);
    EXPECT(orc_kernel_rows(&X, &p, NULL, 1, 1, out) == ORC_EINVAL);
    EXPECT(orc_train(NULL, y, &p, a, F, &r) == ORC_EINVAL);
    EXPECT(orc_train(&X, NULL, &p, a, F, &r) == ORC_EINVAL);
    orc_params bad = p;
    bad.type = 7;
    EXPECT(orc_train(&X, y, &bad, a, F, &r) == ORC_EINVAL);
    bad = p;
    bad.kernel = 9;
    EXPECT(orc_kernel(&X, &X, &bad, out) == ORC_EINVAL);
    EXPECT(orc_responses(&X, y, &p, NULL, F) == ORC_EINVAL);
    int32_t B[4], nB;
    double m, M;
    EXPECT(orc_select(10, y, &p, a, F, 4, NULL, &nB, &m, &M) == ORC_EINVAL);
    (void)B;
    free_data(&D);
}

int main(void)
{
    const int32_t kernels[4] = {ORC_LINEAR, ORC_POLY, ORC_RBF, ORC_SIGMOID};
    for (int k = 0; k < 4; ++k)
        for (int type = 0; type < 2; ++type)
            for (int csr = 0; csr < 2; ++csr) run(type, kernels[k], csr);
    argument_checks();
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle driver: all checks passed\n");
    return 0;
}
