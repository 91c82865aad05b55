/*
 * Drives the argument checks of the C ABI in a build of the library whose
 * host code carries AddressSanitizer and UndefinedBehaviorSanitizer (a CPU
 * test: every call here is refused before any device work, either by the
 * checks or because the device ordinal does not exist).  Exits 0 when every
 * call returned the expected status with a message.
 */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "mi355svm.h"

static int failures = 0;

static void expect(svm_status got, svm_status want, int line)
{
    const char* msg = svm_last_error();
    if (got != want) {
        fprintf(stderr, "line %d: status %d, expected %d (%s)\n", line,
                (int)got, (int)want, msg ? msg : "(null)");
        ++failures;
    } else if (!msg || !msg[0]) {
        fprintf(stderr, "line %d: no error message\n", line);
        ++failures;
    }
}
#define EXPECT(call, want) expect((call), (want), __LINE__)

/* no device, or (on a machine that has one) an ordinal past the last */
static void expect_no_device(svm_status got, int line)
{
    if (got != SVM_E_DEVICE && got != SVM_E_INVALID) {
        fprintf(stderr, "line %d: status %d, expected a refusal\n", line,
                (int)got);
        ++failures;
    }
}

int main(void)
{
    float Xv[40], y[10], bad_y[10];
    for (int i = 0; i < 40; ++i) Xv[i] = (float)((i * 7) % 11) - 5.0f;
    for (int i = 0; i < 10; ++i) {
        y[i] = (i & 1) ? 1.0f : -1.0f;
        bad_y[i] = y[i];
    }
    bad_y[3] = 0.5f;
    int32_t labels[10];
    for (int i = 0; i < 10; ++i) labels[i] = i % 3;
    int64_t rp[11];
    int32_t ci[20];
    float cv[20];
    for (int i = 0; i <= 10; ++i) rp[i] = 2 * i;
    for (int i = 0; i < 20; ++i) {
        ci[i] = i & 3;
        cv[i] = 1.0f + (float)i;
    }

    svm_matrix X;
    memset(&X, 0, sizeof X);
    X.layout = SVM_DENSE;
    X.n = 10;
    X.d = 4;
    X.values = Xv;
    X.ld = 4;
    svm_params p;
    svm_params_default(&p);
    svm_model* m = NULL;

    /* parameters */
    EXPECT(svm_train(&X, y, NULL, &m), SVM_E_INVALID);
    EXPECT(svm_train(&X, y, &p, NULL), SVM_E_INVALID);
    svm_params q = p;
    q.C = 0.0;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.C = NAN;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.tol = -1.0;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.type = 5;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.kernel = 9;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.kernel = SVM_KERNEL_POLY;
    q.degree = 0;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.working_set = 3;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.working_set = 66;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.gamma = INFINITY;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.epsilon = -0.1;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.inner_ratio = 1.0;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.scale = 2;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.lockstep = 99;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.fused = 2;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);
    q = p;
    q.device = -1;
    EXPECT(svm_train(&X, y, &q, &m), SVM_E_INVALID);

    /* matrices */
    EXPECT(svm_train(NULL, y, &p, &m), SVM_E_INVALID);
    svm_matrix B = X;
    B.layout = 7;
    EXPECT(svm_train(&B, y, &p, &m), SVM_E_INVALID);
    B = X;
    B.n = 1;
    EXPECT(svm_train(&B, y, &p, &m), SVM_E_INVALID);
    B = X;
    B.d = 0;
    EXPECT(svm_train(&B, y, &p, &m), SVM_E_INVALID);
    B = X;
    B.ld = 3;
    EXPECT(svm_train(&B, y, &p, &m), SVM_E_INVALID);
    B = X;
    B.values = NULL;
    EXPECT(svm_train(&B, y, &p, &m), SVM_E_INVALID);
    svm_matrix C;
    memset(&C, 0, sizeof C);
    C.layout = SVM_CSR;
    C.n = 10;
    C.d = 4;
    C.row_ptr = rp;
    C.col_idx = ci;
    C.values = cv;
    C.nnz = 20;
    svm_matrix Cb = C;
    Cb.row_ptr = NULL;
    EXPECT(svm_train(&Cb, y, &p, &m), SVM_E_INVALID);
    Cb = C;
    Cb.nnz = -1;
    EXPECT(svm_train(&Cb, y, &p, &m), SVM_E_INVALID);
    Cb = C;
    Cb.col_idx = NULL;
    EXPECT(svm_train(&Cb, y, &p, &m), SVM_E_INVALID);

    /* labels and targets (checked on the host before any device work) */
    EXPECT(svm_train(&X, NULL, &p, &m), SVM_E_INVALID);
    EXPECT(svm_train(&X, bad_y, &p, &m), SVM_E_INVALID);
    float one_class[10];
    for (int i = 0; i < 10; ++i) one_class[i] = 1.0f;
    EXPECT(svm_train(&X, one_class, &p, &m), SVM_E_INVALID);
    q = p;
    q.type = SVM_EPS_SVR;
    float nan_z[10];
    for (int i = 0; i < 10; ++i) nan_z[i] = (float)i;
    nan_z[4] = NAN;
    EXPECT(svm_train(&X, nan_z, &q, &m), SVM_E_INVALID);

    /* one-vs-rest, cross-validation, tuning */
    EXPECT(svm_train_ovr(&X, labels, 1, &p, &m), SVM_E_INVALID);
    int32_t bad_labels[10];
    memcpy(bad_labels, labels, sizeof labels);
    bad_labels[2] = 3;
    EXPECT(svm_train_ovr(&X, bad_labels, 3, &p, &m), SVM_E_INVALID);
    EXPECT(svm_train_ovr(&X, NULL, 3, &p, &m), SVM_E_INVALID);
    svm_cv_stats st;
    EXPECT(svm_cross_validate(&X, y, NULL, 0, &p, 1, NULL, NULL, &st),
           SVM_E_INVALID);
    EXPECT(svm_cross_validate(&X, y, labels, 3, &p, 3, NULL, NULL, &st),
           SVM_E_INVALID);
    EXPECT(svm_cross_validate(&X, y, NULL, 0, &p, 3, NULL, NULL, NULL),
           SVM_E_INVALID);
    int32_t fold[10];
    for (int i = 0; i < 10; ++i) fold[i] = 0;
    EXPECT(svm_cross_validate(&X, y, NULL, 0, &p, 2, fold, NULL, &st),
           SVM_E_INVALID);
    double err[2], Cg[2] = {1.0, -1.0};
    int32_t best = -1;
    EXPECT(svm_tune(&X, y, NULL, 0, &p, 3, NULL, 0, NULL, NULL, NULL, err,
                    &best),
           SVM_E_INVALID);
    EXPECT(svm_tune(&X, y, NULL, 0, &p, 3, NULL, 2, Cg, NULL, NULL, err,
                    &best),
           SVM_E_INVALID);

    /* models and prediction */
    double D[10];
    int32_t L[10];
    EXPECT(svm_predict(NULL, &X, D), SVM_E_INVALID);
    EXPECT(svm_predict_labels(NULL, &X, L), SVM_E_INVALID);
    EXPECT(svm_predict_noalloc(NULL, &X, D, NULL), SVM_E_INVALID);
    svm_model_info info;
    EXPECT(svm_model_get_info(NULL, 0, &info), SVM_E_INVALID);
    EXPECT(svm_model_get(NULL, 0, NULL, NULL, NULL), SVM_E_INVALID);
    svm_model_free(NULL);

    /* test hooks */
    svm_solver* s = NULL;
    EXPECT(svm_test_solver_create(&X, y, &p, NULL), SVM_E_INVALID);
    EXPECT(svm_test_solver_create(&X, bad_y, &p, &s), SVM_E_INVALID);
    double a[10], F[10], g = 0, b = 0, obj = 0;
    int32_t Bv[16], nB = 0, status = 0;
    int64_t it = 0;
    EXPECT(svm_test_set_state(NULL, a, F), SVM_E_INVALID);
    EXPECT(svm_test_get_state(NULL, a, F), SVM_E_INVALID);
    EXPECT(svm_test_select(NULL, Bv, &nB, &g, &b), SVM_E_INVALID);
    EXPECT(svm_test_iterate(NULL, 1, &it, &g), SVM_E_INVALID);
    EXPECT(svm_test_finish(NULL, 0, &g, &b, &obj, &status), SVM_E_INVALID);
    svm_test_solver_free(NULL);

    /* valid arguments: refused for the device ordinal alone */
    q = p;
    q.device = 1000;
    expect_no_device(svm_train(&X, y, &q, &m), __LINE__);
    expect_no_device(svm_train(&C, y, &q, &m), __LINE__);
    expect_no_device(svm_train_ovr(&X, labels, 3, &q, &m), __LINE__);
    expect_no_device(
        svm_cross_validate(&X, y, NULL, 0, &q, 2, NULL, NULL, &st), __LINE__);
    expect_no_device(svm_test_solver_create(&X, y, &q, &s), __LINE__);

    /* the kept row-cache memory: nothing kept, nothing freed (every device
       of the process: no device call when no block is kept); an ordinal
       out of range is refused */
    {
        int64_t freed = -1;
        EXPECT(svm_cache_release(-1, &freed), SVM_OK);
        if (freed != 0) {
            fprintf(stderr, "line %d: freed %lld, expected 0\n", __LINE__,
                    (long long)freed);
            ++failures;
        }
        EXPECT(svm_cache_release(-1, NULL), SVM_OK);
        expect_no_device(svm_cache_release(1000, &freed), __LINE__);
    }

    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("ABI driver: all checks passed\n");
    return 0;
}
