/*
 * mi355svm.h -- C ABI of a kernel-SVM dual solver for one AMD Instinct
 * MI355X (gfx950).
 *
 * The library trains C-SVC and eps-SVR models with the linear, polynomial,
 * RBF or sigmoid kernel by the working-set decomposition of Wang et al.,
 * "Rgtsvm: Support Vector Machines on a GPU in R" (arXiv 1706.05544), and
 * evaluates their decision function.
 * Everything that computes runs in hand-written HIP kernels; this header
 * only moves pointers and sizes.
 *
 * Problem (Section 3, Eq. 2):
 *     min_a  1/2 a^T Q a + p^T a   s.t.  y^T a = 0,  0 <= a_t <= C,
 *     Q_ts = y_t y_s K(x_smp(t), x_smp(s)),  K one of the kernels below.
 *   C-SVC:   one variable per sample, y_t = label in {+1,-1}, p_t = -1.
 *   eps-SVR: two variables per sample (Section 3, "positive and negative
 *            copy"; Eq. 1): copy (i,+) with y = +1, p = eps - z_i and copy
 *            (i,-) with y = -1, p = eps + z_i.
 * Decision function: D(x) = sum_i c_i K(x_i, x) + b with c_i = y_i a_i
 * (C-SVC) or c_i = a_(i,+) - a_(i,-) (eps-SVR).
 *
 * Conventions shared by every call:
 *   - status: 0 OK, > 0 warning (result valid), < 0 error (nothing written,
 *     *out set to NULL where there is one).  svm_last_error() returns a
 *     thread-local message for the last non-OK status.
 *   - All argument validation happens before any device call, so invalid
 *     arguments are reported even on a machine without a GPU.
 *   - Host inputs are read during the call and copied once to the device;
 *     they are never retained.  Device inputs (on_device = 1) are borrowed
 *     for the duration of the call and used on params->stream (dense ones
 *     with ld = d, d a multiple of 4 and 16-byte aligned values are read
 *     in place, not copied; they are never written).
 *   - Calls are synchronous: they return after the device work they queued
 *     has finished.  Models and solvers are not shared between threads
 *     without external locking.
 */
#ifndef MI355SVM_H
#define MI355SVM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SVM_OK = 0,
    SVM_W_MAX_ITER = 1,        /* max_iter reached; model valid, gap > tol */
    SVM_W_NOT_CONVERGED = 2,   /* the gap met tol on the incrementally
                                  updated responses but not, after 3
                                  re-runs, on responses recomputed from
                                  alpha; model valid, gap (recomputed) > tol */
    SVM_E_INVALID = -1,        /* bad argument (message says which) */
    SVM_E_UNSUPPORTED = -2,    /* valid but not implemented (e.g. kernel) */
    SVM_E_NOMEM = -3,          /* device or host allocation failed */
    SVM_E_DEVICE = -4,         /* no usable GPU, or a HIP runtime error */
    SVM_E_INTERNAL = -5
} svm_status;

typedef enum { SVM_C_SVC = 0, SVM_EPS_SVR = 1 } svm_type;

/* The four kernels of Section 3's list, in the e1071 (LIBSVM)
 * parameterisation (the paper names them without formulas):
 *   linear      K(u,v) = u.v
 *   polynomial  K(u,v) = (gamma u.v + coef0)^degree
 *   RBF         K(u,v) = exp(-gamma |u - v|^2)
 *   sigmoid     K(u,v) = tanh(gamma u.v + coef0)
 * Kernel values are computed in fp32 from an fp32 dot product; the
 * sigmoid kernel is not positive semidefinite in general (a pair of
 * non-positive curvature gets the floor 1e-12, as in LIBSVM). */
typedef enum {
    SVM_KERNEL_LINEAR = 0,
    SVM_KERNEL_POLY = 1,
    SVM_KERNEL_RBF = 2,
    SVM_KERNEL_SIGMOID = 3
} svm_kernel;

typedef enum { SVM_DENSE = 0, SVM_CSR = 1 } svm_layout;

/* A feature matrix of n rows and d columns.
 *   dense: values[i*ld + k], fp32, ld >= d.
 *   CSR:   row_ptr[0..n] (row_ptr[0] = 0, nondecreasing, row_ptr[n] = nnz),
 *          col_idx[nnz] sorted and unique within each row, in [0, d),
 *          values[nnz].
 * on_device = 1: every pointer is device memory of params->device. */
typedef struct {
    int32_t layout;
    int32_t on_device;
    int64_t n, d;
    const float *values;
    int64_t ld;
    const int64_t *row_ptr;
    const int32_t *col_idx;
    int64_t nnz;
} svm_matrix;

typedef struct {
    int32_t type;          /* svm_type */
    int32_t kernel;        /* svm_kernel */
    double C;              /* > 0 */
    double epsilon;        /* >= 0, eps-SVR tube half-width */
    double gamma;          /* >= 0; 0 means 1/d (the e1071 default) */
    double tol;            /* > 0; stop when max_{I_up} v - min_{I_low} v <= tol */
    int64_t max_iter;      /* outer iterations; <= 0: max(1e7, 100 N) */
    int32_t working_set;   /* q, even, in [2, 64]; 16 as in Section 3 */
    int32_t device;        /* HIP device ordinal */
    int64_t cache_bytes;   /* kernel-row cache budget; < 0 off; 0 default:
                              the whole K if it fits a quarter of the free
                              device memory, else a quarter of it, at most
                              8 GiB (the memory is kept for the next
                              training: svm_cache_release) */
    void *stream;          /* hipStream_t; NULL: a stream of the library */
    int32_t check_every;   /* outer iterations between host polls (0: 64;
                              fewer near convergence, down to an eighth,
                              from the rate at which the gap falls) */
    double inner_ratio;    /* subproblem stops at local gap <= max(ratio *
                              global gap, tol/2); 0: 0.3 */
    int32_t max_inner;     /* subproblem step cap; 0: 8 q */
    int32_t profile;       /* 1: time the row/update kernel with events
                              (a sample: the launches of one chunk of
                              check_every iterations in four); 2: also the
                              select/solve kernel of those iterations (a
                              timed launch of it costs the loop ~5 us) */
    double coef0;          /* polynomial and sigmoid offset (finite; 0) */
    int32_t degree;        /* polynomial degree, in [1, 64] (3) */
    int32_t scale;         /* 1: standardise each feature (and eps-SVR
                              targets) to mean 0 and sample sd 1 before
                              training, as e1071 does; dense X only; the
                              model applies the same statistics to the rows
                              it predicts (0: inputs used as given) */
    const double *alpha0;  /* warm start for svm_train: N host values (n for
                              C-SVC, 2n for eps-SVR: copy (i,+) then (i,-))
                              with 0 <= a <= C and y^T a = 0 (checked to
                              1e-9 C N when y is in host memory); the solve
                              starts there instead of at 0.  NULL: 0.  Not
                              for one-vs-rest or cross-validation */
    int32_t lockstep;      /* one-vs-rest, cross-validation and svm_tune:
                              up to this many binary problems (classes,
                              folds; in svm_tune also of different grid
                              points) train in lockstep, their outer
                              iterations together, one selection launch (a
                              block per problem) and one pass over X per
                              iteration; each problem's result is the one
                              it has when trained alone without the row
                              cache, which lockstep does not use.  In [0, 4];
                              0 or 1: one problem after another.  Fewer
                              when the working-set rows of more would not
                              fit the row kernel's LDS (2 at d = 784).  > 1
                              needs dense X and working_set = 16, else
                              SVM_E_UNSUPPORTED.  No effect on svm_train.
                              train_ms of a problem then spans its group's
                              run (the groups' problems overlap in time) */
    int32_t fused;         /* 1: every outer iteration as one launch, in
                              which each block merges the selection
                              candidates and solves the subproblem itself
                              while its rows stream (Section 3's loop);
                              dense X and working_set <= 16 only, no row
                              cache.  0 (default): selection and row update
                              as two launches.  The result is the same bit
                              for bit; one launch has been the slower so far
                              (its blocks' selection chains run longer than
                              the stream they hide) */
} svm_params;

/* Result of a k-fold cross-validation. */
typedef struct {
    int32_t folds;
    int32_t status;        /* SVM_OK or SVM_W_MAX_ITER (some fold) */
    int64_t n;             /* rows, each predicted by the model of the folds
                              it is not in */
    int64_t iters;         /* outer iterations over all trainings */
    double accuracy;       /* C-SVC / one-vs-rest: share of correct labels */
    double mse;            /* eps-SVR: mean squared error */
    double scc;            /* eps-SVR: squared correlation of D and targets */
    double error;          /* 1 - accuracy (C-SVC), or mse (eps-SVR) */
    int64_t kernel_rows;   /* kernel rows used over all trainings */
    /* params->profile = 1: the row/update launches that computed rows from
     * X, over all trainings (as in svm_model_info) */
    double row_kernel_ms;
    int64_t row_kernel_launches;
    double row_kernel_bytes;
} svm_cv_stats;

/* Per-output statistics of a trained model. */
typedef struct {
    int32_t type;          /* svm_type */
    int32_t n_outputs;     /* 1, or the number of classes (one-vs-rest) */
    int64_t n_train;       /* training samples */
    int64_t n_features;
    int64_t n_sv;          /* support rows stored (union over outputs) */
    double gamma;          /* resolved gamma */
    int32_t kernel;        /* svm_kernel of the model */
    int32_t degree;        /* its polynomial degree */
    double coef0;          /* its polynomial / sigmoid offset */
    /* the rest refers to the output asked for */
    int32_t status;        /* SVM_OK or SVM_W_MAX_ITER */
    int64_t n_sv_output;   /* samples with non-zero coefficient */
    int64_t n_bounded;     /* variables at C */
    int64_t iters;         /* outer iterations (working sets optimised) */
    double gap;            /* final m - M */
    double b;              /* bias */
    double dual_obj;       /* f(a) of Eq. 2 */
    int64_t kernel_rows;   /* kernel rows K(x_s, X) used (computed + cached) */
    int64_t cache_hits;    /* kernel rows served by the row cache */
    int64_t cache_fills;   /* kernel rows written to the row cache */
    double train_ms;       /* device time from solver start to model ready */
    /* profile = 1: row/update kernel launches that computed the rows from X */
    double row_kernel_ms;        /* summed kernel time */
    int64_t row_kernel_launches; /* launches included in row_kernel_ms */
    int64_t row_kernel_rows;     /* rows of X processed by those launches */
    double row_kernel_bytes;     /* their algorithmic HBM bytes */
    /* profile = 1: launches served entirely from the row cache */
    double cached_kernel_ms;
    int64_t cached_kernel_launches;
    double cached_kernel_bytes;
    /* profile = 2: the select/solve kernel of the same iterations (one
       block: merge, K_BB, subproblem; latency-bound) */
    double select_kernel_ms;
    int64_t select_kernel_launches;
} svm_model_info;

typedef struct svm_model svm_model;  /* opaque, owned by the library */

/* Defaults: C-SVC, RBF, C = 1, eps = 0.1, gamma = 0 (1/d), coef0 = 0,
 * degree = 3, tol = 1e-3, working_set = 16, device 0, NULL stream. */
void svm_params_default(svm_params *p);

/* Train a binary C-SVC (y = labels, each +1 or -1, both present) or an
 * eps-SVR (y = targets z).  y has n entries in the memory space of X.
 * On success *out receives a model the caller frees with svm_model_free. */
svm_status svm_train(const svm_matrix *X, const float *y,
                     const svm_params *p, svm_model **out);

/* One-vs-rest multi-class C-SVC (Section 3, multi-class classification):
 * labels in [0, n_classes), n_classes >= 2; one binary problem per class
 * (class c against the rest), all sharing X on the device. */
svm_status svm_train_ovr(const svm_matrix *X, const int32_t *labels,
                         int32_t n_classes, const svm_params *p,
                         svm_model **out);

/* Decision values D (m x n_outputs, row-major, fp64) for the m rows of X,
 * written to `decision` in the memory space of X (caller-owned). */
svm_status svm_predict(const svm_model *m, const svm_matrix *X,
                       double *decision);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * decision values of svm_predict (bitwise the same kernels and values) for
 * the m dense rows of X, which must be in device memory (layout SVM_DENSE,
 * on_device = 1, any ld >= d), into `decision` (device, m x n_outputs,
 * row-major fp64, caller-owned), queued on `stream` (hipStream_t; NULL:
 * the null stream) and NOT waited for: the values are there when the
 * stream's work up to this call has finished.  The call allocates nothing,
 * frees nothing and does not synchronise with the host: the rows are
 * staged, chunk by chunk, in a static array of 32 MiB per device (held by
 * each GPU the library runs on until the process ends), which every call
 * on that GPU shares, so calls that overlap in time on one GPU race.  X is
 * not checked for finite values (a non-finite row gives non-finite
 * decision values).  Errors: SVM_E_UNSUPPORTED for CSR or host rows, or a
 * row too long for the staging array (over about 8.3 million features);
 * SVM_E_INVALID for a NULL model or output or a different number of
 * features. */
svm_status svm_predict_noalloc(const svm_model *m, const svm_matrix *X,
                               double *decision, void *stream);

/* Labels: +1 / -1 (D >= 0 gives +1) for C-SVC, argmax over classes (ties to
 * the lowest class) for one-vs-rest.  eps-SVR models: SVM_E_INVALID. */
svm_status svm_predict_labels(const svm_model *m, const svm_matrix *X,
                              int32_t *labels);

svm_status svm_model_get_info(const svm_model *m, int32_t output,
                              svm_model_info *info);

/* Host copies of one output: sv_idx[n_sv_output] (training-row indices,
 * increasing) and coef[n_sv_output]; alpha[N] (N = n or 2n) may be NULL. */
svm_status svm_model_get(const svm_model *m, int32_t output, int32_t *sv_idx,
                         double *coef, double *alpha);

void svm_model_free(svm_model *m);

/* Memory management of the library, not an operation of the method.  The
 * device memory of the kernel-row cache (svm_params.cache_bytes) is kept
 * per device between trainings, one block as large as the largest cache
 * used so far on that device, and lent to one training at a time (a
 * training that finds it in use allocates its own): allocating and freeing
 * tens of GB per training would make later allocations wait while the
 * driver clears the freed memory.  This frees the kept block of `device`
 * (device < 0: of every device) unless a training holds it, and writes
 * the bytes freed to *freed (nullable).  Errors: SVM_E_INVALID for a
 * device ordinal out of range, SVM_E_DEVICE without a HIP device. */
svm_status svm_cache_release(int32_t device, int64_t *freed);

/* k-fold cross-validation (Section 3's feature list: "K-fold cross
 * validation", "accuracy or correlation, mean square error").  Give either
 * y (n labels +-1 for C-SVC, or n targets for eps-SVR) with labels = NULL,
 * or labels (n class indices in [0, n_classes)) with y = NULL for
 * one-vs-rest.  fold: n host entries in [0, k), every fold non-empty, or
 * NULL for fold i mod k.  For each fold the model is trained on the other
 * rows (their dual restricted to those rows: the held-out variables stay
 * at 0) and predicts the held-out rows: decision (host, n x n_outputs,
 * nullable) receives every row's decision value from the model that did
 * not see it; stats the metrics over all rows.  With params->scale the
 * data are standardised once over all rows.  y, labels and fold in host
 * memory (X may be on the device).  Returns SVM_W_MAX_ITER when some
 * training stopped at max_iter (results still written). */
svm_status svm_cross_validate(const svm_matrix *X, const float *y,
                              const int32_t *labels, int32_t n_classes,
                              const svm_params *params, int32_t k,
                              const int32_t *fold, double *decision,
                              svm_cv_stats *stats);

/* Grid tuning by cross-validation (Section 3: "tuning parameters ... (C,
 * eps)", e1071's tune): for grid point g the parameters are params with C
 * = C[g], gamma = gamma[g] and epsilon = epsilon[g] (each array nullable:
 * then params' value), and cv_error[g] the k-fold error (1 - accuracy, or
 * the MSE for eps-SVR) on the given folds; *best = the first g of least
 * error.  Same inputs as svm_cross_validate. */
svm_status svm_tune(const svm_matrix *X, const float *y,
                    const int32_t *labels, int32_t n_classes,
                    const svm_params *params, int32_t k, const int32_t *fold,
                    int32_t n_grid, const double *C, const double *gamma,
                    const double *epsilon, double *cv_error, int32_t *best);

const char *svm_last_error(void);

/* ------------------------------------------------------------------------
 * Test hooks: a solver whose state can be set and stepped one phase at a
 * time, so the tests can compare single steps with the CPU oracle from an
 * identical state.  Not needed for training.  Host pointers only.
 * ---------------------------------------------------------------------- */
typedef struct svm_solver svm_solver;

svm_status svm_test_solver_create(const svm_matrix *X, const float *y,
                                  const svm_params *p, svm_solver **out);
void svm_test_solver_free(svm_solver *s);

/* Replace the state: alpha[N] and responses F[n] (fp64). */
svm_status svm_test_set_state(svm_solver *s, const double *alpha,
                              const double *F);
svm_status svm_test_get_state(svm_solver *s, double *alpha, double *F);

/* Working-set selection on the current state: the q/2 largest keys of I_up
 * interleaved with the q/2 smallest of I_low, ties to the lowest index:
 * B[<= q] variable indices, *nB, and m = max_{I_up} v, M = min_{I_low} v. */
svm_status svm_test_select(svm_solver *s, int32_t *B, int32_t *nB, double *m,
                           double *M);

/* Kernel rows K(x_samples[j], X) for k <= 64 samples: out[j*n + i], fp32. */
svm_status svm_test_rows(svm_solver *s, const int32_t *samples, int32_t k,
                         float *out);

/* Solve the subproblem on B from the current state; returns the new
 * alpha_B and the number of inner steps (state unchanged). */
svm_status svm_test_subproblem(svm_solver *s, const int32_t *B, int32_t nB,
                               double inner_tol, int32_t max_inner,
                               double *alpha_B_new, int32_t *steps);

/* Set alpha_B to the given values and update F with the row/update kernel. */
svm_status svm_test_apply(svm_solver *s, const int32_t *B, int32_t nB,
                          const double *alpha_B_new);

/* Run up to k full outer iterations; *iters gets the count, *gap the gap. */
svm_status svm_test_iterate(svm_solver *s, int64_t k, int64_t *iters,
                            double *gap);

/* End a training on the current state as svm_train ends it: recompute F
 * from alpha, re-test the gap and, while it exceeds tol, run the loop again
 * and re-test, at most max_passes (>= 0) times (svm_train uses 3).  *gap,
 * *b (bias: the mean key over free variables, else (m + M) / 2) and
 * *obj (f(a)) come from the recomputed responses; *status is SVM_OK,
 * SVM_W_MAX_ITER or SVM_W_NOT_CONVERGED (the gap still above tol). */
svm_status svm_test_finish(svm_solver *s, int32_t max_passes, double *gap,
                           double *b, double *obj, int32_t *status);

#ifdef __cplusplus
}
#endif
#endif /* MI355SVM_H */
