// C ABI of the MI355X kernel-SVM library: argument validation, status codes,
// the thread-local error message, and dispatch to the solver.  Nothing here
// computes on the data; all arithmetic runs in the HIP kernels.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <memory>
#include <new>
#include <string>

#include "solver.hpp"

namespace {

thread_local std::string g_err;

svm_status fail(svm_status st, const std::string& msg)
{
    g_err = msg;
    return st;
}

bool finite_pos(double v) { return std::isfinite(v) && v > 0.0; }

// The warning status of a training whose model was written, with its
// message (SVM_OK: nothing to say).
svm_status warn(svm_status st, const char* where)
{
    if (st == SVM_W_MAX_ITER)
        return fail(st, std::string("max_iter reached before the gap met tol") +
                            where);
    if (st == SVM_W_NOT_CONVERGED)
        return fail(st, std::string("the gap on the responses recomputed from "
                                    "alpha stayed above tol") +
                            where);
    return SVM_OK;
}

svm_status check_params(const svm_params* p)
{
    if (!p) return fail(SVM_E_INVALID, "params is NULL");
    if (p->type != SVM_C_SVC && p->type != SVM_EPS_SVR)
        return fail(SVM_E_INVALID, "type must be SVM_C_SVC or SVM_EPS_SVR");
    if (p->kernel < SVM_KERNEL_LINEAR || p->kernel > SVM_KERNEL_SIGMOID)
        return fail(SVM_E_INVALID, "unknown kernel");
    if (!std::isfinite(p->coef0))
        return fail(SVM_E_INVALID, "coef0 must be finite");
    if (p->kernel == SVM_KERNEL_POLY && (p->degree < 1 || p->degree > 64))
        return fail(SVM_E_INVALID, "degree must be in [1, 64]");
    if (!finite_pos(p->C)) return fail(SVM_E_INVALID, "C must be finite and > 0");
    if (!std::isfinite(p->epsilon) || p->epsilon < 0)
        return fail(SVM_E_INVALID, "epsilon must be finite and >= 0");
    if (!std::isfinite(p->gamma) || p->gamma < 0)
        return fail(SVM_E_INVALID, "gamma must be finite and >= 0");
    if (!finite_pos(p->tol)) return fail(SVM_E_INVALID, "tol must be finite and > 0");
    if (p->working_set < 2 || p->working_set > msvm::kMaxQ ||
        (p->working_set & 1))
        return fail(SVM_E_INVALID, "working_set must be even and in [2, 64]");
    if (p->device < 0) return fail(SVM_E_INVALID, "device must be >= 0");
    if (p->check_every < 0) return fail(SVM_E_INVALID, "check_every must be >= 0");
    if (!std::isfinite(p->inner_ratio) || p->inner_ratio < 0 ||
        p->inner_ratio >= 1)
        return fail(SVM_E_INVALID, "inner_ratio must be in [0, 1)");
    if (p->max_inner < 0) return fail(SVM_E_INVALID, "max_inner must be >= 0");
    if (p->scale != 0 && p->scale != 1)
        return fail(SVM_E_INVALID, "scale must be 0 or 1");
    if (p->lockstep < 0 || p->lockstep > msvm::kLockMax)
        return fail(SVM_E_INVALID, "lockstep must be in [0, 4]");
    if (p->fused != 0 && p->fused != 1)
        return fail(SVM_E_INVALID, "fused must be 0 or 1");
    return SVM_OK;
}

// Lockstep group size for these features (1: one problem after another).
static int lock_group(const svm_params* p, const msvm::Features& f)
{
    if (p->lockstep <= 1) return 1;
    return std::min<int>(p->lockstep, msvm::Solver::lock_capacity(f, p->type));
}

// lockstep > 1 needs dense features and working sets of 16
static svm_status check_lockstep(const svm_params* p, const svm_matrix* X)
{
    if (p->lockstep > 1 && (X->layout != SVM_DENSE ||
                            p->working_set != 16))
        return fail(SVM_E_UNSUPPORTED,
                    "lockstep needs dense features and working_set = 16");
    return SVM_OK;
}

svm_status check_matrix(const svm_matrix* X, int64_t min_rows)
{
    if (!X) return fail(SVM_E_INVALID, "X is NULL");
    if (X->layout != SVM_DENSE && X->layout != SVM_CSR)
        return fail(SVM_E_INVALID, "unknown layout");
    if (X->n < min_rows)
        return fail(SVM_E_INVALID, min_rows > 1
                                       ? "X needs at least 2 rows"
                                       : "X rows must be >= 0");
    if (X->d < 1 || X->d > (int64_t)1 << 30)
        return fail(SVM_E_INVALID, "d must be in [1, 2^30]");
    if (X->layout == SVM_CSR) {
        if (!X->row_ptr) return fail(SVM_E_INVALID, "CSR row_ptr is NULL");
        if (X->nnz < 0) return fail(SVM_E_INVALID, "CSR nnz must be >= 0");
        if (X->nnz > 0 && (!X->col_idx || !X->values))
            return fail(SVM_E_INVALID, "CSR col_idx or values is NULL");
    } else {
        if (X->n > 0 && !X->values)
            return fail(SVM_E_INVALID, "X values is NULL");
        if (X->ld < X->d) return fail(SVM_E_INVALID, "ld must be >= d");
    }
    if (X->n > ((int64_t)1 << 31) - 1)
        return fail(SVM_E_INVALID, "n must be < 2^31");
    return SVM_OK;
}

svm_status check_device(int dev)
{
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count <= 0)
        return fail(SVM_E_DEVICE, "no HIP device available");
    if (dev >= count) return fail(SVM_E_INVALID, "device ordinal out of range");
    return SVM_OK;
}

svm_status check_host_labels(const float* y, int64_t n, int32_t type)
{
    if (type == SVM_EPS_SVR) {
        for (int64_t i = 0; i < n; ++i)
            if (!std::isfinite(y[i]))
                return fail(SVM_E_INVALID, "targets must be finite");
        return SVM_OK;
    }
    bool pos = false, neg = false;
    for (int64_t i = 0; i < n; ++i) {
        if (y[i] == 1.0f) pos = true;
        else if (y[i] == -1.0f) neg = true;
        else return fail(SVM_E_INVALID, "labels must be +1 or -1");
    }
    if (!pos || !neg) return fail(SVM_E_INVALID, "both classes must be present");
    return SVM_OK;
}

void fill_info(svm_model_info& in, const svm_model& m,
               const msvm::SolveResult& r)
{
    std::memset(&in, 0, sizeof(in));
    in.type = m.type;
    in.n_outputs = m.n_out;
    in.n_train = m.n_train;
    in.n_features = m.d;
    in.gamma = m.gamma;
    in.kernel = m.kf.kind;
    in.degree = m.kf.degree;
    in.coef0 = m.coef0;
    in.status = r.status;
    in.n_sv_output = r.n_sv;
    in.n_bounded = r.n_bounded;
    in.iters = r.iters;
    in.gap = r.gap;
    in.b = r.b;
    in.dual_obj = r.obj;
    in.kernel_rows = r.kernel_rows;
    in.cache_hits = r.cache_served;
    in.cache_fills = r.cache_filled;
    in.train_ms = r.train_ms;
    in.row_kernel_ms = r.row_ms;
    in.row_kernel_launches = r.row_launches;
    in.row_kernel_rows = r.row_rows;
    in.row_kernel_bytes = r.row_bytes;
    in.cached_kernel_ms = r.cached_ms;
    in.cached_kernel_launches = r.cached_launches;
    in.cached_kernel_bytes = r.cached_bytes;
    in.select_kernel_ms = r.select_ms;
    in.select_kernel_launches = r.select_launches;
}

// Leaves HIP's per-thread last-error slot clean on every exit, so that an
// error the library handled (or ignored while freeing) is not reported later
// by a caller's own error check.
struct ClearHipError {
    ~ClearHipError() { (void)hipGetLastError(); }
};

#define GUARD_BEGIN \
    ClearHipError clear_hip_error_on_exit_; \
    try {
#define GUARD_END                                                      \
    }                                                                  \
    catch (const msvm::Error& e) { return fail(e.status, e.msg); }     \
    catch (const std::bad_alloc&) {                                    \
        return fail(SVM_E_NOMEM, "host allocation failed");            \
    }                                                                  \
    catch (const std::exception& e) { return fail(SVM_E_INTERNAL, e.what()); } \
    catch (...) { return fail(SVM_E_INTERNAL, "unknown error"); }

}  // namespace

namespace msvm {
void set_error(svm_status st, const std::string& msg)
{
    (void)st;
    g_err = msg;
}
}  // namespace msvm

struct svm_solver {
    std::unique_ptr<msvm::Context> cx;
    msvm::Features f;
    msvm::DevBuf<float> y;
    std::unique_ptr<msvm::Solver> s;
};

extern "C" {

const char* svm_last_error(void) { return g_err.c_str(); }

void svm_params_default(svm_params* p)
{
    if (!p) return;
    std::memset(p, 0, sizeof(*p));
    p->type = SVM_C_SVC;
    p->kernel = SVM_KERNEL_RBF;
    p->C = 1.0;
    p->epsilon = 0.1;
    p->gamma = 0.0;
    p->tol = 1e-3;
    p->max_iter = 0;
    p->working_set = 16;
    p->device = 0;
    p->cache_bytes = 0;
    p->stream = nullptr;
    p->check_every = 0;
    p->inner_ratio = 0.0;
    p->max_inner = 0;
    p->profile = 0;
    p->coef0 = 0.0;
    p->degree = 3;
}

// A warm start: N finite values in [0, C] with y^T a = 0 (labels in host
// memory only; y == nullptr skips that test).
static svm_status check_warm_start(const double* a, const float* y, int64_t n,
                                   const svm_params* p)
{
    const int64_t N = p->type == SVM_EPS_SVR ? 2 * n : n;
    double s = 0.0;
    for (int64_t t = 0; t < N; ++t) {
        if (!std::isfinite(a[t]) || a[t] < 0.0 || a[t] > p->C)
            return fail(SVM_E_INVALID, "alpha0 must lie in [0, C]");
        if (p->type == SVM_EPS_SVR) s += t < n ? a[t] : -a[t];
        else if (y) s += y[t] > 0 ? a[t] : -a[t];
    }
    if ((p->type == SVM_EPS_SVR || y) &&
        std::fabs(s) > 1e-9 * p->C * (double)N)
        return fail(SVM_E_INVALID, "alpha0 must satisfy y^T alpha = 0");
    return SVM_OK;
}

// Standardises the training features (and, for eps-SVR, the targets) in
// place, keeping the statistics in the model for prediction.
static void scale_training(svm_model& m, msvm::Features& f, float* y_dev,
                           int32_t type, msvm::Context& cx)
{
    msvm::scale_fit(f, cx, m.x_mu, m.x_sd);
    msvm::scale_apply(f, cx, m.x_mu.p, m.x_sd.p);
    m.x_mu_h.resize((size_t)f.d);
    m.x_sd_h.resize((size_t)f.d);
    HIP_TRY(hipMemcpyAsync(m.x_mu_h.data(), m.x_mu.p,
                           (size_t)f.d * sizeof(double), hipMemcpyDeviceToHost,
                           cx.stream));
    HIP_TRY(hipMemcpyAsync(m.x_sd_h.data(), m.x_sd.p,
                           (size_t)f.d * sizeof(double), hipMemcpyDeviceToHost,
                           cx.stream));
    cx.sync();
    if (type == SVM_EPS_SVR && y_dev)
        msvm::scale_targets(y_dev, f.n, cx, &m.y_mu, &m.y_sd);
    m.scaled = true;
}

svm_status svm_train(const svm_matrix* X, const float* y, const svm_params* p,
                     svm_model** out)
{
    if (!out) return fail(SVM_E_INVALID, "out is NULL");
    *out = nullptr;
    svm_status st;
    if ((st = check_params(p)) != SVM_OK) return st;
    if ((st = check_matrix(X, 2)) != SVM_OK) return st;
    if (!y) return fail(SVM_E_INVALID, "y is NULL");
    if (!X->on_device && (st = check_host_labels(y, X->n, p->type)) != SVM_OK)
        return st;
    if (p->alpha0 &&
        (st = check_warm_start(p->alpha0, X->on_device ? nullptr : y, X->n,
                               p)) != SVM_OK)
        return st;
    if ((st = check_device(p->device)) != SVM_OK) return st;
    GUARD_BEGIN
    msvm::Context cx(p->device, p->stream);
    msvm::Features f;
    msvm::load_features(X, f, cx, true);
    msvm::DevBuf<float> yd((size_t)X->n);
    HIP_TRY(hipMemcpyAsync(yd.p, y, (size_t)X->n * sizeof(float),
                           X->on_device ? hipMemcpyDeviceToDevice
                                        : hipMemcpyHostToDevice,
                           cx.stream));
    auto m = std::make_unique<svm_model>();
    if (p->scale) scale_training(*m, f, yd.p, p->type, cx);
    msvm::SolveOptions o = msvm::make_options(p, X->n, X->d);
    msvm::RowCache rc;
    msvm::cache_init(rc, X->n, msvm::one_launch_loop(o, f) ? -1 : p->cache_bytes,
                     cx);
    msvm::Solver s(cx, f, yd.p, o, &rc);
    if (p->alpha0) s.warm_start(p->alpha0);
    msvm::SolveResult r = s.train();

    m->type = p->type;
    m->n_out = 1;
    m->n_train = X->n;
    m->d = X->d;
    m->ldp = f.ldp;
    m->gamma = o.gamma;
    m->kf = msvm::kernel_fn(o);
    m->coef0 = o.coef0;
    m->device = p->device;
    m->b.assign(1, r.b);
    msvm::DevBuf<double> coef((size_t)X->n);
    s.coefficients(coef.p, 1, 0);
    msvm::build_model(*m, cx, f, coef.p, 1);
    m->alpha.resize(1);
    m->alpha[0].resize((size_t)s.N());
    s.get_alpha(m->alpha[0].data());
    m->info.resize(1);
    fill_info(m->info[0], *m, r);
    *out = m.release();
    return warn(r.status, "");
    GUARD_END
}

svm_status svm_train_ovr(const svm_matrix* X, const int32_t* labels,
                         int32_t n_classes, const svm_params* p,
                         svm_model** out)
{
    if (!out) return fail(SVM_E_INVALID, "out is NULL");
    *out = nullptr;
    svm_status st;
    if ((st = check_params(p)) != SVM_OK) return st;
    if (p->type != SVM_C_SVC)
        return fail(SVM_E_INVALID, "one-vs-rest needs type SVM_C_SVC");
    if (p->alpha0)
        return fail(SVM_E_INVALID, "alpha0 is for svm_train only");
    if ((st = check_matrix(X, 2)) != SVM_OK) return st;
    if ((st = check_lockstep(p, X)) != SVM_OK) return st;
    if (!labels) return fail(SVM_E_INVALID, "labels is NULL");
    if (n_classes < 2 || n_classes > 16)
        return fail(SVM_E_INVALID, "n_classes must be in [2, 16]");
    if (!X->on_device) {
        std::vector<int64_t> cnt((size_t)n_classes, 0);
        for (int64_t i = 0; i < X->n; ++i) {
            if (labels[i] < 0 || labels[i] >= n_classes)
                return fail(SVM_E_INVALID, "labels must be in [0, n_classes)");
            cnt[(size_t)labels[i]]++;
        }
        for (int32_t c = 0; c < n_classes; ++c)
            if (cnt[(size_t)c] == 0)
                return fail(SVM_E_INVALID, "every class needs a sample");
    }
    if ((st = check_device(p->device)) != SVM_OK) return st;
    GUARD_BEGIN
    msvm::Context cx(p->device, p->stream);
    msvm::Features f;
    msvm::load_features(X, f, cx, true);
    const int64_t n = X->n;
    msvm::DevBuf<int32_t> ld((size_t)n);
    HIP_TRY(hipMemcpyAsync(ld.p, labels, (size_t)n * sizeof(int32_t),
                           X->on_device ? hipMemcpyDeviceToDevice
                                        : hipMemcpyHostToDevice,
                           cx.stream));
    if (X->on_device) {
        msvm::DevBuf<int32_t> bad(1);
        HIP_TRY(hipMemsetAsync(bad.p, 0, sizeof(int32_t), cx.stream));
        msvm::launch_check_labels(ld.p, n, n_classes, bad.p, cx.stream);
        int32_t hb = 0;
        HIP_TRY(hipMemcpyAsync(&hb, bad.p, sizeof(int32_t),
                               hipMemcpyDeviceToHost, cx.stream));
        cx.sync();
        if (hb) return fail(SVM_E_INVALID, "labels must be in [0, n_classes)");
    }
    auto m = std::make_unique<svm_model>();
    if (p->scale) scale_training(*m, f, nullptr, SVM_C_SVC, cx);
    msvm::SolveOptions o = msvm::make_options(p, n, X->d);
    m->type = SVM_C_SVC;
    m->n_out = n_classes;
    m->n_train = n;
    m->d = X->d;
    m->ldp = f.ldp;
    m->gamma = o.gamma;
    m->kf = msvm::kernel_fn(o);
    m->coef0 = o.coef0;
    m->device = p->device;
    m->b.assign((size_t)n_classes, 0.0);
    m->alpha.resize((size_t)n_classes);
    m->info.resize((size_t)n_classes);
    msvm::DevBuf<double> coef((size_t)(n * n_classes));
    msvm::DevBuf<float> yc((size_t)n);
    std::vector<msvm::SolveResult> res((size_t)n_classes);
    svm_status worst = SVM_OK;
    // one row cache for all classes: the kernel rows do not depend on labels
    msvm::RowCache rc;
    msvm::cache_init(rc, n, msvm::one_launch_loop(o, f) ? -1 : p->cache_bytes,
                     cx);
    auto collect = [&](int32_t c, msvm::Solver& s, const msvm::SolveResult& r) {
        res[(size_t)c] = r;
        s.coefficients(coef.p, n_classes, c);
        m->b[(size_t)c] = r.b;
        m->alpha[(size_t)c].resize((size_t)s.N());
        s.get_alpha(m->alpha[(size_t)c].data());
        if (r.status != SVM_OK) worst = r.status;
    };
    const int L = lock_group(p, f);
    for (int32_t c0 = 0; c0 < n_classes; c0 += L) {
        const int G = std::min<int>(L, n_classes - c0);
        if (G == 1) {
            msvm::launch_ovr_labels(ld.p, n, c0, yc.p, cx.stream);
            msvm::Solver s(cx, f, yc.p, o, L > 1 ? nullptr : &rc);
            collect(c0, s, s.train());
            continue;
        }
        std::vector<std::unique_ptr<msvm::Solver>> ss;
        std::vector<msvm::Solver*> gp;
        for (int j = 0; j < G; ++j) {
            msvm::launch_ovr_labels(ld.p, n, c0 + j, yc.p, cx.stream);
            ss.emplace_back(new msvm::Solver(cx, f, yc.p, o));
            gp.push_back(ss.back().get());
        }
        const std::vector<msvm::SolveResult> rr =
            msvm::Solver::train_lockstep(gp);
        for (int j = 0; j < G; ++j) collect(c0 + j, *gp[j], rr[(size_t)j]);
    }
    msvm::build_model(*m, cx, f, coef.p, n_classes);
    for (int32_t c = 0; c < n_classes; ++c)
        fill_info(m->info[(size_t)c], *m, res[(size_t)c]);
    *out = m.release();
    return warn(worst, " (at least one class)");
    GUARD_END
}

static svm_status predict_impl(const svm_model* mdl, const svm_matrix* X,
                               double* decision, int32_t* labels)
{
    if (!mdl) return fail(SVM_E_INVALID, "model is NULL");
    svm_status st;
    if ((st = check_matrix(X, 0)) != SVM_OK) return st;
    if (X->d != mdl->d)
        return fail(SVM_E_INVALID, "X has a different number of features");
    if (X->n > 0 && !decision && !labels)
        return fail(SVM_E_INVALID, "output is NULL");
    if (labels && mdl->type == SVM_EPS_SVR)
        return fail(SVM_E_INVALID, "labels are undefined for eps-SVR");
    if (X->n == 0) return SVM_OK;
    if ((st = check_device(mdl->device)) != SVM_OK) return st;
    GUARD_BEGIN
    msvm::Context cx(mdl->device, nullptr);
    msvm::Features t;
    msvm::load_features(X, t, cx, true);
    const int64_t m = X->n;
    msvm::DevBuf<double> D((size_t)(m * mdl->n_out));
    msvm::predict_device(*mdl, cx, t, D.p);
    const hipMemcpyKind kind =
        X->on_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost;
    if (decision) {
        HIP_TRY(hipMemcpyAsync(decision, D.p,
                               (size_t)(m * mdl->n_out) * sizeof(double), kind,
                               cx.stream));
    } else {
        msvm::DevBuf<int32_t> L((size_t)m);
        msvm::launch_argmax_labels(D.p, m, mdl->n_out, mdl->type, L.p,
                                   cx.stream);
        HIP_TRY(hipMemcpyAsync(labels, L.p, (size_t)m * sizeof(int32_t), kind,
                               cx.stream));
        cx.sync();
    }
    cx.sync();
    return SVM_OK;
    GUARD_END
}

svm_status svm_predict(const svm_model* m, const svm_matrix* X,
                       double* decision)
{
    if (X && X->n > 0 && !decision)
        return fail(SVM_E_INVALID, "decision is NULL");
    msvm::Range rg("svm_predict");
    return predict_impl(m, X, decision, nullptr);
}

svm_status svm_predict_noalloc(const svm_model* m, const svm_matrix* X,
                               double* decision, void* stream)
{
    if (!m) return fail(SVM_E_INVALID, "model is NULL");
    svm_status st;
    if ((st = check_matrix(X, 0)) != SVM_OK) return st;
    if (X->layout != SVM_DENSE || !X->on_device)
        return fail(SVM_E_UNSUPPORTED,
                    "svm_predict_noalloc takes dense rows in device memory");
    if (X->d != m->d)
        return fail(SVM_E_INVALID, "X has a different number of features");
    if (X->n == 0) return SVM_OK;
    if (!decision) return fail(SVM_E_INVALID, "decision is NULL");
    if (msvm::noalloc_rows_per_chunk(*m, X->values, X->ld) < 1)
        return fail(SVM_E_UNSUPPORTED,
                    "a row of X does not fit the staging array of "
                    "svm_predict_noalloc (32 MiB)");
    if ((st = check_device(m->device)) != SVM_OK) return st;
    GUARD_BEGIN
    HIP_TRY(hipSetDevice(m->device));
    msvm::predict_noalloc(*m, X->values, X->n, X->ld, decision,
                          (hipStream_t)stream);
    return SVM_OK;
    GUARD_END
}

svm_status svm_predict_labels(const svm_model* m, const svm_matrix* X,
                              int32_t* labels)
{
    if (X && X->n > 0 && !labels) return fail(SVM_E_INVALID, "labels is NULL");
    if (m && m->type == SVM_EPS_SVR)
        return fail(SVM_E_INVALID, "labels are undefined for eps-SVR");
    return predict_impl(m, X, nullptr, labels);
}

// ---------------------------------------------------------------------------
// k-fold cross-validation and grid tuning (Section 3's feature list)
// ---------------------------------------------------------------------------

namespace {

// Validation shared by cross-validation and tuning: exactly one of y
// (C-SVC / eps-SVR) and labels (one-vs-rest over n_classes), and the folds.
svm_status check_cv(const svm_matrix* X, const float* y,
                    const int32_t* labels, int32_t n_classes,
                    const svm_params* p, int32_t k, const int32_t* fold)
{
    svm_status st;
    if ((st = check_params(p)) != SVM_OK) return st;
    if (p->alpha0)
        return fail(SVM_E_INVALID, "alpha0 is for svm_train only");
    if ((st = check_matrix(X, 2)) != SVM_OK) return st;
    if ((st = check_lockstep(p, X)) != SVM_OK) return st;
    if ((y != nullptr) == (labels != nullptr))
        return fail(SVM_E_INVALID, "give exactly one of y and labels");
    if (labels) {
        if (p->type != SVM_C_SVC)
            return fail(SVM_E_INVALID, "one-vs-rest needs type SVM_C_SVC");
        if (n_classes < 2 || n_classes > 16)
            return fail(SVM_E_INVALID, "n_classes must be in [2, 16]");
        for (int64_t i = 0; i < X->n; ++i)
            if (labels[i] < 0 || labels[i] >= n_classes)
                return fail(SVM_E_INVALID, "labels must be in [0, n_classes)");
    } else {
        if ((st = check_host_labels(y, X->n, p->type)) != SVM_OK) return st;
    }
    if (k < 2 || (int64_t)k > X->n)
        return fail(SVM_E_INVALID, "folds must be in [2, n]");
    if (fold) {
        std::vector<int64_t> cnt((size_t)k, 0);
        for (int64_t i = 0; i < X->n; ++i) {
            if (fold[i] < 0 || fold[i] >= k)
                return fail(SVM_E_INVALID, "fold entries must be in [0, k)");
            cnt[(size_t)fold[i]]++;
        }
        for (int32_t f = 0; f < k; ++f)
            if (cnt[(size_t)f] == 0)
                return fail(SVM_E_INVALID, "every fold needs a row");
    }
    return check_device(p->device);
}

// Everything a run of cross-validations over one data set shares: the
// feature store (scaled once, as for a training on all rows), the labels
// or targets, the folds and the truth for the metrics.
struct CvData {
    msvm::Features f;
    msvm::DevBuf<float> y;        // targets (scaled for eps-SVR), or +-1
    msvm::DevBuf<float> y_true;   // the targets or labels as given
    msvm::DevBuf<int32_t> labels; // one-vs-rest
    msvm::DevBuf<int32_t> fold;
    double y_mu = 0.0, y_sd = 0.0;
    int32_t n_out = 1;
};

void cv_load(CvData& c, const svm_matrix* X, const float* y,
             const int32_t* labels, int32_t n_classes, const svm_params* p,
             int32_t k, const int32_t* fold, msvm::Context& cx)
{
    const int64_t n = X->n;
    msvm::load_features(X, c.f, cx, true);
    if (p->scale) {
        msvm::DevBuf<double> mu, sd;
        msvm::scale_fit(c.f, cx, mu, sd);
        msvm::scale_apply(c.f, cx, mu.p, sd.p);
    }
    std::vector<int32_t> fh((size_t)n);
    for (int64_t i = 0; i < n; ++i)
        fh[(size_t)i] = fold ? fold[i] : (int32_t)(i % k);
    c.fold.alloc((size_t)n);
    HIP_TRY(hipMemcpyAsync(c.fold.p, fh.data(), (size_t)n * sizeof(int32_t),
                           hipMemcpyHostToDevice, cx.stream));
    c.y.alloc((size_t)n);
    if (labels) {
        c.n_out = n_classes;
        c.labels.alloc((size_t)n);
        HIP_TRY(hipMemcpyAsync(c.labels.p, labels, (size_t)n * sizeof(int32_t),
                               hipMemcpyHostToDevice, cx.stream));
    } else {
        c.y_true.alloc((size_t)n);
        HIP_TRY(hipMemcpyAsync(c.y_true.p, y, (size_t)n * sizeof(float),
                               hipMemcpyHostToDevice, cx.stream));
        HIP_TRY(hipMemcpyAsync(c.y.p, y, (size_t)n * sizeof(float),
                               hipMemcpyHostToDevice, cx.stream));
        if (p->scale && p->type == SVM_EPS_SVR)
            msvm::scale_targets(c.y.p, n, cx, &c.y_mu, &c.y_sd);
    }
    cx.sync();
}

// Totals of the trainings of one cross-validation.
struct CvAcc {
    int64_t iters = 0, kernel_rows = 0, row_launches = 0;
    double row_ms = 0.0, row_bytes = 0.0;
    svm_status worst = SVM_OK;
};

// Metrics of one cross-validation's decision values D (device, n x n_out)
// into stats.
void cv_finish(CvData& c, const svm_params* p, int32_t k, double* D,
               const CvAcc& a, svm_cv_stats* stats, msvm::Context& cx)
{
    const int64_t n = c.f.n;
    if (p->type == SVM_EPS_SVR && c.y_sd > 0.0)
        msvm::launch_affine(D, n, c.y_sd, c.y_mu, cx.stream);
    msvm::DevBuf<double> sums(7);
    msvm::launch_metrics(p->type, c.n_out, D, c.y_true.p, c.labels.p, n,
                         sums.p, cx.stream);
    double h[7];
    HIP_TRY(hipMemcpyAsync(h, sums.p, sizeof(h), hipMemcpyDeviceToHost,
                           cx.stream));
    cx.sync();
    std::memset(stats, 0, sizeof(*stats));
    stats->folds = k;
    stats->n = n;
    stats->status = a.worst;
    stats->iters = a.iters;
    stats->kernel_rows = a.kernel_rows;
    stats->row_kernel_ms = a.row_ms;
    stats->row_kernel_launches = a.row_launches;
    stats->row_kernel_bytes = a.row_bytes;
    const double nn = (double)n;
    if (p->type == SVM_C_SVC) {
        stats->accuracy = h[0] / nn;
        stats->error = 1.0 - stats->accuracy;
    } else {
        stats->mse = h[1] / nn;
        const double num = nn * h[6] - h[2] * h[3];
        const double den = (nn * h[4] - h[2] * h[2]) * (nn * h[5] - h[3] * h[3]);
        stats->scc = den > 0.0 ? num * num / den : 0.0;
        stats->error = stats->mse;
    }
}

// Cross-validations of the parameter sets ps (one D and stats each): k
// trainings each (per class for one-vs-rest), each on the rows outside one
// fold; the decision values of the held-out rows into D[g] (device, n x
// n_out), then the metrics.  One after another with a row cache per
// parameter set, or every (parameter set, fold, class) training in
// lockstep groups.
svm_status cv_run_many(CvData& c, const std::vector<svm_params>& ps,
                       int32_t k, const std::vector<double*>& D,
                       std::vector<svm_cv_stats>& stats, msvm::Context& cx)
{
    const int64_t n = c.f.n;
    const int NG = (int)ps.size();
    std::vector<msvm::SolveOptions> opts;
    for (const auto& p : ps) opts.push_back(msvm::make_options(&p, n, c.f.d));
    std::vector<CvAcc> acc((size_t)NG);
    auto collect = [&](int g, int32_t fo, int32_t cl, msvm::Solver& s,
                       const msvm::SolveResult& r) {
        s.cv_decision(D[(size_t)g], c.n_out, cl, c.fold.p, fo, r.b);
        CvAcc& a = acc[(size_t)g];
        a.iters += r.iters;
        a.kernel_rows += r.kernel_rows;
        a.row_ms += r.row_ms;
        a.row_bytes += r.row_bytes;
        a.row_launches += r.row_launches;
        if (r.status != SVM_OK) a.worst = r.status;
    };
    const int L = lock_group(&ps[0], c.f);
    const int32_t per = k * c.n_out;  // trainings of one parameter set
    if (L == 1) {
        for (int g = 0; g < NG; ++g) {
            msvm::RowCache rc;  // K rows do not depend on fold or class
            msvm::cache_init(rc, n,
                             msvm::one_launch_loop(opts[(size_t)g], c.f)
                                 ? -1
                                 : ps[(size_t)g].cache_bytes,
                             cx);
            for (int32_t t = 0; t < per; ++t) {
                const int32_t fo = t / c.n_out, cl = t % c.n_out;
                if (c.labels.p)
                    msvm::launch_ovr_labels(c.labels.p, n, cl, c.y.p,
                                            cx.stream);
                msvm::Solver s(cx, c.f, c.y.p, opts[(size_t)g], &rc,
                               c.fold.p, fo);
                collect(g, fo, cl, s, s.train());
            }
        }
    } else {
        const int32_t T = NG * per;
        for (int32_t t0 = 0; t0 < T; t0 += L) {
            const int G = std::min<int>(L, T - t0);
            std::vector<std::unique_ptr<msvm::Solver>> ss;
            std::vector<msvm::Solver*> gp;
            for (int j = 0; j < G; ++j) {
                const int32_t t = t0 + j, g = t / per, r = t % per;
                const int32_t fo = r / c.n_out, cl = r % c.n_out;
                if (c.labels.p)
                    msvm::launch_ovr_labels(c.labels.p, n, cl, c.y.p,
                                            cx.stream);
                ss.emplace_back(new msvm::Solver(cx, c.f, c.y.p,
                                                 opts[(size_t)g], nullptr,
                                                 c.fold.p, fo));
                gp.push_back(ss.back().get());
            }
            std::vector<msvm::SolveResult> rr;
            if (G == 1)
                rr.push_back(gp[0]->train());
            else
                rr = msvm::Solver::train_lockstep(gp);
            for (int j = 0; j < G; ++j) {
                const int32_t t = t0 + j, g = t / per, r = t % per;
                collect(g, r / c.n_out, r % c.n_out, *gp[(size_t)j],
                        rr[(size_t)j]);
            }
        }
    }
    stats.assign((size_t)NG, svm_cv_stats{});
    svm_status worst = SVM_OK;
    for (int g = 0; g < NG; ++g) {
        cv_finish(c, &ps[(size_t)g], k, D[(size_t)g], acc[(size_t)g],
                  &stats[(size_t)g], cx);
        if (acc[(size_t)g].worst != SVM_OK) worst = acc[(size_t)g].worst;
    }
    return worst;
}

}  // namespace

svm_status svm_cross_validate(const svm_matrix* X, const float* y,
                              const int32_t* labels, int32_t n_classes,
                              const svm_params* p, int32_t k,
                              const int32_t* fold, double* decision,
                              svm_cv_stats* stats)
{
    if (!stats) return fail(SVM_E_INVALID, "stats is NULL");
    svm_status st;
    if ((st = check_cv(X, y, labels, n_classes, p, k, fold)) != SVM_OK)
        return st;
    GUARD_BEGIN
    msvm::Context cx(p->device, p->stream);
    CvData c;
    cv_load(c, X, y, labels, n_classes, p, k, fold, cx);
    msvm::DevBuf<double> D((size_t)(X->n * c.n_out));
    std::vector<svm_cv_stats> sv;
    st = cv_run_many(c, std::vector<svm_params>(1, *p), k,
                     std::vector<double*>(1, D.p), sv, cx);
    *stats = sv[0];
    if (decision) {
        HIP_TRY(hipMemcpyAsync(decision, D.p,
                               (size_t)(X->n * c.n_out) * sizeof(double),
                               hipMemcpyDeviceToHost, cx.stream));
        cx.sync();
    }
    return warn(st, " (at least one fold)");
    GUARD_END
}

svm_status svm_tune(const svm_matrix* X, const float* y,
                    const int32_t* labels, int32_t n_classes,
                    const svm_params* p, int32_t k, const int32_t* fold,
                    int32_t n_grid, const double* C, const double* gamma,
                    const double* epsilon, double* cv_error, int32_t* best)
{
    if (n_grid < 1) return fail(SVM_E_INVALID, "n_grid must be >= 1");
    if (!cv_error || !best) return fail(SVM_E_INVALID, "outputs are NULL");
    svm_status st;
    if ((st = check_params(p)) != SVM_OK) return st;
    std::vector<svm_params> grid((size_t)n_grid, *p);
    for (int32_t g = 0; g < n_grid; ++g) {
        if (C) grid[(size_t)g].C = C[g];
        if (gamma) grid[(size_t)g].gamma = gamma[g];
        if (epsilon) grid[(size_t)g].epsilon = epsilon[g];
        if ((st = check_params(&grid[(size_t)g])) != SVM_OK) return st;
    }
    if ((st = check_cv(X, y, labels, n_classes, p, k, fold)) != SVM_OK)
        return st;
    GUARD_BEGIN
    msvm::Context cx(p->device, p->stream);
    CvData c;
    cv_load(c, X, y, labels, n_classes, p, k, fold, cx);
    // the decision values of every grid point (their trainings may share
    // lockstep groups)
    const size_t per = (size_t)(X->n * c.n_out);
    msvm::DevBuf<double> D(per * (size_t)n_grid);
    std::vector<double*> Dg;
    for (int32_t g = 0; g < n_grid; ++g) Dg.push_back(D.p + per * (size_t)g);
    std::vector<svm_cv_stats> cs;
    const svm_status worst = cv_run_many(c, grid, k, Dg, cs, cx);
    *best = 0;
    for (int32_t g = 0; g < n_grid; ++g) {
        cv_error[g] = cs[(size_t)g].error;
        if (cv_error[g] < cv_error[*best]) *best = g;  // ties: the first
    }
    return warn(worst, " (at least one fold)");
    GUARD_END
}

svm_status svm_model_get_info(const svm_model* m, int32_t output,
                              svm_model_info* info)
{
    if (!m || !info) return fail(SVM_E_INVALID, "model or info is NULL");
    if (output < 0 || output >= m->n_out)
        return fail(SVM_E_INVALID, "output out of range");
    *info = m->info[(size_t)output];
    info->n_sv = m->n_sv;
    return SVM_OK;
}

svm_status svm_model_get(const svm_model* m, int32_t output, int32_t* sv_idx,
                         double* coef, double* alpha)
{
    if (!m) return fail(SVM_E_INVALID, "model is NULL");
    if (output < 0 || output >= m->n_out)
        return fail(SVM_E_INVALID, "output out of range");
    int64_t k = 0;
    for (int64_t j = 0; j < m->n_sv; ++j) {
        double c = m->coef[(size_t)(j * m->n_out + output)];
        if (c == 0.0) continue;
        if (sv_idx) sv_idx[k] = m->sv_idx[(size_t)j];
        if (coef) coef[k] = c;
        ++k;
    }
    if (alpha) {
        const auto& a = m->alpha[(size_t)output];
        std::memcpy(alpha, a.data(), a.size() * sizeof(double));
    }
    return SVM_OK;
}

void svm_model_free(svm_model* m) { delete m; }

svm_status svm_cache_release(int32_t device, int64_t* freed)
{
    if (freed) *freed = 0;
    svm_status st;
    if (device >= 0 && (st = check_device(device)) != SVM_OK) return st;
    GUARD_BEGIN
    const size_t b = msvm::cache_pool_trim(device);
    if (freed) *freed = (int64_t)b;
    return SVM_OK;
    GUARD_END
}

svm_status svm_test_solver_create(const svm_matrix* X, const float* y,
                                  const svm_params* p, svm_solver** out)
{
    if (!out) return fail(SVM_E_INVALID, "out is NULL");
    *out = nullptr;
    svm_status st;
    if ((st = check_params(p)) != SVM_OK) return st;
    if ((st = check_matrix(X, 2)) != SVM_OK) return st;
    if (X->on_device) return fail(SVM_E_INVALID, "test hooks take host data");
    if (!y) return fail(SVM_E_INVALID, "y is NULL");
    if ((st = check_host_labels(y, X->n, p->type)) != SVM_OK) return st;
    if ((st = check_device(p->device)) != SVM_OK) return st;
    GUARD_BEGIN
    auto s = std::make_unique<svm_solver>();
    s->cx = std::make_unique<msvm::Context>(p->device, p->stream);
    msvm::load_features(X, s->f, *s->cx);
    s->y.alloc((size_t)X->n);
    HIP_TRY(hipMemcpyAsync(s->y.p, y, (size_t)X->n * sizeof(float),
                           hipMemcpyHostToDevice, s->cx->stream));
    s->s = std::make_unique<msvm::Solver>(
        *s->cx, s->f, s->y.p, msvm::make_options(p, X->n, X->d));
    *out = s.release();
    return SVM_OK;
    GUARD_END
}

void svm_test_solver_free(svm_solver* s) { delete s; }

#define SOLVER_CALL(body)                                        \
    if (!s) return fail(SVM_E_INVALID, "solver is NULL");        \
    GUARD_BEGIN body; return SVM_OK;                             \
    GUARD_END

svm_status svm_test_set_state(svm_solver* s, const double* alpha,
                              const double* F)
{
    if (!alpha || !F) return fail(SVM_E_INVALID, "alpha or F is NULL");
    SOLVER_CALL(s->s->set_state(alpha, F))
}

svm_status svm_test_get_state(svm_solver* s, double* alpha, double* F)
{
    SOLVER_CALL(s->s->get_state(alpha, F))
}

svm_status svm_test_select(svm_solver* s, int32_t* B, int32_t* nB, double* m,
                           double* M)
{
    if (!B || !nB || !m || !M) return fail(SVM_E_INVALID, "NULL output");
    SOLVER_CALL(s->s->select(B, nB, m, M))
}

svm_status svm_test_rows(svm_solver* s, const int32_t* samples, int32_t k,
                         float* out)
{
    if (!samples || !out || k < 1 || k > msvm::kMaxQ)
        return fail(SVM_E_INVALID, "need 1..64 samples and an output");
    if (s)
        for (int32_t j = 0; j < k; ++j)
            if (samples[j] < 0 || samples[j] >= s->f.n)
                return fail(SVM_E_INVALID, "sample index out of range");
    SOLVER_CALL(s->s->rows(samples, k, out))
}

svm_status svm_test_subproblem(svm_solver* s, const int32_t* B, int32_t nB,
                               double inner_tol, int32_t max_inner,
                               double* alpha_B_new, int32_t* steps)
{
    if (!B || !alpha_B_new || !steps || nB < 1 || nB > msvm::kMaxQ)
        return fail(SVM_E_INVALID, "need 1..64 variables and outputs");
    if (s)
        for (int32_t j = 0; j < nB; ++j)
            if (B[j] < 0 || B[j] >= s->s->N())
                return fail(SVM_E_INVALID, "variable index out of range");
    SOLVER_CALL(s->s->subproblem(B, nB, inner_tol, max_inner, alpha_B_new,
                                 steps))
}

svm_status svm_test_apply(svm_solver* s, const int32_t* B, int32_t nB,
                          const double* alpha_B_new)
{
    if (!B || !alpha_B_new || nB < 1 || nB > msvm::kMaxQ)
        return fail(SVM_E_INVALID, "need 1..64 variables");
    if (s)
        for (int32_t j = 0; j < nB; ++j)
            if (B[j] < 0 || B[j] >= s->s->N())
                return fail(SVM_E_INVALID, "variable index out of range");
    SOLVER_CALL(s->s->apply(B, nB, alpha_B_new))
}

svm_status svm_test_iterate(svm_solver* s, int64_t k, int64_t* iters,
                            double* gap)
{
    if (!iters || !gap || k < 0) return fail(SVM_E_INVALID, "bad arguments");
    SOLVER_CALL(s->s->iterate(k, iters, gap))
}

svm_status svm_test_finish(svm_solver* s, int32_t max_passes, double* gap,
                           double* b, double* obj, int32_t* status)
{
    if (!gap || !b || !obj || !status || max_passes < 0)
        return fail(SVM_E_INVALID, "bad arguments");
    if (!s) return fail(SVM_E_INVALID, "solver is NULL");
    GUARD_BEGIN
    msvm::SolveResult r;
    s->s->finish_state(max_passes, r);
    *gap = r.gap;
    *b = r.b;
    *obj = r.obj;
    *status = r.status;
    return SVM_OK;
    GUARD_END
}

}  // extern "C"
