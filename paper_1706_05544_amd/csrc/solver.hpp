// Host-side solver state of the MI355X kernel-SVM library.
#pragma once

#include <rocprofiler-sdk-roctx/roctx.h>

#include <memory>
#include <vector>

#include "common.hpp"

namespace msvm {

// A named host range for `rocprofv3 --marker-trace` (phases of a call:
// features, solve loop, finish, model, prediction); without a profiler the
// push and pop do nothing measurable.
struct Range {
    explicit Range(const char* name) { roctxRangePush(name); }
    ~Range() { roctxRangePop(); }
    Range(const Range&) = delete;
    Range& operator=(const Range&) = delete;
};

// RAII device buffer.
template <class T>
struct DevBuf {
    T* p = nullptr;
    size_t count = 0;
    DevBuf() = default;
    explicit DevBuf(size_t n) { alloc(n); }
    DevBuf(const DevBuf&) = delete;
    DevBuf& operator=(const DevBuf&) = delete;
    ~DevBuf() { release(); }
    void alloc(size_t n)
    {
        release();
        if (n == 0) n = 1;
        HIP_TRY(hipMalloc((void**)&p, n * sizeof(T)));
        count = n;
    }
    void release()
    {
        if (p) (void)hipFree(p);
        p = nullptr;
        count = 0;
    }
    size_t bytes() const { return count * sizeof(T); }
};

// Pinned host buffer.
template <class T>
struct HostBuf {
    T* p = nullptr;
    explicit HostBuf(size_t n)
    {
        HIP_TRY(hipHostMalloc((void**)&p, (n ? n : 1) * sizeof(T),
                              hipHostMallocDefault));
    }
    HostBuf(const HostBuf&) = delete;
    HostBuf& operator=(const HostBuf&) = delete;
    ~HostBuf()
    {
        if (p) (void)hipHostFree(p);
    }
};

// The support rows in chunks by column for the factored sparse decision
// path (factor.hip); ok == false: not built.
struct FactSV {
    bool ok = false;
    int32_t nch = 0, ldpm = 0, n_out = 0, fast = 0;
    double sv_nnz = 0.0;  // nonzeros of a support row, on average
    int64_t d = 0;
    DevBuf<int32_t> sv0;
    DevBuf<int64_t> e0;
    DevBuf<uint32_t> map;
    DevBuf<int2> ent;
    DevBuf<double> w, c0;
    DevBuf<float> wf;
};
struct Context;

// Device memory of a kernel-row cache.  The library keeps one block per
// device between trainings and lends it to one cache at a time (grown when
// a cache needs more): freeing and allocating tens of GB per training makes
// a later allocation wait while the driver clears the freed memory.  A
// cache that finds its device's block lent out allocates its own.  The
// block is returned after a device synchronisation, as hipFree would do.
struct CacheRows {
    float* p = nullptr;
    size_t count = 0;
    int device = -1;
    bool lent = false;
    CacheRows() = default;
    CacheRows(const CacheRows&) = delete;
    CacheRows& operator=(const CacheRows&) = delete;
    ~CacheRows() { release(); }
    void alloc(size_t n, int dev);
    void release();
};

// Bytes of the device's kept block while no cache holds it (0 otherwise).
size_t cache_pool_idle_bytes(int device);

// Frees the kept block of a device (every device: device < 0) unless a
// cache holds it; returns the bytes freed.
size_t cache_pool_trim(int device);

// HBM-resident cache of kernel rows K(x_s, .) over all n samples, rows
// padded to ldc floats.  The rows do not depend on the labels, so the
// outputs of a one-vs-rest model share one cache.  Replacement is FIFO and
// decided on the device (slot_of / owner maps, clock).
struct RowCache {
    int64_t slots = 0, ldc = 0;
    CacheRows rows;
    DevBuf<int32_t> slot_of, owner;
    DevBuf<int64_t> clock;
};

// Sizes and clears the cache for n samples.  bytes: 0 = default (the full
// kernel matrix if it fits a quarter of the free device memory, else a
// quarter of it, at most 8 GiB; the device's idle kept block counts as
// free), > 0 = at most that many bytes (clamped likewise), < 0 = no cache.
// Leaves slots = 0 when fewer rows than a working set needs would fit.
void cache_init(RowCache& c, int64_t n, int64_t bytes, Context& cx);

// The device and stream of one call.
struct Context {
    int device = 0;
    hipStream_t stream = nullptr;
    bool own_stream = false;
    Context(int dev, void* stream);
    ~Context();
    void sync();
};

// Dense feature store: X zero-padded to ldp columns, plus squared norms.
// Feature store: dense rows zero-padded to ldp columns, or CSR (int64 row
// pointers, int32 column indices sorted within each row, fp32 values);
// squared norms either way.  ldp is also the width of dense copies of CSR
// rows (the working-set rows, support vectors).
struct Features {
    int64_t n = 0, d = 0, ldp = 0, nnz = 0;
    int64_t maxnz = 0;  // CSR: nonzeros of the longest row
    bool csr = false;
    DevBuf<float> X, sq;
    // dense device input already in the padded layout (ld = ldp = d, 16-byte
    // aligned): used in place for the duration of the call, not copied
    const float* Xb = nullptr;
    const float* x() const { return Xb ? Xb : X.p; }
    DevBuf<int64_t> rp;
    DevBuf<int32_t> ci;
    DevBuf<float> cv;
    // the rows again, sliced by kSellRows for the row kernel (empty when the
    // row lengths are so uneven that the padding would pass 4 x nnz, or when
    // d > 65536)
    DevBuf<int64_t> so;
    DevBuf<uint16_t> sci;  // 16-bit column indices (d <= 65536)
    DevBuf<float> scv;
};

// Uploads X (host or device) into the padded layout and computes norms.
// Throws Error{SVM_E_INVALID} if a value is not finite.
// borrow: dense device input already in the padded layout is used in place
// (the caller's buffer must outlive f; only for calls that return before
// the caller regains it).
void load_features(const svm_matrix* M, Features& f, Context& cx,
                   bool borrow = false);

int64_t padded_ld(int64_t d);

struct SolveOptions {
    int32_t type;
    int32_t kernel, degree;
    double C, eps, gamma, coef0, tol;
    int64_t max_iter;
    int32_t q;
    int32_t check_every;
    double inner_ratio;
    int32_t max_inner;
    int32_t profile;  // 0 none, 1 row launches, 2 also the select launches
    int32_t fused;       // svm_params.fused
    int64_t cache_req;   // svm_params.cache_bytes
};

SolveOptions make_options(const svm_params* p, int64_t n, int64_t d);

// The kernel of the options as the kernels take it.
KernelFn kernel_fn(const SolveOptions& o);

// Whether a solve of these options on these features runs one launch per
// outer iteration (k_iter) instead of a selection launch and a row launch
// (the row cache serves only the latter).
bool one_launch_loop(const SolveOptions& o, const Features& f);

// Result of one binary (or SVR) solve.
struct SolveResult {
    svm_status status = SVM_OK;
    int64_t iters = 0;
    double gap = 0, m = 0, M = 0, b = 0, obj = 0;
    int64_t n_free = 0, n_bounded = 0, n_sv = 0;
    int64_t kernel_rows = 0;
    int64_t cache_served = 0, cache_filled = 0;
    double train_ms = 0;
    // profiled row-kernel launches: computed from X, and served from cache
    double row_ms = 0, cached_ms = 0;
    int64_t row_launches = 0, row_rows = 0, cached_launches = 0;
    double row_bytes = 0, cached_bytes = 0;
    // profiled select/solve launches of the same iterations
    double select_ms = 0;
    int64_t select_launches = 0;
};

class Solver {
public:
    // y: device pointer to n labels (+-1) or targets.  Features are shared.
    // fold (device, n entries) and held: rows with fold[i] == held are held
    // out of the training (cross-validation); fold == nullptr: none.
    Solver(Context& cx, const Features& f, const float* y_dev,
           const SolveOptions& o, RowCache* cache = nullptr,
           const int32_t* fold = nullptr, int32_t held = -1);

    // Full training run: initial keys, iterations, final recompute, bias.
    SolveResult train();

    // Training of several solvers in lockstep (one-vs-rest classes,
    // cross-validation folds, grid points): their outer iterations advance
    // together, one selection launch (a block per solver) and one pass over
    // X per iteration (k_lock).  Each result is the one train() gives
    // without the row cache.  The solvers share the features and the
    // stream, are of one type and kernel kind, have working sets of 16,
    // dense features and no row cache; at most lock_capacity() of them.
    static std::vector<SolveResult> train_lockstep(
        const std::vector<Solver*>& group);
    // Problems one lockstep pass can carry for these features (their
    // working-set rows share the row kernel's LDS): 1 .. kLockMax.
    static int lock_capacity(const Features& f, int32_t type);

    // Expansion coefficients c_i over all n samples, written to
    // c[i * stride + off] (device).
    void coefficients(double* c, int32_t stride, int32_t off);

    // Host copy of alpha (N values).
    void get_alpha(double* out);

    // Start the next train() from alpha (N host values, feasible): the
    // state bytes and F are derived from it.
    void warm_start(const double* alpha_h);

    // After train(): decision values F_i + b of the rows with fold[i] ==
    // held, to out[i * stride + off] (device).
    void cv_decision(double* out, int32_t stride, int32_t off,
                     const int32_t* fold, int32_t held, double b);

    // ---- test hooks ----
    void set_state(const double* alpha_h, const double* F_h);
    void get_state(double* alpha_h, double* F_h);
    void select(int32_t* B, int32_t* nB, double* m, double* M);
    void rows(const int32_t* samples, int32_t k, float* out_h);
    void subproblem(const int32_t* B, int32_t nB, double inner_tol,
                    int32_t max_inner, double* alpha_B, int32_t* steps);
    void apply(const int32_t* B, int32_t nB, const double* alpha_B);
    void iterate(int64_t k, int64_t* iters, double* gap);
    // The end of a training on the current state: F recomputed from alpha,
    // the gap re-tested and the loop re-run at most max_passes times, then
    // bias, objective and counts.
    void finish_state(int max_passes, SolveResult& r);

    int64_t N() const { return N_; }

private:
    hipEvent_t start(bool keys);
    void finish(SolveResult& r, bool conv, hipEvent_t t0,
                int max_passes = 3);
    void launch_keys();
    void launch_hot_rows(hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
    void launch_solve(int32_t mode, hipEvent_t e0 = nullptr,
                      hipEvent_t e1 = nullptr);
    void launch_select_only();
    bool run_loop(SolveResult& r);
    // one launch per outer iteration: initial records, the loop
    void launch_keys_fused();
    bool run_loop_fused(SolveResult& r);
    // the loop of the solver's kind, from the current state
    bool loop(SolveResult& r);
    void recompute_responses();
    void read_ws(WorkingSet& w);
    // CSR: compact working-set columns of a launch with nbc column blocks
    // (-1 for dense features), and the by-column working set in the args
    int csr_cols(int nbc) const;
    void set_csr(RowArgs& a, int nbc) const;
    void set_csr(SelArgs& a, int nbc);

    Context& cx_;
    const Features& f_;
    SolveOptions o_;
    int64_t n_, N_;
    KernelFn kf_;
    int half_, nblk_cols_, tiles_, nb_;
    // one launch per outer iteration: blocks (= candidate records), tiles
    // per row wave, tiles of the record-writing k_rows launch on that grid;
    // the second responses buffer, the double-buffered records, the ticket
    bool fused_ = false;
    int nbi_ = 0, tilesi_ = 0, tilesk_ = 0;
    DevBuf<double> F2_, irk_;
    DevBuf<int32_t> iri_;
    DevBuf<uint32_t> ticket_;
    DevBuf<double> F_, alpha_;
    DevBuf<uint8_t> st_;
    DevBuf<float> y_;
    DevBuf<WorkingSet> ws_;
    DevBuf<float> xS_;
    DevBuf<int32_t> xsc_cols_;  // CSR: the working set by column
    DevBuf<float> xsc_;
    DevBuf<double> ckey_;
    DevBuf<int32_t> cidx_;
    DevBuf<Summary> sum_;
    DevBuf<double> cvec_;
    DevBuf<int32_t> cblk_, sv_idx_;
    DevBuf<double> sv_coef_;
    DevBuf<int64_t> sv_cnt_;
    DevBuf<float> sv_rows_, sv_sq_;
    DevBuf<float> rows_out_;
    // sparse decision path of the recompute: support rows by column
    int ch_cap_ = 0;
    DevBuf<int32_t> ch_ncol_, ch_cols_;
    DevBuf<float> ch_tab_;
    FactSV fc_;
    DevBuf<int32_t> self_sv_;
    RowCache* cache_ = nullptr;
    double row_ms_ = 0, cached_ms_ = 0, row_bytes_ = 0, cached_bytes_ = 0;
    int64_t row_launches_ = 0, row_rows_ = 0, cached_launches_ = 0;
    double select_ms_ = 0;
    int64_t select_launches_ = 0;
};

}  // namespace msvm

// The opaque model of the C ABI.
struct svm_model {
    int32_t type = 0;
    int32_t n_out = 1;
    int64_t n_train = 0, d = 0, ldp = 0;
    // trained on standardised data: the features' means and standard
    // deviations (a constant column has sd 0 and is left as it is), and
    // for eps-SVR the targets' (decision values are mapped back)
    bool scaled = false;
    msvm::DevBuf<double> x_mu, x_sd;
    std::vector<double> x_mu_h, x_sd_h;
    double y_mu = 0.0, y_sd = 1.0;
    double gamma = 0, coef0 = 0;
    msvm::KernelFn kf{};
    int device = 0;
    int64_t n_sv = 0;
    msvm::DevBuf<float> SV, sqsv;
    msvm::DevBuf<double> coef_dev, b_dev;
    // CSR training set with sparse rows: the support rows by column in
    // chunks of 16, for the sparse decision path (ch_cap == 0: none)
    int32_t ch_cap = 0;
    msvm::DevBuf<int32_t> ch_ncol, ch_cols;
    msvm::DevBuf<float> ch_tab;
    // the same rows in chunks by column for the factored path (CSR models
    // whose rows are sparse enough)
    msvm::FactSV fc;
    std::vector<int32_t> sv_idx;             // union, increasing
    std::vector<double> coef;                // n_sv x n_out
    std::vector<double> b;                   // n_out
    std::vector<std::vector<double>> alpha;  // per output, N values
    std::vector<svm_model_info> info;        // per output
};

namespace msvm {

// Dense copies of rows idx[0..k) of f (dense or CSR) and their norms.
void gather_rows(const Features& f, const int32_t* idx, int64_t k, float* out,
                 float* sq_out, hipStream_t s);

// Decision sums of a (support rows, coefficients, outputs set) for every
// row of t: dense rows directly; sparse CSR rows through the sparse path
// when a carries the support rows by column; other CSR rows through dense
// chunks of rows.
void predict_rows(PredictArgs a, const Features& t, hipStream_t s,
                  const FactSV* fc = nullptr);

// Builds fc for support rows idx[0..nsv) of the CSR features f, with
// coefficients coef (device, nsv x n_out), and writes their norms to sqsv
// (device, nsv).  Leaves fc.ok false where the factored path does not apply:
// dense features, more than 4 outputs, support rows holding on average more
// than a tenth of the columns, a row longer than a chunk, a map over
// fc_map_bytes_limit(), or SVM_SPARSE_PATH=table in the environment.
// With query rows given, it is built only if the rule below takes it for
// them.  predict_rows takes the factored path for query rows t when a
// query row and a support row share fewer than kFcMatchMax columns on
// average (nnz(t)/n(t) * fc.sv_nnz / d), else the table path (the
// factored path pays per shared column about what the table path pays per
// pair); SVM_SPARSE_PATH=factor takes it whenever it is built (a developer
// switch for comparing the two paths).
void build_fact(FactSV& fc, const Features& f, const int32_t* idx,
                int64_t nsv, const double* coef, int32_t n_out,
                const KernelFn& kf, Context& cx, float* sqsv,
                const Features* query = nullptr);

// Capacity (columns per chunk of 16 rows) of the by-column support rows of
// the sparse decision path for a CSR training set, or 0 when its rows are
// not sparse enough (more than 32 nonzeros a row on average) or a chunk's
// table would not fit the kernel's LDS.
int sparse_chunk_cap(const Features& f);

// Builds the by-column support rows: support row j is row idx[j] of f, and
// its norm goes to sq_out[j] (when given).  Sizes the buffers.
void build_sv_chunks(const Features& f, const int32_t* idx, int64_t nsv,
                     int cap, DevBuf<int32_t>& ncol, DevBuf<int32_t>& cols,
                     DevBuf<float>& tab, float* sq_out, hipStream_t s);

// Builds the model arrays from the n x n_out coefficient matrix (device).
void build_model(svm_model& m, Context& cx, const Features& f,
                 const double* coef_dev, int32_t n_out);

// Decision values for X (m x n_out) into `out` (device); t is scaled with
// the model's statistics first when the model was trained on scaled data.
void predict_device(const svm_model& mdl, Context& cx, Features& t,
                    double* out);

// Allocation-free decision values (noalloc.hip): the m dense rows of X
// (device, leading dimension ld) staged in a static per-device array of
// noalloc_scratch_bytes(), chunk by chunk, decision values to out
// (device, m x n_out), all on stream s with no allocation and no host
// synchronisation.
void predict_noalloc(const svm_model& mdl, const float* X, int64_t m,
                     int64_t ld, double* out, hipStream_t s);
// whether the rows are copied (padded, scaled) into the array, and how many
// rows one chunk takes (< 1: a row does not fit)
bool noalloc_needs_copy(const svm_model& mdl, const float* X, int64_t ld);
int64_t noalloc_rows_per_chunk(const svm_model& mdl, const float* X,
                               int64_t ld);
size_t noalloc_scratch_bytes();

// Standardisation (dense features only): per-feature mean and sample
// standard deviation of f (device, d values each), and their application
// to a feature store (its norms recomputed).  Targets: the same for the n
// values of y (mean and sd returned on the host).
void scale_fit(const Features& f, Context& cx, DevBuf<double>& mu,
               DevBuf<double>& sd);
void scale_apply(Features& f, Context& cx, const double* mu,
                 const double* sd);
void scale_targets(float* y_dev, int64_t n, Context& cx, double* mu,
                   double* sd);

}  // namespace msvm
