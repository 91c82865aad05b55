// Internal declarations of the MI355X kernel-SVM library (not installed).
//
// Data layout in HBM (one device):
//   X    n x ldp fp32, row-major, ldp = d rounded up to a multiple of 4 and
//        zero-padded, so that every lane can load aligned float4 pieces.
//   sq   n fp32 squared norms |x_i|^2 (summed in fp64, rounded once).
//   F    n fp64 responses F_i = sum_t y_t a_t K(x_i, x_smp(t)).
//   a    N fp64 dual variables; st N bytes of state (label sign, I_up, I_low).
//   z    n fp32 targets (eps-SVR only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/mi355svm.h"

namespace msvm {

constexpr int kMaxQ = 64;          // largest working set
constexpr int kMaxHalf = kMaxQ / 2;
constexpr int kRowThreads = 256;   // row/update kernel: 4 waves
constexpr int kSellRows = 16;      // rows per slice of the sliced CSR copy
constexpr int kSelThreads = 1024;  // select/solve kernel: one block
constexpr int kBlockTop = 2;       // candidates per side kept per row group
constexpr int kSelRecords = 2;     // row-group records held per thread
constexpr int kSelPerThread = kSelRecords * kBlockTop;  // per side
constexpr double kTau = 1e-12;     // curvature floor of a degenerate pair

// how the row kernel of an iteration gets K(x_i, x_s) (set by the selection)
enum : int32_t {
    PATH_STREAM = 0,  // computed from X
    PATH_INSERT = 1,  // computed from X; rows of missing samples go to the cache
    PATH_CACHED = 2   // every sample of the working set is cached: rows read
};
constexpr int kPathLog = 256;  // iterations of path history kept (profiling)

// state byte of a dual variable
constexpr uint8_t ST_YPOS = 1;  // y_t = +1
constexpr uint8_t ST_UP = 2;    // t in I_up
constexpr uint8_t ST_LOW = 4;   // t in I_low

// Device-resident description of the current working set.  Written by the
// select/solve kernel, read by the row/update kernel of the same iteration.
struct WorkingSet {
    int32_t done;      // 0 running, 1 converged (gap <= tol), 2 iteration cap
    int32_t nB;        // variables in B
    int32_t nS;        // distinct samples of B (slots)
    int32_t pad0;
    int64_t iter;      // outer iterations performed
    int64_t rows;      // kernel rows evaluated (sum of nS)
    double gap, m, M;
    int32_t B[kMaxQ];
    int32_t S[kMaxQ];     // sample of each slot
    int32_t slotB[kMaxQ]; // slot of each variable of B
    float sS[kMaxQ];      // squared norm of each slot's sample
    double coef[kMaxQ];   // change of the expansion coefficient per slot
    double alphaB[kMaxQ]; // new alpha_B (written by the solve)
    int32_t steps;        // inner steps of the last subproblem
    int32_t pad1;
    int64_t inner_total;  // inner steps summed over iterations
    int64_t rescans;      // iterations that rescanned exhausted blocks
    int64_t slow_selects; // iterations that fell back to a full scan
    int64_t prof[12];     // select/solve phase times (wall-clock ticks)
    // kernel-row cache
    int32_t path;             // PATH_* of the current iteration
    int32_t pad2;
    int32_t cslot[kMaxQ];     // cache slot of each working-set slot (cached:
                              // source; insert: destination or -1)
    int64_t cache_served;     // kernel rows read from the cache
    int64_t cache_filled;     // kernel rows written to the cache
    uint8_t path_log[kPathLog];  // path of iteration t at [t % kPathLog]
    uint8_t fill_log[kPathLog];  // rows written to the cache by iteration t
    uint8_t ns_log[kPathLog];    // distinct samples of iteration t
};

// Final reductions of a state (bias and objective).
struct Summary {
    double sum_free_v;  // sum of v_t over free variables
    double obj2;        // sum_t a_t y_t (r_t + v_t); f = -obj2 / 2
    int64_t n_free;
    int64_t n_bounded;
};

// row/update kernel modes
enum : int32_t {
    RU_UPDATE = 1,      // F += sum_s coef_s K(x_i, x_s)
    RU_ROWS = 2,        // write K(x_s, x_i) to rows_out (tests)
    RU_CAND = 4,        // keys and per-block candidates
    RU_CHECK_DONE = 8   // return at once if the solve has finished
};

// select/solve kernel modes
enum : int32_t {
    SS_SOLVE = 1,       // build B, solve, write the new working set
    SS_CHECK_DONE = 2,
    SS_GIVEN_B = 4,     // B is taken from ws->B (tests)
    SS_NO_WRITE = 8,    // leave alpha/state untouched (tests)
    SS_SET_ALPHA = 16   // alpha_B taken from ws->alphaB instead of solved
};

// The kernel function (Section 3's list, e1071 parameterisation):
// kind = svm_kernel; RBF exp(-gamma |u - v|^2) = 2^(-gexp |u - v|^2) with
// gexp = gamma log2(e); linear u.v; polynomial (gamma u.v + coef0)^degree;
// sigmoid tanh(gamma u.v + coef0).
struct KernelFn {
    int32_t kind;
    int32_t degree;
    float gexp;
    float gamma;
    float coef0;
};

struct RowArgs {
    const float* X;       // dense rows, or nullptr for CSR
    const int64_t* rp;    // CSR rows (rp == nullptr: dense)
    const int32_t* ci;
    const float* cv;
    // CSR rows sliced by kSellRows (so == nullptr: walk rp/ci/cv instead):
    // nonzero k of row i at so[i / kSellRows] + kSellRows * k + i % kSellRows
    const int64_t* so;
    const uint16_t* sci;  // column indices (below 65536) of the sliced copy
    const float* scv;
    const float* sq;
    double* F;
    const uint8_t* st;
    const float* z;
    const WorkingSet* ws;
    const float* xS;      // kMaxQ x ldp rows of the working-set samples
    // CSR: the working set by column (written by the selection): the column
    // of each of csr_cols compact rows (-1: unused), and the rows
    // (csr_cols + 1 of 16 * nblk_cols floats; unused rows and the last are 0)
    const int32_t* xsc_cols;
    const float* xsc;
    int32_t csr_cols;
    double* cand_key;     // [blocks][2][kBlockTop]: up scores v, low -v
    int32_t* cand_idx;
    float* rows_out;      // nS x n (tests)
    float* cache;         // kernel-row cache rows (stride ldc), or nullptr
    int64_t ldc;
    int64_t n, ldp;
    double eps;
    KernelFn kf;
    int32_t half;
    int32_t tiles;        // 16-row tiles per wave
    int32_t mode;
    int32_t nS_override;  // >= 0: use this many slots (tests), else ws->nS
};

struct SelArgs {
    const double* cand_key;
    const int32_t* cand_idx;
    int32_t nb, half;     // nb: candidate records (one per k_rows block)
    WorkingSet* ws;
    double* alpha;
    uint8_t* st;
    const double* F;
    const float* z;
    const float* X;       // dense rows, or nullptr for CSR
    const int64_t* rp;    // CSR rows (rp == nullptr: dense)
    const int32_t* ci;
    const float* cv;
    const float* sq;
    float* xS;
    int32_t* xsc_cols;    // CSR: the working set by column (see RowArgs)
    float* xsc;
    int32_t csr_cols;
    int64_t n, ldp;
    double C, eps, tol;
    KernelFn kf;
    double inner_ratio;
    double inner_tol_override;  // >= 0: fixed inner tolerance (tests)
    int32_t max_inner;
    int64_t max_iter;
    int32_t mode;
    int32_t group_rows;   // rows behind one candidate record (a k_rows block)
    int32_t slice;        // features per LDS slice of the working-set rows
    // kernel-row cache (cache_slots == 0: none)
    const float* cache;   // cache_slots rows of ldc floats
    int64_t ldc, cache_slots;
    int32_t* slot_of;     // n: cache slot of each sample, or -1
    int32_t* owner;       // cache_slots: sample held by each slot, or -1
    int64_t* clock;       // next replacement candidate (FIFO)
};

struct PredictArgs {
    const float* Xt;      // m x ldp test rows
    const float* sqt;
    int64_t m, ldp;
    const float* SV;      // nsv x ldp support rows
    const float* sqsv;
    int64_t nsv;
    const double* coef;   // nsv x n_out
    const double* b;      // n_out or nullptr
    int32_t n_out;
    const int32_t* sv_train_idx;  // with self_match: K(x_i, x_i) = 1 exactly
    int32_t self_match;
    int64_t row_base;     // training-set index of query row 0 (self_match)
    const int32_t* self_sv;  // factored sparse path: training row -> its
                             // support row or -1 (nullptr: no self pairs)
    // dense paths: the support rows are split into nrange ranges of whole
    // 64-row tiles (predict_ranges(nsv), so a row's value does not depend
    // on the batch it comes in); with nrange > 1 each range's sums go to
    // part (nrange x m x n_out) and a second kernel adds them in range
    // order, with b
    int32_t nrange;
    double* part;
    double* out;          // m x n_out
    KernelFn kf;
    // sparse path: CSR query rows, and the support rows by column in
    // chunks of 16 (chunk k: support rows 16k .. 16k + 15)
    const int64_t* rpt;
    const int32_t* cit;
    const float* cvt;
    const int32_t* ch_ncol;  // columns some row of the chunk holds
    const int32_t* ch_cols;  // nchunk x ch_cap: those columns, increasing
    const float* ch_tab;     // nchunk x ch_cap x 16: their values (0: none)
    int32_t ch_cap;
};

// One outer iteration per launch (k_iter, dense features, q <= 16): every
// block merges the previous launch's candidate records, solves the
// subproblem and updates its rows; F and the records are double-buffered by
// launch parity; the last block (ticket) writes alpha_B, the state bytes of
// B and the working-set record.
constexpr int kIterMaxRecords = 1024;  // blocks (candidate records) at most
struct IterArgs {
    const float* X;       // dense rows
    const float* sq;
    const float* z;       // labels (C-SVC) or targets (eps-SVR)
    const double* F_in;   // responses after the previous launch
    double* F_out;        // responses after this one
    double* alpha;
    uint8_t* st;
    const double* rk_in;  // candidate records of the previous launch
    const int32_t* ri_in;
    double* rk_out;       // this launch's (one per block)
    int32_t* ri_out;
    WorkingSet* ws;
    uint32_t* ticket;     // 0 between launches
    int64_t n, ldp;
    int32_t nb;           // blocks = candidate records
    int32_t half;
    int32_t tiles;        // 16-row tiles per row wave
    int32_t group_rows;   // most rows of a block
    double C, eps, tol;
    KernelFn kf;
    double inner_ratio;
    int32_t max_inner;
    int64_t max_iter;
};

// Several problems over one stream of X (k_lock): problem p's working set
// is staged at rows 16p .. 16p + 15 of xS; the rest is per problem.  Every
// problem has the same n, features and kernel kind.
constexpr int kLockMax = 4;
struct LockArgs {
    const float* X;       // dense rows
    const float* sq;
    const float* xS;      // P x 16 rows of ldp floats
    int64_t n, ldp;
    int32_t tiles;        // 16-row tiles per wave
    double* F[kLockMax];
    const uint8_t* st[kLockMax];
    const float* z[kLockMax];
    const WorkingSet* ws[kLockMax];
    double* cand_key[kLockMax];  // as RowArgs, one table per problem
    int32_t* cand_idx[kLockMax];
    KernelFn kf[kLockMax];
    double eps[kLockMax];
};

// Building the support rows by column (see PredictArgs), from CSR rows:
// support row j is CSR row idx[j] (idx == nullptr: row j).  cap bounds the
// columns of a chunk (16 times the longest row, at most ldp).
struct ChunkArgs {
    const int64_t* rp;
    const int32_t* ci;
    const float* cv;
    const float* sq;       // norms of the CSR rows
    const int32_t* idx;
    int64_t nsv, ldp;
    int32_t cap;
    int32_t* ncol;         // ceil(nsv / 16)
    int32_t* cols;         // ceil(nsv / 16) x cap
    float* tab;            // ceil(nsv / 16) x cap x 16
    float* sq_out;         // nsv: norms of the support rows (or nullptr)
};

// The sparse decision path by column (factor.hip).  With s_x = |x|^2, the
// RBF value of a pair factors as K(x, v) = e^(-g s_x) e^(-g s_v) e^(2g x.v),
// and x.v = 0 for every pair of rows with no column in common, so
//   D(x) = e^(-g s_x) C0 + sum over the support rows v sharing a column
//          with x of (c_v K(x, v) - e^(-g s_x) w_v),
// with w_v = c_v e^(-g s_v) and C0 = sum_v w_v (the other kernels:
// e^(-g s) -> 1 and w_v = c_v K of a zero dot product).  The support rows
// are split into chunks of consecutive rows (at most kFcSvMax); a chunk holds
// its nonzeros by column (CSC: for every column the chunk's rows that hold
// it, in increasing order, as (local row, value)), and a dense map from
// column to (first entry << kFcLenBits | count).  A wave takes query rows
// one at a time: it adds each product x_c v_c into an LDS accumulator of the
// chunk's rows (walk 1), then reads back and clears the accumulator at every
// row it touched (walk 2), which visits each overlapping pair once.
constexpr int kFcSvMax = 2048;     // support rows of a chunk
constexpr int kFcLenBits = 12;     // bits of the count in a map entry
constexpr int64_t kFcEntMax = (int64_t)1 << 20;  // entries of a chunk
// bound on gexp |x|^2 of the factored RBF form (rows above it, or a model
// with a support row above it, take the direct formula)
constexpr float kFcSafe = 63.0f;
// the factored path serves query rows that share fewer columns than this
// with a support row on average (measured on the C5 shape, 20 of 1000
// columns per row: 0.4 shared columns a pair, both paths 103 ms for 1M
// rows against 44k support rows)
constexpr double kFcMatchMax = 0.3;
struct FactArgs {
    const int64_t* rpt;   // m query rows (CSR)
    const int32_t* cit;
    const float* cvt;
    const float* sqt;
    int64_t m;
    int64_t row_base;     // index of query row 0 in self_sv
    const int32_t* self_sv;  // query row -> its own support row, or -1
                             // (recompute of F: K(x_i, x_i) = 1), or nullptr
    int32_t nch;          // chunks
    int32_t ldpm;         // columns of a map row
    const int32_t* ch_sv0;   // nch + 1: first support row of each chunk
    const int64_t* ch_e0;    // nch + 1: first entry of each chunk
    const uint32_t* map;     // nch x ldpm
    const int2* ent;         // (local support row, value bits)
    const float* sqsv;       // nsv norms
    const double* coef;      // nsv x n_out
    const double* w;         // nsv x n_out (see above)
    const float* wf;         // nsv: w of output 0 in fp32
    const double* c0;        // n_out
    const double* b;         // n_out or nullptr
    int32_t n_out;
    int32_t fast;         // 1: e^(-g s) of every support row is in range
    double* out;          // m x n_out
    KernelFn kf;
};
// Building the chunks: support row j is CSR row idx[j] of (rp, ci, cv).
struct FactBuildArgs {
    const int64_t* rp;
    const int32_t* ci;
    const float* cv;
    const int32_t* idx;
    int32_t nch, ldpm;
    const int32_t* ch_sv0;
    const int64_t* ch_e0;
    uint32_t* map;
    int2* ent;
};

// ---- launch wrappers (kernels.hip / predict.hip) ----
void launch_pad_copy(const float* src, int64_t ld, int64_t n, int64_t d,
                     float* dst, int64_t ldp, hipStream_t s);
void launch_norms(const float* X, int64_t n, int64_t ldp, float* sq,
                  int32_t* bad_flag, hipStream_t s);
// fold == nullptr: every row trains; else rows with fold[i] == held are
// held out (alpha = 0, outside I_up and I_low)
void launch_init_state(int32_t type, const float* y, int64_t n,
                       const int32_t* fold, int32_t held, uint8_t* st,
                       int32_t* bad_flag, hipStream_t s);
void launch_cv_decision(const double* F, int64_t n, double b,
                        const int32_t* fold, int32_t held, double* out,
                        int32_t stride, int32_t off, hipStream_t s);
// per-column mean and sample standard deviation (n - 1) of n x d (leading
// dimension ld) in fp64; part holds col_stats_partials(n, d) doubles
void launch_col_stats(const float* X, int64_t n, int64_t ld, int64_t d,
                      double* part, double* mu, double* sd, hipStream_t s);
int64_t col_stats_partials(int64_t n, int64_t d);
void launch_scale_apply(float* X, int64_t n, int64_t ld, int64_t d,
                        const double* mu, const double* sd, hipStream_t s);
void launch_affine(double* D, int64_t m, double a, double b, hipStream_t s);
void launch_metrics(int32_t type, int32_t n_out, const double* D,
                    const float* y, const int32_t* labels, int64_t n,
                    double* out, hipStream_t s);
void launch_ovr_labels(const int32_t* labels, int64_t n, int32_t cls,
                       float* y, hipStream_t s);
void launch_check_labels(const int32_t* labels, int64_t n, int32_t ncls,
                         int32_t* bad_flag, hipStream_t s);
void launch_check_finite(const float* v, int64_t n, int32_t* bad_flag,
                         hipStream_t s);
void launch_rows(const RowArgs& a, int nblocks, int nblk_cols, bool svr,
                 hipStream_t s, hipEvent_t e0 = nullptr,
                 hipEvent_t e1 = nullptr);
// csr_cols < 0: dense features; else the compact working-set columns (CSR)
size_t rows_lds_bytes(int nblk_cols, int64_t ldp, int tiles, bool svr,
                      int csr_cols);
int rows_blocks_per_cu(int nblk_cols, bool svr, size_t lds, bool csr);
// Resident blocks per compute unit of (kernel, block size, dynamic LDS)
// from the runtime, at least 1; asked once per process and kept (the
// library builds for one architecture).
int occupancy_memo(const void* kernel, int threads, size_t lds);
// Raises a kernel's dynamic LDS limit to at least lds bytes (never lowers
// it; thread-safe); false when the device refuses.
bool raise_dynamic_lds(const void* kernel, size_t lds);
void launch_select(const SelArgs& a, int nblk_cols, bool svr, hipStream_t s,
                   hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// one block per problem (P <= kLockMax entries, each with working sets of
// 16), the arguments passed by value in the launch
void launch_select_group(const SelArgs* args, int P, bool svr, hipStream_t s);
// lockstep row/update kernel of P problems (dense features, q = 16 each)
void launch_lock(const LockArgs& a, int P, int nblocks, bool svr,
                 hipStream_t s, hipEvent_t e0 = nullptr,
                 hipEvent_t e1 = nullptr);
size_t lock_lds_bytes(int P, int64_t ldp, int tiles, bool svr);
int lock_blocks_per_cu(int P, bool svr, size_t lds);
// one outer iteration (k_iter): nblocks = a.nb blocks
void launch_iter(const IterArgs& a, int nblocks, bool svr, hipStream_t s,
                 hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
size_t iter_lds_bytes(int64_t ldp, int tiles, bool svr);
int iter_blocks_per_cu(bool svr, size_t lds);
void launch_state_from_alpha(int32_t type, const float* y, const double* a,
                             int64_t n, double C, uint8_t* st, hipStream_t s);
void launch_coef(int32_t type, const double* a, const uint8_t* st, int64_t n,
                 double* c, hipStream_t s);
void launch_coef_strided(int32_t type, const double* a, const uint8_t* st,
                         int64_t n, double* c, int32_t stride, int32_t off,
                         hipStream_t s);
// out: 1 + kSummaryBlocks entries (the result at out[0], partial sums
// after it)
constexpr int kSummaryBlocks = 256;
void launch_summary(int32_t type, const double* a, const uint8_t* st,
                    const double* F, const float* z, int64_t n, double C,
                    double eps, Summary* out, hipStream_t s);
// compaction of rows with any non-zero coefficient over n_out columns
void launch_compact(const double* coef, int64_t n, int32_t n_out,
                    int32_t* blk_cnt, int32_t* idx_out, double* coef_out,
                    int64_t* count_out, hipStream_t s);
void launch_gather_rows(const float* X, const float* sq, int64_t ldp,
                        const int32_t* idx, int64_t k, float* out,
                        float* sq_out, hipStream_t s);
void launch_predict(const PredictArgs& a, hipStream_t s);
// ranges of support rows of the dense decision kernels (1 to 8, set by the
// number of support rows only), and the doubles of part they need for m rows
int32_t predict_ranges(int64_t nsv);
int64_t predict_part_doubles(int64_t nsv, int64_t m, int32_t n_out);
void launch_sv_chunks(const ChunkArgs& a, hipStream_t s);
void launch_predict_sparse(const PredictArgs& a, hipStream_t s);
// LDS of the sparse decision kernel, and whether it fits
size_t predict_sparse_lds_bytes(int64_t ldp, int cap);
bool predict_sparse_fits(int64_t ldp, int cap);
// sparse decision path by column (factor.hip)
// nonzeros of each support row, and its norm (sq_out[j] = sq[idx[j]])
void launch_fc_nnz(const int64_t* rp, const float* sq, const int32_t* idx,
                   int64_t nsv, int32_t* nz, float* sq_out, hipStream_t s);
void launch_fc_build(const FactBuildArgs& a, hipStream_t s);
// w = coef x (RBF: 2^(-gexp s_v); else K of a zero dot), wf = its first
// column in fp32, c0 = column sums
// of w (fixed order), and the largest gexp s_v into *gs_max (float bits)
void launch_fc_weights(const double* coef, const float* sqsv, int64_t nsv,
                       int32_t n_out, const KernelFn& kf, double* w,
                       float* wf, double* c0, uint32_t* gs_max, hipStream_t s);
void launch_fc_self(const int32_t* sv_idx, int64_t nsv, int64_t n,
                    int32_t* self_sv, hipStream_t s);
void launch_predict_fact(const FactArgs& a, hipStream_t s);
size_t fc_map_bytes_limit();
void launch_csr_compact(const float* xS, int32_t nS, int64_t ldp,
                        int32_t qs, int32_t csr_cols, int32_t* xsc_cols,
                        float* xsc, hipStream_t s);
void launch_csr_check_norms(const int64_t* rp, const int32_t* ci,
                            const float* cv, int64_t n, int64_t d,
                            int64_t nnz, float* sq, int32_t* bad,
                            hipStream_t s);
// sliced copy of CSR rows (kSellRows rows per slice): so[0 .. ns] (the
// offsets, ns = ceil(n / kSellRows)), then the entries
void launch_sell_offsets(const int64_t* rp, int64_t n, int64_t* so,
                         hipStream_t s);
void launch_sell_fill(const int64_t* rp, const int32_t* ci, const float* cv,
                      int64_t n, const int64_t* so, uint16_t* sci, float* scv,
                      hipStream_t s);
// dense copies of CSR rows (idx == nullptr: rows r0 .. r0 + k - 1)
void launch_gather_rows_csr(const int64_t* rp, const int32_t* ci,
                            const float* cv, const float* sq, int64_t ldp,
                            const int32_t* idx, int64_t r0, int64_t k,
                            float* out, float* sq_out, hipStream_t s);
void launch_argmax_labels(const double* D, int64_t m, int32_t n_out,
                          int32_t type, int32_t* labels, hipStream_t s);
void launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s);

int64_t compact_blocks(int64_t n);

// ---- errors ----
struct Error {
    svm_status status;
    std::string msg;
};

void set_error(svm_status st, const std::string& msg);

#define HIP_TRY(expr)                                                     \
    do {                                                                  \
        hipError_t e_ = (expr);                                           \
        if (e_ != hipSuccess) {                                           \
            throw ::msvm::Error{e_ == hipErrorOutOfMemory ? SVM_E_NOMEM   \
                                                          : SVM_E_DEVICE, \
                                std::string(#expr) + ": " +               \
                                    hipGetErrorString(e_)};               \
        }                                                                 \
    } while (0)

}  // namespace msvm
