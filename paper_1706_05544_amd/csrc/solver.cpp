// Host side of the working-set dual solve: buffers, the iteration loop,
// the final recompute of the responses, bias, objective and the model.
#include "solver.hpp"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>

namespace msvm {

// ---------------------------------------------------------------------------
// context and features
// ---------------------------------------------------------------------------

Context::Context(int dev, void* s) : device(dev)
{
    HIP_TRY(hipSetDevice(dev));
    stream = (hipStream_t)s;  // NULL: the device's default stream
}

Context::~Context()
{
    if (own_stream && stream) {
        (void)hipStreamSynchronize(stream);
        (void)hipStreamDestroy(stream);
    }
}

void Context::sync() { HIP_TRY(hipStreamSynchronize(stream)); }

int64_t padded_ld(int64_t d) { return (d + 3) / 4 * 4; }

static void load_csr(const svm_matrix* M, Features& f, Context& cx)
{
    f.csr = true;
    f.nnz = M->nnz;
    f.rp.alloc((size_t)(f.n + 1));
    f.ci.alloc((size_t)f.nnz);
    f.cv.alloc((size_t)f.nnz);
    f.sq.alloc((size_t)f.n);
    const hipMemcpyKind kind =
        M->on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    HIP_TRY(hipMemcpyAsync(f.rp.p, M->row_ptr,
                           (size_t)(f.n + 1) * sizeof(int64_t), kind,
                           cx.stream));
    if (f.nnz > 0) {
        HIP_TRY(hipMemcpyAsync(f.ci.p, M->col_idx,
                               (size_t)f.nnz * sizeof(int32_t), kind,
                               cx.stream));
        HIP_TRY(hipMemcpyAsync(f.cv.p, M->values, (size_t)f.nnz * sizeof(float),
                               kind, cx.stream));
    }
    DevBuf<int32_t> bad(2);
    HIP_TRY(hipMemsetAsync(bad.p, 0, 2 * sizeof(int32_t), cx.stream));
    launch_csr_check_norms(f.rp.p, f.ci.p, f.cv.p, f.n, f.d, f.nnz, f.sq.p,
                           bad.p, cx.stream);
    // slice offsets from the row pointers (used only once these are valid)
    const int64_t ns = (f.n + kSellRows - 1) / kSellRows;
    f.so.alloc((size_t)(ns + 1));
    launch_sell_offsets(f.rp.p, f.n, f.so.p, cx.stream);
    int32_t hbv[2] = {0, 0};
    int64_t sell_total = 0;
    HIP_TRY(hipMemcpyAsync(hbv, bad.p, 2 * sizeof(int32_t),
                           hipMemcpyDeviceToHost, cx.stream));
    HIP_TRY(hipMemcpyAsync(&sell_total, f.so.p + ns, sizeof(int64_t),
                           hipMemcpyDeviceToHost, cx.stream));
    cx.sync();
    const int32_t hb = hbv[0];
    f.maxnz = hbv[1];
    if (hb & 2)
        throw Error{SVM_E_INVALID,
                    "CSR row pointers must start at 0, not decrease and end at "
                    "nnz"};
    if (hb & 4)
        throw Error{SVM_E_INVALID,
                    "CSR column indices must be in [0, d), sorted and unique "
                    "within each row"};
    if (hb & 1)
        throw Error{SVM_E_INVALID,
                    "X holds a value that is not finite (or whose square "
                    "overflows fp32)"};
    if (sell_total > 0 && sell_total <= 4 * f.nnz + 64 * kSellRows &&
        f.d <= 65536) {
        f.sci.alloc((size_t)sell_total);
        f.scv.alloc((size_t)sell_total);
        launch_sell_fill(f.rp.p, f.ci.p, f.cv.p, f.n, f.so.p, f.sci.p,
                         f.scv.p, cx.stream);
    } else {
        f.so.release();
    }
}

void load_features(const svm_matrix* M, Features& f, Context& cx, bool borrow)
{
    Range rg("svm features (copy, norms, checks)");
    f.n = M->n;
    f.d = M->d;
    f.ldp = padded_ld(M->d);
    if (M->layout == SVM_CSR) {
        load_csr(M, f, cx);
        return;
    }
    f.sq.alloc((size_t)f.n);
    const hipMemcpyKind kind =
        M->on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    f.Xb = nullptr;
    if (borrow && M->on_device && f.n > 0 && f.ldp == f.d && M->ld == f.d &&
        ((uintptr_t)M->values & 15) == 0) {
        f.Xb = static_cast<const float*>(M->values);
        f.X.release();
    } else {
        f.X.alloc((size_t)(f.n * f.ldp));
    }
    if (f.n > 0 && !f.Xb) {
        if (f.ldp == f.d && M->ld == f.d) {
            HIP_TRY(hipMemcpyAsync(f.X.p, M->values,
                                   (size_t)(f.n * f.d) * sizeof(float), kind,
                                   cx.stream));
        } else if (M->on_device) {
            launch_pad_copy(M->values, M->ld, f.n, f.d, f.X.p, f.ldp,
                            cx.stream);
        } else {
            HIP_TRY(hipMemsetAsync(f.X.p, 0, f.X.bytes(), cx.stream));
            HIP_TRY(hipMemcpy2DAsync(f.X.p, (size_t)f.ldp * sizeof(float),
                                     M->values, (size_t)M->ld * sizeof(float),
                                     (size_t)f.d * sizeof(float),
                                     (size_t)f.n, kind, cx.stream));
        }
    }
    DevBuf<int32_t> bad(1);
    HIP_TRY(hipMemsetAsync(bad.p, 0, sizeof(int32_t), cx.stream));
    launch_norms(f.x(), f.n, f.ldp, f.sq.p, bad.p, cx.stream);
    int32_t hb = 0;
    HIP_TRY(hipMemcpyAsync(&hb, bad.p, sizeof(int32_t),
                           hipMemcpyDeviceToHost, cx.stream));
    cx.sync();
    if (hb)
        throw Error{SVM_E_INVALID,
                    "X holds a value that is not finite (or whose square "
                    "overflows fp32)"};
}

SolveOptions make_options(const svm_params* p, int64_t n, int64_t d)
{
    SolveOptions o{};
    o.type = p->type;
    o.C = p->C;
    o.eps = p->type == SVM_EPS_SVR ? p->epsilon : 0.0;
    o.kernel = p->kernel;
    o.degree = p->kernel == SVM_KERNEL_POLY ? p->degree : 1;
    o.coef0 = p->coef0;
    o.gamma = p->gamma > 0 ? p->gamma : 1.0 / (double)d;
    o.tol = p->tol;
    const int64_t N = p->type == SVM_EPS_SVR ? 2 * n : n;
    o.max_iter = p->max_iter > 0 ? p->max_iter
                                 : std::max<int64_t>(10000000, 100 * N);
    o.q = p->working_set;
    // (the per-iteration path history covers kPathLog iterations)
    o.check_every = p->check_every > 0 ? std::min(p->check_every, kPathLog)
                                       : 64;
    o.inner_ratio = p->inner_ratio > 0 ? p->inner_ratio : 0.3;
    o.max_inner = p->max_inner > 0 ? p->max_inner : 8 * p->working_set;
    o.profile = p->profile < 0 ? 0 : (p->profile > 2 ? 2 : p->profile);
    o.fused = p->fused;
    o.cache_req = p->cache_bytes;
    return o;
}

bool one_launch_loop(const SolveOptions& o, const Features& f)
{
    // (asked for only: on the shapes measured so far it is slower, the
    // selection chain of a block under 512 concurrent ones taking longer
    // than the stream it hides)
    return o.fused > 0 && !f.csr && o.q <= 16;
}

KernelFn kernel_fn(const SolveOptions& o)
{
    KernelFn k{};
    k.kind = o.kernel;
    k.degree = o.degree;
    k.gexp = (float)(o.gamma * 1.4426950408889634);  // gamma log2(e)
    k.gamma = (float)o.gamma;
    k.coef0 = (float)o.coef0;
    return k;
}

// ---------------------------------------------------------------------------
// solver
// ---------------------------------------------------------------------------

namespace {

struct CachePool {
    std::mutex mu;
    float* p = nullptr;
    size_t bytes = 0;
    bool lent = false;
};

constexpr int kPoolDevices = 64;

CachePool& pool_of(int dev)
{
    static CachePool pools[kPoolDevices];
    if (dev < 0 || dev >= kPoolDevices)
        throw Error{SVM_E_INVALID, "device ordinal out of range"};
    return pools[dev];
}

// wait for the device's work (on its own current-device setting)
void sync_device(int dev)
{
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) cur = -1;
    if (cur != dev) (void)hipSetDevice(dev);
    (void)hipDeviceSynchronize();
    if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
}

}  // namespace

void CacheRows::alloc(size_t n, int dev)
{
    release();
    if (n == 0) n = 1;
    const size_t b = n * sizeof(float);
    CachePool& pl = pool_of(dev);
    std::lock_guard<std::mutex> g(pl.mu);
    if (!pl.lent) {
        if (pl.bytes < b) {
            if (pl.p) (void)hipFree(pl.p);
            pl.p = nullptr;
            pl.bytes = 0;
            HIP_TRY(hipMalloc((void**)&pl.p, b));
            pl.bytes = b;
        }
        pl.lent = true;
        p = pl.p;
        lent = true;
    } else {
        HIP_TRY(hipMalloc((void**)&p, b));
    }
    count = n;
    device = dev;
}

void CacheRows::release()
{
    if (!p) return;
    if (lent) {
        // no kernel of this cache may still read the block when the next
        // cache gets it
        sync_device(device);
        CachePool& pl = pool_of(device);
        std::lock_guard<std::mutex> g(pl.mu);
        pl.lent = false;
    } else {
        (void)hipFree(p);
    }
    p = nullptr;
    count = 0;
    lent = false;
}

size_t cache_pool_idle_bytes(int device)
{
    CachePool& pl = pool_of(device);
    std::lock_guard<std::mutex> g(pl.mu);
    return pl.lent ? 0 : pl.bytes;
}

size_t cache_pool_trim(int device)
{
    size_t freed = 0;
    for (int d = device < 0 ? 0 : device;
         d < (device < 0 ? kPoolDevices : device + 1); ++d) {
        CachePool& pl = pool_of(d);
        std::lock_guard<std::mutex> g(pl.mu);
        if (pl.lent || !pl.p) continue;
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) cur = -1;
        if (cur != d) (void)hipSetDevice(d);
        (void)hipFree(pl.p);
        if (cur >= 0 && cur != d) (void)hipSetDevice(cur);
        freed += pl.bytes;
        pl.p = nullptr;
        pl.bytes = 0;
    }
    return freed;
}

void cache_init(RowCache& c, int64_t n, int64_t bytes, Context& cx)
{
    c.slots = 0;
    if (const char* e = getenv("SVM_CACHE_BYTES"))  // developer override
        bytes = atoll(e);
    if (bytes < 0 || n <= 0) return;
    c.ldc = (n + 3) / 4 * 4;
    const int64_t row = c.ldc * (int64_t)sizeof(float);
    size_t free_b = 0, total_b = 0;
    HIP_TRY(hipMemGetInfo(&free_b, &total_b));
    free_b += cache_pool_idle_bytes(cx.device);  // kept for the cache
    // default: the whole K when it fits a quarter of the free memory (the
    // cache then keeps every row it computes); otherwise a quarter of the
    // free memory, at most 8 GiB.  An explicit budget may use the free
    // memory but 2 GiB (left to the caller).
    int64_t cap = std::min<int64_t>((int64_t)(free_b / 4), (int64_t)8 << 30);
    if (n * row <= (int64_t)(free_b / 4)) cap = n * row;
    if (bytes > 0)
        cap = std::min<int64_t>(bytes,
                                std::max<int64_t>((int64_t)free_b -
                                                      ((int64_t)2 << 30), 0));
    const int64_t slots = std::min<int64_t>(n, cap / row);
    // a working set reads up to kMaxQ slots and the replacement needs a
    // free one besides them
    if (slots <= kMaxQ && slots < n) return;
    if (slots < 2) return;
    // (+16 floats: the row kernel reads whole 16-row tiles, up to 15 rows
    // past the last sample, and the last row has nothing after it)
    c.rows.alloc((size_t)(slots * c.ldc + 16), cx.device);
    c.slot_of.alloc((size_t)n);
    c.owner.alloc((size_t)slots);
    c.clock.alloc(1);
    HIP_TRY(hipMemsetAsync(c.slot_of.p, 0xFF, c.slot_of.bytes(), cx.stream));
    HIP_TRY(hipMemsetAsync(c.owner.p, 0xFF, c.owner.bytes(), cx.stream));
    HIP_TRY(hipMemsetAsync(c.clock.p, 0, c.clock.bytes(), cx.stream));
    c.slots = slots;
}

Solver::Solver(Context& cx, const Features& f, const float* y_dev,
               const SolveOptions& o, RowCache* cache, const int32_t* fold,
               int32_t held)
    : cx_(cx), f_(f), o_(o), cache_(cache && cache->slots > 0 ? cache : nullptr)
{
    n_ = f.n;
    N_ = o.type == SVM_EPS_SVR ? 2 * n_ : n_;
    kf_ = kernel_fn(o);
    half_ = o.q / 2;
    nblk_cols_ = o.q <= 16 ? 1 : (o.q <= 32 ? 2 : 4);
    // Grid: every block of k_rows resident at once (occupancy from the
    // runtime); units of 32 rows (two 16-row tiles) are shared out evenly
    // over the blocks, and a block's tiles over its waves: at most
    // `tiles_` tiles per wave.
    constexpr int kWaves = kRowThreads / 64;
    const bool svr = o.type == SVM_EPS_SVR;
    constexpr size_t kLdsMax = 160 * 1024;
    if (f.csr && o.q > 32)
        throw Error{SVM_E_UNSUPPORTED,
                    "CSR input supports working sets of at most 32"};
    if (rows_lds_bytes(nblk_cols_, f.ldp, 1, svr, csr_cols(nblk_cols_)) > kLdsMax)
        throw Error{SVM_E_UNSUPPORTED,
                    "too many features for the dense row kernel's LDS tile"};
    int cus = 0;
    HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                                  cx.device));
    const int64_t units = (n_ + 31) / 32;
    const int64_t tiles_total = (n_ + 15) / 16;
    // tiles per wave with nb blocks
    auto wave_tiles = [&](int64_t nb) {
        const int64_t block_tiles = 2 * ((units + nb - 1) / nb);
        return (int)((block_tiles + kWaves - 1) / kWaves);
    };
    // The LDS of a block grows with the tiles per wave (row data is staged),
    // and the resident blocks shrink with the LDS: iterate to a fixed point
    // (tiles only grow, so this ends).
    tiles_ = 1;
    int64_t cap_blocks = 1;
    for (int it = 0; it < 8; ++it) {
        const size_t lds = rows_lds_bytes(nblk_cols_, f.ldp, tiles_, svr, csr_cols(nblk_cols_));
        cap_blocks = (int64_t)cus * rows_blocks_per_cu(nblk_cols_, svr, lds, f.csr);
        const int t = wave_tiles(std::min(cap_blocks, units));
        if (t <= tiles_) break;
        tiles_ = t;
    }
    // as many blocks as are resident (fewer when there are fewer tiles);
    // one candidate record per block, at most kSelRecords per select thread
    const int64_t rec_cap = (int64_t)kSelThreads * kSelRecords;
    int64_t nb = std::min(cap_blocks, (tiles_total + kWaves - 1) / kWaves);
    if (const char* e = getenv("SVM_TILES")) {  // tuning override
        const int64_t t = std::max(1, std::min(4096, atoi(e)));
        nb = (tiles_total + kWaves * t - 1) / (kWaves * t);
    }
    nb = std::max<int64_t>(1, std::min({nb, rec_cap, units}));
    tiles_ = wave_tiles(nb);
    if (rows_lds_bytes(nblk_cols_, f.ldp, tiles_, svr, csr_cols(nblk_cols_)) > kLdsMax ||
        (int64_t)16 * tiles_ * f.ldp * 4 >= ((int64_t)1 << 31))
        throw Error{SVM_E_UNSUPPORTED,
                    "training set too large for the dense row kernel"};
    nb_ = (int)nb;
    ch_cap_ = sparse_chunk_cap(f);

    // One launch per outer iteration: as many k_iter blocks as are
    // resident (at most kIterMaxRecords, one candidate record each), the
    // rows of a block over its 3 row waves.
    if (one_launch_loop(o, f)) {
        auto iter_tiles = [&](int64_t nbk) {
            const int64_t block_tiles = 2 * ((units + nbk - 1) / nbk);
            return (int)((block_tiles + 2) / 3);
        };
        int T = 1;
        int64_t nbk = 1;
        bool ok = true;
        for (int it = 0; it < 8; ++it) {
            const size_t lds = iter_lds_bytes(f.ldp, T, svr);
            if (lds > kLdsMax) {
                ok = false;
                break;
            }
            const int64_t cap =
                (int64_t)cus * iter_blocks_per_cu(svr, lds);
            nbk = std::max<int64_t>(
                1, std::min<int64_t>({cap, units, (int64_t)kIterMaxRecords}));
            const int t = iter_tiles(nbk);
            if (t <= T) break;
            T = t;
        }
        T = iter_tiles(nbk);
        const int tk = wave_tiles(nbk);  // the k_rows launch on that grid
        if (ok && iter_lds_bytes(f.ldp, T, svr) <= kLdsMax &&
            rows_lds_bytes(1, f.ldp, tk, svr, -1) <= kLdsMax &&
            (int64_t)16 * std::max(T, tk) * f.ldp * 4 < ((int64_t)1 << 31)) {
            fused_ = true;
            nbi_ = (int)nbk;
            tilesi_ = T;
            tilesk_ = tk;
            cache_ = nullptr;  // (the row cache serves the two-launch loop)
        }
    }

    F_.alloc((size_t)n_);
    alpha_.alloc((size_t)N_);
    st_.alloc((size_t)N_);
    y_.alloc((size_t)n_);
    ws_.alloc(1);
    xS_.alloc((size_t)kMaxQ * f.ldp);
    if (f.csr) {
        xsc_cols_.alloc((size_t)f.ldp);
        xsc_.alloc((size_t)(f.ldp + 1) * kMaxQ);
    }
    ckey_.alloc((size_t)nb_ * 2 * kBlockTop);
    cidx_.alloc((size_t)nb_ * 2 * kBlockTop);
    if (fused_) {
        F2_.alloc((size_t)n_);
        irk_.alloc((size_t)2 * nbi_ * 2 * kBlockTop);
        iri_.alloc((size_t)2 * nbi_ * 2 * kBlockTop);
        ticket_.alloc(1);
    }
    sum_.alloc(1 + kSummaryBlocks);
    cvec_.alloc((size_t)n_);
    cblk_.alloc((size_t)compact_blocks(n_));
    sv_idx_.alloc((size_t)n_);
    sv_coef_.alloc((size_t)n_);
    sv_cnt_.alloc(1);

    hipStream_t s = cx_.stream;
    HIP_TRY(hipMemcpyAsync(y_.p, y_dev, (size_t)n_ * sizeof(float),
                           hipMemcpyDeviceToDevice, s));
    HIP_TRY(hipMemsetAsync(F_.p, 0, F_.bytes(), s));
    HIP_TRY(hipMemsetAsync(alpha_.p, 0, alpha_.bytes(), s));
    HIP_TRY(hipMemsetAsync(ws_.p, 0, sizeof(WorkingSet), s));
    HIP_TRY(hipMemsetAsync(xS_.p, 0, xS_.bytes(), s));
    if (fused_) HIP_TRY(hipMemsetAsync(ticket_.p, 0, ticket_.bytes(), s));
    DevBuf<int32_t> bad(1);
    HIP_TRY(hipMemsetAsync(bad.p, 0, sizeof(int32_t), s));
    launch_init_state(o.type, y_.p, n_, fold, held, st_.p, bad.p, s);
    int32_t hb = 0;
    HIP_TRY(hipMemcpyAsync(&hb, bad.p, sizeof(int32_t), hipMemcpyDeviceToHost,
                           s));
    cx_.sync();
    if (o.type == SVM_C_SVC) {
        if (hb & 1) throw Error{SVM_E_INVALID, "labels must be +1 or -1"};
        if ((hb & 6) != 6)
            throw Error{SVM_E_INVALID, "both classes must be present"};
    } else if (hb & 1) {
        throw Error{SVM_E_INVALID, "targets must be finite"};
    }
}

int Solver::csr_cols(int nbc) const
{
    if (!f_.csr) return -1;
    // the columns of the working set: at most its samples' nonzeros and d
    const int64_t c = std::min<int64_t>(f_.ldp,
                                        (int64_t)16 * nbc * std::max<int64_t>(1, f_.maxnz));
    return (int)c;
}

void Solver::set_csr(RowArgs& a, int nbc) const
{
    a.so = f_.so.p;
    a.sci = f_.sci.p;
    a.scv = f_.scv.p;
    a.csr_cols = csr_cols(nbc);
    a.xsc_cols = xsc_cols_.p;
    a.xsc = xsc_.p;
}

void Solver::set_csr(SelArgs& a, int nbc)
{
    a.csr_cols = csr_cols(nbc);
    a.xsc_cols = xsc_cols_.p;
    a.xsc = xsc_.p;
}

void Solver::launch_keys()
{
    RowArgs a{};
    a.X = f_.x();
    a.rp = f_.rp.p;
    a.ci = f_.ci.p;
    a.cv = f_.cv.p;
    a.sq = f_.sq.p;
    a.F = F_.p;
    a.st = st_.p;
    a.z = y_.p;
    a.ws = ws_.p;
    a.xS = xS_.p;
    set_csr(a, nblk_cols_);
    a.cand_key = ckey_.p;
    a.cand_idx = cidx_.p;
    a.n = n_;
    a.ldp = f_.ldp;
    a.eps = o_.eps;
    a.kf = kf_;
    a.half = half_;
    a.tiles = tiles_;
    a.mode = RU_CAND;
    a.nS_override = 0;
    launch_rows(a, nb_, nblk_cols_, o_.type == SVM_EPS_SVR, cx_.stream);
}

// The first candidate records of the one-launch loop (k_rows, keys only,
// on k_iter's grid: the same row range per block, so the records belong to
// the row groups k_iter's rescans assume), into parity 0.
void Solver::launch_keys_fused()
{
    RowArgs a{};
    a.X = f_.x();
    a.sq = f_.sq.p;
    a.F = F_.p;
    a.st = st_.p;
    a.z = y_.p;
    a.ws = ws_.p;
    a.xS = xS_.p;
    a.csr_cols = -1;
    a.cand_key = irk_.p;
    a.cand_idx = iri_.p;
    a.n = n_;
    a.ldp = f_.ldp;
    a.eps = o_.eps;
    a.kf = kf_;
    a.half = half_;
    a.tiles = tilesk_;
    a.mode = RU_CAND;
    a.nS_override = 0;
    launch_rows(a, nbi_, 1, o_.type == SVM_EPS_SVR, cx_.stream);
}

void Solver::launch_hot_rows(hipEvent_t e0, hipEvent_t e1)
{
    RowArgs a{};
    a.X = f_.x();
    a.rp = f_.rp.p;
    a.ci = f_.ci.p;
    a.cv = f_.cv.p;
    a.sq = f_.sq.p;
    a.F = F_.p;
    a.st = st_.p;
    a.z = y_.p;
    a.ws = ws_.p;
    a.xS = xS_.p;
    set_csr(a, nblk_cols_);
    a.cand_key = ckey_.p;
    a.cand_idx = cidx_.p;
    a.n = n_;
    a.ldp = f_.ldp;
    a.eps = o_.eps;
    a.kf = kf_;
    a.half = half_;
    a.tiles = tiles_;
    a.mode = RU_UPDATE | RU_CAND | RU_CHECK_DONE;
    a.nS_override = -1;
    if (cache_) {
        a.cache = cache_->rows.p;
        a.ldc = cache_->ldc;
    }
    launch_rows(a, nb_, nblk_cols_, o_.type == SVM_EPS_SVR, cx_.stream, e0,
                e1);
}

void Solver::launch_solve(int32_t mode, hipEvent_t e0, hipEvent_t e1)
{
    SelArgs a{};
    a.cand_key = ckey_.p;
    a.cand_idx = cidx_.p;
    a.nb = nb_;
    a.half = half_;
    a.ws = ws_.p;
    a.alpha = alpha_.p;
    a.st = st_.p;
    a.F = F_.p;
    a.z = y_.p;
    a.X = f_.x();
    a.rp = f_.rp.p;
    a.ci = f_.ci.p;
    a.cv = f_.cv.p;
    a.sq = f_.sq.p;
    a.xS = xS_.p;
    set_csr(a, nblk_cols_);
    a.n = n_;
    a.ldp = f_.ldp;
    a.C = o_.C;
    a.eps = o_.eps;
    a.tol = o_.tol;
    a.kf = kf_;
    a.inner_ratio = o_.inner_ratio;
    a.inner_tol_override = -1.0;
    a.max_inner = o_.max_inner;
    a.max_iter = o_.max_iter;
    a.mode = mode;
    a.group_rows = (kRowThreads / 64) * 16 * tiles_;  // most rows of a block
    if (cache_) {
        a.cache = cache_->rows.p;
        a.ldc = cache_->ldc;
        a.cache_slots = cache_->slots;
        a.slot_of = cache_->slot_of.p;
        a.owner = cache_->owner.p;
        a.clock = cache_->clock.p;
    }
    launch_select(a, nblk_cols_, o_.type == SVM_EPS_SVR, cx_.stream, e0, e1);
}

void Solver::launch_select_only() { launch_solve(0); }

void Solver::read_ws(WorkingSet& w)
{
    HIP_TRY(hipMemcpyAsync(&w, ws_.p, sizeof(WorkingSet),
                           hipMemcpyDeviceToHost, cx_.stream));
    cx_.sync();
}

// Chunks of the iteration loop whose row launches are timed in profiling
// mode: one in kProfileEvery.
constexpr int64_t kProfileEvery = 4;

// Queue chunks of `check_every` iterations, two chunks in flight, and poll
// the done flag of the older chunk.  Iterations queued after convergence
// return at their first instruction.
bool Solver::run_loop(SolveResult& r)
{
    const int K = o_.check_every;
    HostBuf<WorkingSet> hs(2);
    hipEvent_t ev[2];
    HIP_TRY(hipEventCreateWithFlags(&ev[0], hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&ev[1], hipEventDisableTiming));
    std::vector<hipEvent_t> pe;
    if (o_.profile) {
        // per iteration of the two chunks in flight: the row launch's two
        // events, then the select launch's two
        pe.resize((size_t)8 * K);
        // device-scope release only: the events time the kernel, not a
        // flush of the caches to host-visible memory
        for (auto& e : pe)
            HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    }
    WorkingSet w0;
    read_ws(w0);
    int64_t last_iter = w0.iter;

    // profiling: the row launches of one chunk in kProfileEvery carry the
    // events (a launch with events costs the loop about 1.4 us more), so
    // the timed launches are a sample spread over the whole solve
    int64_t chunk_no = 0;
    bool timed[2] = {false, false};
    int kc[2] = {K, K};  // iterations queued in each chunk
    double gmin = -1.0;  // smallest gap polled so far, and its iteration
    int64_t it_min = 0;
    auto enqueue = [&](int slot, int kk) {
        timed[slot] = o_.profile && chunk_no % kProfileEvery == 0;
        ++chunk_no;
        kc[slot] = kk;
        for (int k = 0; k < kk; ++k) {
            // the events are part of the kernel's own dispatch, so they
            // bracket its execution, not the queue around it
            const size_t e = (size_t)(slot * K + k) * 4;
            if (timed[slot]) {
                if (o_.profile >= 2)
                    launch_solve(SS_SOLVE | SS_CHECK_DONE, pe[e + 2],
                                 pe[e + 3]);
                else
                    launch_solve(SS_SOLVE | SS_CHECK_DONE);
                launch_hot_rows(pe[e], pe[e + 1]);
            } else {
                launch_solve(SS_SOLVE | SS_CHECK_DONE);
                launch_hot_rows();
            }
        }
        HIP_TRY(hipMemcpyAsync(&hs.p[slot], ws_.p, sizeof(WorkingSet),
                               hipMemcpyDeviceToHost, cx_.stream));
        HIP_TRY(hipEventRecord(ev[slot], cx_.stream));
    };

    enqueue(0, K);
    enqueue(1, K);
    int cur = 0;
    for (;;) {
        HIP_TRY(hipEventSynchronize(ev[cur]));
        const WorkingSet& w = hs.p[cur];
        if (timed[cur]) {
            int64_t real = std::min<int64_t>(w.iter - last_iter, kc[cur]);
            // algorithmic bytes of a launch: computed from X, the features,
            // norm, F read and written and the state byte(s) (eps-SVR: and
            // the target) of every row, plus the rows written to the cache;
            // served from the cache, the nS cached rows instead of X and
            // the norms
            const bool svr = o_.type == SVM_EPS_SVR;
            const double per_row = 16.0 + (svr ? 6.0 : 1.0);
            for (int64_t k = 0; k < real; ++k) {
                const size_t e = (size_t)(cur * K + k) * 4;
                float ms = 0.f;
                HIP_TRY(hipEventElapsedTime(&ms, pe[e], pe[e + 1]));
                if (o_.profile >= 2) {
                    float sms = 0.f;
                    HIP_TRY(hipEventElapsedTime(&sms, pe[e + 2], pe[e + 3]));
                    select_ms_ += sms;
                    select_launches_ += 1;
                }
                const int64_t t = (last_iter + k + 1) % kPathLog;
                if (w.path_log[t] == PATH_CACHED) {
                    cached_ms_ += ms;
                    cached_launches_ += 1;
                    cached_bytes_ +=
                        (double)n_ * (per_row + 4.0 * (double)w.ns_log[t]);
                } else {
                    // the features: dense 4d per row; CSR 8 per nonzero
                    // and the row pointers, or in the sliced copy 6 per
                    // nonzero (16-bit column) and the slice offsets
                    const bool sl = f_.csr && f_.so.p != nullptr;
                    const double feat =
                        !f_.csr ? 4.0 * (double)f_.d * (double)n_
                        : sl    ? 6.0 * (double)f_.nnz +
                                   8.0 * (double)((n_ + kSellRows - 1) /
                                                      kSellRows + 1)
                                : 8.0 * (double)f_.nnz + 8.0 * (double)(n_ + 1);
                    row_ms_ += ms;
                    row_launches_ += 1;
                    row_rows_ += n_;
                    row_bytes_ += feat + (double)n_ * (per_row + 4.0 +
                                                       4.0 * w.fill_log[t]);
                }
            }
        }
        if (w.done) break;
        if (w.iter == last_iter) {
            cx_.sync();
            for (auto& e : pe) (void)hipEventDestroy(e);
            (void)hipEventDestroy(ev[0]);
            (void)hipEventDestroy(ev[1]);
            throw Error{SVM_E_INTERNAL, "solver state made no progress"};
        }
        last_iter = w.iter;
        // Near the end the chunks shrink: the launches queued behind the
        // converged iteration return at once but still cost a launch each
        // (about 5 us a pair), and a whole chunk is in flight when the host
        // sees convergence.  The iterations still to go are estimated from
        // the rate at which the smallest gap seen so far has been falling
        // (log scale); a chunk is then about half of them, at least K / 8.
        // The device stops at the same iteration whatever the chunking.
        int next = K;
        if (w.gap > o_.tol && gmin > 0.0 && w.gap < gmin) {
            const double rate = std::log(gmin / w.gap) /
                                (double)std::max<int64_t>(w.iter - it_min, 1);
            const double togo = std::log(w.gap / o_.tol) / rate;
            if (togo < 2.0 * K)
                next = std::max(std::max(K / 8, 1),
                                std::min(K, (int)(0.5 * togo)));
        }
        if (gmin <= 0.0 || w.gap < gmin) {
            gmin = w.gap;
            it_min = w.iter;
        }
        enqueue(cur, next);
        cur ^= 1;
    }
    cx_.sync();
    for (auto& e : pe) (void)hipEventDestroy(e);
    (void)hipEventDestroy(ev[0]);
    (void)hipEventDestroy(ev[1]);
    WorkingSet w;
    read_ws(w);
    r.iters = w.iter;
    r.gap = w.gap;
    r.m = w.m;
    r.M = w.M;
    r.kernel_rows = w.rows;
    r.status = w.done == 2 ? SVM_W_MAX_ITER : SVM_OK;
    return w.done == 1;
}

// The one-launch loop: chunks of `check_every` k_iter launches, two chunks
// in flight, the done flag of the older chunk polled.  Launch k of the
// chunk sequence reads the responses and records of parity k % 2 and writes
// the other; the responses end in F_ (copied there when the number of
// iterations was odd).
bool Solver::run_loop_fused(SolveResult& r)
{
    const int K = o_.check_every;
    HostBuf<WorkingSet> hs(2);
    hipEvent_t ev[2];
    HIP_TRY(hipEventCreateWithFlags(&ev[0], hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&ev[1], hipEventDisableTiming));
    std::vector<hipEvent_t> pe;
    if (o_.profile) {
        pe.resize((size_t)4 * K);
        for (auto& e : pe)
            HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    }
    WorkingSet w0;
    read_ws(w0);
    const int64_t iter_start = w0.iter;
    int64_t last_iter = w0.iter;
    const int64_t units = (n_ + 31) / 32;
    IterArgs a{};
    a.X = f_.x();
    a.sq = f_.sq.p;
    a.z = y_.p;
    a.alpha = alpha_.p;
    a.st = st_.p;
    a.ws = ws_.p;
    a.ticket = ticket_.p;
    a.n = n_;
    a.ldp = f_.ldp;
    a.nb = nbi_;
    a.half = half_;
    a.tiles = tilesi_;
    a.group_rows = (int32_t)std::min<int64_t>(
        n_, 32 * ((units + nbi_ - 1) / nbi_));
    a.C = o_.C;
    a.eps = o_.eps;
    a.tol = o_.tol;
    a.kf = kf_;
    a.inner_ratio = o_.inner_ratio;
    a.max_inner = o_.max_inner;
    a.max_iter = o_.max_iter;
    const size_t rec = (size_t)nbi_ * 2 * kBlockTop;
    int64_t launched = 0;
    const bool svr = o_.type == SVM_EPS_SVR;

    int64_t chunk_no = 0;  // (profiling: one chunk in kProfileEvery)
    bool timed[2] = {false, false};
    auto enqueue = [&](int slot) {
        timed[slot] = o_.profile && chunk_no % kProfileEvery == 0;
        ++chunk_no;
        for (int k = 0; k < K; ++k) {
            const int par = (int)(launched & 1);
            a.F_in = par ? F2_.p : F_.p;
            a.F_out = par ? F_.p : F2_.p;
            a.rk_in = irk_.p + par * rec;
            a.ri_in = iri_.p + par * rec;
            a.rk_out = irk_.p + (1 - par) * rec;
            a.ri_out = iri_.p + (1 - par) * rec;
            if (timed[slot])
                launch_iter(a, nbi_, svr, cx_.stream,
                            pe[(size_t)(slot * K + k) * 2],
                            pe[(size_t)(slot * K + k) * 2 + 1]);
            else
                launch_iter(a, nbi_, svr, cx_.stream);
            ++launched;
        }
        HIP_TRY(hipMemcpyAsync(&hs.p[slot], ws_.p, sizeof(WorkingSet),
                               hipMemcpyDeviceToHost, cx_.stream));
        HIP_TRY(hipEventRecord(ev[slot], cx_.stream));
    };

    enqueue(0);
    enqueue(1);
    int cur = 0;
    for (;;) {
        HIP_TRY(hipEventSynchronize(ev[cur]));
        const WorkingSet& w = hs.p[cur];
        if (timed[cur]) {
            const int64_t real = std::min<int64_t>(w.iter - last_iter, K);
            const double per_row = 16.0 + (svr ? 6.0 : 1.0);
            for (int64_t k = 0; k < real; ++k) {
                float ms = 0.f;
                HIP_TRY(hipEventElapsedTime(
                    &ms, pe[(size_t)(cur * K + k) * 2],
                    pe[(size_t)(cur * K + k) * 2 + 1]));
                row_ms_ += ms;
                row_launches_ += 1;
                row_rows_ += n_;
                row_bytes_ += 4.0 * (double)f_.d * (double)n_ +
                              (double)n_ * (per_row + 4.0);
            }
        }
        if (w.done) break;
        if (w.iter == last_iter) {
            cx_.sync();
            for (auto& e : pe) (void)hipEventDestroy(e);
            (void)hipEventDestroy(ev[0]);
            (void)hipEventDestroy(ev[1]);
            throw Error{SVM_E_INTERNAL, "solver state made no progress"};
        }
        last_iter = w.iter;
        enqueue(cur);
        cur ^= 1;
    }
    cx_.sync();
    for (auto& e : pe) (void)hipEventDestroy(e);
    (void)hipEventDestroy(ev[0]);
    (void)hipEventDestroy(ev[1]);
    WorkingSet w;
    read_ws(w);
    // iteration k (counted from this call's start) wrote F2_ when odd
    if ((w.iter - iter_start) & 1)
        HIP_TRY(hipMemcpyAsync(F_.p, F2_.p, (size_t)n_ * sizeof(double),
                               hipMemcpyDeviceToDevice, cx_.stream));
    r.iters = w.iter;
    r.gap = w.gap;
    r.m = w.m;
    r.M = w.M;
    r.kernel_rows = w.rows;
    r.status = w.done == 2 ? SVM_W_MAX_ITER : SVM_OK;
    return w.done == 1;
}

bool Solver::loop(SolveResult& r)
{
    if (!fused_) return run_loop(r);  // (candidates from launch_keys)
    launch_keys_fused();
    return run_loop_fused(r);
}

void Solver::recompute_responses()
{
    hipStream_t s = cx_.stream;
    launch_coef(o_.type, alpha_.p, st_.p, n_, cvec_.p, s);
    launch_compact(cvec_.p, n_, 1, cblk_.p, sv_idx_.p, sv_coef_.p,
                   sv_cnt_.p, s);
    int64_t nsv = 0;
    HIP_TRY(hipMemcpyAsync(&nsv, sv_cnt_.p, sizeof(int64_t),
                           hipMemcpyDeviceToHost, s));
    cx_.sync();
    if (nsv == 0) {
        HIP_TRY(hipMemsetAsync(F_.p, 0, F_.bytes(), s));
        return;
    }
    PredictArgs a{};
    if (sv_sq_.count < (size_t)nsv) sv_sq_.alloc((size_t)nsv);
    if (f_.csr)
        build_fact(fc_, f_, sv_idx_.p, nsv, sv_coef_.p, 1, kf_, cx_,
                   sv_sq_.p, &f_);
    if (fc_.ok) {
        if (self_sv_.count < (size_t)n_) self_sv_.alloc((size_t)n_);
        launch_fc_self(sv_idx_.p, nsv, n_, self_sv_.p, s);
        a.self_sv = self_sv_.p;
    } else if (ch_cap_ > 0) {
        build_sv_chunks(f_, sv_idx_.p, nsv, ch_cap_, ch_ncol_, ch_cols_,
                        ch_tab_, sv_sq_.p, s);
        a.ch_ncol = ch_ncol_.p;
        a.ch_cols = ch_cols_.p;
        a.ch_tab = ch_tab_.p;
        a.ch_cap = ch_cap_;
    } else {
        if (sv_rows_.count < (size_t)(nsv * f_.ldp))
            sv_rows_.alloc((size_t)(nsv * f_.ldp));
        gather_rows(f_, sv_idx_.p, nsv, sv_rows_.p, sv_sq_.p, s);
        a.SV = sv_rows_.p;
    }
    a.sqsv = sv_sq_.p;
    a.nsv = nsv;
    a.coef = sv_coef_.p;
    a.b = nullptr;
    a.n_out = 1;
    a.sv_train_idx = sv_idx_.p;
    a.self_match = 1;
    a.out = F_.p;
    a.kf = kf_;
    predict_rows(a, f_, s, fc_.ok ? &fc_ : nullptr);
}

SolveResult Solver::train()
{
    SolveResult r;
    hipEvent_t t0 = start(!fused_);
    bool conv;
    {
        Range rg("svm solve loop");
        conv = loop(r);
    }
    Range rg("svm finish (recompute, gap, bias, objective)");
    finish(r, conv, t0);
    return r;
}

hipEvent_t Solver::start(bool keys)
{
    hipEvent_t t0;
    HIP_TRY(hipEventCreate(&t0));
    HIP_TRY(hipEventRecord(t0, cx_.stream));
    if (keys) launch_keys();
    return t0;
}

void Solver::finish(SolveResult& r, bool conv, hipEvent_t t0, int max_passes)
{
    hipEvent_t t1;
    HIP_TRY(hipEventCreate(&t1));
    // The incremental responses accumulate rounding over many updates: F is
    // recomputed from alpha and the gap re-tested on it.  A solve that met
    // tol only on the incremental responses continues from the recomputed
    // ones, at most max_passes times; the gap, m and M reported (and the
    // bias and objective below) always come from recomputed responses, and
    // SVM_OK only from a gap measured on them.
    for (int pass = 0;; ++pass) {
        recompute_responses();
        launch_keys();
        launch_select_only();
        WorkingSet w;
        read_ws(w);
        r.gap = w.gap;
        r.m = w.m;
        r.M = w.M;
        if (!conv || w.gap <= o_.tol) break;  // (max_iter: status stands)
        if (pass >= max_passes) {
            r.status = SVM_W_NOT_CONVERGED;
            break;
        }
        launch_fill_i32(&ws_.p->done, 0, 1, cx_.stream);
        conv = loop(r);
    }

    launch_summary(o_.type, alpha_.p, st_.p, F_.p, y_.p, n_, o_.C, o_.eps,
                   sum_.p, cx_.stream);
    Summary sm;
    HIP_TRY(hipMemcpyAsync(&sm, sum_.p, sizeof(Summary),
                           hipMemcpyDeviceToHost, cx_.stream));
    int64_t nsv = 0;
    HIP_TRY(hipMemcpyAsync(&nsv, sv_cnt_.p, sizeof(int64_t),
                           hipMemcpyDeviceToHost, cx_.stream));
    HIP_TRY(hipEventRecord(t1, cx_.stream));
    cx_.sync();
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, t0, t1));
    (void)hipEventDestroy(t0);
    (void)hipEventDestroy(t1);

    r.n_free = sm.n_free;
    r.n_bounded = sm.n_bounded;
    r.b = sm.n_free > 0 ? sm.sum_free_v / (double)sm.n_free
                        : 0.5 * (r.m + r.M);
    r.obj = -0.5 * sm.obj2;
    r.n_sv = nsv;
    r.train_ms = ms;
    r.row_ms = row_ms_;
    r.row_launches = row_launches_;
    r.row_rows = row_rows_;
    r.row_bytes = row_bytes_;
    r.cached_ms = cached_ms_;
    r.cached_launches = cached_launches_;
    r.cached_bytes = cached_bytes_;
    r.select_ms = select_ms_;
    r.select_launches = select_launches_;
    WorkingSet w;
    read_ws(w);
    r.kernel_rows = w.rows;
    r.cache_served = w.cache_served;
    r.cache_filled = w.cache_filled;
    r.iters = w.iter;
    if (const char* e = getenv("SVM_LOG")) {
        if (atoi(e) > 0 && fused_ && w.prof[4] > 0) {
            const double k = 10.0 / (double)w.prof[4];  // 100 MHz ticks -> ns
            fprintf(stderr,
                    "[mi355svm] one launch per iteration: iters=%lld "
                    "blocks=%d tiles=%d rescans=%lld; phases of the last "
                    "block (us): merge %.2f rescans %.2f build %.2f stage "
                    "%.2f solve %.2f rows %.2f tail %.2f; kernel %.2f "
                    "us/launch (%lld timed)\n",
                    (long long)w.iter, nbi_, tilesi_, (long long)w.rescans,
                    1e-3 * k * w.prof[0], 1e-3 * k * w.prof[1],
                    1e-3 * k * w.prof[2], 1e-3 * k * w.prof[3],
                    1e-3 * k * w.prof[5], 1e-3 * k * w.prof[6],
                    1e-3 * k * w.prof[7],
                    row_launches_ ? 1e3 * row_ms_ / row_launches_ : 0.0,
                    (long long)row_launches_);
        } else if (atoi(e) > 0 && w.prof[4] > 0) {
            const double k = 10.0 / (double)w.prof[4];  // 100 MHz ticks -> ns
            fprintf(stderr,
                    "[mi355svm] iters=%lld rows=%lld (cache: served %lld "
                    "filled %lld) inner=%.1f/iter rescans=%lld slow=%lld "
                    "select(us): merge %.2f (bound %.2f rank %.2f groups "
                    "%.2f rescans %.2f) kss %.2f (build %.2f stage %.2f) "
                    "inner %.2f write %.2f; rows kernel %.2f us/launch "
                    "(%lld timed), cached %.2f us/launch (%lld)\n",
                    (long long)w.iter, (long long)w.rows,
                    (long long)w.cache_served, (long long)w.cache_filled,
                    (double)w.inner_total / (double)w.prof[4],
                    (long long)w.rescans, (long long)w.slow_selects,
                    1e-3 * k * w.prof[0], 1e-3 * k * w.prof[5],
                    1e-3 * k * w.prof[8], 1e-3 * k * w.prof[9],
                    1e-3 * k * w.prof[10], 1e-3 * k * w.prof[1],
                    1e-3 * k * w.prof[6], 1e-3 * k * w.prof[7],
                    1e-3 * k * w.prof[2], 1e-3 * k * w.prof[3],
                    row_launches_ ? 1e3 * row_ms_ / row_launches_ : 0.0,
                    (long long)row_launches_,
                    cached_launches_ ? 1e3 * cached_ms_ / cached_launches_
                                     : 0.0,
                    (long long)cached_launches_);
        }
    }
}

int Solver::lock_capacity(const Features& f, int32_t type)
{
    constexpr size_t kLdsMax = 160 * 1024;
    const bool svr = type == SVM_EPS_SVR;
    int P = kLockMax;
    while (P > 1 && lock_lds_bytes(P, f.ldp, 1, svr) > kLdsMax) --P;
    return P;
}

std::vector<SolveResult> Solver::train_lockstep(
    const std::vector<Solver*>& g)
{
    const int G = (int)g.size();
    std::vector<SolveResult> res(G);
    if (G == 0) return res;
    Solver& s0 = *g[0];
    Context& cx = s0.cx_;
    const Features& f = s0.f_;
    const bool svr = s0.o_.type == SVM_EPS_SVR;
    const int64_t n = s0.n_;
    if (G > lock_capacity(f, s0.o_.type))
        throw Error{SVM_E_INTERNAL, "lockstep group too large"};
    for (Solver* s : g) {
        if (&s->f_ != &f || &s->cx_ != &cx || s->o_.type != s0.o_.type ||
            s->kf_.kind != s0.kf_.kind || s->o_.q != 16 || f.csr ||
            s->cache_ != nullptr)
            throw Error{SVM_E_INTERNAL, "solvers cannot run in lockstep"};
    }
    hipStream_t st = cx.stream;

    // Grid of the lockstep pass for all G problems (as the constructor
    // does for k_rows): every block resident, units of 32 rows shared out
    // evenly; fewer problems later reuse it (their LDS is smaller).
    constexpr int kWaves = kRowThreads / 64;
    constexpr size_t kLdsMax = 160 * 1024;
    int cus = 0;
    HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                                  cx.device));
    const int64_t units = (n + 31) / 32, tiles_total = (n + 15) / 16;
    auto wave_tiles = [&](int64_t nb) {
        const int64_t block_tiles = 2 * ((units + nb - 1) / nb);
        return (int)((block_tiles + kWaves - 1) / kWaves);
    };
    int tiles = 1;
    int64_t cap_blocks = 1;
    for (int it = 0; it < 8; ++it) {
        const size_t lds = lock_lds_bytes(G, f.ldp, tiles, svr);
        cap_blocks = (int64_t)cus * lock_blocks_per_cu(G, svr, lds);
        const int t = wave_tiles(std::min(cap_blocks, units));
        if (t <= tiles) break;
        tiles = t;
    }
    const int64_t rec_cap = (int64_t)kSelThreads * kSelRecords;
    int64_t nb = std::min(cap_blocks, (tiles_total + kWaves - 1) / kWaves);
    nb = std::max<int64_t>(1, std::min({nb, rec_cap, units}));
    tiles = wave_tiles(nb);
    // the staged rows of many features leave little LDS for the row data:
    // more blocks (not all resident at once), fewer tiles per wave
    while (lock_lds_bytes(G, f.ldp, tiles, svr) > kLdsMax &&
           nb < std::min(rec_cap, units)) {
        nb = std::min({2 * nb, rec_cap, units});
        tiles = wave_tiles(nb);
    }
    if (lock_lds_bytes(G, f.ldp, tiles, svr) > kLdsMax ||
        (int64_t)16 * tiles * f.ldp * 4 >= ((int64_t)1 << 31))
        throw Error{SVM_E_UNSUPPORTED,
                    "training set too large for the lockstep row kernel"};

    // the group's working-set rows (problem at position p: rows 16p ..),
    // candidate tables of the lockstep grid, selection arguments
    DevBuf<float> xs((size_t)kLockMax * 16 * f.ldp);
    HIP_TRY(hipMemsetAsync(xs.p, 0, xs.bytes(), st));
    std::vector<DevBuf<double>> ck(G);
    std::vector<DevBuf<int32_t>> ci(G);
    for (int p = 0; p < G; ++p) {
        ck[p].alloc((size_t)nb * 2 * kBlockTop);
        ci[p].alloc((size_t)nb * 2 * kBlockTop);
    }
    std::vector<SelArgs> hsel(kLockMax);
    HostBuf<WorkingSet> hws((size_t)2 * G);
    std::vector<int> act(G);
    for (int p = 0; p < G; ++p) act[p] = p;
    LockArgs la{};

    // arguments of the active problems, by position
    auto build = [&]() {
        la = LockArgs{};
        la.X = f.x();
        la.sq = f.sq.p;
        la.xS = xs.p;
        la.n = n;
        la.ldp = f.ldp;
        la.tiles = tiles;
        for (int q = 0; q < (int)act.size(); ++q) {
            Solver& s = *g[act[q]];
            la.F[q] = s.F_.p;
            la.st[q] = s.st_.p;
            la.z[q] = s.y_.p;
            la.ws[q] = s.ws_.p;
            la.cand_key[q] = ck[act[q]].p;
            la.cand_idx[q] = ci[act[q]].p;
            la.kf[q] = s.kf_;
            la.eps[q] = s.o_.eps;
            SelArgs a{};
            a.cand_key = ck[act[q]].p;
            a.cand_idx = ci[act[q]].p;
            a.nb = (int32_t)nb;
            a.half = s.half_;
            a.ws = s.ws_.p;
            a.alpha = s.alpha_.p;
            a.st = s.st_.p;
            a.F = s.F_.p;
            a.z = s.y_.p;
            a.X = f.x();
            a.sq = f.sq.p;
            a.xS = xs.p + (size_t)q * 16 * f.ldp;
            a.csr_cols = -1;
            a.n = n;
            a.ldp = f.ldp;
            a.C = s.o_.C;
            a.eps = s.o_.eps;
            a.tol = s.o_.tol;
            a.kf = s.kf_;
            a.inner_ratio = s.o_.inner_ratio;
            a.inner_tol_override = -1.0;
            a.max_inner = s.o_.max_inner;
            a.max_iter = s.o_.max_iter;
            a.mode = SS_SOLVE | SS_CHECK_DONE;
            a.group_rows = kWaves * 16 * tiles;  // most rows of a block
            hsel[q] = a;
        }
    };

    std::vector<hipEvent_t> t0(G);
    for (int p = 0; p < G; ++p) t0[p] = g[p]->start(false);
    // the first candidates: a pass with empty working sets (F + 0)
    build();
    launch_lock(la, G, (int)nb, svr, st);

    const int K = s0.o_.check_every;
    const bool prof = s0.o_.profile;
    hipEvent_t ev[2];
    HIP_TRY(hipEventCreateWithFlags(&ev[0], hipEventDisableTiming));
    HIP_TRY(hipEventCreateWithFlags(&ev[1], hipEventDisableTiming));
    std::vector<hipEvent_t> pe;
    if (prof) {
        pe.resize((size_t)4 * K);
        for (auto& e : pe)
            HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    }
    auto cleanup = [&]() {
        for (auto& e : pe) (void)hipEventDestroy(e);
        (void)hipEventDestroy(ev[0]);
        (void)hipEventDestroy(ev[1]);
    };
    std::vector<int64_t> last(G, 0);
    std::vector<int> ran(2, 0);  // problems in each chunk
    // (profiling: one chunk in kProfileEvery, chunk j being iterations
    // [jK, (j + 1)K) of every problem of the group, as in a problem's own
    // loop)
    int64_t chunk_no = 0;
    bool timed[2] = {false, false};
    auto enqueue = [&](int slot) {
        const int P = (int)act.size();
        ran[slot] = P;
        timed[slot] = prof && chunk_no % kProfileEvery == 0;
        ++chunk_no;
        for (int k = 0; k < K; ++k) {
            launch_select_group(hsel.data(), P, svr, st);
            if (timed[slot])
                launch_lock(la, P, (int)nb, svr, st,
                            pe[(size_t)(slot * K + k) * 2],
                            pe[(size_t)(slot * K + k) * 2 + 1]);
            else
                launch_lock(la, P, (int)nb, svr, st);
        }
        for (int q = 0; q < P; ++q)
            HIP_TRY(hipMemcpyAsync(&hws.p[(size_t)slot * G + act[q]],
                                   g[act[q]]->ws_.p, sizeof(WorkingSet),
                                   hipMemcpyDeviceToHost, st));
        HIP_TRY(hipEventRecord(ev[slot], st));
    };

    // Algorithmic bytes of a lockstep launch: X and the norms once, and
    // each problem's F (read and written) and state bytes (eps-SVR: and
    // its targets); shared bytes and the time are split evenly over the
    // problems of the launch.
    const double own = 16.0 + (svr ? 6.0 : 1.0);
    const double shared = 4.0 * (double)f.d * (double)n + 4.0 * (double)n;
    auto account = [&](int slot, const std::vector<int64_t>& adv) {
        if (!timed[slot]) return;
        const int P = ran[slot];
        for (int k = 0; k < K; ++k) {
            int pk = 0;
            for (int q = 0; q < P; ++q) pk += adv[act[q]] > k;
            if (pk == 0) continue;
            float ms = 0.f;
            HIP_TRY(hipEventElapsedTime(&ms, pe[(size_t)(slot * K + k) * 2],
                                        pe[(size_t)(slot * K + k) * 2 + 1]));
            for (int q = 0; q < P; ++q) {
                if (adv[act[q]] <= k) continue;
                Solver& s = *g[act[q]];
                s.row_ms_ += ms / pk;
                s.row_launches_ += 1;
                s.row_rows_ += n;
                s.row_bytes_ += shared / pk + (double)n * own;
            }
        }
    };

    try {
        enqueue(0);
        enqueue(1);
        int cur = 0;
        for (;;) {
            HIP_TRY(hipEventSynchronize(ev[cur]));
            std::vector<int64_t> adv(G, 0);
            bool moved = false, changed = false;
            std::vector<int> next;
            for (int p : act) {
                const WorkingSet& w = hws.p[(size_t)cur * G + p];
                adv[p] = w.iter - last[p];
                moved |= adv[p] > 0;
                last[p] = w.iter;
                if (w.done)
                    changed = true;
                else
                    next.push_back(p);
            }
            account(cur, adv);
            if (next.empty()) break;
            if (!moved) throw Error{SVM_E_INTERNAL,
                                    "solver state made no progress"};
            if (changed) {
                // drain the chunk in flight (its problem set is the old
                // one), then restart the pipeline with the rest
                cx.sync();
                const int o = cur ^ 1;
                std::vector<int64_t> adv2(G, 0);
                next.clear();
                for (int p : act) {
                    const WorkingSet& w = hws.p[(size_t)o * G + p];
                    adv2[p] = w.iter - last[p];
                    last[p] = w.iter;
                    if (!w.done) next.push_back(p);
                }
                account(o, adv2);
                if (next.empty()) break;
                act = next;
                build();
                enqueue(0);
                enqueue(1);
                cur = 0;
                continue;
            }
            enqueue(cur);
            cur ^= 1;
        }
        cx.sync();
    } catch (...) {
        cx.sync();
        cleanup();
        for (auto& e : t0) (void)hipEventDestroy(e);
        throw;
    }
    cleanup();

    std::vector<char> conv(G);
    for (int p = 0; p < G; ++p) {
        WorkingSet w;
        g[p]->read_ws(w);
        SolveResult& r = res[p];
        r.iters = w.iter;
        r.gap = w.gap;
        r.m = w.m;
        r.M = w.M;
        r.kernel_rows = w.rows;
        r.status = w.done == 2 ? SVM_W_MAX_ITER : SVM_OK;
        conv[p] = w.done == 1;
    }
    for (int p = 0; p < G; ++p) g[p]->finish(res[p], conv[p], t0[p]);
    return res;
}

void Solver::coefficients(double* c, int32_t stride, int32_t off)
{
    launch_coef_strided(o_.type, alpha_.p, st_.p, n_, c, stride, off,
                        cx_.stream);
}

void Solver::cv_decision(double* out, int32_t stride, int32_t off,
                         const int32_t* fold, int32_t held, double b)
{
    launch_cv_decision(F_.p, n_, b, fold, held, out, stride, off, cx_.stream);
}

void Solver::get_alpha(double* out)
{
    HIP_TRY(hipMemcpyAsync(out, alpha_.p, (size_t)N_ * sizeof(double),
                           hipMemcpyDeviceToHost, cx_.stream));
    cx_.sync();
}

// ---- test hooks ----

void Solver::set_state(const double* alpha_h, const double* F_h)
{
    hipStream_t s = cx_.stream;
    HIP_TRY(hipMemcpyAsync(alpha_.p, alpha_h, (size_t)N_ * sizeof(double),
                           hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemcpyAsync(F_.p, F_h, (size_t)n_ * sizeof(double),
                           hipMemcpyHostToDevice, s));
    launch_state_from_alpha(o_.type, y_.p, alpha_.p, n_, o_.C, st_.p, s);
    HIP_TRY(hipMemsetAsync(ws_.p, 0, sizeof(WorkingSet), s));
    cx_.sync();
}

void Solver::warm_start(const double* alpha_h)
{
    hipStream_t s = cx_.stream;
    HIP_TRY(hipMemcpyAsync(alpha_.p, alpha_h, (size_t)N_ * sizeof(double),
                           hipMemcpyHostToDevice, s));
    launch_state_from_alpha(o_.type, y_.p, alpha_.p, n_, o_.C, st_.p, s);
    recompute_responses();
    HIP_TRY(hipMemsetAsync(ws_.p, 0, sizeof(WorkingSet), s));
    cx_.sync();
}

void Solver::get_state(double* alpha_h, double* F_h)
{
    if (alpha_h)
        HIP_TRY(hipMemcpyAsync(alpha_h, alpha_.p, (size_t)N_ * sizeof(double),
                               hipMemcpyDeviceToHost, cx_.stream));
    if (F_h)
        HIP_TRY(hipMemcpyAsync(F_h, F_.p, (size_t)n_ * sizeof(double),
                               hipMemcpyDeviceToHost, cx_.stream));
    cx_.sync();
}

void Solver::select(int32_t* B, int32_t* nB, double* m, double* M)
{
    launch_keys();
    launch_select_only();
    WorkingSet w;
    read_ws(w);
    *nB = w.nB;
    for (int i = 0; i < w.nB; ++i) B[i] = w.B[i];
    *m = w.m;
    *M = w.M;
}

void Solver::rows(const int32_t* samples, int32_t k, float* out_h)
{
    hipStream_t s = cx_.stream;
    WorkingSet w;
    read_ws(w);
    w.nS = k;
    for (int j = 0; j < k; ++j) {
        w.S[j] = samples[j];
        HIP_TRY(hipMemcpyAsync(&w.sS[j], f_.sq.p + samples[j], sizeof(float),
                               hipMemcpyDeviceToHost, s));
    }
    DevBuf<int32_t> sidx((size_t)k);
    HIP_TRY(hipMemcpyAsync(sidx.p, samples, (size_t)k * sizeof(int32_t),
                           hipMemcpyHostToDevice, s));
    gather_rows(f_, sidx.p, k, xS_.p, nullptr, s);
    const int nbc = k <= 16 ? 1 : (k <= 32 ? 2 : 4);
    if (f_.csr)
        launch_csr_compact(xS_.p, k, f_.ldp, 16 * nbc, csr_cols(nbc),
                           xsc_cols_.p, xsc_.p, s);
    cx_.sync();
    HIP_TRY(hipMemcpyAsync(ws_.p, &w, sizeof(WorkingSet),
                           hipMemcpyHostToDevice, s));
    cx_.sync();
    if (rows_out_.count < (size_t)(k * n_)) rows_out_.alloc((size_t)(k * n_));
    RowArgs a{};
    a.X = f_.x();
    a.rp = f_.rp.p;
    a.ci = f_.ci.p;
    a.cv = f_.cv.p;
    a.sq = f_.sq.p;
    a.F = F_.p;
    a.st = st_.p;
    a.z = y_.p;
    a.ws = ws_.p;
    a.xS = xS_.p;
    set_csr(a, nbc);
    a.rows_out = rows_out_.p;
    a.n = n_;
    a.ldp = f_.ldp;
    a.eps = o_.eps;
    a.kf = kf_;
    a.half = half_;
    a.tiles = tiles_;
    a.mode = RU_ROWS;
    a.nS_override = k;
    if (rows_lds_bytes(nbc, f_.ldp, tiles_, o_.type == SVM_EPS_SVR,
                       csr_cols(nbc)) >
        160 * 1024)
        throw Error{SVM_E_UNSUPPORTED, "too many features for the row tile"};
    launch_rows(a, nb_, nbc, o_.type == SVM_EPS_SVR, s);
    HIP_TRY(hipMemcpyAsync(out_h, rows_out_.p,
                           (size_t)(k * n_) * sizeof(float),
                           hipMemcpyDeviceToHost, s));
    cx_.sync();
}

void Solver::subproblem(const int32_t* B, int32_t nB, double inner_tol,
                        int32_t max_inner, double* alpha_B, int32_t* steps)
{
    hipStream_t s = cx_.stream;
    WorkingSet w;
    read_ws(w);
    w.nB = nB;
    for (int i = 0; i < nB; ++i) w.B[i] = B[i];
    w.done = 0;
    HIP_TRY(hipMemcpyAsync(ws_.p, &w, sizeof(WorkingSet),
                           hipMemcpyHostToDevice, s));
    cx_.sync();
    SelArgs a{};
    a.ws = ws_.p;
    a.alpha = alpha_.p;
    a.st = st_.p;
    a.F = F_.p;
    a.z = y_.p;
    a.X = f_.x();
    a.rp = f_.rp.p;
    a.ci = f_.ci.p;
    a.cv = f_.cv.p;
    a.sq = f_.sq.p;
    a.xS = xS_.p;
    set_csr(a, nB <= 16 ? 1 : (nB <= 32 ? 2 : 4));
    a.n = n_;
    a.ldp = f_.ldp;
    a.C = o_.C;
    a.eps = o_.eps;
    a.tol = o_.tol;
    a.kf = kf_;
    a.inner_ratio = o_.inner_ratio;
    a.inner_tol_override = inner_tol;
    a.max_inner = max_inner;
    a.max_iter = o_.max_iter;
    a.half = half_;
    a.group_rows = (kRowThreads / 64) * 16 * tiles_;  // most rows of a block
    a.mode = SS_GIVEN_B | SS_SOLVE | SS_NO_WRITE;
    int nbc = nB <= 16 ? 1 : (nB <= 32 ? 2 : 4);
    launch_select(a, nbc, o_.type == SVM_EPS_SVR, s);
    read_ws(w);
    for (int i = 0; i < nB; ++i) alpha_B[i] = w.alphaB[i];
    *steps = w.steps;
}

void Solver::apply(const int32_t* B, int32_t nB, const double* alpha_B)
{
    hipStream_t s = cx_.stream;
    WorkingSet w;
    read_ws(w);
    w.nB = nB;
    w.done = 0;
    for (int i = 0; i < nB; ++i) {
        w.B[i] = B[i];
        w.alphaB[i] = alpha_B[i];
    }
    HIP_TRY(hipMemcpyAsync(ws_.p, &w, sizeof(WorkingSet),
                           hipMemcpyHostToDevice, s));
    cx_.sync();
    SelArgs a{};
    a.ws = ws_.p;
    a.alpha = alpha_.p;
    a.st = st_.p;
    a.F = F_.p;
    a.z = y_.p;
    a.X = f_.x();
    a.rp = f_.rp.p;
    a.ci = f_.ci.p;
    a.cv = f_.cv.p;
    a.sq = f_.sq.p;
    a.xS = xS_.p;
    set_csr(a, nB <= 16 ? 1 : (nB <= 32 ? 2 : 4));
    a.n = n_;
    a.ldp = f_.ldp;
    a.C = o_.C;
    a.eps = o_.eps;
    a.tol = o_.tol;
    a.kf = kf_;
    a.inner_ratio = o_.inner_ratio;
    a.inner_tol_override = 0.0;
    a.max_inner = 0;
    a.max_iter = o_.max_iter;
    a.half = half_;
    a.group_rows = (kRowThreads / 64) * 16 * tiles_;  // most rows of a block
    a.mode = SS_GIVEN_B | SS_SOLVE | SS_SET_ALPHA;
    int nbc = nB <= 16 ? 1 : (nB <= 32 ? 2 : 4);
    launch_select(a, nbc, o_.type == SVM_EPS_SVR, s);
    RowArgs r{};
    r.X = f_.x();
    r.rp = f_.rp.p;
    r.ci = f_.ci.p;
    r.cv = f_.cv.p;
    r.sq = f_.sq.p;
    r.F = F_.p;
    r.st = st_.p;
    r.z = y_.p;
    r.ws = ws_.p;
    r.xS = xS_.p;
    set_csr(r, nbc);
    r.cand_key = ckey_.p;
    r.cand_idx = cidx_.p;
    r.n = n_;
    r.ldp = f_.ldp;
    r.eps = o_.eps;
    r.kf = kf_;
    r.half = half_;
    r.tiles = tiles_;
    r.mode = RU_UPDATE;
    r.nS_override = -1;
    if (rows_lds_bytes(nbc, f_.ldp, tiles_, o_.type == SVM_EPS_SVR,
                       csr_cols(nbc)) >
        160 * 1024)
        throw Error{SVM_E_UNSUPPORTED, "too many features for the row tile"};
    launch_rows(r, nb_, nbc, o_.type == SVM_EPS_SVR, s);
    cx_.sync();
}

void Solver::finish_state(int max_passes, SolveResult& r)
{
    hipEvent_t t0 = start(false);
    finish(r, true, t0, max_passes);
}

void Solver::iterate(int64_t k, int64_t* iters, double* gap)
{
    launch_keys();
    for (int64_t i = 0; i < k; ++i) {
        launch_solve(SS_SOLVE | SS_CHECK_DONE);
        launch_hot_rows();
    }
    WorkingSet w;
    read_ws(w);
    *iters = w.iter;
    *gap = w.gap;
}

// ---------------------------------------------------------------------------
// model
// ---------------------------------------------------------------------------

void build_model(svm_model& m, Context& cx, const Features& f,
                 const double* coef_dev, int32_t n_out)
{
    Range rg("svm model (support vectors)");
    hipStream_t s = cx.stream;
    const int64_t n = f.n;
    DevBuf<int32_t> blk((size_t)compact_blocks(n)), idx((size_t)n);
    DevBuf<double> cc((size_t)(n * n_out));
    DevBuf<int64_t> cnt(1);
    launch_compact(coef_dev, n, n_out, blk.p, idx.p, cc.p, cnt.p, s);
    int64_t nsv = 0;
    HIP_TRY(hipMemcpyAsync(&nsv, cnt.p, sizeof(int64_t),
                           hipMemcpyDeviceToHost, s));
    cx.sync();
    m.n_sv = nsv;
    m.SV.alloc((size_t)(nsv * f.ldp));
    m.sqsv.alloc((size_t)nsv);
    m.coef_dev.alloc((size_t)(nsv * n_out));
    m.b_dev.alloc((size_t)n_out);
    gather_rows(f, idx.p, nsv, m.SV.p, m.sqsv.p, s);
    m.ch_cap = sparse_chunk_cap(f);
    if (m.ch_cap > 0)
        build_sv_chunks(f, idx.p, nsv, m.ch_cap, m.ch_ncol, m.ch_cols,
                        m.ch_tab, nullptr, s);
    // (the training rows stand in for the query rows in the path rule)
    if (f.csr)
        build_fact(m.fc, f, idx.p, nsv, cc.p, n_out, m.kf, cx, m.sqsv.p, &f);
    m.sv_idx.resize((size_t)nsv);
    m.coef.resize((size_t)(nsv * n_out));
    if (nsv > 0) {
        HIP_TRY(hipMemcpyAsync(m.coef_dev.p, cc.p,
                               (size_t)(nsv * n_out) * sizeof(double),
                               hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipMemcpyAsync(m.sv_idx.data(), idx.p,
                               (size_t)nsv * sizeof(int32_t),
                               hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(m.coef.data(), cc.p,
                               (size_t)(nsv * n_out) * sizeof(double),
                               hipMemcpyDeviceToHost, s));
    }
    HIP_TRY(hipMemcpyAsync(m.b_dev.p, m.b.data(),
                           (size_t)n_out * sizeof(double),
                           hipMemcpyHostToDevice, s));
    cx.sync();
}

void scale_fit(const Features& f, Context& cx, DevBuf<double>& mu,
               DevBuf<double>& sd)
{
    if (f.csr)
        throw Error{SVM_E_UNSUPPORTED,
                    "scaling needs dense features (centring a sparse matrix "
                    "would fill it)"};
    mu.alloc((size_t)f.d);
    sd.alloc((size_t)f.d);
    DevBuf<double> part((size_t)col_stats_partials(f.n, f.d));
    launch_col_stats(f.x(), f.n, f.ldp, f.d, part.p, mu.p, sd.p, cx.stream);
    cx.sync();
}

void scale_apply(Features& f, Context& cx, const double* mu, const double* sd)
{
    if (f.csr)
        throw Error{SVM_E_UNSUPPORTED,
                    "a model trained on scaled data predicts dense rows only"};
    if (f.Xb) {  // scaled in place: the caller's rows are copied first
        f.X.alloc((size_t)(f.n * f.ldp));
        HIP_TRY(hipMemcpyAsync(f.X.p, f.Xb, f.X.bytes(),
                               hipMemcpyDeviceToDevice, cx.stream));
        f.Xb = nullptr;
    }
    launch_scale_apply(f.X.p, f.n, f.ldp, f.d, mu, sd, cx.stream);
    DevBuf<int32_t> bad(1);
    HIP_TRY(hipMemsetAsync(bad.p, 0, sizeof(int32_t), cx.stream));
    launch_norms(f.X.p, f.n, f.ldp, f.sq.p, bad.p, cx.stream);
    int32_t hb = 0;
    HIP_TRY(hipMemcpyAsync(&hb, bad.p, sizeof(int32_t), hipMemcpyDeviceToHost,
                           cx.stream));
    cx.sync();
    if (hb)
        throw Error{SVM_E_INVALID,
                    "a scaled value is not finite (or its square overflows "
                    "fp32)"};
}

void scale_targets(float* y_dev, int64_t n, Context& cx, double* mu,
                   double* sd)
{
    DevBuf<double> m(1), s(1), part((size_t)col_stats_partials(n, 1));
    launch_col_stats(y_dev, n, 1, 1, part.p, m.p, s.p, cx.stream);
    launch_scale_apply(y_dev, n, 1, 1, m.p, s.p, cx.stream);
    HIP_TRY(hipMemcpyAsync(mu, m.p, sizeof(double), hipMemcpyDeviceToHost,
                           cx.stream));
    HIP_TRY(hipMemcpyAsync(sd, s.p, sizeof(double), hipMemcpyDeviceToHost,
                           cx.stream));
    cx.sync();
    if (!(*sd > 0.0)) *sd = 0.0;  // constant targets: left as they are
}

void predict_device(const svm_model& mdl, Context& cx, Features& t,
                    double* out)
{
    if (mdl.scaled) scale_apply(t, cx, mdl.x_mu.p, mdl.x_sd.p);
    PredictArgs a{};
    a.SV = mdl.SV.p;
    a.sqsv = mdl.sqsv.p;
    a.nsv = mdl.n_sv;
    a.coef = mdl.coef_dev.p;
    a.b = mdl.b_dev.p;
    a.n_out = mdl.n_out;
    a.sv_train_idx = nullptr;
    a.self_match = 0;
    a.out = out;
    a.kf = mdl.kf;
    if (mdl.ch_cap > 0) {
        a.ch_ncol = mdl.ch_ncol.p;
        a.ch_cols = mdl.ch_cols.p;
        a.ch_tab = mdl.ch_tab.p;
        a.ch_cap = mdl.ch_cap;
    }
    predict_rows(a, t, cx.stream, mdl.fc.ok ? &mdl.fc : nullptr);
    if (mdl.scaled && mdl.type == SVM_EPS_SVR && mdl.y_sd > 0.0)
        launch_affine(out, t.n * mdl.n_out, mdl.y_sd, mdl.y_mu, cx.stream);
}

int sparse_chunk_cap(const Features& f)
{
    if (!f.csr || f.n <= 0 || f.nnz > 32 * f.n) return 0;
    const int64_t cap =
        std::min<int64_t>(f.ldp, 16 * std::max<int64_t>(1, f.maxnz));
    return predict_sparse_fits(f.ldp, (int)cap) ? (int)cap : 0;
}

void build_sv_chunks(const Features& f, const int32_t* idx, int64_t nsv,
                     int cap, DevBuf<int32_t>& ncol, DevBuf<int32_t>& cols,
                     DevBuf<float>& tab, float* sq_out, hipStream_t s)
{
    const int64_t nch = (nsv + 15) / 16;
    if (ncol.count < (size_t)nch) ncol.alloc((size_t)nch);
    if (cols.count < (size_t)(nch * cap)) cols.alloc((size_t)(nch * cap));
    if (tab.count < (size_t)(nch * cap * 16))
        tab.alloc((size_t)(nch * cap * 16));
    ChunkArgs c{};
    c.rp = f.rp.p;
    c.ci = f.ci.p;
    c.cv = f.cv.p;
    c.sq = f.sq.p;
    c.idx = idx;
    c.nsv = nsv;
    c.ldp = f.ldp;
    c.cap = cap;
    c.ncol = ncol.p;
    c.cols = cols.p;
    c.tab = tab.p;
    c.sq_out = sq_out;
    launch_sv_chunks(c, s);
}

void gather_rows(const Features& f, const int32_t* idx, int64_t k, float* out,
                 float* sq_out, hipStream_t s)
{
    if (f.csr)
        launch_gather_rows_csr(f.rp.p, f.ci.p, f.cv.p, f.sq.p, f.ldp, idx, 0,
                               k, out, sq_out, s);
    else
        launch_gather_rows(f.x(), f.sq.p, f.ldp, idx, k, out, sq_out, s);
}

// SVM_SPARSE_PATH: 1 = "table" (the factored path is not built), 2 =
// "factor" (taken whenever built), 0 = unset (chosen by the rule)
static int sparse_path_switch()
{
    const char* e = getenv("SVM_SPARSE_PATH");  // developer switch
    if (!e) return 0;
    const std::string v(e);
    return v == "table" ? 1 : v == "factor" ? 2 : 0;
}

static bool use_fact(const FactSV* fc, const Features& t)
{
    if (!fc || !fc->ok || t.n <= 0) return false;
    if (sparse_path_switch() == 2) return true;
    const double shared = (double)t.nnz / (double)t.n * fc->sv_nnz /
                          (double)std::max<int64_t>(fc->d, 1);
    return shared < kFcMatchMax;
}

void build_fact(FactSV& fc, const Features& f, const int32_t* idx,
                int64_t nsv, const double* coef, int32_t n_out,
                const KernelFn& kf, Context& cx, float* sqsv,
                const Features* query)
{
    fc.ok = false;
    if (!f.csr || nsv <= 0 || n_out < 1 || n_out > 4) return;
    if (sparse_path_switch() == 1) return;
    hipStream_t s = cx.stream;
    DevBuf<int32_t> nzd((size_t)nsv);
    launch_fc_nnz(f.rp.p, f.sq.p, idx, nsv, nzd.p, sqsv, s);
    std::vector<int32_t> nz((size_t)nsv);
    HIP_TRY(hipMemcpyAsync(nz.data(), nzd.p, (size_t)nsv * sizeof(int32_t),
                           hipMemcpyDeviceToHost, s));
    cx.sync();
    // chunks of consecutive support rows: at most kFcSvMax rows and
    // kFcEntMax nonzeros each
    std::vector<int32_t> sv0{0};
    std::vector<int64_t> e0{0};
    int64_t tot = 0, ce = 0;
    int32_t cs = 0;
    for (int64_t j = 0; j < nsv; ++j) {
        const int64_t z = nz[(size_t)j];
        if (z > kFcEntMax) return;
        if (cs == kFcSvMax || ce + z > kFcEntMax) {
            sv0.push_back((int32_t)j);
            e0.push_back(e0.back() + ce);
            ce = 0;
            cs = 0;
        }
        ce += z;
        ++cs;
        tot += z;
    }
    sv0.push_back((int32_t)nsv);
    e0.push_back(e0.back() + ce);
    // the factored path pays per entry that a query row meets; rows that
    // hold a large share of the columns are cheaper through the table path
    if ((double)tot > 0.1 * (double)f.d * (double)nsv) return;
    fc.sv_nnz = (double)tot / (double)nsv;
    fc.d = f.d;
    fc.ok = true;  // (for the rule only)
    const bool take = !query || use_fact(&fc, *query);
    fc.ok = false;
    if (!take) return;
    const int32_t nch = (int32_t)(sv0.size() - 1);
    const int64_t ldpm = (f.ldp + 3) & ~(int64_t)3;
    if ((size_t)nch * (size_t)ldpm * 4 > fc_map_bytes_limit()) return;
    fc.sv0.alloc((size_t)nch + 1);
    fc.e0.alloc((size_t)nch + 1);
    fc.map.alloc((size_t)nch * (size_t)ldpm);
    fc.ent.alloc((size_t)std::max<int64_t>(tot, 1));
    fc.w.alloc((size_t)(nsv * n_out));
    fc.wf.alloc((size_t)nsv);
    fc.c0.alloc((size_t)n_out);
    HIP_TRY(hipMemcpyAsync(fc.sv0.p, sv0.data(), sv0.size() * sizeof(int32_t),
                           hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemcpyAsync(fc.e0.p, e0.data(), e0.size() * sizeof(int64_t),
                           hipMemcpyHostToDevice, s));
    FactBuildArgs b{};
    b.rp = f.rp.p;
    b.ci = f.ci.p;
    b.cv = f.cv.p;
    b.idx = idx;
    b.nch = nch;
    b.ldpm = (int32_t)ldpm;
    b.ch_sv0 = fc.sv0.p;
    b.ch_e0 = fc.e0.p;
    b.map = fc.map.p;
    b.ent = fc.ent.p;
    launch_fc_build(b, s);
    DevBuf<uint32_t> gs(1);
    HIP_TRY(hipMemsetAsync(gs.p, 0, sizeof(uint32_t), s));
    launch_fc_weights(coef, sqsv, nsv, n_out, kf, fc.w.p, fc.wf.p, fc.c0.p,
                      gs.p, s);
    uint32_t gsh = 0;
    HIP_TRY(hipMemcpyAsync(&gsh, gs.p, sizeof(uint32_t),
                           hipMemcpyDeviceToHost, s));
    cx.sync();
    float gmax = 0.0f;
    std::memcpy(&gmax, &gsh, sizeof(float));
    fc.nch = nch;
    fc.ldpm = (int32_t)ldpm;
    fc.n_out = n_out;
    fc.fast = gmax <= kFcSafe ? 1 : 0;
    fc.ok = true;
}

void predict_rows(PredictArgs a, const Features& t, hipStream_t s,
                  const FactSV* fc)
{
    a.ldp = t.ldp;
    a.nrange = predict_ranges(a.nsv);
    if (!t.csr) {
        a.Xt = t.x();
        a.sqt = t.sq.p;
        a.m = t.n;
        a.row_base = 0;
        DevBuf<double> part;
        if (a.nrange > 1 && t.n > 0) {
            part.alloc((size_t)predict_part_doubles(a.nsv, t.n, a.n_out));
            a.part = part.p;
        }
        launch_predict(a, s);
        // the partial sums are freed when the stream has used them
        if (part.p) HIP_TRY(hipStreamSynchronize(s));
        return;
    }
    if (t.nnz <= 32 * t.n && use_fact(fc, t)) {
        FactArgs f{};
        f.rpt = t.rp.p;
        f.cit = t.ci.p;
        f.cvt = t.cv.p;
        f.sqt = t.sq.p;
        f.m = t.n;
        f.row_base = 0;
        f.self_sv = a.self_sv;
        f.nch = fc->nch;
        f.ldpm = fc->ldpm;
        f.ch_sv0 = fc->sv0.p;
        f.ch_e0 = fc->e0.p;
        f.map = fc->map.p;
        f.ent = fc->ent.p;
        f.sqsv = a.sqsv;
        f.coef = a.coef;
        f.w = fc->w.p;
        f.wf = fc->wf.p;
        f.c0 = fc->c0.p;
        f.b = a.b;
        f.n_out = a.n_out;
        f.fast = fc->fast;
        f.out = a.out;
        f.kf = a.kf;
        if (fc->ldpm < ((t.ldp + 3) & ~(int64_t)3))
            throw Error{SVM_E_INTERNAL, "query rows wider than the model"};
        launch_predict_fact(f, s);
        return;
    }
    if (a.ch_tab && t.nnz <= 32 * t.n) {
        a.rpt = t.rp.p;
        a.cit = t.ci.p;
        a.cvt = t.cv.p;
        a.sqt = t.sq.p;
        a.m = t.n;
        a.row_base = 0;
        launch_predict_sparse(a, s);
        return;
    }
    if (!a.SV)
        throw Error{SVM_E_INTERNAL, "no dense support rows for this input"};
    // CSR rows: dense chunks of up to 256 MB
    const int64_t row_bytes = t.ldp * (int64_t)sizeof(float);
    int64_t chunk = std::max<int64_t>(64, ((int64_t)256 << 20) / row_bytes);
    chunk = std::min<int64_t>(chunk, t.n);
    if (chunk <= 0) return;
    DevBuf<float> buf((size_t)(chunk * t.ldp));
    DevBuf<double> part;
    if (a.nrange > 1) {
        part.alloc((size_t)predict_part_doubles(a.nsv, chunk, a.n_out));
        a.part = part.p;
    }
    double* out0 = a.out;
    for (int64_t r0 = 0; r0 < t.n; r0 += chunk) {
        const int64_t k = std::min<int64_t>(chunk, t.n - r0);
        launch_gather_rows_csr(t.rp.p, t.ci.p, t.cv.p, t.sq.p, t.ldp, nullptr,
                               r0, k, buf.p, nullptr, s);
        a.Xt = buf.p;
        a.sqt = t.sq.p + r0;
        a.m = k;
        a.row_base = r0;
        a.out = out0 + r0 * a.n_out;
        launch_predict(a, s);
    }
    // the chunk buffers are freed when the stream has used them
    HIP_TRY(hipStreamSynchronize(s));
}

}  // namespace msvm
