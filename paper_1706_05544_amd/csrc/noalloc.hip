// Decision function without device allocation, for callers that cannot
// allocate (code under HIP graph capture, tight serving loops).
//
// svm_predict stages the query rows in buffers it allocates (a padded copy
// of X, their norms, the partial sums over ranges of support rows, the
// decision values).  This variant stages what it needs in one static
// per-device array instead and writes the decision values straight to the
// caller's buffer; the kernels are the same (k_pad_copy, k_scale_apply,
// k_norms, the decision kernels), so the values are bitwise those of
// svm_predict.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "solver.hpp"

namespace msvm {

// The staging memory.  Each GPU the library runs on holds its own copy
// until the process ends; every call on a GPU shares it, so calls that
// overlap on one GPU race.  Nothing in it is read before the call writes
// it (norms and padded rows are written whole, chunk by chunk, on the
// call's stream before they are read).
constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr size_t kScratchHead = 256;  // the norms kernel's (unread) flag
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch[kMaxDevices] = {};

// Device address of the staging array on device dev (current): looked up
// once per device.  The array's name is not a device address in host code.
static unsigned char* scratch_of(int dev)
{
    if (dev < 0 || dev >= kMaxDevices)
        throw Error{SVM_E_DEVICE, "device ordinal out of range"};
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) throw Error{SVM_E_DEVICE, "no address for the staging array"};
        g_scratch[dev] = p;
    }
    return static_cast<unsigned char*>(g_scratch[dev]);
}

bool noalloc_needs_copy(const svm_model& mdl, const float* X, int64_t ld)
{
    // k_predict reads rows of ldp floats (aligned float4 pieces, the
    // columns past d zero): the caller's rows serve as they are when they
    // have that layout and the model takes them unscaled
    return mdl.scaled || ld != mdl.ldp || mdl.ldp != mdl.d ||
           ((uintptr_t)X & 15) != 0;
}

int64_t noalloc_rows_per_chunk(const svm_model& mdl, const float* X,
                               int64_t ld)
{
    const bool copy = noalloc_needs_copy(mdl, X, ld);
    // a staged row, its norm and its partial sums over the support ranges
    const int64_t row = (copy ? mdl.ldp * 4 : 0) + 4 +
                        predict_part_doubles(mdl.n_sv, 1, mdl.n_out) * 8;
    int64_t rows = (int64_t)(kScratchBytes - kScratchHead - 512) / row;
    if (rows >= 64) rows &= ~(int64_t)63;
    return rows;
}

size_t noalloc_scratch_bytes() { return kScratchBytes; }

void predict_noalloc(const svm_model& mdl, const float* X, int64_t m,
                     int64_t ld, double* out, hipStream_t s)
{
    if (m <= 0) return;
    unsigned char* base = scratch_of(mdl.device);
    const int64_t d = mdl.d, ldp = mdl.ldp;
    const bool copy = noalloc_needs_copy(mdl, X, ld);
    const int64_t chunk = noalloc_rows_per_chunk(mdl, X, ld);
    if (chunk < 1)
        throw Error{SVM_E_UNSUPPORTED,
                    "a row of X does not fit the 32 MiB staging array"};
    int32_t* bad = reinterpret_cast<int32_t*>(base);  // never read
    float* sq = reinterpret_cast<float*>(base + kScratchHead);
    const size_t sq_bytes = ((size_t)chunk * 4 + 255) & ~(size_t)255;
    const size_t part_bytes =
        ((size_t)predict_part_doubles(mdl.n_sv, chunk, mdl.n_out) * 8 + 255) &
        ~(size_t)255;
    double* part =
        reinterpret_cast<double*>(base + kScratchHead + sq_bytes);
    float* rows = reinterpret_cast<float*>(base + kScratchHead + sq_bytes +
                                           part_bytes);
    if (kScratchHead + sq_bytes + part_bytes +
            (copy ? (size_t)chunk * ldp * 4 : 0) >
        kScratchBytes)
        throw Error{SVM_E_INTERNAL, "staging layout"};

    PredictArgs a{};
    a.SV = mdl.SV.p;
    a.sqsv = mdl.sqsv.p;
    a.nsv = mdl.n_sv;
    a.coef = mdl.coef_dev.p;
    a.b = mdl.b_dev.p;
    a.n_out = mdl.n_out;
    a.sv_train_idx = nullptr;
    a.self_match = 0;
    a.kf = mdl.kf;
    a.ldp = ldp;
    a.nrange = predict_ranges(mdl.n_sv);
    a.part = a.nrange > 1 ? part : nullptr;
    for (int64_t r0 = 0; r0 < m; r0 += chunk) {
        const int64_t k = m - r0 < chunk ? m - r0 : chunk;
        const float* src = X + r0 * ld;
        const float* Xt = src;
        if (copy) {
            launch_pad_copy(src, ld, k, d, rows, ldp, s);
            if (mdl.scaled)
                launch_scale_apply(rows, k, ldp, d, mdl.x_mu.p, mdl.x_sd.p,
                                   s);
            Xt = rows;
        }
        launch_norms(Xt, k, ldp, sq, bad, s);
        a.Xt = Xt;
        a.sqt = sq;
        a.m = k;
        a.row_base = r0;
        a.out = out + r0 * mdl.n_out;
        launch_predict(a, s);
    }
    if (mdl.scaled && mdl.type == SVM_EPS_SVR && mdl.y_sd > 0.0)
        launch_affine(out, m * mdl.n_out, mdl.y_sd, mdl.y_mu, s);
    HIP_TRY(hipPeekAtLastError());
}

}  // namespace msvm
