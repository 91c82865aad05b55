// HIP kernels of the feature store, the state set-up and the model
// extraction of the working-set dual solve (gfx950).
#include <hip/hip_ext.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

#include "common.hpp"
#include "device.hpp"

namespace msvm {

// ---------------------------------------------------------------------------
// feature store
// ---------------------------------------------------------------------------

__global__ void k_pad_copy(const float* src, int64_t ld, int64_t n, int64_t d,
                           float* dst, int64_t ldp)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t total = n * ldp;
    for (; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = i / ldp, c = i - r * ldp;
        dst[i] = c < d ? src[r * ld + c] : 0.0f;
    }
}

void launch_pad_copy(const float* src, int64_t ld, int64_t n, int64_t d,
                     float* dst, int64_t ldp, hipStream_t s)
{
    if (n <= 0) return;
    int64_t blocks = (n * ldp + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    k_pad_copy<<<(unsigned)blocks, 256, 0, s>>>(src, ld, n, d, dst, ldp);
}

// Squared norms: 16 lanes per row, fp64 partial sums, fixed reduction order.
// A non-finite row (NaN, Inf, or a square that overflows) sets *bad.
__global__ void k_norms(const float* X, int64_t n, int64_t ldp, float* sq,
                        int32_t* bad)
{
    int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
    int sub = threadIdx.x & 15;
    if (row >= n) return;
    const float* x = X + row * ldp;
    double acc = 0.0;
    for (int64_t k = sub; k < ldp; k += 16) {
        double v = (double)x[k];
        acc += v * v;
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 16);
    if (sub == 0) {
        float f = (float)acc;
        sq[row] = f;
        if (!isfinite(f)) atomicOr(bad, 1);
    }
}

void launch_norms(const float* X, int64_t n, int64_t ldp, float* sq,
                  int32_t* bad, hipStream_t s)
{
    if (n <= 0) return;
    int64_t blocks = (n * 16 + 255) / 256;
    k_norms<<<(unsigned)blocks, 256, 0, s>>>(X, n, ldp, sq, bad);
}

__global__ void k_check_finite(const float* v, int64_t n, int32_t* bad)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n && !isfinite(v[i])) atomicOr(bad, 1);
}

void launch_check_finite(const float* v, int64_t n, int32_t* bad,
                         hipStream_t s)
{
    if (n <= 0) return;
    k_check_finite<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(v, n, bad);
}

// Initial state bytes for alpha = 0.  C-SVC: label +1 -> I_up, -1 -> I_low;
// a label other than +-1 sets bit 0 of *bad, each class seen sets bit 1
// (+1) or bit 2 (-1).  eps-SVR: positive copies in I_up, negative in I_low.
// State bytes at alpha = 0.  A row held out of the training (fold[i] ==
// held, cross-validation) keeps only its label bit: its variables stay at
// 0 outside I_up and I_low, so no working set takes them and the solve is
// the dual restricted to the other rows.  bad: 1 an invalid label or
// target, 2 / 4 a positive / negative training row seen.
__global__ __launch_bounds__(256) void k_init_state(int32_t type,
                                                   const float* y, int64_t n,
                                                   const int32_t* fold,
                                                   int32_t held, uint8_t* st,
                                                   int32_t* bad)
{
    __shared__ int wflags[4];
    int flags = 0;  // 1 bad value, 2 a training +1, 4 a training -1
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * 256) {
        const bool train = !fold || fold[i] != held;
        const uint8_t up = train ? ST_UP : 0, low = train ? ST_LOW : 0;
        if (type == SVM_C_SVC) {
            const float v = y[i];
            if (v == 1.0f) {
                st[i] = ST_YPOS | up;
                flags |= train ? 2 : 0;
            } else if (v == -1.0f) {
                st[i] = low;
                flags |= train ? 4 : 0;
            } else {
                st[i] = 0;
                flags |= 1;
            }
        } else {
            st[i] = ST_YPOS | up;
            st[n + i] = low;
            flags |= isfinite(y[i]) ? 0 : 1;
        }
    }
    // one atomic per block (atomics on one address serialise)
    const int w = (__ballot(flags & 1) ? 1 : 0) | (__ballot(flags & 2) ? 2 : 0) |
                  (__ballot(flags & 4) ? 4 : 0);
    if ((threadIdx.x & 63) == 0) wflags[threadIdx.x >> 6] = w;
    __syncthreads();
    if (threadIdx.x == 0) {
        const int f = wflags[0] | wflags[1] | wflags[2] | wflags[3];
        if (f) atomicOr(bad, f);
    }
}

void launch_init_state(int32_t type, const float* y, int64_t n,
                       const int32_t* fold, int32_t held, uint8_t* st,
                       int32_t* bad, hipStream_t s)
{
    const int64_t nb = std::max<int64_t>(
        1, std::min<int64_t>(512, (n + 255) / 256));
    k_init_state<<<(unsigned)nb, 256, 0, s>>>(type, y, n, fold, held, st,
                                              bad);
}

// Decision values of the rows held out of a training: out[i * stride +
// off] = F_i + b for fold[i] == held (F_i = sum_j c_j K(x_j, x_i) over the
// trained coefficients, recomputed from alpha at the end of the solve).
__global__ void k_cv_decision(const double* F, int64_t n, double b,
                              const int32_t* fold, int32_t held, double* out,
                              int32_t stride, int32_t off)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n && fold[i] == held) out[i * stride + off] = F[i] + b;
}

void launch_cv_decision(const double* F, int64_t n, double b,
                        const int32_t* fold, int32_t held, double* out,
                        int32_t stride, int32_t off, hipStream_t s)
{
    if (n > 0)
        k_cv_decision<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(
            F, n, b, fold, held, out, stride, off);
}

// ---------------------------------------------------------------------------
// scaling (standardisation of the features and, for eps-SVR, the targets)
// ---------------------------------------------------------------------------

constexpr int kStatRows = 256;  // rows of one partial sum

// part[b * d + c] = sum over rows b * kStatRows .. of x_rc (mu == nullptr)
// or of (x_rc - mu_c)^2, in fp64 and row order.
__global__ void k_col_partial(const float* X, int64_t n, int64_t ld,
                              int64_t d, const double* mu, double* part)
{
    const int64_t r0 = (int64_t)blockIdx.x * kStatRows;
    const int64_t r1 = min(r0 + kStatRows, n);
    for (int64_t c = threadIdx.x; c < d; c += blockDim.x) {
        const double m = mu ? mu[c] : 0.0;
        double acc = 0.0;
        for (int64_t r = r0; r < r1; ++r) {
            const double v = (double)X[r * ld + c];
            if (mu) {
                const double e = v - m;
                acc += e * e;
            } else {
                acc += v;
            }
        }
        part[(int64_t)blockIdx.x * d + c] = acc;
    }
}

// mode 0: mu_c = (sum of the partials) / n; mode 1: sd_c = sqrt(sum / (n-1))
// (the partials summed in block order)
__global__ void k_col_finish(const double* part, int64_t nblk, int64_t d,
                             int64_t n, int32_t mode, double* out)
{
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= d) return;
    double s = 0.0;
    for (int64_t b = 0; b < nblk; ++b) s += part[b * d + c];
    out[c] = mode == 0 ? s / (double)n : sqrt(s / (double)(n - 1));
}

void launch_col_stats(const float* X, int64_t n, int64_t ld, int64_t d,
                      double* part, double* mu, double* sd, hipStream_t s)
{
    const int64_t nblk = (n + kStatRows - 1) / kStatRows;
    const unsigned g = (unsigned)((d + 255) / 256);
    k_col_partial<<<(unsigned)nblk, 256, 0, s>>>(X, n, ld, d, nullptr, part);
    k_col_finish<<<g, 256, 0, s>>>(part, nblk, d, n, 0, mu);
    k_col_partial<<<(unsigned)nblk, 256, 0, s>>>(X, n, ld, d, mu, part);
    k_col_finish<<<g, 256, 0, s>>>(part, nblk, d, n, 1, sd);
}

int64_t col_stats_partials(int64_t n, int64_t d)
{
    return (n + kStatRows - 1) / kStatRows * d;
}

// x_rc = (x_rc - mu_c) / sd_c in fp64, rounded once to fp32; a constant
// column (sd_c = 0) is left as it is.
__global__ void k_scale_apply(float* X, int64_t n, int64_t ld, int64_t d,
                              const double* mu, const double* sd)
{
    const int64_t total = n * d;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = e / d, c = e - r * d;
        const double s = sd[c];
        if (s > 0.0) {
            float* x = X + r * ld + c;
            *x = (float)(((double)*x - mu[c]) / s);
        }
    }
}

void launch_scale_apply(float* X, int64_t n, int64_t ld, int64_t d,
                        const double* mu, const double* sd, hipStream_t s)
{
    const int64_t total = n * d;
    if (total <= 0) return;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
    k_scale_apply<<<(unsigned)blocks, 256, 0, s>>>(X, n, ld, d, mu, sd);
}

// D = D * a + b (the decision values of a model trained on scaled targets,
// back in the units of the targets)
__global__ void k_affine(double* D, int64_t m, double a, double b)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < m) D[i] = fma(D[i], a, b);
}

void launch_affine(double* D, int64_t m, double a, double b, hipStream_t s)
{
    if (m > 0)
        k_affine<<<(unsigned)((m + 255) / 256), 256, 0, s>>>(D, m, a, b);
}

// Quality of decision values against the truth (cross-validation):
// out[0] correct labels (C-SVC: sign, D >= 0 is +1, against y; one-vs-rest:
// argmax, ties to the lowest class, against labels), out[1] sum (D - y)^2,
// out[2..6] sum D, sum y, sum D^2, sum y^2, sum D y.  One block, fp64,
// a fixed reduction order.
__global__ __launch_bounds__(1024) void k_metrics(int32_t type, int32_t n_out,
                                                  const double* D,
                                                  const float* y,
                                                  const int32_t* labels,
                                                  int64_t n, double* out)
{
    __shared__ double sh[7][1024];
    const int tid = threadIdx.x;
    double acc[7] = {0, 0, 0, 0, 0, 0, 0};
    for (int64_t i = tid; i < n; i += 1024) {
        if (n_out > 1) {
            int best = 0;
            double bv = D[i * n_out];
            for (int o = 1; o < n_out; ++o)
                if (D[i * n_out + o] > bv) {
                    bv = D[i * n_out + o];
                    best = o;
                }
            acc[0] += best == labels[i] ? 1.0 : 0.0;
            continue;
        }
        const double d = D[i], t = (double)y[i];
        if (type == SVM_C_SVC) acc[0] += (d >= 0.0 ? 1.0 : -1.0) == t ? 1.0 : 0.0;
        acc[1] += (d - t) * (d - t);
        acc[2] += d;
        acc[3] += t;
        acc[4] += d * d;
        acc[5] += t * t;
        acc[6] += d * t;
    }
    for (int k = 0; k < 7; ++k) sh[k][tid] = acc[k];
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (tid < w)
            for (int k = 0; k < 7; ++k) sh[k][tid] += sh[k][tid + w];
        __syncthreads();
    }
    if (tid < 7) out[tid] = sh[tid][0];
}

void launch_metrics(int32_t type, int32_t n_out, const double* D,
                    const float* y, const int32_t* labels, int64_t n,
                    double* out, hipStream_t s)
{
    k_metrics<<<1, 1024, 0, s>>>(type, n_out, D, y, labels, n, out);
}

__global__ void k_ovr_labels(const int32_t* labels, int64_t n, int32_t cls,
                             float* y)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) y[i] = labels[i] == cls ? 1.0f : -1.0f;
}

void launch_ovr_labels(const int32_t* labels, int64_t n, int32_t cls,
                       float* y, hipStream_t s)
{
    k_ovr_labels<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(labels, n, cls,
                                                             y);
}

__global__ void k_check_labels(const int32_t* labels, int64_t n,
                               int32_t ncls, int32_t* bad)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n && (labels[i] < 0 || labels[i] >= ncls)) atomicOr(bad, 1);
}

void launch_check_labels(const int32_t* labels, int64_t n, int32_t ncls,
                         int32_t* bad, hipStream_t s)
{
    k_check_labels<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(labels, n,
                                                               ncls, bad);
}

__global__ void k_fill_i32(int32_t* p, int32_t v, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

void launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s)
{
    if (n <= 0) return;
    k_fill_i32<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(p, v, n);
}

bool raise_dynamic_lds(const void* kernel, size_t lds)
{
    static std::mutex mu;
    static std::map<const void*, size_t> lim;
    std::lock_guard<std::mutex> g(mu);
    size_t& cur = lim[kernel];
    if (lds <= cur) return true;
    if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    cur = lds;
    return true;
}

int occupancy_memo(const void* kernel, int threads, size_t lds)
{
    static std::mutex mu;
    static std::map<std::tuple<const void*, int, size_t>, int> memo;
    const auto key = std::make_tuple(kernel, threads, lds);
    std::lock_guard<std::mutex> g(mu);
    const auto it = memo.find(key);
    if (it != memo.end()) return it->second;
    int bpc = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&bpc, kernel, threads,
                                                     lds) != hipSuccess) {
        (void)hipGetLastError();
        bpc = 0;
    }
    const int r = bpc > 0 ? bpc : 1;
    memo[key] = r;
    return r;
}

// State bytes from a given alpha (test hooks).
__global__ void k_state_from_alpha(int32_t type, const float* y,
                                   const double* a, int64_t n, double C,
                                   uint8_t* st)
{
    int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t N = type == SVM_EPS_SVR ? 2 * n : n;
    if (t >= N) return;
    double yt = type == SVM_EPS_SVR ? (t < n ? 1.0 : -1.0)
                                    : (y[t] > 0.0f ? 1.0 : -1.0);
    st[t] = state_bits(yt, a[t], C);
}

void launch_state_from_alpha(int32_t type, const float* y, const double* a,
                             int64_t n, double C, uint8_t* st, hipStream_t s)
{
    int64_t N = type == SVM_EPS_SVR ? 2 * n : n;
    k_state_from_alpha<<<(unsigned)((N + 255) / 256), 256, 0, s>>>(
        type, y, a, n, C, st);
}

// ---------------------------------------------------------------------------
// coefficients, summary, compaction
// ---------------------------------------------------------------------------

// c_i = y_i a_i (C-SVC) or a_(i,+) - a_(i,-) (eps-SVR), written with a
// stride so that several outputs can share one n x n_out matrix.
__global__ void k_coef(int32_t type, const double* a, const uint8_t* st,
                       int64_t n, double* c, int32_t stride, int32_t off)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    double v;
    if (type == SVM_EPS_SVR) v = a[i] - a[n + i];
    else v = (st[i] & ST_YPOS) ? a[i] : -a[i];
    c[i * stride + off] = v;
}

void launch_coef(int32_t type, const double* a, const uint8_t* st, int64_t n,
                 double* c, hipStream_t s)
{
    k_coef<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(type, a, st, n, c, 1,
                                                       0);
}

void launch_coef_strided(int32_t type, const double* a, const uint8_t* st,
                         int64_t n, double* c, int32_t stride, int32_t off,
                         hipStream_t s)
{
    k_coef<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(type, a, st, n, c,
                                                       stride, off);
}

// Bias and objective ingredients, one block, fixed reduction order.
// Per-block partial sums of a state (bias and objective terms) over a
// fixed split of the N variables, then their sum in a fixed tree order:
// the same bits on every run.
__global__ __launch_bounds__(1024) void k_summary(int32_t type,
                                                  const double* a,
                                                  const uint8_t* st,
                                                  const double* F,
                                                  const float* z, int64_t n,
                                                  double C, double eps,
                                                  Summary* part)
{
    __shared__ double s_v[1024], s_o[1024];
    __shared__ int64_t s_f[1024], s_b[1024];
    const int tid = threadIdx.x;
    const int64_t N = type == SVM_EPS_SVR ? 2 * n : n;
    const int64_t t0 = (int64_t)blockIdx.x * N / gridDim.x;
    const int64_t t1 = ((int64_t)blockIdx.x + 1) * N / gridDim.x;
    double sv = 0.0, so = 0.0;
    int64_t nf = 0, nbd = 0;
    for (int64_t t = t0 + tid; t < t1; t += 1024) {
        const int64_t sm = t >= n ? t - n : t;
        double yv, rv;
        if (type == SVM_EPS_SVR) {
            yv = t < n ? 1.0 : -1.0;
            rv = t < n ? (double)z[sm] - eps : (double)z[sm] + eps;
        } else {
            yv = (st[t] & ST_YPOS) ? 1.0 : -1.0;
            rv = yv;
        }
        const double at = a[t];
        const double v = rv - F[sm];
        if (at > 0.0 && at < C) {
            sv += v;
            ++nf;
        }
        if (at == C) ++nbd;
        so += at * yv * (rv + v);
    }
    s_v[tid] = sv;
    s_o[tid] = so;
    s_f[tid] = nf;
    s_b[tid] = nbd;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (tid < w) {
            s_v[tid] += s_v[tid + w];
            s_o[tid] += s_o[tid + w];
            s_f[tid] += s_f[tid + w];
            s_b[tid] += s_b[tid + w];
        }
        __syncthreads();
    }
    if (tid == 0) {
        Summary& o = part[blockIdx.x];
        o.sum_free_v = s_v[0];
        o.obj2 = s_o[0];
        o.n_free = s_f[0];
        o.n_bounded = s_b[0];
    }
}

__global__ __launch_bounds__(kSummaryBlocks) void k_summary_finish(
    const Summary* part, int nb, Summary* out)
{
    __shared__ double s_v[kSummaryBlocks], s_o[kSummaryBlocks];
    __shared__ int64_t s_f[kSummaryBlocks], s_b[kSummaryBlocks];
    const int tid = threadIdx.x;
    const bool in = tid < nb;
    s_v[tid] = in ? part[tid].sum_free_v : 0.0;
    s_o[tid] = in ? part[tid].obj2 : 0.0;
    s_f[tid] = in ? part[tid].n_free : 0;
    s_b[tid] = in ? part[tid].n_bounded : 0;
    __syncthreads();
    for (int w = kSummaryBlocks / 2; w > 0; w >>= 1) {
        if (tid < w) {
            s_v[tid] += s_v[tid + w];
            s_o[tid] += s_o[tid + w];
            s_f[tid] += s_f[tid + w];
            s_b[tid] += s_b[tid + w];
        }
        __syncthreads();
    }
    if (tid == 0) {
        out->sum_free_v = s_v[0];
        out->obj2 = s_o[0];
        out->n_free = s_f[0];
        out->n_bounded = s_b[0];
    }
}

void launch_summary(int32_t type, const double* a, const uint8_t* st,
                    const double* F, const float* z, int64_t n, double C,
                    double eps, Summary* out, hipStream_t s)
{
    const int64_t N = type == SVM_EPS_SVR ? 2 * n : n;
    const int nb = (int)std::max<int64_t>(
        1, std::min<int64_t>(kSummaryBlocks, (N + 4095) / 4096));
    k_summary<<<nb, 1024, 0, s>>>(type, a, st, F, z, n, C, eps, out + 1);
    k_summary_finish<<<1, kSummaryBlocks, 0, s>>>(out + 1, nb, out);
}

constexpr int kCompactThreads = 1024;

int64_t compact_blocks(int64_t n)
{
    return (n + kCompactThreads - 1) / kCompactThreads;
}

__device__ __forceinline__ bool row_nonzero(const double* coef, int64_t i,
                                            int32_t n_out)
{
    bool nz = false;
    for (int o = 0; o < n_out; ++o) nz |= coef[i * n_out + o] != 0.0;
    return nz;
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_count(
    const double* coef, int64_t n, int32_t n_out, int32_t* blk_cnt)
{
    __shared__ int32_t wc[kCompactThreads / 64];
    const int64_t i = (int64_t)blockIdx.x * kCompactThreads + threadIdx.x;
    const bool f = i < n && row_nonzero(coef, i, n_out);
    const unsigned long long m = __ballot(f);
    if ((threadIdx.x & 63) == 0) wc[threadIdx.x >> 6] = __popcll(m);
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t c = 0;
        for (int w = 0; w < kCompactThreads / 64; ++w) c += wc[w];
        blk_cnt[blockIdx.x] = c;
    }
}

__global__ __launch_bounds__(1024) void k_compact_scan(int32_t* blk_cnt,
                                                      int64_t nblk,
                                                      int64_t* total)
{
    __shared__ int wsum[1024 / 64];
    const int tot = block_exclusive_scan<1024>(blk_cnt, nblk, wsum);
    if (threadIdx.x == 0) *total = tot;
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_scatter(
    const double* coef, int64_t n, int32_t n_out, const int32_t* blk_off,
    int32_t* idx_out, double* coef_out)
{
    __shared__ int32_t wc[kCompactThreads / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t i = (int64_t)blockIdx.x * kCompactThreads + threadIdx.x;
    const bool f = i < n && row_nonzero(coef, i, n_out);
    const unsigned long long m = __ballot(f);
    if (lane == 0) wc[wave] = __popcll(m);
    __syncthreads();
    int32_t base = blk_off[blockIdx.x];
    for (int w = 0; w < wave; ++w) base += wc[w];
    const unsigned long long below =
        lane == 0 ? 0ull : (m & ((1ull << lane) - 1ull));
    if (f) {
        int32_t pos = base + __popcll(below);
        idx_out[pos] = (int32_t)i;
        for (int o = 0; o < n_out; ++o)
            coef_out[(int64_t)pos * n_out + o] = coef[i * n_out + o];
    }
}

void launch_compact(const double* coef, int64_t n, int32_t n_out,
                    int32_t* blk_cnt, int32_t* idx_out, double* coef_out,
                    int64_t* count_out, hipStream_t s)
{
    int64_t nblk = compact_blocks(n);
    if (nblk == 0) return;
    k_compact_count<<<(unsigned)nblk, kCompactThreads, 0, s>>>(coef, n, n_out,
                                                               blk_cnt);
    k_compact_scan<<<1, 1024, 0, s>>>(blk_cnt, nblk, count_out);
    k_compact_scatter<<<(unsigned)nblk, kCompactThreads, 0, s>>>(
        coef, n, n_out, blk_cnt, idx_out, coef_out);
}

__global__ void k_gather_rows(const float* X, const float* sq, int64_t ldp,
                              const int32_t* idx, int64_t k, float* out,
                              float* sq_out)
{
    const int64_t q4 = ldp >> 2;
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; e < k * q4; e += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = e / q4, c4 = e - r * q4;
        int64_t src = idx[r];
        *reinterpret_cast<float4*>(out + r * ldp + 4 * c4) =
            ld4(X + src * ldp + 4 * c4);
        if (c4 == 0 && sq_out) sq_out[r] = sq[src];
    }
}

void launch_gather_rows(const float* X, const float* sq, int64_t ldp,
                        const int32_t* idx, int64_t k, float* out,
                        float* sq_out, hipStream_t s)
{
    if (k <= 0) return;
    int64_t blocks = (k * (ldp >> 2) + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    k_gather_rows<<<(unsigned)blocks, 256, 0, s>>>(X, sq, ldp, idx, k, out,
                                                   sq_out);
}

// ---------------------------------------------------------------------------
// CSR feature store
// ---------------------------------------------------------------------------

// Checks the CSR structure of row i and computes its squared norm (fp64
// sum, rounded once).  bad |= 1: a value not finite (or a norm past fp32),
// 2: row pointers, 4: column indices out of range, unsorted or repeated.
// bad[0]: flags (1 value, 2 pointers, 4 columns); bad[1]: the longest row
__global__ void k_csr_check_norms(const int64_t* rp, const int32_t* ci,
                                  const float* cv, int64_t n, int64_t d,
                                  int64_t nnz, float* sq, int32_t* bad)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0 && (rp[0] != 0 || rp[n] != nnz)) atomicOr(bad, 2);
    if (i >= n) return;
    const int64_t p0 = rp[i], p1 = rp[i + 1];
    int32_t flags = 0;
    double s = 0.0;
    if (p0 < 0 || p1 < p0 || p1 > nnz) {
        flags |= 2;  // (the entries are not read)
    } else {
        int32_t prev = -1;
        for (int64_t k = p0; k < p1; ++k) {
            const int32_t c = ci[k];
            const float v = cv[k];
            if (c < 0 || (int64_t)c >= d || c <= prev) flags |= 4;
            prev = c;
            if (!isfinite(v)) flags |= 1;
            s += (double)v * (double)v;
        }
    }
    const float f = (float)s;
    if (!isfinite(f)) flags |= 1;
    sq[i] = f;
    if (flags) atomicOr(bad, flags);
    if (!(flags & 2) && p1 > p0)
        atomicMax(bad + 1, (int32_t)min(p1 - p0, (int64_t)INT32_MAX));
}

// The working set by column from its dense rows xS (nS rows of ldp floats):
// see compact_by_column.  One block.
__global__ __launch_bounds__(1024) void k_csr_compact(
    const float* xS, int32_t nS, int64_t ldp, int32_t qs, int32_t csr_cols,
    int32_t* xsc_cols, float* xsc)
{
    __shared__ int cnt;
    if (threadIdx.x == 0) cnt = 0;
    __syncthreads();
    compact_by_column(
        [&](int s, int64_t c) { return xS[(int64_t)s * ldp + c]; }, nS, ldp,
        qs, csr_cols, xsc_cols, xsc, &cnt);
}

void launch_csr_compact(const float* xS, int32_t nS, int64_t ldp,
                        int32_t qs, int32_t csr_cols, int32_t* xsc_cols,
                        float* xsc, hipStream_t s)
{
    k_csr_compact<<<1, 1024, 0, s>>>(xS, nS, ldp, qs, csr_cols, xsc_cols,
                                     xsc);
}

void launch_csr_check_norms(const int64_t* rp, const int32_t* ci,
                            const float* cv, int64_t n, int64_t d,
                            int64_t nnz, float* sq, int32_t* bad,
                            hipStream_t s)
{
    const int64_t blocks = (n + 255) / 256;
    k_csr_check_norms<<<(unsigned)(blocks > 0 ? blocks : 1), 256, 0, s>>>(
        rp, ci, cv, n, d, nnz, sq, bad);
}

// ---------------------------------------------------------------------------
// Sliced copy of the CSR rows for the row kernel
// ---------------------------------------------------------------------------
//
// Slices of kSellRows consecutive rows.  Slice s holds nonzero k of its row t
// at so[s] + kSellRows * k + t for k below the slice width (the most
// nonzeros of its rows); entries past the end of a row are (column 0, value
// 0).  A row keeps its nonzeros in column order.  The row kernel walks one
// row per lane: a load of nonzero k of 64 rows then reads four 64-byte runs
// instead of 64 scattered words.

// so[s] = kSellRows * (width of slice s), for the scan below
__global__ void k_sell_widths(const int64_t* rp, int64_t n, int64_t* so)
{
    const int64_t ns = (n + kSellRows - 1) / kSellRows;
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= ns) return;
    int64_t w = 0;
    for (int t = 0; t < kSellRows; ++t) {
        const int64_t i = s * kSellRows + t;
        if (i < n) w = max(w, rp[i + 1] - rp[i]);
    }
    so[s] = kSellRows * max(w, (int64_t)0);
}

// Exclusive scan of so[0 .. ns) in place; so[ns] = the total.  One block:
// each thread sums a contiguous run, the run sums are scanned in LDS, then
// each thread rewrites its run.
__global__ __launch_bounds__(1024) void k_sell_scan(int64_t* so, int64_t ns)
{
    __shared__ int64_t part[1024];
    const int t = threadIdx.x;
    const int64_t run = (ns + 1023) / 1024;
    const int64_t b = min((int64_t)t * run, ns), e = min(b + run, ns);
    int64_t acc = 0;
    for (int64_t k = b; k < e; ++k) acc += so[k];
    part[t] = acc;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int64_t v = t >= off ? part[t - off] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    acc = part[t] - acc;  // exclusive prefix of this run
    for (int64_t k = b; k < e; ++k) {
        const int64_t w = so[k];
        so[k] = acc;
        acc += w;
    }
    if (t == 1023) so[ns] = part[1023];
}

// One thread per row: its nonzeros, then the padding of its slice.
__global__ void k_sell_fill(const int64_t* rp, const int32_t* ci,
                            const float* cv, int64_t n, const int64_t* so,
                            uint16_t* sci, float* scv)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t s = i / kSellRows, t = i - s * kSellRows;
    const int64_t w = (so[s + 1] - so[s]) / kSellRows;
    const int64_t p0 = rp[i], nz = rp[i + 1] - p0;
    for (int64_t k = 0; k < w; ++k) {
        const int64_t dst = so[s] + kSellRows * k + t;
        sci[dst] = k < nz ? (uint16_t)ci[p0 + k] : (uint16_t)0;
        scv[dst] = k < nz ? cv[p0 + k] : 0.0f;
    }
}

void launch_sell_offsets(const int64_t* rp, int64_t n, int64_t* so,
                         hipStream_t s)
{
    const int64_t ns = (n + kSellRows - 1) / kSellRows;
    if (ns > 0)
        k_sell_widths<<<(unsigned)((ns + 255) / 256), 256, 0, s>>>(rp, n, so);
    k_sell_scan<<<1, 1024, 0, s>>>(so, ns);
}

void launch_sell_fill(const int64_t* rp, const int32_t* ci, const float* cv,
                      int64_t n, const int64_t* so, uint16_t* sci, float* scv,
                      hipStream_t s)
{
    if (n > 0)
        k_sell_fill<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(rp, ci, cv, n,
                                                              so, sci, scv);
}

// Dense rows (ldp wide, zero-filled) of CSR rows: row r of the output is
// source row idx[r] (idx == nullptr: row r0 + r), with its norm.  One block
// per output row.
__global__ void k_gather_rows_csr(const int64_t* rp, const int32_t* ci,
                                  const float* cv, const float* sq,
                                  int64_t ldp, const int32_t* idx, int64_t r0,
                                  int64_t k, float* out, float* sq_out)
{
    for (int64_t r = blockIdx.x; r < k; r += gridDim.x) {
        const int64_t src = idx ? (int64_t)idx[r] : r0 + r;
        float* row = out + r * ldp;
        for (int64_t c = threadIdx.x; c < ldp; c += blockDim.x) row[c] = 0.0f;
        __syncthreads();
        const int64_t p0 = rp[src], p1 = rp[src + 1];
        for (int64_t q = p0 + threadIdx.x; q < p1; q += blockDim.x)
            row[ci[q]] = cv[q];
        if (threadIdx.x == 0 && sq_out) sq_out[r] = sq[src];
        __syncthreads();
    }
}

void launch_gather_rows_csr(const int64_t* rp, const int32_t* ci,
                            const float* cv, const float* sq, int64_t ldp,
                            const int32_t* idx, int64_t r0, int64_t k,
                            float* out, float* sq_out, hipStream_t s)
{
    if (k <= 0) return;
    const int64_t blocks = k < 65536 ? k : 65536;
    k_gather_rows_csr<<<(unsigned)blocks, 256, 0, s>>>(rp, ci, cv, sq, ldp, idx,
                                                       r0, k, out, sq_out);
}

__global__ void k_labels(const double* D, int64_t m, int32_t n_out,
                         int32_t* labels)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= m) return;
    if (n_out == 1) {
        labels[i] = D[i] >= 0.0 ? 1 : -1;
        return;
    }
    int32_t best = 0;
    double bv = D[i * n_out];
    for (int o = 1; o < n_out; ++o) {
        double v = D[i * n_out + o];
        if (v > bv) {
            bv = v;
            best = o;
        }
    }
    labels[i] = best;
}

void launch_argmax_labels(const double* D, int64_t m, int32_t n_out,
                          int32_t type, int32_t* labels, hipStream_t s)
{
    (void)type;
    if (m <= 0) return;
    k_labels<<<(unsigned)((m + 255) / 256), 256, 0, s>>>(D, m, n_out, labels);
}

}  // namespace msvm
