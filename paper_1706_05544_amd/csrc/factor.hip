// Sparse decision function by column (gfx950): D(x) = sum_j c_j K(sv_j, x) + b
// for CSR query rows against CSR support rows, and the recompute of the
// responses F after a CSR training, with work that grows with the pairs of
// rows that share a column rather than with all pairs.
//
// Pairs with no column in common have x.v = 0, so the RBF value of such a
// pair is e^(-g s_x) e^(-g s_v): summed over all support rows this is
// e^(-g s_x) C0 with C0 = sum_v c_v e^(-g s_v), one constant per output.
// Only the pairs that share a column need their dot product and kernel
// value, and they enter as the difference from that constant term.  The
// dot products of one query row against one chunk of support rows are
// accumulated in LDS (one fp32 slot per support row of the chunk, walk 1),
// then read back and cleared at exactly the slots that were touched
// (walk 2, an atomic exchange with 0: a support row that shares several
// columns with the query row is visited once, at its first entry).
//
// No barrier: every wave owns its LDS accumulator and its query rows, and
// walks all chunks (entries and maps are read from global memory, where
// the chunk that the waves of a CU are walking stays in L2).  Per row and
// chunk the partial sums are reduced across the wave in a fixed order and
// added in chunk order, so the values do not depend on timing.
#include "common.hpp"
#include "device.hpp"

namespace msvm {

constexpr int kFcWaves = 4;     // waves of a block (independent)
constexpr int kFcRW = 16;       // query rows of a wave
constexpr int kFcGroup = 8;     // entry loads issued together
constexpr uint32_t kFcLenMask = (1u << kFcLenBits) - 1;
// Rows with gexp * |x|^2 above kFcSafe take the direct formula, so that
// e^(-g s_x) and the factor 2^(2 gexp x.v) stay inside fp64 and fp32 range
// (2 gexp x.v <= gexp (|x|^2 + |v|^2) <= 2 kFcSafe < 128 when both sides
// are within the bound).
static_assert(kFcSvMax <= (int)kFcLenMask, "count field of a map entry");
static_assert(kFcEntMax <= ((int64_t)1 << (32 - kFcLenBits)),
              "start field of a map entry");

// inclusive prefix sum over the wave
__device__ __forceinline__ int fc_scan(int v, int lane)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(v, o);
        if (lane >= o) v += u;
    }
    return v;
}

// The segment (query nonzero) holding flattened position p: the largest k
// with E_k <= p, where E (the segments' first positions, one per lane) does
// not decrease over the lanes and E_0 = 0.  Every lane takes part.
__device__ __forceinline__ int fc_seg(int E, int p)
{
    int k = 0;
#pragma unroll
    for (int s = 32; s > 0; s >>= 1) {
        const int e = __shfl(E, k + s);
        if (e <= p) k += s;
    }
    return k;
}

// One group of at most 64 nonzeros of a query row against a chunk: the
// lane's nonzero (column, value), its segment of the chunk's entries and
// the flattened layout (T positions in all).
struct FcGroup {
    float xv;
    int E, off, T;
};

__device__ __forceinline__ FcGroup fc_group(const FactArgs& a,
                                            const uint32_t* mp, int64_t gb,
                                            int nzg, int lane)
{
    FcGroup g;
    int col = 0;
    g.xv = 0.0f;
    uint32_t mm = 0;
    if (lane < nzg) {
        col = a.cit[gb + lane];
        g.xv = a.cvt[gb + lane];
        mm = mp[col];
    }
    const int len = (int)(mm & kFcLenMask), st = (int)(mm >> kFcLenBits);
    const int inc = fc_scan(len, lane);
    g.T = __builtin_amdgcn_readlane(inc, 63);
    g.E = inc - len;
    g.off = st - g.E;
    return g;
}

// Per-row constants of walk 2.
struct FcRow {
    float sx;      // |x|^2
    double A;      // e^(-g s_x) (RBF), else 1
    double invA;   // 1 / A (the row's own support row, factored form)
    int64_t js;    // the row's own support row, or -1
    bool fast;     // factored RBF form
};

// The term of a support row v (local to the chunk at sv0) whose dot
// product d with the query row was taken from the accumulator (and the
// slot cleared) at its first visit; wv is w_v of output 0 in fp32.
template <int NOUT>
__device__ __forceinline__ void fc_term(const FactArgs& a, const FcRow& R,
                                        int sv0, int v, float d, float wv,
                                        double (&part)[NOUT])
{
    const int64_t j = (int64_t)sv0 + v;
    const int n_out = a.n_out;
    if (R.fast) {
        if (j == R.js) {
            // K(x_i, x_i) = 1: c_v - A w_v, in units of A
#pragma unroll
            for (int o = 0; o < NOUT; ++o)
                if (o < n_out)
                    part[o] += a.coef[j * n_out + o] * R.invA -
                               a.w[j * n_out + o];
        } else {
            // c_v K - A w_v = A w_v (2^(2 gexp d) - 1)
            const float t =
                __builtin_amdgcn_exp2f(2.0f * a.kf.gexp * d) - 1.0f;
            if (NOUT == 1) {
                part[0] += (double)(t * wv);
            } else {
#pragma unroll
                for (int o = 0; o < NOUT; ++o)
                    if (o < n_out)
                        part[o] = fma((double)t, a.w[j * n_out + o], part[o]);
            }
        }
    } else {
        float K;
        if (a.kf.kind == SVM_KERNEL_RBF) {
            K = rbf_from_dot(R.sx, a.sqsv[j], d, a.kf.gexp);
            if (j == R.js) K = 1.0f;
        } else {
            K = kernel_of_dot(a.kf, d);
        }
#pragma unroll
        for (int o = 0; o < NOUT; ++o)
            if (o < n_out)
                part[o] += a.coef[j * n_out + o] * (double)K -
                           R.A * a.w[j * n_out + o];
    }
}

// wave sum in a fixed order (every lane receives it)
__device__ __forceinline__ double fc_wave_sum(double v)
{
    v = row_sum_f64(v);
    return (rl_f64(v, 0) + rl_f64(v, 16)) + (rl_f64(v, 32) + rl_f64(v, 48));
}

__device__ __forceinline__ int fc_wave_max(int v)
{
    v = max(v, dpp_i32<kDppRor8>(v));
    v = max(v, dpp_i32<kDppRor4>(v));
    v = max(v, dpp_i32<kDppRor2>(v));
    v = max(v, dpp_i32<kDppRor1>(v));
    return max(max(rl_i32(v, 0), rl_i32(v, 16)),
               max(rl_i32(v, 32), rl_i32(v, 48)));
}

// A row of at most 64 nonzeros against one chunk.  Lane l serves nonzero
// k = l / spp of the row: entries st_k + sub, st_k + sub + spp, ... of its
// column's list (sub = l % spp), kFcGroup of them per step with their loads
// issued together.
template <int NOUT>
__device__ __forceinline__ void fc_chunk(const FactArgs& a, const FcRow& R,
                                         int sv0, const int2* ent,
                                         uint32_t mm, bool act, int sub,
                                         int spp, float xk, float* sp,
                                         double (&part)[NOUT])
{
    const int len = act ? (int)(mm & kFcLenMask) : 0;
    const int st = (int)(mm >> kFcLenBits);
    const int maxlen = fc_wave_max(len);
    if (maxlen == 0) return;
    constexpr int G = kFcGroup;
    // walk 1: x_c v_c into the slots
    for (int it0 = 0; it0 * spp < maxlen; it0 += G) {
        int2 en[G];
#pragma unroll
        for (int u = 0; u < G; ++u) {
            const int j = sub + (it0 + u) * spp;
            en[u] = j < len ? ent[st + j] : make_int2(0, 0);
        }
#pragma unroll
        for (int u = 0; u < G; ++u) {
            const int j = sub + (it0 + u) * spp;
            if (j < len)
                atomicAdd(&sp[en[u].x], xk * __int_as_float(en[u].y));
        }
    }
    // walk 2: each touched slot taken once (and cleared)
    const float* wf = a.wf + sv0;
    for (int it0 = 0; it0 * spp < maxlen; it0 += G) {
        int v[G];
#pragma unroll
        for (int u = 0; u < G; ++u) {
            const int j = sub + (it0 + u) * spp;
            v[u] = j < len ? ent[st + j].x : -1;
        }
        float d[G], wv[G];
#pragma unroll
        for (int u = 0; u < G; ++u) {
            d[u] = v[u] >= 0 ? atomicExch(&sp[v[u]], 0.0f) : 0.0f;
            wv[u] = (NOUT == 1 && d[u] != 0.0f) ? wf[v[u]] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < G; ++u)
            if (d[u] != 0.0f)
                fc_term<NOUT>(a, R, sv0, v[u], d[u], wv[u], part);
    }
}

// The general case (more than 64 nonzeros): the row's nonzeros in groups of
// 64, each group's entries flattened over the lanes (binary search of the
// position in the segments' prefix sums); walk 1 over every group before
// walk 2.
template <bool ADD>
__device__ __forceinline__ int fc_visit(const FcGroup& g, const int2* ent,
                                        float* sp, int p)
{
    const int k = fc_seg(g.E, p);
    const int off = __shfl(g.off, k);
    const float x = __shfl(g.xv, k);
    int v = -1;
    if (p < g.T) {
        const int2 en = ent[p + off];
        v = en.x;
        if (ADD) atomicAdd(&sp[v], x * __int_as_float(en.y));
    }
    return v;
}

template <int NOUT>
__device__ void fc_long_row(const FactArgs& a, const FcRow& R, int64_t k0,
                            int64_t k1, int sv0, const int2* ent,
                            const uint32_t* mp, float* sp, int lane,
                            double (&part)[NOUT])
{
    for (int64_t gb = k0; gb < k1; gb += 64) {
        const FcGroup g =
            fc_group(a, mp, gb, (int)min<int64_t>(64, k1 - gb), lane);
        for (int p0 = 0; p0 < g.T; p0 += 64)
            fc_visit<true>(g, ent, sp, p0 + lane);
    }
    for (int64_t gb = k0; gb < k1; gb += 64) {
        const FcGroup g =
            fc_group(a, mp, gb, (int)min<int64_t>(64, k1 - gb), lane);
        for (int p0 = 0; p0 < g.T; p0 += 64) {
            const int v = fc_visit<false>(g, ent, sp, p0 + lane);
            const float d = v >= 0 ? atomicExch(&sp[v], 0.0f) : 0.0f;
            if (d != 0.0f)
                fc_term<NOUT>(a, R, sv0, v, d,
                              NOUT == 1 ? a.wf[(int64_t)sv0 + v] : 0.0f, part);
        }
    }
}

// One wave, its query rows against every chunk: chunk by chunk (all
// resident waves walk the same few chunks at a time, which stay in L2),
// each row's terms of a chunk reduced across the wave (fixed order) and
// added to the row's sum in LDS in chunk order.
template <int NOUT>
__global__ __launch_bounds__(kFcWaves * 64) void k_predict_fact(FactArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    float* sp = reinterpret_cast<float*>(smem) + wave * kFcSvMax;
    double* rs = reinterpret_cast<double*>(smem + kFcWaves * kFcSvMax * 4) +
                 wave * kFcRW * (NOUT + 1);
    double* rA = rs + kFcRW * NOUT;  // per row: e^(-g s_x) (RBF), else 1
    for (int i = lane; i < kFcSvMax; i += 64) sp[i] = 0.0f;
    const int64_t r0 = ((int64_t)blockIdx.x * kFcWaves + wave) * kFcRW;
    const int rows = (int)min<int64_t>(kFcRW, a.m - r0);
    if (rows <= 0) return;  // (no barrier in this kernel)
    const bool rbf = a.kf.kind == SVM_KERNEL_RBF;
    const int n_out = a.n_out;
    if (lane < rows) {
        const float sx = a.sqt[r0 + lane];
        rA[lane] = rbf ? exp2(-(double)a.kf.gexp * (double)sx) : 1.0;
#pragma unroll
        for (int o = 0; o < NOUT; ++o) rs[lane * NOUT + o] = 0.0;
    }
    for (int g = 0; g < a.nch; ++g) {
        const int sv0 = a.ch_sv0[g], sv1 = a.ch_sv0[g + 1];
        const int2* ent = a.ent + a.ch_e0[g];
        const uint32_t* mp = a.map + (int64_t)g * a.ldpm;
        for (int rr = 0; rr < rows; ++rr) {
            const int64_t r = r0 + rr;
            const int64_t k0 = a.rpt[r], k1 = a.rpt[r + 1];
            const int64_t nz = k1 - k0;
            if (nz == 0) continue;
            FcRow R;
            R.sx = a.sqt[r];
            R.A = rA[rr];
            R.fast = rbf && a.fast && a.kf.gexp * R.sx <= kFcSafe;
            R.js = -1;
            R.invA = 0.0;
            if (a.self_sv) {
                const int js = a.self_sv[r + a.row_base];
                if (js >= sv0 && js < sv1) {
                    R.js = js;
                    if (R.fast) R.invA = 1.0 / R.A;
                }
            }
            double part[NOUT];
#pragma unroll
            for (int o = 0; o < NOUT; ++o) part[o] = 0.0;
            if (nz > 64) {
                fc_long_row<NOUT>(a, R, k0, k1, sv0, ent, mp, sp, lane, part);
            } else {
                // lane -> (nonzero k, slot sub); every lane of a nonzero
                // reads its column's map entry itself
                const int nzi = (int)nz;
                const int spp = 64 / nzi;
                const int k = lane / spp, sub = lane - k * spp;
                const bool act = k < nzi;
                const int col = act ? a.cit[k0 + k] : 0;
                const float xk = act ? a.cvt[k0 + k] : 0.0f;
                fc_chunk<NOUT>(a, R, sv0, ent, mp[col], act, sub, spp, xk,
                               sp, part);
            }
#pragma unroll
            for (int o = 0; o < NOUT; ++o) {
                if (o < n_out) {
                    const double t = fc_wave_sum(part[o]);
                    if (lane == 0) rs[rr * NOUT + o] += t;
                }
            }
        }
    }
    // D = A C0 + (factored rows: A) sum of the terms + b
    if (lane < rows) {
        const int64_t r = r0 + lane;
        const float sx = a.sqt[r];
        const bool fast = rbf && a.fast && a.kf.gexp * sx <= kFcSafe;
        for (int o = 0; o < n_out; ++o) {
            const double t = rs[lane * NOUT + o];
            a.out[r * n_out + o] = rA[lane] * a.c0[o] +
                                   (fast ? rA[lane] * t : t) +
                                   (a.b ? a.b[o] : 0.0);
        }
    }
}

static size_t fc_lds_bytes(int nout)
{
    return (size_t)kFcWaves * kFcSvMax * 4 +
           (size_t)kFcWaves * kFcRW * (nout + 1) * 8;
}

void launch_predict_fact(const FactArgs& a, hipStream_t s)
{
    if (a.m <= 0) return;
    if (a.n_out < 1 || a.n_out > 4)
        throw Error{SVM_E_INTERNAL, "factored decision path: 1 to 4 outputs"};
    const int64_t per = (int64_t)kFcWaves * kFcRW;
    const unsigned blocks = (unsigned)((a.m + per - 1) / per);
    if (a.n_out == 1)
        k_predict_fact<1><<<blocks, kFcWaves * 64, fc_lds_bytes(1), s>>>(a);
    else
        k_predict_fact<4><<<blocks, kFcWaves * 64, fc_lds_bytes(4), s>>>(a);
}

// ---- building the chunks ----

__global__ void k_fc_nnz(const int64_t* rp, const float* sq,
                         const int32_t* idx, int64_t nsv, int32_t* nz,
                         float* sq_out)
{
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nsv;
         j += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = idx ? (int64_t)idx[j] : j;
        nz[j] = (int32_t)(rp[r + 1] - rp[r]);
        if (sq_out) sq_out[j] = sq[r];
    }
}

void launch_fc_nnz(const int64_t* rp, const float* sq, const int32_t* idx,
                   int64_t nsv, int32_t* nz, float* sq_out, hipStream_t s)
{
    if (nsv <= 0) return;
    const unsigned blocks = (unsigned)std::min<int64_t>((nsv + 255) / 256,
                                                        4096);
    k_fc_nnz<<<blocks, 256, 0, s>>>(rp, sq, idx, nsv, nz, sq_out);
}

// One block per chunk: column counts (LDS), their exclusive scan (the
// first entry of each column), the map row, then the entries in the order
// (column, support row): one wave walks the chunk's rows in order and
// takes each nonzero's slot from an LDS cursor, so that every column lists
// its rows increasing (the same layout on every build).
constexpr int kFcBuildThreads = 256;
__global__ __launch_bounds__(kFcBuildThreads) void k_fc_build(FactBuildArgs a)
{
    extern __shared__ __align__(16) int fc_cnt[];  // ldpm
    __shared__ int wsum[kFcBuildThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = blockIdx.x;
    const int s0 = a.ch_sv0[g], s1 = a.ch_sv0[g + 1];
    const int64_t e0 = a.ch_e0[g];
    const int ldpm = a.ldpm;
    for (int c = tid; c < ldpm; c += kFcBuildThreads) fc_cnt[c] = 0;
    __syncthreads();
    for (int s = s0 + wave; s < s1; s += kFcBuildThreads / 64) {
        const int64_t r = a.idx ? (int64_t)a.idx[s] : s;
        for (int64_t p = a.rp[r] + lane; p < a.rp[r + 1]; p += 64)
            atomicAdd(&fc_cnt[a.ci[p]], 1);
    }
    __syncthreads();
    // counts -> (start << kFcLenBits) | count, and cursors at the starts
    const int total = block_exclusive_scan<kFcBuildThreads>(fc_cnt, ldpm,
                                                            wsum);
    uint32_t* mp = a.map + (int64_t)g * ldpm;
    for (int c = tid; c < ldpm; c += kFcBuildThreads) {
        const int st = fc_cnt[c];
        const int nx = c + 1 < ldpm ? fc_cnt[c + 1] : total;
        mp[c] = ((uint32_t)st << kFcLenBits) | (uint32_t)(nx - st);
    }
    __syncthreads();
    if (wave == 0) {
        for (int s = s0; s < s1; ++s) {
            const int64_t r = a.idx ? (int64_t)a.idx[s] : s;
            const int64_t p0 = a.rp[r], p1 = a.rp[r + 1];
            for (int64_t p = p0 + lane; p < p1; p += 64) {
                const int c = a.ci[p];
                const int pos = atomicAdd(&fc_cnt[c], 1);
                a.ent[e0 + pos] = make_int2(s - s0, __float_as_int(a.cv[p]));
            }
        }
    }
}

void launch_fc_build(const FactBuildArgs& a, hipStream_t s)
{
    if (a.nch <= 0) return;
    k_fc_build<<<(unsigned)a.nch, kFcBuildThreads, (size_t)a.ldpm * 4, s>>>(
        a);
}

// w (grid-stride) and the largest gexp * s_v (one atomic per block)
__global__ void k_fc_w(const double* coef, const float* sqsv, int64_t nsv,
                       int32_t n_out, KernelFn kf, double* w, float* wf,
                       uint32_t* gs_max)
{
    const bool rbf = kf.kind == SVM_KERNEL_RBF;
    const double k0 = rbf ? 0.0 : (double)kernel_of_dot(kf, 0.0f);
    float mx = 0.0f;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nsv;
         j += (int64_t)gridDim.x * blockDim.x) {
        const float s = sqsv[j];
        mx = fmaxf(mx, kf.gexp * s);
        const double f = rbf ? exp2(-(double)kf.gexp * (double)s) : k0;
        for (int o = 0; o < n_out; ++o)
            w[j * n_out + o] = coef[j * n_out + o] * f;
        wf[j] = (float)(coef[j * n_out] * f);
    }
    for (int off = 32; off > 0; off >>= 1)
        mx = fmaxf(mx, __shfl_xor(mx, off));
    if ((threadIdx.x & 63) == 0) atomicMax(gs_max, __float_as_uint(mx));
}

// c0[o] = sum_j w[j][o]: one block, thread t sums j = t, t + 1024, ... in
// order, then a fixed tree
__global__ __launch_bounds__(1024) void k_fc_c0(const double* w, int64_t nsv,
                                                int32_t n_out, double* c0)
{
    __shared__ double red[1024];
    const int tid = threadIdx.x;
    for (int o = 0; o < n_out; ++o) {
        double s = 0.0;
        for (int64_t j = tid; j < nsv; j += 1024) s += w[j * n_out + o];
        red[tid] = s;
        __syncthreads();
        for (int h = 512; h > 0; h >>= 1) {
            if (tid < h) red[tid] += red[tid + h];
            __syncthreads();
        }
        if (tid == 0) c0[o] = red[0];
        __syncthreads();
    }
}

void launch_fc_weights(const double* coef, const float* sqsv, int64_t nsv,
                       int32_t n_out, const KernelFn& kf, double* w,
                       float* wf, double* c0, uint32_t* gs_max, hipStream_t s)
{
    if (nsv > 0) {
        const unsigned blocks =
            (unsigned)std::min<int64_t>((nsv + 255) / 256, 2048);
        k_fc_w<<<blocks, 256, 0, s>>>(coef, sqsv, nsv, n_out, kf, w, wf,
                                      gs_max);
    }
    k_fc_c0<<<1, 1024, 0, s>>>(w, nsv, n_out, c0);
}

__global__ void k_fc_self_set(const int32_t* sv_idx, int64_t nsv,
                              int32_t* self_sv)
{
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nsv;
         j += (int64_t)gridDim.x * blockDim.x)
        self_sv[sv_idx[j]] = (int32_t)j;
}

void launch_fc_self(const int32_t* sv_idx, int64_t nsv, int64_t n,
                    int32_t* self_sv, hipStream_t s)
{
    if (n <= 0) return;
    launch_fill_i32(self_sv, -1, n, s);
    if (nsv <= 0) return;
    const unsigned blocks =
        (unsigned)std::min<int64_t>((nsv + 255) / 256, 4096);
    k_fc_self_set<<<blocks, 256, 0, s>>>(sv_idx, nsv, self_sv);
}

size_t fc_map_bytes_limit() { return (size_t)1 << 30; }

}  // namespace msvm
