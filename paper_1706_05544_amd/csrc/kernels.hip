// HIP kernels of the working-set dual solve (gfx950).
//
// One outer iteration of the decomposition (Section 3: pick a working set
// of 16 coefficients by the largest partial derivatives under the
// constraints, optimise them from the local gradient, update the responses)
// is two launches:
//
//   k_select  one block of 1024 threads.  Merges the per-block candidates of
//             the previous k_rows into the global working set B (the q/2
//             largest keys of I_up interleaved with the q/2 smallest keys of
//             I_low), tests the gap m - M against tol, computes the kernel
//             block K_BB on the matrix cores and solves the subproblem on B
//             with maximal-violating-pair steps.  Writes the new alpha_B, the
//             state bytes and the coefficient change of each distinct sample.
//   k_rows    the whole grid.  Streams X once: for each 16-row tile, the dot
//             products with the (at most 16 per column block) working-set
//             samples on the matrix cores (16x16x4 fp32), the RBF epilogue,
//             F_i += sum_s dc_s K(x_i, x_s) in fp64, the keys v of the
//             variables of the tile and the per-block top-q/2 candidates of
//             each side for the next k_select.
#include <hip/hip_ext.h>

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
__global__ void k_init_state(int32_t type, const float* y, int64_t n,
                             uint8_t* st, int32_t* bad)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    if (type == SVM_C_SVC) {
        float v = y[i];
        if (v == 1.0f) {
            st[i] = ST_YPOS | ST_UP;
            atomicOr(bad, 2);
        } else if (v == -1.0f) {
            st[i] = ST_LOW;
            atomicOr(bad, 4);
        } else {
            st[i] = 0;
            atomicOr(bad, 1);
        }
    } else {
        st[i] = ST_YPOS | ST_UP;
        st[n + i] = ST_LOW;
        if (!isfinite(y[i])) atomicOr(bad, 1);
    }
}

void launch_init_state(int32_t type, const float* y, int64_t n, uint8_t* st,
                       int32_t* bad, hipStream_t s)
{
    k_init_state<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(type, y, n, st,
                                                             bad);
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
// row / update kernel
// ---------------------------------------------------------------------------


// LDS row stride of the per-wave feature slab buffer (64 columns + pad)
constexpr int kSlabStride = 68;
// feature slabs in flight per wave of k_rows
constexpr int kRing = 4;
constexpr int kRowWaves = kRowThreads / 64;

// LDS row stride of a staged working-set sample: ldp rounded up to whole
// 16-feature chunks (zero-filled) plus a pad of 4 against bank conflicts.
__host__ __device__ inline int rows_xs_stride(int64_t ldp)
{
    return (int)(((ldp + 15) & ~(int64_t)15) + 4);
}

// Per-wave LDS bytes for the row data of 16 * tiles rows: F (fp64), the
// squared norm, for eps-SVR the target, and the state byte of each copy.
__host__ __device__ inline int rows_aux_bytes(int tiles, bool svr)
{
    return ((16 * tiles * (svr ? 18 : 13)) + 15) & ~15;
}

__host__ __device__ inline size_t rows_aux_offset(int nblk_cols, int64_t ldp)
{
    return (size_t)nblk_cols * 16 * rows_xs_stride(ldp) * sizeof(float) +
           (size_t)kRowWaves * 16 * kSlabStride * sizeof(float);
}

size_t rows_lds_bytes(int nblk_cols, int64_t ldp, int tiles, bool svr)
{
    return rows_aux_offset(nblk_cols, ldp) +
           (size_t)kRowWaves * rows_aux_bytes(tiles, svr);
}

// Running best two (score, variable) of one lane, in the order of better().
struct Top2 {
    double k1 = -INFINITY, k2 = -INFINITY;
    int32_t i1 = INT_MAX, i2 = INT_MAX;
    __device__ __forceinline__ void push(double k, int32_t i)
    {
        if (better(k, i, k1, i1)) {
            k2 = k1;
            i2 = i1;
            k1 = k;
            i1 = i;
        } else if (better(k, i, k2, i2)) {
            k2 = k;
            i2 = i;
        }
    }
};

// Both sides at once (independent chains interleave): writes the wave's best
// two up scores to ok[0..1] and best two low scores to ok[2..3].
__device__ __forceinline__ void wave_top2_pair(Top2 u, Top2 l, double* ok,
                                               int32_t* oi)
{
    double ku = u.k1, kl = l.k1;
    int32_t iu = u.i1, il = l.i1;
    wave_best_pair(ku, iu, kl, il);
    const bool mu = u.i1 == iu && u.k1 == ku;
    const bool ml = l.i1 == il && l.k1 == kl;
    double ku2 = mu ? u.k2 : u.k1, kl2 = ml ? l.k2 : l.k1;
    int32_t iu2 = mu ? u.i2 : u.i1, il2 = ml ? l.i2 : l.i1;
    wave_best_pair(ku2, iu2, kl2, il2);
    if ((threadIdx.x & 63) == 0) {
        ok[0] = ku;
        oi[0] = iu;
        ok[1] = ku2;
        oi[1] = iu2;
        ok[2] = kl;
        oi[2] = il;
        ok[3] = kl2;
        oi[3] = il2;
    }
}

// Row/update kernel.  Each wave owns 16 * tiles consecutive rows.
//
// Its row data (F, norms, state bytes, targets) is read once into a
// wave-private LDS area, updated there and F is written back, coalesced, at
// the end: the feature stream is then the only global traffic in the main
// loop, and every load in it is unconditional (buffer range checks give the
// zeros of ragged tails), so the loads stay in flight across slabs.
//
// Features go through 64-column slabs: the global loads are row-contiguous
// (16 lanes cover 256 B of one row, 4 rows per instruction) and run kRing
// slabs ahead; each slab passes through a wave-private LDS buffer and is read
// back in the matrix-core operand layout (lane (g, nl): row nl, columns
// 16c + 4g .. +3 of chunk c), which is the library-wide chunk order, so every
// K value matches the other kernels bitwise.
template <bool SVR, int NBLK, int MODE>
__global__ __launch_bounds__(kRowThreads) void k_rows(RowArgs a)
{
    constexpr bool UPD = (MODE & RU_UPDATE) != 0;
    constexpr bool ROWS = (MODE & RU_ROWS) != 0;
    constexpr bool CAND = (MODE & RU_CAND) != 0;
    constexpr bool XS = UPD || ROWS;  // the working-set samples are needed
    constexpr int kXsEarly = 2;       // staging loads issued with the stream
    extern __shared__ __align__(16) unsigned char smem[];
    const WorkingSet* ws = a.ws;
    if ((MODE & RU_CHECK_DONE) && ws->done) return;

    const int tid = threadIdx.x, lane = tid & 63;
    // wave-uniform by construction; said so, so that the buffer resources
    // built from it live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, nl = lane & 15;
    const int T = a.tiles, RW = 16 * T;
    const int64_t n = a.n;
    const int ldp = (int)a.ldp;
    const int xstride = rows_xs_stride(ldp);
    float* xsl = reinterpret_cast<float*>(smem);

    // working-set slot b * 16 + nl of this lane (slots past nS contribute 0)
    const int nS = XS ? (a.nS_override >= 0 ? a.nS_override : ws->nS) : 0;
    double cf[NBLK];
    float ssl[NBLK];
    int32_t sidx[NBLK];
#pragma unroll
    for (int b = 0; b < NBLK; ++b) {
        const int slot = b * 16 + nl;  // < kMaxQ: always inside the arrays
        const bool ok = slot < nS;
        const double c = ws->coef[slot];
        const float s = ws->sS[slot];
        const int32_t i = ws->S[slot];
        cf[b] = (ok && UPD) ? c : 0.0;
        ssl[b] = ok ? s : 0.0f;
        sidx[b] = ok ? i : -1;
    }

    // rows of this wave: rw0 .. rw0 + nw - 1, in Tw tiles of 16
    const int64_t rw0 = ((int64_t)blockIdx.x * kRowWaves + wave) * RW;
    const int nw = rw0 >= n ? 0 : (int)min((int64_t)RW, n - rw0);
    const int Tw = (nw + 15) >> 4;
    unsigned char* aux =
        smem + rows_aux_offset(NBLK, ldp) + wave * rows_aux_bytes(T, SVR);
    double* Fw = reinterpret_cast<double*>(aux);
    float* sqw = reinterpret_cast<float*>(aux + 8 * RW);
    float* zw = reinterpret_cast<float*>(aux + 12 * RW);
    uint8_t* stw = aux + (SVR ? 16 : 12) * RW;  // copy (i,-) at stw[RW + r]

    // row data of rows k0 .. k0 + 255 of the wave: issue, then store to LDS
    struct AuxRegs {
        double f[4];
        float q[4], z[4];
        uint8_t s0[4], s1[4];
    };
    const Rsrc rF = make_rsrc(a.F + rw0, (int64_t)nw * 8);
    auto aux_issue = [&](int k0, AuxRegs& x) {
        const Rsrc rQ = make_rsrc(a.sq + rw0, (int64_t)nw * 4);
        const Rsrc rS0 = make_rsrc(a.st + rw0, nw);
        const Rsrc rS1 = make_rsrc(a.st + n + rw0, SVR ? nw : 0);
        const Rsrc rZ = make_rsrc(a.z + rw0, SVR ? (int64_t)nw * 4 : 0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t r = (uint32_t)(k0 + 64 * j + lane);
            x.f[j] = (UPD || CAND) ? bld_f64(rF, 8 * r) : 0.0;
            x.q[j] = XS ? bld_f32(rQ, 4 * r) : 0.0f;
            x.s0[j] = CAND ? bld_u8(rS0, r) : 0;
            x.s1[j] = (SVR && CAND) ? bld_u8(rS1, r) : 0;
            x.z[j] = (SVR && CAND) ? bld_f32(rZ, 4 * r) : 0.0f;
        }
    };
    auto aux_store = [&](int k0, const AuxRegs& x) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = k0 + 64 * j + lane;
            if (r < RW) {
                Fw[r] = x.f[j];
                sqw[r] = x.q[j];
                stw[r] = x.s0[j];
                if (SVR) {
                    stw[RW + r] = x.s1[j];
                    zw[r] = x.z[j];
                }
            }
        }
    };

    Top2 up, lo;  // this lane's best candidates of each side
    auto push = [&](int lr, double Fn) {
        const int32_t row = (int32_t)(rw0 + lr);
        const uint8_t s0 = stw[lr];
        const double r0 = SVR ? (double)zw[lr] - a.eps
                              : ((s0 & ST_YPOS) ? 1.0 : -1.0);
        const double v0 = r0 - Fn;
        if (s0 & ST_UP) up.push(v0, row);
        if (s0 & ST_LOW) lo.push(-v0, row);
        if (SVR) {
            const uint8_t s1 = stw[RW + lr];
            const double v1 = ((double)zw[lr] + a.eps) - Fn;
            if (s1 & ST_UP) up.push(v1, (int32_t)(n + row));
            if (s1 & ST_LOW) lo.push(-v1, (int32_t)(n + row));
        }
    };

    if (XS) {
        // Staged working-set rows: every slot (finite values past nS),
        // zero-filled to whole 16-feature chunks.
        const int q4 = (xstride - 4) >> 2;  // float4 per staged row
        const int xs_total = NBLK * 16 * q4;
        const Rsrc rXs = make_rsrc(a.xS, (int64_t)NBLK * 16 * ldp * 4);
        auto xs_off = [&](int e) -> uint32_t {
            const int slot = e / q4, c4 = e - slot * q4;
            return (e < xs_total && 4 * c4 < ldp)
                       ? (uint32_t)((slot * ldp + 4 * c4) * 4)
                       : kOob;
        };
        auto xs_put = [&](int e, float4 v) {
            const int slot = e / q4, c4 = e - slot * q4;
            if (e < xs_total)
                *reinterpret_cast<float4*>(xsl + slot * xstride + 4 * c4) = v;
        };

        const int nslab = (ldp + 63) >> 6;
        const Rsrc rX = make_rsrc(a.X + rw0 * ldp, (int64_t)nw * ldp * 4);
        float* wbuf = xsl + NBLK * 16 * xstride + wave * (16 * kSlabStride);
        const uint32_t step4 = (uint32_t)(16 * ldp);  // 4 rows, in bytes
        int fti = 0, fsl = 0;  // next slab to fetch
        auto fetch = [&](float4 (&v)[4]) {
            const int col = fsl * 64 + 4 * nl;
            const bool ok = fti < Tw && col < ldp;
            const uint32_t o = (uint32_t)(((16 * fti + g) * ldp + col) * 4);
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                v[rr] = bld_f4(rX, ok ? o + rr * step4 : kOob);
            if (++fsl == nslab) {
                fsl = 0;
                ++fti;
            }
        };

        // Everything the first slabs need is requested at once: the first
        // staging loads, the row data and kRing feature slabs.
        float4 xv[kXsEarly];
#pragma unroll
        for (int i = 0; i < kXsEarly; ++i)
            xv[i] = bld_f4(rXs, xs_off(tid + i * kRowThreads));
        AuxRegs ar;
        aux_issue(0, ar);
        float4 ring[kRing][4];
#pragma unroll
        for (int j = 0; j < kRing; ++j) fetch(ring[j]);
#pragma unroll
        for (int i = 0; i < kXsEarly; ++i) xs_put(tid + i * kRowThreads, xv[i]);
        aux_store(0, ar);
        for (int k0 = 256; k0 < RW; k0 += 256) {
            aux_issue(k0, ar);
            aux_store(k0, ar);
        }
        for (int e = tid + kXsEarly * kRowThreads; e < xs_total;
             e += kRowThreads)
            xs_put(e, bld_f4(rXs, xs_off(e)));
        __syncthreads();

        floatx4 acc[NBLK];
        auto epilogue = [&](int ti) {
            const int lr = 16 * ti + 4 * g;
            const float4 q4v = *reinterpret_cast<const float4*>(sqw + lr);
            const float qv[4] = {q4v.x, q4v.y, q4v.z, q4v.w};
            double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int b = 0; b < NBLK; ++b) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float kv = rbf_from_dot(qv[v], ssl[b], acc[b][v], a.gexp);
                    if (rw0 + lr + v == (int64_t)sidx[b]) kv = 1.0f;
                    part[v] = fma(cf[b], (double)kv, part[v]);
                    if (ROWS && b * 16 + nl < nS && lr + v < nw)
                        a.rows_out[(int64_t)(b * 16 + nl) * n + rw0 + lr + v] =
                            kv;
                }
            }
            const int orl = lr + (nl & 3);  // row owned by lanes nl < 4
            double Fn = 0.0;
            if (UPD || CAND) Fn = Fw[orl];
            if (UPD) {
#pragma unroll
                for (int v = 0; v < 4; ++v) part[v] = row_sum_f64(part[v]);
                Fn += pick4(part, nl & 3);
                if (nl < 4) Fw[orl] = Fn;
            }
            if (CAND && nl < 4 && orl < nw) push(orl, Fn);
        };

        int pti = 0, psl = 0;  // slab being processed
        for (int s0 = 0; s0 < Tw * nslab; s0 += kRing) {
            // all kRing slots every trip (slabs past the end are zeros and
            // touch no memory), so the loads in flight are countable
#pragma unroll
            for (int j = 0; j < kRing; ++j) {
                if (psl == 0) {
#pragma unroll
                    for (int b = 0; b < NBLK; ++b)
                        acc[b] = floatx4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    *reinterpret_cast<float4*>(
                        wbuf + (4 * rr + g) * kSlabStride + 4 * nl) =
                        ring[j][rr];
                fetch(ring[j]);  // refill the slot kRing slabs ahead
                __builtin_amdgcn_wave_barrier();
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int ch = psl * 4 + c;
                    if (ch * 16 < ldp) {  // chunk present (uniform)
                        const float4 av =
                            ld4(wbuf + nl * kSlabStride + c * 16 + 4 * g);
#pragma unroll
                        for (int b = 0; b < NBLK; ++b) {
                            const float4 bv = ld4(xsl + (b * 16 + nl) * xstride +
                                                  ch * 16 + 4 * g);
                            acc[b] = mfma_chunk(acc[b], av, bv);
                        }
                    }
                }
                __builtin_amdgcn_wave_barrier();
                if (psl == nslab - 1 && pti < Tw) epilogue(pti);
                if (++psl == nslab) {
                    psl = 0;
                    ++pti;
                }
            }
        }
        if (UPD)
            for (int r = lane; r < nw; r += 64) bst_f64(rF, 8 * r, Fw[r]);
    } else if (CAND) {
        AuxRegs ar;
        for (int k0 = 0; k0 < RW; k0 += 256) {
            aux_issue(k0, ar);
            aux_store(k0, ar);
        }
        for (int ti = 0; ti < Tw; ++ti) {
            const int orl = 16 * ti + 4 * g + (nl & 3);
            if (nl < 4 && orl < nw) push(orl, Fw[orl]);
        }
    }

    if (!CAND) return;
    // the best two of each side over this wave's rows; a variable outside
    // the global top q/2 never needs more (k_select rescans a row group
    // whose two candidates were both taken)
    const size_t wid = (size_t)blockIdx.x * kRowWaves + wave;
    wave_top2_pair(up, lo, a.cand_key + wid * 2 * kBlockTop,
                   a.cand_idx + wid * 2 * kBlockTop);
}

template <bool SVR, int NBLK, int MODE>
static void rows_dispatch(const RowArgs& a, int nblocks, hipStream_t s,
                          hipEvent_t e0, hipEvent_t e1)
{
    const size_t lds = rows_lds_bytes(NBLK, a.ldp, a.tiles, SVR);
    static size_t lds_allowed = 64 * 1024;
    if (lds > lds_allowed) {
        hipError_t e = hipFuncSetAttribute(
            (const void*)k_rows<SVR, NBLK, MODE>,
            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            throw Error{SVM_E_UNSUPPORTED,
                        "row tile needs more LDS than the device allows"};
        }
        lds_allowed = lds;
    }
    if (e0) {
        hipExtLaunchKernelGGL(k_rows<SVR, NBLK, MODE>, dim3(nblocks),
                              dim3(kRowThreads), (uint32_t)lds, s, e0, e1, 0,
                              a);
    } else {
        k_rows<SVR, NBLK, MODE><<<nblocks, kRowThreads, lds, s>>>(a);
    }
}

constexpr int kModeHot = RU_UPDATE | RU_CAND | RU_CHECK_DONE;

template <bool SVR, int NBLK>
static void rows_mode(const RowArgs& a, int nblocks, hipStream_t s,
                      hipEvent_t e0, hipEvent_t e1)
{
    switch (a.mode) {
        case kModeHot:
            rows_dispatch<SVR, NBLK, kModeHot>(a, nblocks, s, e0, e1);
            break;
        case RU_CAND:
            rows_dispatch<SVR, NBLK, RU_CAND>(a, nblocks, s, e0, e1);
            break;
        case RU_ROWS:
            rows_dispatch<SVR, NBLK, RU_ROWS>(a, nblocks, s, e0, e1);
            break;
        case RU_UPDATE:
            rows_dispatch<SVR, NBLK, RU_UPDATE>(a, nblocks, s, e0, e1);
            break;
        default: throw Error{SVM_E_INTERNAL, "bad row kernel mode"};
    }
}

template <bool SVR, int NBLK>
static int rows_occupancy(size_t lds)
{
    int bpc = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &bpc, (const void*)k_rows<SVR, NBLK, kModeHot>, kRowThreads,
            lds) != hipSuccess) {
        (void)hipGetLastError();
        return 1;
    }
    return bpc > 0 ? bpc : 1;
}

int rows_blocks_per_cu(int nblk_cols, bool svr, size_t lds)
{
    switch (nblk_cols * 2 + (svr ? 1 : 0)) {
        case 2: return rows_occupancy<false, 1>(lds);
        case 3: return rows_occupancy<true, 1>(lds);
        case 4: return rows_occupancy<false, 2>(lds);
        case 5: return rows_occupancy<true, 2>(lds);
        case 8: return rows_occupancy<false, 4>(lds);
        case 9: return rows_occupancy<true, 4>(lds);
        default: return 1;
    }
}

void launch_rows(const RowArgs& a, int nblocks, int nblk_cols, bool svr,
                 hipStream_t s, hipEvent_t e0, hipEvent_t e1)
{
    if (nblocks <= 0) return;
    // byte offsets inside one wave's rows must stay below 2^31
    if ((int64_t)16 * a.tiles * a.ldp * 4 >= ((int64_t)1 << 31))
        throw Error{SVM_E_UNSUPPORTED, "row group too large for the row kernel"};
    switch (nblk_cols * 2 + (svr ? 1 : 0)) {
        case 2: rows_mode<false, 1>(a, nblocks, s, e0, e1); break;
        case 3: rows_mode<true, 1>(a, nblocks, s, e0, e1); break;
        case 4: rows_mode<false, 2>(a, nblocks, s, e0, e1); break;
        case 5: rows_mode<true, 2>(a, nblocks, s, e0, e1); break;
        case 8: rows_mode<false, 4>(a, nblocks, s, e0, e1); break;
        case 9: rows_mode<true, 4>(a, nblocks, s, e0, e1); break;
        default: throw Error{SVM_E_INTERNAL, "bad column-block count"};
    }
}

// ---------------------------------------------------------------------------
// select / solve kernel
// ---------------------------------------------------------------------------

__device__ __forceinline__ int64_t sample_of(bool svr, int64_t t, int64_t n)
{
    return (svr && t >= n) ? t - n : t;
}

// Scores of variable t on both sides, recomputed from the responses exactly
// as k_rows computes them: up = v (t in I_up), low = -v (t in I_low).
template <bool SVR>
__device__ __forceinline__ void var_scores(const SelArgs& a, int64_t t,
                                           double& up, double& lo)
{
    const int64_t n = a.n;
    const int64_t sm = sample_of(SVR, t, n);
    const uint8_t s = a.st[t];
    double r;
    if (SVR) r = t < n ? (double)a.z[sm] - a.eps : (double)a.z[sm] + a.eps;
    else r = (s & ST_YPOS) ? 1.0 : -1.0;
    const double v = r - a.F[sm];
    up = (s & ST_UP) ? v : -INFINITY;
    lo = (s & ST_LOW) ? -v : -INFINITY;
}

// Survivor-list capacity per side of the threshold filter in k_select.
constexpr int kSurv = 1024;

// Top-`half` of entries (k[0..M), i[0..M)) by rank: entry e goes to slot
// rank(e) = #{f : f better than e}; entries are distinct (key, index) pairs
// so ranks are unique.  Run by threads [tl, tl+nt).
__device__ __forceinline__ void rank_select(const double* k, const int32_t* i,
                                            int M, int half, double* ok,
                                            int32_t* oi, int tl, int nt)
{
    for (int e = tl; e < M; e += nt) {
        const double ke = k[e];
        const int32_t ie = i[e];
        if (ke == -INFINITY) continue;
        int r = 0;
        for (int f = 0; f < M; ++f) r += better(k[f], i[f], ke, ie) ? 1 : 0;
        if (r < half) {
            ok[r] = ke;
            oi[r] = ie;
        }
    }
}

__device__ __forceinline__ int lanes_below(unsigned long long m)
{
    return __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((unsigned)m, 0));
}

// Exact top-`half` over `count` entries produced by get(e, key, index), by
// `half` block-wide rounds (each: the best entry after the previous winner).
// All threads of the block take part; thread 0 writes ok/oi.
template <class Get>
__device__ void block_rounds(int64_t count, Get get, int half, double* ok,
                             int32_t* oi, double (*rk)[kSelThreads / 64],
                             int32_t (*ri)[kSelThreads / 64])
{
    constexpr int NW = kSelThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double pk = INFINITY;
    int32_t pi = -1;
    for (int k = 0; k < half; ++k) {
        double bk = -INFINITY;
        int32_t bi = INT_MAX;
        for (int64_t e = tid; e < count; e += kSelThreads) {
            double key;
            int32_t t;
            get(e, key, t);
            if (after(key, t, pk, pi) && better(key, t, bk, bi)) {
                bk = key;
                bi = t;
            }
        }
        wave_best_fast(bk, bi);
        if (lane == 0) {
            rk[k & 1][wave] = bk;
            ri[k & 1][wave] = bi;
        }
        __syncthreads();
        bk = rk[k & 1][0];
        bi = ri[k & 1][0];
        for (int w = 1; w < NW; ++w)
            if (better(rk[k & 1][w], ri[k & 1][w], bk, bi)) {
                bk = rk[k & 1][w];
                bi = ri[k & 1][w];
            }
        pk = bk;
        pi = bi;
        if (tid == 0) {
            ok[k] = bk;
            oi[k] = bi;
        }
    }
    __syncthreads();
}

template <bool SVR, int NBLK>
__global__ __launch_bounds__(kSelThreads) void k_select(SelArgs a)
{
    WorkingSet* ws = a.ws;
    if ((a.mode & SS_CHECK_DONE) && ws->done) return;
    const uint64_t t_start = wall_clock64();

    constexpr int NW = kSelThreads / 64;
    constexpr int QS = NBLK * 16;  // slots covered by K_SS
    __shared__ double upk[kMaxHalf], lok[kMaxHalf];
    __shared__ int32_t upi[kMaxHalf], loi[kMaxHalf];
    __shared__ double rmax[2][NW * 4];
    __shared__ double theta[2];
    __shared__ double svk[2][kSurv];
    __shared__ int32_t svi[2][kSurv];
    __shared__ int32_t nsv[2];
    __shared__ int32_t exb[2][kMaxHalf];
    __shared__ int32_t nex[2];
    __shared__ double keepk[kMaxHalf];
    __shared__ int32_t keepi[kMaxHalf];
    __shared__ int32_t nkeep;
    __shared__ double rk[2][NW];
    __shared__ int32_t ri[2][NW];
    __shared__ int32_t shB[kMaxQ], shSlot[kMaxQ], shS[kMaxQ];
    __shared__ float shsS[kMaxQ];
    __shared__ float KSS[QS][QS + 1];
    __shared__ double shDc[kMaxQ];
    __shared__ int32_t shNB, shNS, shGo, shSlow;
    __shared__ double shGap;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = a.half;
    const int64_t n = a.n, ldp = a.ldp;
    const bool given = (a.mode & SS_GIVEN_B) != 0;

    if (!given) {
        // (1) the per-group candidates
        const int cnt = a.nb * kBlockTop;
        double ku[kSelPerThread], kl[kSelPerThread];
        int32_t iu[kSelPerThread], il[kSelPerThread];
#pragma unroll
        for (int j = 0; j < kSelPerThread; ++j) {
            const int e = tid + j * kSelThreads;
            if (e < cnt) {
                const int blk = e / kBlockTop, k = e - blk * kBlockTop;
                const size_t bu = (size_t)blk * 2 * kBlockTop;
                ku[j] = a.cand_key[bu + k];
                iu[j] = a.cand_idx[bu + k];
                kl[j] = a.cand_key[bu + kBlockTop + k];
                il[j] = a.cand_idx[bu + kBlockTop + k];
            } else {
                ku[j] = kl[j] = -INFINITY;
                iu[j] = il[j] = INT_MAX;
            }
        }
        // (2) maxima of every 16-lane row: distinct candidates, so the
        // half-th largest of them bounds the half-th best key from below
        double mu = -INFINITY, ml = -INFINITY;
#pragma unroll
        for (int j = 0; j < kSelPerThread; ++j) {
            mu = fmax(mu, ku[j]);
            ml = fmax(ml, kl[j]);
        }
        mu = row_max_f64(mu);
        ml = row_max_f64(ml);
        if ((lane & 15) == 0) {
            rmax[0][wave * 4 + (lane >> 4)] = mu;
            rmax[1][wave * 4 + (lane >> 4)] = ml;
        }
        if (tid < 2) nsv[tid] = 0;
        if (tid < kMaxHalf) {
            upk[tid] = lok[tid] = -INFINITY;
            upi[tid] = loi[tid] = INT_MAX;
        }
        __syncthreads();
        if (wave == 0) {
            // lane l holds row maximum l; theta = the largest x_l with at
            // least `half` row maxima >= x_l (-inf if there is none)
            for (int side = 0; side < 2; ++side) {
                const double x = rmax[side][lane];
                int c = 0;
                for (int j = 0; j < NW * 4; ++j) c += rmax[side][j] >= x;
                double th = (c >= half && x != -INFINITY) ? x : -INFINITY;
                th = fmax(fmax(rl_f64(row_max_f64(th), 0),
                               rl_f64(row_max_f64(th), 16)),
                          fmax(rl_f64(row_max_f64(th), 32),
                               rl_f64(row_max_f64(th), 48)));
                if (lane == 0) theta[side] = th;
            }
        }
        __syncthreads();
        // (3) keep the candidates at or above the bound
        {
            const double th0 = theta[0], th1 = theta[1];
#pragma unroll
            for (int j = 0; j < kSelPerThread; ++j) {
                for (int side = 0; side < 2; ++side) {
                    const double kv = side ? kl[j] : ku[j];
                    const int32_t iv = side ? il[j] : iu[j];
                    const double th = side ? th1 : th0;
                    const bool keep = kv != -INFINITY && kv >= th;
                    const unsigned long long m = __ballot(keep);
                    if (m == 0) continue;
                    int base = 0;
                    if (lane == 0) base = atomicAdd(&nsv[side], __popcll(m));
                    base = __builtin_amdgcn_readfirstlane(base);
                    const int pos = base + lanes_below(m);
                    if (keep && pos < kSurv) {
                        svk[side][pos] = kv;
                        svi[side][pos] = iv;
                    }
                }
            }
        }
        __syncthreads();
        const int M0 = nsv[0], M1 = nsv[1];
        const bool overflow = M0 > kSurv || M1 > kSurv;
        if (!overflow) {
            // (4) rank the survivors: side 0 on threads [0,512), side 1 on
            // the rest
            const int hs = kSelThreads / 2;
            if (tid < hs) rank_select(svk[0], svi[0], M0, half, upk, upi, tid, hs);
            else rank_select(svk[1], svi[1], M1, half, lok, loi, tid - hs, hs);
            __syncthreads();
        } else {
            // (4') too many ties at the bound (e.g. alpha = 0): exact block
            // rounds over all candidates
            for (int side = 0; side < 2; ++side) {
                auto get = [&](int64_t e, double& key, int32_t& t) {
                    const int64_t blk = e / kBlockTop, k = e - blk * kBlockTop;
                    const size_t o = (size_t)blk * 2 * kBlockTop +
                                     (side ? kBlockTop : 0) + k;
                    key = a.cand_key[o];
                    t = a.cand_idx[o];
                };
                block_rounds(cnt, get, half, side ? lok : upk,
                             side ? loi : upi, rk, ri);
            }
            if (tid == 0) ws->slow_selects += 1;
        }
        // (5) row groups whose whole candidate list was taken may hold
        // more: wave 0 finds them (lane-parallel)
        const uint32_t grows = (uint32_t)a.group_rows;
        if (wave == 0) {
            for (int side = 0; side < 2; ++side) {
                const double* kk = side ? lok : upk;
                const int32_t* ii = side ? loi : upi;
                const bool valid = lane < half && kk[lane] != -INFINITY;
                const int32_t b =
                    valid ? (int32_t)((uint32_t)sample_of(SVR, ii[lane], n) / grows)
                          : -1 - lane;
                int c = 0;
                bool first = true;
                for (int j = 0; j < half; ++j) {
                    const int32_t bj = rl_i32(b, j);
                    c += bj == b;
                    first &= !(j < lane && bj == b);
                }
                const bool ex = valid && c >= kBlockTop && first;
                const unsigned long long m = __ballot(ex);
                if (ex) exb[side][lanes_below(m)] = b;
                if (lane == 0) nex[side] = __popcll(m);
            }
        }
        __syncthreads();
        if (nex[0] + nex[1] > 0) {
            // (6) rare: exact block rounds over the winners outside those
            // groups plus every variable of the groups (keys from F)
            const uint32_t NV = SVR ? 2 : 1;
            for (int side = 0; side < 2; ++side) {
                const int ne = nex[side];
                if (ne == 0) continue;
                double* kk = side ? lok : upk;
                int32_t* ii = side ? loi : upi;
                if (tid == 0) {
                    int c = 0;
                    for (int k = 0; k < half; ++k) {
                        if (kk[k] == -INFINITY) continue;
                        const int32_t b =
                            (int32_t)((uint32_t)sample_of(SVR, ii[k], n) / grows);
                        bool ex = false;
                        for (int x = 0; x < ne; ++x) ex |= exb[side][x] == b;
                        if (!ex) {
                            keepk[c] = kk[k];
                            keepi[c] = ii[k];
                            ++c;
                        }
                    }
                    nkeep = c;
                }
                __syncthreads();
                const int nk = nkeep;
                const uint32_t per = grows * NV;
                auto get = [&](int64_t e, double& key, int32_t& t) {
                    if (e < nk) {
                        key = keepk[e];
                        t = keepi[e];
                        return;
                    }
                    const uint32_t q = (uint32_t)(e - nk);
                    const uint32_t x = q / per, o = q - x * per;
                    const int64_t row = (int64_t)exb[side][x] * grows + (o % grows);
                    key = -INFINITY;
                    t = INT_MAX;
                    if (row < n) {
                        const int64_t tt = o < grows ? row : n + row;
                        double u, l;
                        var_scores<SVR>(a, tt, u, l);
                        key = side ? l : u;
                        t = (int32_t)tt;
                    }
                };
                block_rounds((int64_t)nk + (int64_t)ne * per, get, half, kk, ii,
                             rk, ri);
            }
            if (tid == 0) ws->rescans += 1;
        }
    }
    const uint64_t t_merge = wall_clock64();

    // (8) working set, distinct samples (wave 0, lane-parallel)
    if (wave == 0) {
        int go = 0, nB = 0;
        double gap = 0.0;
        if (!given) {
            const bool valid = upk[0] != -INFINITY && lok[0] != -INFINITY;
            const double m = upk[0], M = -lok[0];
            gap = valid ? m - M : 0.0;
            bool build = true;
            if (a.mode & SS_SOLVE) {
                if (!valid || gap <= a.tol) {
                    if (lane == 0) ws->done = 1;
                    build = false;
                } else if (ws->iter >= a.max_iter) {
                    if (lane == 0) ws->done = 2;
                    build = false;
                }
            }
            if (lane == 0) {
                ws->gap = gap;
                ws->m = valid ? m : 0.0;
                ws->M = valid ? M : 0.0;
            }
            if (build) {
                // lanes [0,half): up list, [half,2half): low list; position
                // in the interleaved order U0 L0 U1 L1 ...
                const bool isU = lane < half;
                const bool inL = lane >= half && lane < 2 * half;
                const int k = isU ? lane : lane - half;
                const double key = isU ? upk[k] : (inL ? lok[k] : -INFINITY);
                const int32_t idx = isU ? upi[k] : (inL ? loi[k] : INT_MAX);
                bool keep = (isU || inL) && key != -INFINITY;
                if (keep) {
                    // drop a variable already placed earlier in the order
                    if (isU) {
                        for (int j = 0; j < k; ++j)
                            keep &= !(lok[j] != -INFINITY && loi[j] == idx);
                    } else {
                        for (int j = 0; j <= k; ++j)
                            keep &= !(upk[j] != -INFINITY && upi[j] == idx);
                    }
                }
                const unsigned long long m = __ballot(keep);
                const unsigned long long mu = m & ((1ull << half) - 1ull);
                const unsigned long long ml = (m >> half) & ((1ull << half) - 1ull);
                const unsigned long long below = (1ull << k) - 1ull;
                int pos = __popcll(mu & below) + __popcll(ml & below);
                if (!isU) pos += (int)((mu >> k) & 1ull);
                int32_t* dst = (a.mode & SS_SOLVE) ? shB : ws->B;
                if (keep) dst[pos] = idx;
                nB = __popcll(m);
                if (a.mode & SS_SOLVE) go = 1;
                else if (lane == 0) ws->nB = nB;
            }
        } else {
            nB = ws->nB;
            if (lane < nB) shB[lane] = ws->B[lane];
            gap = ws->gap;
            go = (a.mode & SS_SOLVE) ? 1 : 0;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        int nS = 0;
        if (go) {
            // slot of each variable: rank of the first occurrence of its
            // sample (eps-SVR: both copies of a sample share one slot)
            const bool act = lane < nB;
            const int32_t s = act ? (int32_t)sample_of(SVR, shB[lane], n) : -1;
            int firstpos = lane;
            if (SVR && act)
                for (int j = lane - 1; j >= 0; --j)
                    if ((int32_t)sample_of(SVR, shB[j], n) == s) firstpos = j;
            const unsigned long long fm = __ballot(act && firstpos == lane);
            const unsigned long long bl =
                firstpos >= 64 ? ~0ull : ((1ull << firstpos) - 1ull);
            const int slot = __popcll(fm & bl);
            if (act) {
                shSlot[lane] = slot;
                if (firstpos == lane) shS[slot] = s;
            }
            nS = __popcll(fm);
        }
        if (lane == 0) {
            shGo = go;
            shNB = nB;
            shNS = nS;
            shGap = gap;
        }
    }
    __syncthreads();
    if (!shGo) {
        if (tid == 0) ws->prof[0] += (int64_t)(t_merge - t_start);
        return;
    }
    const int nB = shNB, nS = shNS;

    // (9) state of B for the subproblem (wave 0, loads issued early)
    const bool act = wave == 0 && lane < nB;
    const int32_t t = act ? shB[lane] : INT_MAX;
    const int sl = act ? shSlot[lane] : 0;
    const int64_t sm = act ? sample_of(SVR, t, n) : 0;
    double al = act ? a.alpha[t] : 0.0;
    double yv = 1.0, rv = 0.0, v = 0.0;
    if (act) {
        if (SVR) {
            yv = t < n ? 1.0 : -1.0;
            rv = t < n ? (double)a.z[sm] - a.eps : (double)a.z[sm] + a.eps;
        } else {
            yv = (a.st[t] & ST_YPOS) ? 1.0 : -1.0;
            rv = yv;
        }
        v = rv - a.F[sm];
    }

    // (10) K_SS on the matrix cores (same operand order as k_rows) while
    // the other waves copy the working-set rows for the next k_rows
    if (wave < NBLK * NBLK) {
        const int g = lane >> 4, nl = lane & 15;
        const int bi = wave / NBLK, bj = wave - bi * NBLK;
        const int sa = bi * 16 + nl, sb = bj * 16 + nl;
        const bool va = sa < nS, vb = sb < nS;
        const float* xa = a.X + (int64_t)(va ? shS[sa] : 0) * ldp;
        const float* xb = a.X + (int64_t)(vb ? shS[sb] : 0) * ldp;
        float sqa[4];
#pragma unroll
        for (int vv = 0; vv < 4; ++vv) {
            const int ia = bi * 16 + 4 * g + vv;
            sqa[vv] = ia < nS ? a.sq[shS[ia]] : 0.0f;
        }
        const float sqb = vb ? a.sq[shS[sb]] : 0.0f;
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
        for (int64_t c0 = 0; c0 < ldp; c0 += 16) {
            const int64_t col = c0 + 4 * g;
            const bool cv = col < ldp;
            float4 av = (va && cv) ? ld4(xa + col) : zero4();
            float4 bv = (vb && cv) ? ld4(xb + col) : zero4();
            acc = mfma_chunk(acc, av, bv);
        }
#pragma unroll
        for (int vv = 0; vv < 4; ++vv) {
            const int ia = bi * 16 + 4 * g + vv, ib = bj * 16 + nl;
            if (ia < nS && ib < nS)
                KSS[ia][ib] = ia == ib ? 1.0f
                                       : rbf_from_dot(sqa[vv], sqb, acc[vv],
                                                      a.gexp);
        }
        if (bi == 0 && bj == 0 && g == 0 && vb) shsS[sb] = sqb;
        if (NBLK > 1 && bi == 0 && g == 0 && vb) shsS[sb] = sqb;
    }
    {
        // copy by the waves without a K_SS block (by every wave if all of
        // them have one)
        constexpr int GW = NBLK * NBLK < NW ? NBLK * NBLK : 0;
        if (wave >= GW) {
            const int q4 = (int)(ldp >> 2);
            const int nt = (NW - GW) * 64;
            for (int e = tid - GW * 64; e < nS * q4; e += nt) {
                const int slot = e / q4, c4 = e - slot * q4;
                *reinterpret_cast<float4*>(a.xS + (int64_t)slot * ldp +
                                           4 * c4) =
                    ld4(a.X + (int64_t)shS[slot] * ldp + 4 * c4);
            }
        }
    }
    __syncthreads();
    const uint64_t t_kss = wall_clock64();

    if (wave != 0) return;

    // (11) subproblem: maximal-violating-pair steps restricted to B
    const double a0 = al;
    if ((a.mode & SS_SET_ALPHA) && act) al = ws->alphaB[lane];
    const double C = a.C;
    const double itol = a.inner_tol_override >= 0.0
                            ? a.inner_tol_override
                            : fmax(a.inner_ratio * shGap, 0.5 * a.tol);
    int steps = 0;
    for (; steps < a.max_inner; ++steps) {
        const bool up = act && ((yv > 0 && al < C) || (yv < 0 && al > 0));
        const bool lo = act && ((yv > 0 && al > 0) || (yv < 0 && al < C));
        double bu = up ? v : -INFINITY, bl = lo ? -v : -INFINITY;
        int32_t iu = up ? t : INT_MAX, il = lo ? t : INT_MAX;
        if (NBLK == 1) {
            row_best(bu, iu);
            row_best(bl, il);
            bu = rl_f64(bu, 0);
            iu = rl_i32(iu, 0);
            bl = rl_f64(bl, 0);
            il = rl_i32(il, 0);
        } else {
            wave_best_fast(bu, iu);
            wave_best_fast(bl, il);
        }
        if (bu == -INFINITY || bl == -INFINITY) break;
        const double vi = bu, vj = -bl;
        if (!(vi - vj > itol)) break;
        const int Li =
            __ffsll((unsigned long long)__ballot(act && t == iu)) - 1;
        const int Lj =
            __ffsll((unsigned long long)__ballot(act && t == il)) - 1;
        const double ali = rl_f64(al, Li), alj = rl_f64(al, Lj);
        const double yi = rl_f64(yv, Li), yj = rl_f64(yv, Lj);
        const int si = rl_i32(sl, Li), sj = rl_i32(sl, Lj);
        const double kij = (double)KSS[si][sj];
        const double kai = (double)KSS[sl][si], kaj = (double)KSS[sl][sj];
        double a2 = (double)KSS[si][si] + (double)KSS[sj][sj] - 2.0 * kij;
        if (a2 <= 0.0) a2 = kTau;
        double s = (vi - vj) / a2;
        const double Ui = yi > 0 ? C - ali : ali;
        const double Lb = yj > 0 ? alj : C - alj;
        bool ci = false, cj = false;
        if (Ui <= s) {
            s = Ui;
            ci = true;
        }
        if (Lb <= s) {
            s = Lb;
            cj = true;
            ci = (Ui == s);
        }
        if (lane == Li) {
            al += yi * s;
            if (ci) al = yi > 0 ? C : 0.0;
        }
        if (lane == Lj) {
            al -= yj * s;
            if (cj) al = yj > 0 ? 0.0 : C;
        }
        if (act) v -= s * (kai - kaj);
    }
    const uint64_t t_inner = wall_clock64();

    if (act) ws->alphaB[lane] = al;
    if (!(a.mode & SS_NO_WRITE)) {
        if (act) {
            a.alpha[t] = al;
            a.st[t] = state_bits(yv, al, C);
        }
        shDc[lane] = act ? yv * (al - a0) : 0.0;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (lane < nS) {
            double c = 0.0;
            for (int b = 0; b < nB; ++b)
                if (shSlot[b] == lane) c += shDc[b];
            ws->coef[lane] = c;
            ws->S[lane] = shS[lane];
            ws->sS[lane] = shsS[lane];
        }
        if (act) {
            ws->B[lane] = t;
            ws->slotB[lane] = sl;
        }
        if (lane == 0) {
            ws->nB = nB;
            ws->nS = nS;
            if (!given) ws->iter += 1;
            ws->rows += nS;
        }
    }
    if (lane == 0) {
        ws->steps = steps;
        ws->inner_total += steps;
        ws->prof[0] += (int64_t)(t_merge - t_start);
        ws->prof[1] += (int64_t)(t_kss - t_merge);
        ws->prof[2] += (int64_t)(t_inner - t_kss);
        ws->prof[3] += (int64_t)(wall_clock64() - t_inner);
        ws->prof[4] += 1;
    }
}

void launch_select(const SelArgs& a, int nblk_cols, bool svr, hipStream_t s)
{
    switch (nblk_cols * 2 + (svr ? 1 : 0)) {
        case 2: k_select<false, 1><<<1, kSelThreads, 0, s>>>(a); break;
        case 3: k_select<true, 1><<<1, kSelThreads, 0, s>>>(a); break;
        case 4: k_select<false, 2><<<1, kSelThreads, 0, s>>>(a); break;
        case 5: k_select<true, 2><<<1, kSelThreads, 0, s>>>(a); break;
        case 8: k_select<false, 4><<<1, kSelThreads, 0, s>>>(a); break;
        case 9: k_select<true, 4><<<1, kSelThreads, 0, s>>>(a); break;
        default: throw Error{SVM_E_INTERNAL, "bad column-block count"};
    }
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
__global__ __launch_bounds__(1024) void k_summary(int32_t type,
                                                  const double* a,
                                                  const uint8_t* st,
                                                  const double* F,
                                                  const float* z, int64_t n,
                                                  double C, double eps,
                                                  Summary* out)
{
    __shared__ double s_v[1024], s_o[1024];
    __shared__ int64_t s_f[1024], s_b[1024];
    const int tid = threadIdx.x;
    const int64_t N = type == SVM_EPS_SVR ? 2 * n : n;
    double sv = 0.0, so = 0.0;
    int64_t nf = 0, nbd = 0;
    for (int64_t t = tid; t < N; t += 1024) {
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
    k_summary<<<1, 1024, 0, s>>>(type, a, st, F, z, n, C, eps, out);
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

__global__ void k_compact_scan(int32_t* blk_cnt, int64_t nblk,
                               int64_t* total)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int64_t acc = 0;
    for (int64_t b = 0; b < nblk; ++b) {
        int32_t c = blk_cnt[b];
        blk_cnt[b] = (int32_t)acc;
        acc += c;
    }
    *total = acc;
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
    k_compact_scan<<<1, 64, 0, s>>>(blk_cnt, nblk, count_out);
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
        if (c4 == 0) sq_out[r] = sq[src];
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
