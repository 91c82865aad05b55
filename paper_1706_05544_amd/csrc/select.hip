// Select/solve kernel of the working-set dual solve (gfx950).
//
// k_select is one block of 1024 threads per outer iteration (Section 3: pick
// a working set of 16 coefficients by the largest partial derivatives under
// the constraints and optimise them from the local gradient).  It merges the
// per-wave candidates of the previous k_rows into the global working set B
// (the q/2 largest keys of I_up interleaved with the q/2 smallest keys of
// I_low), tests the gap m - M against tol, computes the kernel block K_BB on
// the matrix cores and solves the subproblem on B with maximal-violating-pair
// steps.  It writes the new alpha_B, the state bytes, the coefficient change
// of each distinct sample and the working-set rows for the next k_rows.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.hpp"
#include "device.hpp"

namespace msvm {

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

// Top `half` of (k[0..M), i[0..M)) in the order of better(), by `half`
// rounds over one wave (entries are distinct (key, index) pairs); lane 0
// writes ok/oi.  The first 256 entries are held in registers.
__device__ void wave_top(const double* k, const int32_t* i, int M, int half,
                         double* ok, int32_t* oi)
{
    const int lane = threadIdx.x & 63;
    double ck[4];
    int32_t ci[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int e = lane + 64 * j;
        ck[j] = e < M ? k[e] : -INFINITY;
        ci[j] = e < M ? i[e] : INT_MAX;
    }
    double pk = INFINITY;
    int32_t pi = -1;
    for (int r = 0; r < half; ++r) {
        double bk = -INFINITY;
        int32_t bi = INT_MAX;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (after(ck[j], ci[j], pk, pi) && better(ck[j], ci[j], bk, bi)) {
                bk = ck[j];
                bi = ci[j];
            }
        for (int e = lane + 256; e < M; e += 64) {
            const double ke = k[e];
            const int32_t ie = i[e];
            if (after(ke, ie, pk, pi) && better(ke, ie, bk, bi)) {
                bk = ke;
                bi = ie;
            }
        }
        wave_best_fast(bk, bi);
        if (lane == 0) {
            ok[r] = bk;
            oi[r] = bi;
        }
        pk = bk;
        pi = bi;
    }
}

// Largest list (per side) ranked by pairs in one pass.
constexpr int kPairSmall = 64;

// Top `half` of each side's entries (k[s][0..M_s), i[s][0..M_s)), M_s <=
// kSelThreads / LPE, by ranks computed all at once: LPE threads share one
// entry, each compares it with a slice of the others, and a sum over the
// LPE threads gives its rank (the number of entries before it in the order
// of better(); entries are distinct, so ranks are unique).  Run by the
// whole block.
template <int LPE>
__device__ __forceinline__ void pair_rank_top(const double (*k)[kSurv],
                                              const int32_t (*i)[kSurv],
                                              int M0, int M1, int half,
                                              double* ku, int32_t* iu,
                                              double* kl, int32_t* il)
{
    constexpr int E = kSelThreads / LPE;  // entries covered
    constexpr int F = E / LPE;            // comparisons per thread
    const int tid = threadIdx.x;
    // thread (e, l) compares entry e with entries l, l + LPE, ...: the
    // LPE lanes of an entry read consecutive entries (no LDS bank
    // conflicts), and the count does not depend on the split
    const int e = tid / LPE, f0 = tid % LPE;
    // first entry of this wave: a wave whose entries are all past a side's
    // list skips that side
    const int e_wave = (tid & ~63) / LPE;
#pragma unroll
    for (int side = 0; side < 2; ++side) {
        const int M = side ? M1 : M0;
        if (e_wave >= M) continue;  // uniform over the wave
        const bool ve = e < M;
        const double ke = k[side][ve ? e : 0];
        const int32_t ie = i[side][ve ? e : 0];
        int c = 0;
#pragma unroll 8
        for (int j = 0; j < F; ++j) {
            const int f = f0 + LPE * j;
            const double kf = k[side][f];
            const int32_t iff = i[side][f];
            c += (f < M && better(kf, iff, ke, ie)) ? 1 : 0;
        }
        if (LPE == 16) {
            c = row_sum_i32(c);
        } else {
#pragma unroll
            for (int o = 1; o < LPE; o <<= 1) c += __shfl_xor(c, o);
        }
        if (ve && tid % LPE == 0 && c < half) {
            (side ? kl : ku)[c] = ke;
            (side ? il : iu)[c] = ie;
        }
    }
}

// Exact top `half` of each side's entries (k[s][0..M_s), i[s][0..M_s)),
// M_s <= kSurv, into (ku, iu) and (kl, il).  A list longer than one pair
// pass ranks cheaply is cut first: the half-th best of its first 64
// entries bounds the half-th best of the whole list from below, so the
// entries at or above it (at least `half` of them) hold the top `half`;
// they are compacted in place and ranked.  Run by the whole block; k and i
// are overwritten.
__device__ __forceinline__ void top_half(double (*k)[kSurv], int32_t (*i)[kSurv], int M0,
                         int M1, int half, double* ku, int32_t* iu, double* kl,
                         int32_t* il, int32_t* shM)
{
    const int tid = threadIdx.x, lane = tid & 63;
    if (M0 > kPairSmall || M1 > kPairSmall) {
        pair_rank_top<16>(k, i, min(M0, kPairSmall), min(M1, kPairSmall), half,
                          ku, iu, kl, il);
        if (tid < 2) shM[tid] = 0;
        __syncthreads();
        double ke[2];
        int32_t ie[2];
        bool keep[2];
#pragma unroll
        for (int side = 0; side < 2; ++side) {
            const int M = side ? M1 : M0;
            const double bk = (side ? kl : ku)[half - 1];
            const int32_t bi = (side ? il : iu)[half - 1];
            const bool in = tid < M;
            ke[side] = in ? k[side][tid] : -INFINITY;
            ie[side] = in ? i[side][tid] : INT_MAX;
            keep[side] = in && (M <= kPairSmall || !after(ke[side], ie[side], bk, bi));
        }
        __syncthreads();  // every entry read before the in-place writes
#pragma unroll
        for (int side = 0; side < 2; ++side) {
            const unsigned long long m = __ballot(keep[side]);
            if (m == 0) continue;
            int base = 0;
            if (lane == 0) base = atomicAdd(&shM[side], __popcll(m));
            base = __builtin_amdgcn_readfirstlane(base);
            if (keep[side]) {
                const int pos = base + lanes_below(m);
                k[side][pos] = ke[side];
                i[side][pos] = ie[side];
            }
        }
        __syncthreads();
        M0 = shM[0];
        M1 = shM[1];
    }
    const int lm = max(M0, M1);
    if (lm <= kPairSmall) {
        pair_rank_top<16>(k, i, M0, M1, half, ku, iu, kl, il);
    } else if (lm <= 2 * kPairSmall) {
        pair_rank_top<8>(k, i, M0, M1, half, ku, iu, kl, il);
    } else {
        const int wave = tid >> 6;
        if (wave == 0) wave_top(k[0], i[0], M0, half, ku, iu);
        if (wave == 1) wave_top(k[1], i[1], M1, half, kl, il);
    }
    __syncthreads();
}

// Exact top-`half` over `count` entries produced by get(e, key, index), by
// `half` block-wide rounds (each: the best entry after the previous winner).
// Up to kRoundRegs entries per thread are fetched once and kept in
// registers; larger counts fetch in every round.  All threads of the block
// take part; thread 0 writes ok/oi.
constexpr int kRoundRegs = 4;
template <class Get>
__device__ void block_rounds(int64_t count, Get get, int half, double* ok,
                             int32_t* oi, double (*rk)[kSelThreads / 64],
                             int32_t (*ri)[kSelThreads / 64])
{
    constexpr int NW = kSelThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool held = count <= (int64_t)kRoundRegs * kSelThreads;
    double hk[kRoundRegs];
    int32_t hi[kRoundRegs];
#pragma unroll
    for (int j = 0; j < kRoundRegs; ++j) {
        const int64_t e = tid + (int64_t)j * kSelThreads;
        hk[j] = -INFINITY;
        hi[j] = INT_MAX;
        if (held && e < count) get(e, hk[j], hi[j]);
    }
    double pk = INFINITY;
    int32_t pi = -1;
    for (int k = 0; k < half; ++k) {
        double bk = -INFINITY;
        int32_t bi = INT_MAX;
        if (held) {
#pragma unroll
            for (int j = 0; j < kRoundRegs; ++j)
                if (after(hk[j], hi[j], pk, pi) && better(hk[j], hi[j], bk, bi)) {
                    bk = hk[j];
                    bi = hi[j];
                }
        } else {
            for (int64_t e = tid; e < count; e += kSelThreads) {
                double key;
                int32_t t;
                get(e, key, t);
                if (after(key, t, pk, pi) && better(key, t, bk, bi)) {
                    bk = key;
                    bi = t;
                }
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

// Best (key, lane) of each side over a 16-lane row (NBLK = 1) or the wave,
// both sides interleaved; results are wave-uniform.  Ties go to the lowest
// lane.
template <int NBLK>
__device__ __forceinline__ void best_two_sides(double& ku, int& lu, double& kl,
                                               int& ll)
{
    if (NBLK == 1) {
        const double mu = row_max_f64(ku), ml = row_max_f64(kl);
        const int cu = row_min_i32(ku == mu ? lu : INT_MAX);
        const int cl = row_min_i32(kl == ml ? ll : INT_MAX);
        ku = rl_f64(mu, 0);
        kl = rl_f64(ml, 0);
        lu = rl_i32(cu, 0);
        ll = rl_i32(cl, 0);
    } else {
        wave_best_pair(ku, lu, kl, ll);
    }
}

// Features per LDS slice of the working-set rows in k_select.
int select_slice(int nblk_cols, int64_t ldp)
{
    const int64_t ldp16 = (ldp + 15) & ~(int64_t)15;
    const int64_t budget = 96 * 1024;  // bytes of dynamic LDS
    int64_t w = (budget / ((int64_t)nblk_cols * 16 * 4) - 4) & ~(int64_t)15;
    w = std::min<int64_t>(w, ldp16);
    return (int)std::max<int64_t>(16, w);
}

// Dynamic LDS of the CSR working set in the selection: the column index
// (ldp int32) and the by-column table ((csr_cols + 1) rows of 16 * nblk_cols
// floats).
__host__ __device__ inline size_t select_csr_lds_bytes(int nblk_cols,
                                                       int64_t ldp,
                                                       int csr_cols)
{
    return (size_t)((ldp + 3) & ~(int64_t)3) * 4 +
           (size_t)(csr_cols + 1) * nblk_cols * 16 * 4;
}

// LDS limit of the CSR working set in the selection.
constexpr size_t kSelCsrLds = 112 * 1024;

// The slots' nonzero lists (csr_cols int32 after the table: csr_cols /
// (16 nblk_cols) entries a slot) when they fit the limit besides it.
__host__ __device__ inline bool select_csr_lists(int nblk_cols, int64_t ldp,
                                                 int csr_cols)
{
    return select_csr_lds_bytes(nblk_cols, ldp, csr_cols) +
               (size_t)csr_cols * 4 <=
           kSelCsrLds;
}

static size_t select_lds_bytes(int nblk_cols, int slice)
{
    return (size_t)nblk_cols * 16 * (slice + 4) * sizeof(float);
}

// Value of the lane R places along this lane's 16-lane row (a row rotate:
// every lane has a source, so none keeps its old value); R = 1 .. 15 meet
// every other lane of the row once.  Needs the whole row active.
template <int R>
__device__ __forceinline__ int row_rot(int v)
{
    return __builtin_amdgcn_mov_dpp(v, 0x120 + R, 0xF, 0xF, false);
}

template <int R = 1, class Fn>
__device__ __forceinline__ void for_row_rotations(Fn&& fn)
{
    if constexpr (R < 16) {
        fn(std::integral_constant<int, R>{});
        // one rotation at a time (hoisting them all would hold 15 values)
        __builtin_amdgcn_sched_barrier(0);
        for_row_rotations<R + 1>(fn);
    }
}

// Exclusive scan in place of the 0/1 flags v[0..L), L <= kSelThreads, by
// the whole block (one flag a thread: a ballot and a count of the lanes
// below, no shuffle chain); returns the number of flags set.  Longer lists
// take the general block scan.
__device__ __forceinline__ int flag_exclusive_scan(int* v, int64_t L,
                                                   int* wsum)
{
    if (L > kSelThreads) return block_exclusive_scan<kSelThreads>(v, L, wsum);
    constexpr int NW = kSelThreads / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool in = tid < L;
    const unsigned long long m = __ballot(in && v[in ? tid : 0] != 0);
    if (lane == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const int x = wsum[w];
        off += w < wave ? x : 0;
        tot += x;
    }
    if (in) v[tid] = off + lanes_below(m);
    __syncthreads();
    return tot;
}

template <bool SVR, int NBLK>
__device__ __forceinline__ void select_body(const SelArgs& a)
{
    WorkingSet* ws = a.ws;
    // (SS_CHECK_DONE) ws->done is tested once the record loads are in flight
    const int32_t done0 = (a.mode & SS_CHECK_DONE) ? ws->done : 0;
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
    __shared__ double rk[2][NW];
    __shared__ int32_t ri[2][NW];
    __shared__ int32_t shB[kMaxQ], shSlot[kMaxQ], shS[kMaxQ];
    __shared__ int32_t shCandPos[kMaxQ], shSlotCand[kMaxQ];
    __shared__ int64_t shRpC[kMaxQ][2];  // CSR: row pointers of candidate c
    __shared__ float shSqCand[kMaxQ];  // squared norm of each candidate
    __shared__ int32_t shPos[kMaxQ];  // position in B of the i-th smallest
    __shared__ float shsS[kMaxQ];
    __shared__ float KSS[QS][QS + 1];
    __shared__ double shDc[kMaxQ];
    __shared__ int32_t shNB, shNS, shGo, shDone;
    __shared__ int32_t shNoList;       // CSR: a slot's row is longer than LM
    __shared__ int32_t shLen[kMaxQ];   // CSR: nonzeros of each slot's row

    __shared__ double shGap, shMx, shMn;
    extern __shared__ __align__(16) float xst[];  // QS x (slice + 4)

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = a.half;
    const int64_t n = a.n, ldp = a.ldp;
    const bool given = (a.mode & SS_GIVEN_B) != 0;
    if (given && done0) return;
    // (1) the candidate records of the row groups (best two up keys, best
    // two low keys, their variables): thread t loads records t, t +
    // kSelThreads, ... with 16-byte loads, issued before anything else
    static_assert(kBlockTop == 2, "candidate record layout");
    double ku[kSelPerThread], kl[kSelPerThread];
    int32_t iu[kSelPerThread], il[kSelPerThread];
#pragma unroll
    for (int j = 0; j < kSelRecords; ++j) {
        const int r = tid + j * kSelThreads;
        double2 k01 = make_double2(-INFINITY, -INFINITY);
        double2 k23 = k01;
        int4 ix = make_int4(INT_MAX, INT_MAX, INT_MAX, INT_MAX);
        if (!given && r < a.nb) {
            const double* rk0 = a.cand_key + 4 * (size_t)r;
            k01 = *reinterpret_cast<const double2*>(rk0);
            k23 = *reinterpret_cast<const double2*>(rk0 + 2);
            ix = *reinterpret_cast<const int4*>(a.cand_idx + 4 * (size_t)r);
        }
        ku[2 * j] = k01.x;
        ku[2 * j + 1] = k01.y;
        kl[2 * j] = k23.x;
        kl[2 * j + 1] = k23.y;
        iu[2 * j] = ix.x;
        iu[2 * j + 1] = ix.y;
        il[2 * j] = ix.z;
        il[2 * j + 1] = ix.w;
    }
    const int64_t iter0 = ws->iter;  // issued early, used in (8)
    // Counters: read now and written back once by thread 0 at the exit, so
    // that no read-modify-write of global memory waits on the way.  Global
    // stores are likewise left to the exit: a barrier after a store waits
    // for it.
    int64_t c_rows = 0, c_inner = 0, c_resc = 0, c_slow = 0;
    int64_t c_prof[12] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    // ends of the merge phases: bound, rank, exhausted groups
    uint64_t t_c1 = t_start, t_c2 = t_start, t_c3 = t_start;
    if (tid == 0) {
        c_rows = ws->rows;
        c_inner = ws->inner_total;
        c_resc = ws->rescans;
        c_slow = ws->slow_selects;
#pragma unroll
        for (int k = 0; k < 12; ++k) c_prof[k] = ws->prof[k];
    }
    if (tid == 0) shDone = 0;
    // Wave 1's cache state (used after K_SS), read now: a scalar load
    // issued later would be waited for by the next barrier, while here its
    // round trip overlaps the records'.
    const bool use_cache =
        a.cache_slots > 0 && (a.mode & SS_SOLVE) && !given && wave == 1;
    int64_t clk0 = 0, c_served = 0, c_filled = 0;
    if (use_cache) clk0 = *a.clock;
    if (wave == 1) {
        c_served = ws->cache_served;
        c_filled = ws->cache_filled;
    }
    // (7) prefetch (dense input): waves 1.. stage the first feature slice
    // of the winners' rows in LDS, row c for candidate c, and their norms,
    // while wave 0 builds the working set
    constexpr int PT = kSelThreads - 64;  // prefetching threads
    bool pf = false;  // uniform: the winners' first slice is staged
    const int ldp16 = (int)((ldp + 15) & ~(int64_t)15);
    const int pq4 = min(a.slice, ldp16) >> 2;  // float4 per row of the slice

    if (!given) {
        if (tid < kMaxHalf) {
            upk[tid] = lok[tid] = -INFINITY;
            upi[tid] = loi[tid] = INT_MAX;
        }
        if (done0) return;  // uniform over the block
        const int cnt = a.nb * kBlockTop;
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
        __syncthreads();
        if (wave < 2) {
            // wave `side`, lane l: row maximum l of that side; theta = the
            // largest x_l with at least `half` row maxima >= x_l (-inf if
            // there is none)
            {
                const int side = wave;
                const double x = rmax[side][lane];
                int c = 0;
#pragma unroll 16
                for (int j = 0; j < NW * 4; ++j) c += rmax[side][j] >= x;
                double th = (c >= half && x != -INFINITY) ? x : -INFINITY;
                th = row_max_f64(th);
                th = fmax(fmax(rl_f64(th, 0), rl_f64(th, 16)),
                          fmax(rl_f64(th, 32), rl_f64(th, 48)));
                if (lane == 0) theta[side] = th;
            }
        }
        __syncthreads();
        t_c1 = wall_clock64();
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
            // (4) rank the survivors: side 0 on threads [0,512), side 1
            // on the rest
            top_half(svk, svi, M0, M1, half, upk, upi, lok, loi, nsv);
        } else {
            // (4') too many ties at the bound (e.g. alpha = 0): exact
            // block rounds over all candidates
            for (int side = 0; side < 2; ++side) {
                auto get = [&](int64_t e, double& key, int32_t& t) {
                    const int64_t blk = e / kBlockTop,
                                  k = e - blk * kBlockTop;
                    const size_t o = (size_t)blk * 2 * kBlockTop +
                                     (side ? kBlockTop : 0) + k;
                    key = a.cand_key[o];
                    t = a.cand_idx[o];
                };
                block_rounds(cnt, get, half, side ? lok : upk,
                             side ? loi : upi, rk, ri);
            }
            if (tid == 0) c_slow += 1;
        }
        t_c2 = wall_clock64();
        // (5) row groups whose whole candidate list was taken may hold
        // more: wave 0 finds them (lane-parallel).  Group b (k_rows block
        // b) holds the units [b TU / nb, (b + 1) TU / nb) of the TU units
        // of 32 rows; it has at most grows rows.
        const uint32_t grows = (uint32_t)a.group_rows;
        int32_t wgrp = -1;  // wave 0: the group of this lane's winner
        const int64_t TU = (n + 31) >> 5, NB = a.nb;
        // group of a row: floor(((row / 32 + 1) NB - 1) / TU), through an
        // fp64 quotient corrected to the exact integer
        auto group_of = [&](int64_t row) -> int32_t {
            const int64_t x = ((row >> 5) + 1) * NB - 1;
            int64_t g = (int64_t)((double)x / (double)TU);
            if (g * TU > x) --g;
            else if ((g + 1) * TU <= x) ++g;
            return (int32_t)g;
        };
        auto group_start = [&](int64_t b) -> int64_t {
            return 32 * (b * TU / NB);
        };
        if (wave == 0) {
            // lanes [0, 32): the up winners, [32, 64): the low winners
            const int side = lane >> 5, k = lane & 31;
            const double* kk = side ? lok : upk;
            const int32_t* ii = side ? loi : upi;
            const bool valid = k < half && kk[k] != -INFINITY;
            const int32_t b =
                valid ? group_of(sample_of(SVR, ii[k], n)) : -1 - lane;
            wgrp = b;
            int c = 0;
            bool first = true;
            if (half <= 16) {
                // a side's winners sit in one 16-lane row (rows 0 and 2):
                // the row rotations meet every other winner of the side
                uint32_t same = k < half ? (1u << k) : 0u;
                for_row_rotations([&](auto r) {
                    constexpr int R = decltype(r)::value;
                    const int m = row_rot<R>(lane & 15);
                    const int32_t bm = row_rot<R>(b);
                    same |= (m < half && bm == b) ? (1u << m) : 0u;
                });
                c = __popc(same);
                first = (same & ((1u << k) - 1u)) == 0u;
            } else {
                for (int j = 0; j < half; ++j) {
                    const int32_t bu = rl_i32(b, j), bl = rl_i32(b, 32 + j);
                    const int32_t bj = side ? bl : bu;
                    c += bj == b;
                    first &= !(j < k && bj == b);
                }
            }
            const bool ex = valid && c >= kBlockTop && first;
            const unsigned long long m = __ballot(ex);
            const unsigned long long ms = side ? (m >> 32) : (m & 0xffffffffull);
            if (ex) exb[side][__popcll(ms & ((1ull << k) - 1ull))] = b;
            if (k == 0) nex[side] = __popcll(ms);
        }
        __syncthreads();
        t_c3 = wall_clock64();
        if (nex[0] + nex[1] > 0) {
            // (6) rare: the exact best `half` of the winners outside those
            // groups plus every variable of the groups (keys from F); a
            // side without such groups keeps its winners.  Staged and
            // ranked like the survivors when they fit, else by rounds.
            const uint32_t NV = SVR ? 2 : 1;
            const uint32_t per = grows * NV;
            if (wave == 0) {
                // the winners outside the exhausted groups, in order (lane
                // layout and groups as in (5))
                const int side = lane >> 5, k = lane & 31;
                const int ne = nex[side];
                const double* kk = side ? lok : upk;
                const int32_t* ii = side ? loi : upi;
                const bool valid = k < half && kk[k] != -INFINITY;
                bool ex = false;
                for (int x = 0; x < ne; ++x) ex |= exb[side][x] == wgrp;
                const bool keep = valid && !ex;
                const unsigned long long m = __ballot(keep);
                const unsigned long long ms =
                    side ? (m >> 32) : (m & 0xffffffffull);
                if (keep) {
                    const int pos = __popcll(ms & ((1ull << k) - 1ull));
                    svk[side][pos] = kk[k];
                    svi[side][pos] = ii[k];
                }
                if (k == 0) nsv[side] = __popcll(ms);
            }
            __syncthreads();
            const int nk0 = nsv[0], nk1 = nsv[1];
            const int64_t tot0 = nk0 + (int64_t)nex[0] * per;
            const int64_t tot1 = nk1 + (int64_t)nex[1] * per;
            // variable e - nk of the exhausted groups of a side
            auto group_var = [&](int side, int64_t q, double& key,
                                 int32_t& t) {
                const uint32_t x = (uint32_t)(q / per),
                               o = (uint32_t)(q - (int64_t)x * per);
                const int64_t b = exb[side][x];
                const int64_t row = group_start(b) + (o % grows);
                key = -INFINITY;
                t = INT_MAX;
                if (row < min(n, group_start(b + 1))) {
                    const int64_t tt = o < grows ? row : n + row;
                    double u, l;
                    var_scores<SVR>(a, tt, u, l);
                    key = side ? l : u;
                    t = (int32_t)tt;
                }
            };
            if (tot0 <= kSurv && tot1 <= kSurv) {
#pragma unroll
                for (int side = 0; side < 2; ++side) {
                    const int nk = side ? nk1 : nk0;
                    const int64_t tot = side ? tot1 : tot0;
                    if (tid >= nk && tid < tot) {
                        double key;
                        int32_t t;
                        group_var(side, tid - nk, key, t);
                        svk[side][tid] = key;
                        svi[side][tid] = t;
                    }
                }
                __syncthreads();
                top_half(svk, svi, (int)tot0, (int)tot1, half, upk, upi, lok,
                         loi, nsv);
            } else {
                for (int side = 0; side < 2; ++side) {
                    if (nex[side] == 0) continue;
                    const int nk = side ? nk1 : nk0;
                    if (tid < nk) {
                        keepk[tid] = svk[side][tid];
                        keepi[tid] = svi[side][tid];
                    }
                    __syncthreads();
                    auto get = [&](int64_t e, double& key, int32_t& t) {
                        if (e < nk) {
                            key = keepk[e];
                            t = keepi[e];
                        } else {
                            group_var(side, e - nk, key, t);
                        }
                    };
                    block_rounds(side ? tot1 : tot0, get, half,
                                 side ? lok : upk, side ? loi : upi, rk, ri);
                }
            }
            if (tid == 0) c_resc += 1;
        }
    }
    const uint64_t t_merge = wall_clock64();

    // CSR input: wave 1 reads the row pointers of the winners (candidate
    // c: up winner c for c < half, else low winner c - half) while wave 0
    // builds the working set, so that the staging of the working-set rows
    // starts from them
    const bool pfr = !given && a.rp && (a.mode & SS_SOLVE);  // uniform
    if (pfr && wave == 1 && lane < 2 * half) {
        const int c = lane;
        const double key = c < half ? upk[c] : lok[c - half];
        const int32_t idx = c < half ? upi[c] : loi[c - half];
        const int64_t smp =
            key != -INFINITY ? sample_of(SVR, idx, n) : 0;
        const int64_t r0 = a.rp[smp], r1 = a.rp[smp + 1];
        shRpC[c][0] = r0;
        shRpC[c][1] = r1;
    }
    // candidate c: up winner c (c < half) or low winner c - half
    pf = !given && !a.rp && (a.mode & SS_SOLVE) && 2 * half * pq4 <= 4 * PT;
    if (pf && wave != 0) {
        const int pwst = a.slice + 4;
        float4 xv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = tid - 64 + j * PT;
            const bool in = e < 2 * half * pq4;
            const int c = in ? e / pq4 : 0;
            const int c4 = e - c * pq4;
            const double key = c < half ? upk[c] : lok[c - half];
            const int32_t idx = c < half ? upi[c] : loi[c - half];
            const bool ok = in && key != -INFINITY && 4 * c4 < ldp;
            // unconditional loads (an address inside X when unused)
            xv[j] = ld4(a.X + (ok ? sample_of(SVR, idx, n) * ldp + 4 * c4 : 0));
            if (!ok) xv[j] = zero4();
        }
        float q = 0.0f;
        const int cq = tid - 64;
        if (cq < 2 * half) {
            const int32_t idx = cq < half ? upi[cq] : loi[cq - half];
            const bool ok = (cq < half ? upk[cq] : lok[cq - half]) != -INFINITY;
            q = a.sq[ok ? sample_of(SVR, idx, n) : 0];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = tid - 64 + j * PT;
            if (e < 2 * half * pq4) {
                const int c = e / pq4, c4 = e - c * pq4;
                *reinterpret_cast<float4*>(xst + c * pwst + 4 * c4) = xv[j];
            }
        }
        if (cq < 2 * half) shSqCand[cq] = q;
    }

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
                    if (lane == 0) shDone = 1;
                    build = false;
                } else if (iter0 >= a.max_iter) {
                    if (lane == 0) shDone = 2;
                    build = false;
                }
            }
            if (lane == 0) {
                shMx = valid ? m : 0.0;
                shMn = valid ? M : 0.0;
            }
            if (build) {
                // lanes [0,half): up list, [half,2half): low list; position
                // in the interleaved order U0 L0 U1 L1 ...
                const bool isU = lane < half;
                const bool inL = lane >= half && lane < 2 * half;
                const int k = isU ? lane : lane - half;
                const double key = isU ? upk[k] : (inL ? lok[k] : -INFINITY);
                const bool ent = (isU || inL) && key != -INFINITY;
                const int32_t idx =
                    ent ? (isU ? upi[k] : loi[k]) : INT_MAX;  // none: no match
                bool keep = ent;
                // drop a variable already placed earlier in the order: up
                // entry k follows low entries 0..k-1, low entry k follows up
                // entries 0..k (entries compared through registers)
                if (2 * half <= 16) {
                    // both lists in the first 16-lane row: each lane meets
                    // every other entry by the 15 row rotations (no chain
                    // of readlanes)
                    int dup = 0;
                    const int lo = isU ? half : 0;  // partners it checks:
                    const int hi = isU ? half + k : k + 1;  // lanes [lo, hi)
                    for_row_rotations([&](auto r) {
                        constexpr int R = decltype(r)::value;
                        const int m = row_rot<R>(lane & 15);
                        const int32_t im = row_rot<R>(idx);
                        dup |= (m >= lo && m < hi && im == idx) ? 1 : 0;
                    });
                    if (dup) keep = false;
                } else {
                    for (int j = 0; j < half; ++j) {
                        const int32_t uj = rl_i32(idx, j),
                                      lj = rl_i32(idx, half + j);
                        if (isU && j < k && lj == idx) keep = false;
                        if (inL && j <= k && uj == idx) keep = false;
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
                if (lane < 2 * half) shCandPos[lane] = keep ? pos : -1;
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
        __builtin_amdgcn_wave_barrier();
        int nS = 0;
        if (go) {
            // slot of each variable: rank of the first occurrence of its
            // sample (eps-SVR: both copies of a sample share one slot)
            const bool act = lane < nB;
            const int32_t t = act ? shB[lane] : INT_MAX;
            const int32_t s = act ? (int32_t)sample_of(SVR, t, n) : -1;
            int firstpos = lane;
            const bool row16 = nB <= 16;  // B in the first 16-lane row
            if (SVR && row16) {
                // the lanes of B holding the same sample, by row rotations
                uint32_t same = 0;
                for_row_rotations([&](auto r) {
                    constexpr int R = decltype(r)::value;
                    const int m = row_rot<R>(lane & 15);
                    const int32_t sm = row_rot<R>(s);
                    same |= (m < nB && sm == s) ? (1u << m) : 0u;
                });
                if (act) firstpos = __builtin_ctz(same | (1u << lane));
            } else if (SVR) {
                for (int j = 0; j < nB; ++j) {
                    const int32_t sj = rl_i32(s, j);
                    if (act && j < firstpos && sj == s) firstpos = j;
                }
            }
            const unsigned long long fm = __ballot(act && firstpos == lane);
            const unsigned long long bl =
                firstpos >= 64 ? ~0ull : ((1ull << firstpos) - 1ull);
            const int slot = __popcll(fm & bl);
            // order of the variable among B by index (the subproblem runs
            // its variables in increasing index order: lowest lane = lowest
            // index on ties)
            int p = 0;
            if (row16) {
                for_row_rotations([&](auto r) {
                    constexpr int R = decltype(r)::value;
                    const int m = row_rot<R>(lane & 15);
                    const int32_t tm = row_rot<R>(t);
                    p += (m < nB && tm < t) ? 1 : 0;
                });
            } else {
                for (int j = 0; j < nB; ++j) p += rl_i32(t, j) < t ? 1 : 0;
            }
            if (act) {
                shSlot[lane] = slot;
                if (firstpos == lane) shS[slot] = s;
                shPos[p] = lane;
            }
            nS = __popcll(fm);
            __builtin_amdgcn_wave_barrier();
            if (!given && lane < 2 * half) {
                // a candidate of each slot (twins of one sample: either)
                const int cp = shCandPos[lane];
                if (cp >= 0) shSlotCand[shSlot[cp]] = lane;
            }
        }
        if (lane == 0) {
            shGo = go;
            shNB = nB;
            shNS = nS;
            shGap = gap;
        }
    }
    __syncthreads();
    const uint64_t t_build = wall_clock64();
    // state written at every exit (threads 0 and 1)
    auto finish = [&](int64_t t_end) {
        if (tid == 0) {
            if (!given) {
                if (shDone) ws->done = shDone;
                ws->gap = shGap;
                ws->m = shMx;
                ws->M = shMn;
            }
            ws->slow_selects = c_slow;
            ws->rescans = c_resc;
            (void)t_end;
        }
    };
    if (!shGo) {
        finish(0);
        if (tid == 0) ws->prof[0] = c_prof[0] + (int64_t)(t_merge - t_start);
        return;
    }
    const int nB = shNB, nS = shNS;

    // (9) state of B for the subproblem (wave 0, loads issued early).  The
    // variable of rank p by index sits in lane p; with q <= 16 it sits in
    // lane p of both row 0 (its up side) and row 1 (its low side), so that
    // one row reduction serves both sides of a step.
    constexpr bool DUP = NBLK == 1;
    const int p = DUP ? (lane & 15) : lane;
    const int prow = lane >> 4;
    const bool act = wave == 0 && p < nB && (!DUP || prow < 2);
    const bool own = act && (!DUP || prow == 0);  // writes the results
    const int bpos = act ? shPos[p] : 0;          // position in B
    const int32_t t = act ? shB[bpos] : INT_MAX;
    const int sl = act ? shSlot[bpos] : 0;
    const int64_t sm = act ? sample_of(SVR, t, n) : 0;
    // The state of B is loaded here and used only by the subproblem: the
    // loads are unconditional (index 0 for lanes without a variable) and
    // their values pass an empty asm at the subproblem, so that the
    // compiler neither branches around them nor computes from them early
    // (either makes wave 0 wait for them before the next barrier).
    const int64_t t_l = act ? t : 0, sm_l = act ? sm : 0;
    double al_b = a.alpha[t_l];
    double F_b = a.F[sm_l];
    float z_b = SVR ? a.z[sm_l] : 0.0f;
    uint32_t st_b = SVR ? 0u : (uint32_t)a.st[t_l];

    uint64_t t_stage = 0;
    // Kernel-row cache (wave 1): the slot of each working-set sample,
    // looked up while the working-set rows load.
    int32_t hslot = -1;
    if (use_cache && lane < nS) hslot = a.slot_of[shS[lane]];

    // (10) K_SS.  CSR input: the working set by column (below).  Dense input: on the matrix cores (same operand
    // order as k_rows): the working-set rows pass through LDS in feature
    // slices: every thread loads a piece into LDS; then the NBLK^2
    // matrix-core waves accumulate the slice while the other waves copy it
    // to xS (the rows of the next k_rows).
    int csrE = 0;  // CSR: the columns of the working set's table
    if (a.rp) {
        // CSR: the working set by column.  cidx[c] flags, then numbers in
        // increasing column order, the columns some sample holds; tab[e *
        // QS + s] = x_s[column e].  K_SS sums over the columns in that
        // order, the products that involve a zero adding nothing: these
        // are the row kernel's sums over the nonzeros of sample ia, bit for
        // bit.  The table (padded with zero rows to csr_cols + 1) also goes
        // to the row kernel.
        int* cidx = reinterpret_cast<int*>(xst);
        float* tab = xst + ((ldp + 3) & ~(int64_t)3);
        const int CC = a.csr_cols;
        // Per slot, the table rows of its nonzeros in column order (LM
        // entries a slot): K_SS[a][b] then runs over the nonzeros of sample
        // a, the row kernel's own fma sequence for row a and slot b, instead
        // of over every column of the table.  Used when every slot's row
        // fits LM entries (csr_cols = 16 nblk_cols x the longest row when
        // that is below d).
        const int LM = CC / QS;
        int* lst = reinterpret_cast<int*>(tab + (int64_t)(CC + 1) * QS);
        const bool lfit = select_csr_lists(NBLK, ldp, CC) && LM > 0;
        if (tid == 0) shNoList = lfit ? 0 : 1;
        for (int64_t c = tid; c < ldp; c += kSelThreads) cidx[c] = 0;
        for (int64_t e = tid; e < (int64_t)(CC + 1) * QS; e += kSelThreads)
            tab[e] = 0.0f;
        // sample rows: a wave per slot (two at most: nS <= 32), the first
        // 256 nonzeros of a row held in registers from one load round,
        // the rest of a longer row loaded again where needed
        static_assert(NW * 2 >= 32, "two CSR slots per wave");
        int32_t hc[2][4];
        float hv[2][4];
        int64_t hp0[2], hp1[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int slot = wave + k * NW;
            if (pfr) {
                // those of a candidate of the slot, read during the build
                const int c = slot < nS ? shSlotCand[slot] : 0;
                hp0[k] = slot < nS ? shRpC[c][0] : 0;
                hp1[k] = slot < nS ? shRpC[c][1] : hp0[k];
            } else {
                const int64_t smp = slot < nS ? shS[slot] : 0;
                hp0[k] = a.rp[smp];
                hp1[k] = slot < nS ? a.rp[smp + 1] : hp0[k];
            }
        }
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t q = hp0[k] + lane + 64 * j;
                hc[k][j] = q < hp1[k] ? a.ci[q] : 0;
                hv[k][j] = q < hp1[k] ? a.cv[q] : 0.0f;
            }
        auto for_rest = [&](auto fn) {  // nonzeros past the first 256
#pragma unroll
            for (int k = 0; k < 2; ++k)
                for (int64_t q = hp0[k] + 256 + lane; q < hp1[k]; q += 64)
                    fn(wave + k * NW, a.ci[q], a.cv[q]);
        };
        float sqa = 0.0f, sqb = 0.0f;
        if (tid < nS * nS) {
            const int ia = tid / nS, ib = tid - ia * nS;
            sqa = a.sq[shS[ia]];
            sqb = a.sq[shS[ib]];
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 2; ++k) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (hp0[k] + lane + 64 * j < hp1[k]) cidx[hc[k][j]] = 1;
            const int slot = wave + k * NW;
            if (lane == 0 && slot < nS) {
                shLen[slot] = (int32_t)(hp1[k] - hp0[k]);
                if (hp1[k] - hp0[k] > LM) shNoList = 1;
            }
        }
        for_rest([&](int, int32_t c, float) { cidx[c] = 1; });
        __syncthreads();
        const int E = flag_exclusive_scan(cidx, ldp, ri[0]);
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (hp0[k] + lane + 64 * j < hp1[k])
                    tab[(int64_t)cidx[hc[k][j]] * QS + wave + k * NW] = hv[k][j];
        for_rest([&](int slot, int32_t c, float v) {
            tab[(int64_t)cidx[c] * QS + slot] = v;
        });
        const bool lists = shNoList == 0;  // uniform: set before a barrier
        if (lists) {
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int slot = wave + k * NW;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t q = hp0[k] + lane + 64 * j;
                    if (q < hp1[k])
                        lst[slot * LM + (int)(q - hp0[k])] = cidx[hc[k][j]];
                }
                for (int64_t q = hp0[k] + 256 + lane; q < hp1[k]; q += 64)
                    lst[slot * LM + (int)(q - hp0[k])] = cidx[a.ci[q]];
            }
        }
        __syncthreads();
        for (int e = tid; e < nS * nS; e += kSelThreads) {
            const int ia = e / nS, ib = e - ia * nS;
            float k = 1.0f;
            if ((ia != ib || !kernel_self_is_one(a.kf)) && lists) {
                // over the nonzeros of sample ia in column order: the row
                // kernel's fma sequence for row ia and slot ib (eight
                // nonzeros' loads issued ahead of their fmas)
                const int* la = lst + ia * LM;
                const int na = shLen[ia];
                float acc = 0.0f;
                int j = 0;
                for (; j + 8 <= na; j += 8) {
                    int e8[8];
                    float va[8], vb[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) e8[u] = la[j + u];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        va[u] = tab[e8[u] * QS + ia];
                        vb[u] = tab[e8[u] * QS + ib];
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) acc = fmaf(va[u], vb[u], acc);
                }
                for (; j < na; ++j) {
                    const int r = la[j];
                    acc = fmaf(tab[r * QS + ia], tab[r * QS + ib], acc);
                }
                const float qa = e == tid ? sqa : a.sq[shS[ia]];
                const float qb = e == tid ? sqb : a.sq[shS[ib]];
                k = kernel_from_dot(a.kf, qa, qb, acc);
            } else if (ia != ib || !kernel_self_is_one(a.kf)) {
                // the sum in column order (the row kernel's order), eight
                // columns' loads issued ahead of their fmas
                float acc = 0.0f;
                int r = 0;
                for (; r + 8 <= E; r += 8) {
                    float va[8], vb[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        va[u] = tab[(r + u) * QS + ia];
                        vb[u] = tab[(r + u) * QS + ib];
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) acc = fmaf(va[u], vb[u], acc);
                }
                for (; r < E; ++r)
                    acc = fmaf(tab[r * QS + ia], tab[r * QS + ib], acc);
                const float qa = e == tid ? sqa : a.sq[shS[ia]];
                const float qb = e == tid ? sqb : a.sq[shS[ib]];
                k = kernel_from_dot(a.kf, qa, qb, acc);
            }
            KSS[ia][ib] = k;
        }
        // (the table and its columns go to the row kernel after the last
        // barrier, from the waves that do not solve: a barrier waits for
        // the stores before it)
        csrE = E;
        // norm of slot tid: the sqb of pair (0, tid), loaded above
        if (tid < nS) shsS[tid] = sqb;
        t_stage = wall_clock64();
    } else {
        const int g = lane >> 4, nl = lane & 15;
        const int bi = wave / NBLK, bj = wave - bi * NBLK;
        const int sa = bi * 16 + nl, sb = bj * 16 + nl;
        const bool mw = wave < NBLK * NBLK;
        const bool va = mw && sa < nS, vb = mw && sb < nS;
        float sqa[4] = {0.f, 0.f, 0.f, 0.f};
        float sqb = 0.f;
        if (mw && !pf) {
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) {
                const int ia = bi * 16 + 4 * g + vv;
                sqa[vv] = a.sq[ia < nS ? shS[ia] : 0];
            }
            sqb = a.sq[vb ? shS[sb] : 0];
        }
        const int W = a.slice, wst = W + 4;
        // copy waves: those without a K_SS block, or all of them.  With a
        // single slice the copy waits until after the last barrier (waves
        // 1.. copy while wave 0 solves), so that no barrier waits for it.
        constexpr int GW = NBLK * NBLK < NW ? NBLK * NBLK : 0;
        const bool one_slice = W >= ldp16;
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
        t_stage = wall_clock64();
        for (int c0 = 0; c0 < ldp16; c0 += W) {
            const int wc = min(W, ldp16 - c0), q4 = wc >> 2, tot = nS * q4;
            // the first slice is staged already when prefetched (LDS row
            // of a slot: that of a candidate of it)
            const bool bycand = c0 == 0 && pf;
            for (int e0 = tid; e0 < tot && !bycand; e0 += 4 * kSelThreads) {
                float4 xv[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int e = e0 + j * kSelThreads;
                    const bool in = e < tot;
                    const int slot = in ? e / q4 : 0;
                    const int c4 = e - slot * q4;
                    const int64_t col = c0 + 4 * c4;
                    const bool ok = in && col < ldp;
                    // unconditional loads (an address inside X when unused)
                    xv[j] = ld4(a.X + (ok ? (int64_t)shS[slot] * ldp + col : 0));
                    if (!ok) xv[j] = zero4();
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int e = e0 + j * kSelThreads;
                    if (e < tot) {
                        const int slot = e / q4, c4 = e - slot * q4;
                        *reinterpret_cast<float4*>(xst + slot * wst + 4 * c4) =
                            xv[j];
                    }
                }
            }
            __syncthreads();
            if (c0 == 0) {
                t_stage = wall_clock64();
                if (mw && pf) {
#pragma unroll
                    for (int vv = 0; vv < 4; ++vv) {
                        const int ia = bi * 16 + 4 * g + vv;
                        sqa[vv] = shSqCand[shSlotCand[ia < nS ? ia : 0]];
                    }
                    sqb = shSqCand[shSlotCand[vb ? sb : 0]];
                }
            }
            if (mw) {
                const int ra = bycand ? shSlotCand[va ? sa : 0] : sa;
                const int rb = bycand ? shSlotCand[vb ? sb : 0] : sb;
                for (int cc = 0; cc < wc; cc += 16) {
                    float4 av = ld4(xst + ra * wst + cc + 4 * g);
                    float4 bv = ld4(xst + rb * wst + cc + 4 * g);
                    if (!va) av = zero4();
                    if (!vb) bv = zero4();
                    acc = mfma_chunk(acc, av, bv);
                }
            }
            if (!one_slice) {
                if (wave >= GW) {
                    for (int e = tid - GW * 64; e < tot;
                         e += kSelThreads - GW * 64) {
                        const int slot = e / q4, c4 = e - slot * q4;
                        const int64_t col = c0 + 4 * c4;
                        if (col < ldp)
                            *reinterpret_cast<float4*>(
                                a.xS + (int64_t)slot * ldp + col) =
                                ld4(xst +
                                    (bycand ? shSlotCand[slot] : slot) * wst +
                                    4 * c4);
                    }
                }
                __syncthreads();
            }
        }
        if (mw) {
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) {
                const int ia = bi * 16 + 4 * g + vv, ib = bj * 16 + nl;
                if (ia < nS && ib < nS)
                    KSS[ia][ib] = (ia == ib && kernel_self_is_one(a.kf))
                                      ? 1.0f
                                      : kernel_from_dot(a.kf, sqa[vv], sqb,
                                                        acc[vv]);
            }
            if (bi == 0 && g == 0 && vb) shsS[sb] = sqb;
        }
    }
    __syncthreads();
    const uint64_t t_kss = wall_clock64();

    if (wave != 0) {
        if (wave == 1 && (a.mode & SS_SOLVE) && !given) {
            // The path of this iteration's row kernel (while wave 0
            // solves): a working set whose samples are all cached is served
            // from the cache; otherwise each missing sample gets a slot
            // (FIFO, never a slot this working set reads) and the row
            // kernel fills it.
            int path = PATH_STREAM, nfill = 0;
            int32_t cslot = -1;
            if (use_cache) {
                const int32_t hs = lane < nS ? hslot : -2;
                const unsigned long long missm = __ballot(lane < nS && hs < 0);
                int64_t clk = clk0;
                // rows stop going to a cache that serves almost nothing (a
                // working set whose samples rarely all recur): the fills
                // cost HBM writes and the two paths give the same bits.  A
                // cache with a slot for every sample never evicts, so it
                // keeps filling: every working set whose samples have all
                // been used before is then served.
                const bool fill = a.cache_slots >= a.n || iter0 < 512 ||
                                  c_served * 8 >= c_filled;
                if (missm == 0) {
                    path = PATH_CACHED;
                    cslot = hs;
                } else if (fill) {
                    path = PATH_INSERT;
                    unsigned long long mm = missm;
                    while (mm) {
                        const int k = __ffsll(mm) - 1;
                        mm &= mm - 1;
                        int32_t v;
                        do {
                            v = (int32_t)clk;
                            clk = clk + 1 >= a.cache_slots ? 0 : clk + 1;
                        } while (__ballot(lane < nS && hs == v) != 0);
                        if (lane == k) cslot = v;
                    }
                    nfill = __popcll(missm);
                    if (lane < nS && cslot >= 0) {
                        const int32_t smp = shS[lane];
                        const int32_t old = a.owner[cslot];
                        if (old >= 0) a.slot_of[old] = -1;
                        a.owner[cslot] = smp;
                        a.slot_of[smp] = cslot;
                    }
                    if (lane == 0) *a.clock = clk;
                }
            }
            if (lane < nS) ws->cslot[lane] = cslot;
            if (lane == 0) {
                ws->path = path;
                const int64_t t = (iter0 + 1) % kPathLog;
                ws->path_log[t] = (uint8_t)path;
                ws->fill_log[t] = (uint8_t)nfill;
                ws->ns_log[t] = (uint8_t)nS;
                ws->cache_served = c_served + (path == PATH_CACHED ? nS : 0);
                ws->cache_filled = c_filled + nfill;
            }
        }
        if (a.rp && a.xsc) {
            // the CSR table and its columns for the row kernel (cidx and
            // tab are still in LDS)
            const int* cidx = reinterpret_cast<const int*>(xst);
            const float* tab = xst + ((ldp + 3) & ~(int64_t)3);
            const int CC = a.csr_cols, E = csrE;
            constexpr int CT = kSelThreads - 64;  // copying threads
            for (int64_t c = tid - 64; c < ldp; c += CT) {
                const int e = cidx[c];
                const bool used = (c + 1 < ldp ? cidx[c + 1] : E) > e;
                if (used && e < CC) a.xsc_cols[e] = (int32_t)c;
            }
            for (int e = E + tid - 64; e < CC; e += CT) a.xsc_cols[e] = -1;
            const int64_t n4 = (int64_t)(CC + 1) * QS / 4;
            for (int64_t e = tid - 64; e < n4; e += CT)
                *reinterpret_cast<float4*>(a.xsc + 4 * e) = ld4(tab + 4 * e);
        }
        const int ldp16 = (int)((ldp + 15) & ~(int64_t)15);
        const int W = a.slice;
        if (!a.rp && W >= ldp16) {
            const int q4 = ldp16 >> 2, wst = W + 4;
            for (int e = tid - 64; e < nS * q4; e += kSelThreads - 64) {
                const int slot = e / q4, c4 = e - slot * q4;
                const int64_t col = 4 * c4;
                if (col < ldp)
                    *reinterpret_cast<float4*>(a.xS + (int64_t)slot * ldp +
                                               col) =
                        ld4(xst + (pf ? shSlotCand[slot] : slot) * wst + 4 * c4);
            }
        }
        return;
    }

    // (11) subproblem: maximal-violating-pair steps restricted to B
    asm volatile("" : "+v"(al_b), "+v"(F_b), "+v"(z_b), "+v"(st_b));
    double al = act ? al_b : 0.0;
    double yv = 1.0, rv = 0.0, v = 0.0;
    if (act) {
        if (SVR) {
            yv = t < n ? 1.0 : -1.0;
            rv = t < n ? (double)z_b - a.eps : (double)z_b + a.eps;
        } else {
            yv = (st_b & ST_YPOS) ? 1.0 : -1.0;
            rv = yv;
        }
        v = rv - F_b;
    }
    const double a0 = al;
    if ((a.mode & SS_SET_ALPHA) && act) al = ws->alphaB[bpos];
    const double C = a.C;
    const double itol = a.inner_tol_override >= 0.0
                            ? a.inner_tol_override
                            : fmax(a.inner_ratio * shGap, 0.5 * a.tol);
    // q <= 16: each lane holds the K_SS row of its slot in registers, and
    // a step takes K(s, s_i), K(s, s_j) from there (uniform register
    // index) and K_ii, K_jj, K_ij from lanes i and j: the same stored
    // values as the LDS reads, without an LDS round trip on the step's
    // chain
    float krow[DUP ? QS : 1];
    if (DUP) {
#pragma unroll
        for (int c = 0; c < QS; ++c) krow[c] = KSS[sl][c];
    }
    int steps = 0;
    for (; steps < a.max_inner; ++steps) {
        const bool up = act && ((yv > 0 && al < C) || (yv < 0 && al > 0));
        const bool lo = act && ((yv > 0 && al > 0) || (yv < 0 && al < C));
        double bu, bl;
        int Li, Lj;
        if (DUP) {
            // row 0: up scores v, row 1: low scores -v; ties to the lowest
            // lane = the lowest index
            const bool lside = prow == 1;
            const double key =
                lside ? (lo ? -v : -INFINITY) : (up ? v : -INFINITY);
            const int idx = (lside ? lo : up) ? p : INT_MAX;
            const double M = row_max_f64(key);
            const unsigned long long hit = __ballot(key == M && idx != INT_MAX);
            bu = rl_f64(M, 0);
            bl = rl_f64(M, 16);
            Li = __builtin_ctzll((hit & 0xFFFFull) | 0x10000ull);
            Lj = __builtin_ctzll(((hit >> 16) & 0xFFFFull) | 0x10000ull);
        } else {
            bu = up ? v : -INFINITY;
            bl = lo ? -v : -INFINITY;
            Li = up ? lane : INT_MAX;
            Lj = lo ? lane : INT_MAX;
            wave_best_pair(bu, Li, bl, Lj);
        }
        if (bu == -INFINITY || bl == -INFINITY) break;
        const double vi = bu, vj = -bl;
        if (!(vi - vj > itol)) break;
        // the room of each lane's variable as the up one (ucap) and as the
        // low one (lcap), taken from lanes i and j; lanes i and j update
        // their own alpha with their own label
        const double ucap = yv > 0 ? C - al : al;
        const double lcap = yv > 0 ? al : C - al;
        const double Ui = rl_f64(ucap, Li), Lb = rl_f64(lcap, Lj);
        const int si = rl_i32(sl, Li), sj = rl_i32(sl, Lj);
        double kij, kai, kaj, kii, kjj;
        if (DUP) {
            const float fi = krow[si], fj = krow[sj];  // K(s, s_i), K(s, s_j)
            kai = (double)fi;
            kaj = (double)fj;
            kij = (double)__int_as_float(rl_i32(__float_as_int(fj), Li));
            kii = (double)__int_as_float(rl_i32(__float_as_int(fi), Li));
            kjj = (double)__int_as_float(rl_i32(__float_as_int(fj), Lj));
        } else {
            kij = (double)KSS[si][sj];
            kai = (double)KSS[sl][si];
            kaj = (double)KSS[sl][sj];
            kii = (double)KSS[si][si];
            kjj = (double)KSS[sj][sj];
        }
        double a2 = kii + kjj - 2.0 * kij;
        if (a2 <= 0.0) a2 = kTau;
        double s = (vi - vj) / a2;
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
        if (act && p == Li) {
            al += yv * s;
            if (ci) al = yv > 0 ? C : 0.0;
        }
        if (act && p == Lj) {
            al -= yv * s;
            if (cj) al = yv > 0 ? 0.0 : C;
        }
        if (act) v -= s * (kai - kaj);
    }
    const uint64_t t_inner = wall_clock64();

    if (own) ws->alphaB[bpos] = al;
    if (!(a.mode & SS_NO_WRITE)) {
        const double dc = own ? yv * (al - a0) : 0.0;
        if (own) {
            a.alpha[t] = al;
            a.st[t] = state_bits(yv, al, C);
            shDc[p] = dc;
        }
        // the change of the coefficient of each slot: the one variable of
        // the slot, or (eps-SVR) the sum of both copies of its sample
        int partner = -1;
        if (SVR && DUP) {
            // variable p sits in lane p of its row: the row rotations meet
            // every other variable (a sample has at most one twin)
            uint32_t pm = 0;
            for_row_rotations([&](auto r) {
                constexpr int R = decltype(r)::value;
                const int m = row_rot<R>(lane & 15);
                const int slm = row_rot<R>(sl);
                pm |= (m < nB && slm == sl) ? (1u << m) : 0u;
            });
            partner = pm ? __builtin_ctz(pm) : -1;
        } else if (SVR) {
            for (int j = 0; j < nB; ++j)
                if (j != p && rl_i32(sl, j) == sl) partner = j;
        }
        __builtin_amdgcn_wave_barrier();
        if (own && (partner < 0 || p < partner))
            ws->coef[sl] = dc + (partner >= 0 ? shDc[partner] : 0.0);
        if (lane < nS) {
            ws->S[lane] = shS[lane];
            ws->sS[lane] = shsS[lane];
        }
        if (lane < nB) {
            ws->B[lane] = shB[lane];
            ws->slotB[lane] = shSlot[lane];
        }
        if (lane == 0) {
            ws->nB = nB;
            ws->nS = nS;
            if (!given) ws->iter = iter0 + 1;
            ws->rows = c_rows + nS;
        }
    }
    finish(0);
    if (lane == 0) {
        ws->steps = steps;
        ws->inner_total = c_inner + steps;
        ws->prof[0] = c_prof[0] + (int64_t)(t_merge - t_start);
        ws->prof[1] = c_prof[1] + (int64_t)(t_kss - t_merge);
        ws->prof[2] = c_prof[2] + (int64_t)(t_inner - t_kss);
        ws->prof[3] = c_prof[3] + (int64_t)(wall_clock64() - t_inner);
        ws->prof[4] = c_prof[4] + 1;
        ws->prof[5] = c_prof[5] + (int64_t)(t_c1 - t_start);
        ws->prof[6] = c_prof[6] + (int64_t)(t_build - t_merge);
        ws->prof[7] = c_prof[7] + (int64_t)(t_stage - t_build);
        ws->prof[8] = c_prof[8] + (int64_t)(t_c2 - t_c1);
        ws->prof[9] = c_prof[9] + (int64_t)(t_c3 - t_c2);
        ws->prof[10] = c_prof[10] + (int64_t)(t_merge - t_c3);
    }
}

template <bool SVR, int NBLK>
__global__ __launch_bounds__(kSelThreads) void k_select(SelArgs a)
{
    select_body<SVR, NBLK>(a);
}

// One problem per block: several selections of problems that advance in
// lockstep (working sets of 16 each).  The arguments travel in the launch.
struct SelGroup {
    SelArgs a[kLockMax];
};

template <bool SVR>
__global__ __launch_bounds__(kSelThreads) void k_select_group(SelGroup g)
{
    select_body<SVR, 1>(g.a[blockIdx.x]);
}

template <bool SVR, int NBLK>
static void select_dispatch(const SelArgs& a, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1)
{
    const size_t lds =
        a.rp ? select_csr_lds_bytes(NBLK, a.ldp, a.csr_cols) +
                   (select_csr_lists(NBLK, a.ldp, a.csr_cols)
                        ? (size_t)a.csr_cols * 4
                        : 0)
             : select_lds_bytes(NBLK, a.slice);
    if (!raise_dynamic_lds((const void*)k_select<SVR, NBLK>, lds))
        throw Error{SVM_E_UNSUPPORTED,
                    "select tile needs more LDS than the device allows"};
    if (e0 || e1)  // timed: the events are part of the dispatch
        hipExtLaunchKernelGGL(k_select<SVR, NBLK>, dim3(1), dim3(kSelThreads),
                              lds, s, e0, e1, 0, a);
    else
        k_select<SVR, NBLK><<<1, kSelThreads, lds, s>>>(a);
}

void launch_select_group(const SelArgs* args, int P, bool svr, hipStream_t s)
{
    if (P <= 0 || P > kLockMax)
        throw Error{SVM_E_INTERNAL, "bad lockstep selection"};
    SelGroup g{};
    const int slice =
        args[0].slice > 0 ? args[0].slice : select_slice(1, args[0].ldp);
    for (int p = 0; p < P; ++p) {
        if (args[p].rp || args[p].ldp != args[0].ldp)
            throw Error{SVM_E_INTERNAL, "bad lockstep selection"};
        g.a[p] = args[p];
        g.a[p].slice = slice;
    }
    const size_t lds = select_lds_bytes(1, slice);
    const void* fn = svr ? (const void*)k_select_group<true>
                         : (const void*)k_select_group<false>;
    if (!raise_dynamic_lds(fn, lds))
        throw Error{SVM_E_UNSUPPORTED,
                    "select tile needs more LDS than the device allows"};
    if (svr)
        k_select_group<true><<<P, kSelThreads, lds, s>>>(g);
    else
        k_select_group<false><<<P, kSelThreads, lds, s>>>(g);
}

void launch_select(const SelArgs& a0, int nblk_cols, bool svr, hipStream_t s,
                   hipEvent_t e0, hipEvent_t e1)
{
    SelArgs a = a0;
    if (a.slice <= 0) a.slice = select_slice(nblk_cols, a.ldp);
    if (a.rp) {
        // CSR: the working set by column is whole in LDS
        a.slice = (int)((a.ldp + 15) & ~(int64_t)15);
        if (select_csr_lds_bytes(nblk_cols, a.ldp, a.csr_cols) > kSelCsrLds)
            throw Error{SVM_E_UNSUPPORTED,
                        "too many features for a CSR working set in LDS"};
    }
    switch (nblk_cols * 2 + (svr ? 1 : 0)) {
        case 2: select_dispatch<false, 1>(a, s, e0, e1); break;
        case 3: select_dispatch<true, 1>(a, s, e0, e1); break;
        case 4: select_dispatch<false, 2>(a, s, e0, e1); break;
        case 5: select_dispatch<true, 2>(a, s, e0, e1); break;
        case 8: select_dispatch<false, 4>(a, s, e0, e1); break;
        case 9: select_dispatch<true, 4>(a, s, e0, e1); break;
        default: throw Error{SVM_E_INTERNAL, "bad column-block count"};
    }
}

}  // namespace msvm
