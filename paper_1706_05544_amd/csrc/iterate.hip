// One outer iteration of the working-set solve per launch (gfx950): dense
// features, working sets of at most 16 variables.
//
// Section 3's loop is: pick the working set B by the largest violations,
// optimise B from the local gradient, update the responses of all n
// samples.  The two-launch loop (k_select, then k_rows) runs the pick and
// the subproblem on one block while the rest of the chip idles, then
// streams X.  Here every block of the launch repeats the pick and the
// subproblem for itself (a few microseconds of latency-bound work on data
// that sits in L2) while the feature rows of its own tiles are already on
// their way, so the stream of X overlaps the selection chain instead of
// following it:
//
//   1. every block reads the candidate records the previous launch wrote
//      (best two keys of each side per row group) and merges them into the
//      exact top q/2 of I_up and of I_low (rescanning the rows of a group
//      whose two candidates of a side were both taken), with the gap test;
//   2. wave 0 builds B and its distinct samples, gathers their rows, forms
//      K_BB on the matrix cores and solves the subproblem; waves 1..3, which
//      own the block's rows, meanwhile take the first feature slabs of
//      their tiles through the matrix cores;
//   3. after one barrier the row waves apply F_i += sum_s dc_s K(x_i, x_s),
//      compute the keys of their variables (the new state of B's variables
//      patched in from the block's own solve) and the block writes its
//      candidate record for the next launch;
//   4. the last block to finish (an atomic ticket, no waiting) writes what
//      must be written once: alpha_B, the state bytes of B and the working-
//      set record.
//
// Every block computes the same B and the same alpha_B bit for bit (the
// same inputs, the same code), and the kernel values, the F update order
// and the selection are those of k_select and k_rows, so a solve takes the
// same iterations to the same result.  F and the candidate records are
// double-buffered by launch parity: a block reads the previous launch's
// values of rows that other blocks are updating.
#include <hip/hip_ext.h>

#include "common.hpp"
#include "device.hpp"
#include "rowtile.hpp"

namespace msvm {

constexpr int kIterThreads = 256;              // 4 waves
constexpr int kIterWaves = kIterThreads / 64;
constexpr int kIterRowWaves = kIterWaves - 1;  // waves 1..3 own the rows
constexpr int kIterRecs = kIterMaxRecords / kIterThreads;  // per thread
constexpr int kIterXsBatch = 4;  // working-set loads issued first, per thread
constexpr int kIterRescanRegs = 4;  // rescan entries per thread in registers

// per-wave LDS bytes of the row data of 16 * tiles rows (F, norm, target,
// state bytes), as in k_rows
__host__ __device__ inline int iter_aux_bytes(int tiles, bool svr)
{
    return ((16 * tiles * (svr ? 18 : 13)) + 15) & ~15;
}

// dot products of tiles completed before the subproblem's coefficients are
// known: up to kRing tiles of a row wave, a floatx4 per lane each
constexpr int kHeldBytes = kRing * 64 * 16;

size_t iter_lds_bytes(int64_t ldp, int tiles, bool svr)
{
    return (size_t)16 * rows_xs_stride(ldp) * sizeof(float) +         // x_S
           (size_t)kIterRowWaves * 16 * kSlabStride * sizeof(float) +  // slabs
           (size_t)kIterRowWaves * iter_aux_bytes(tiles, svr) +        // rows
           (size_t)kIterRowWaves * kHeldBytes +                        // held
           (size_t)kIterWaves * 4 * (8 + 4);                           // recs
}

__device__ __forceinline__ int64_t iter_sample(bool svr, int64_t t, int64_t n)
{
    return (svr && t >= n) ? t - n : t;
}

// Exact top `half` of `count` entries of one side given by get(e, key,
// idx), by `half` block-wide rounds (each the best entry after the previous
// winner); thread 0 writes ok/oi.  xk / xi: LDS for the exchange.
template <class Get>
__device__ __forceinline__ void iter_rounds(int64_t count, Get get, int half,
                                            double* ok, int32_t* oi,
                                            double (*xk)[kIterWaves],
                                            int32_t (*xi)[kIterWaves])
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double pk = INFINITY;
    int32_t pi = -1;
    for (int r = 0; r < half; ++r) {
        double bk = -INFINITY;
        int32_t bi = INT_MAX;
        for (int64_t e = tid; e < count; e += kIterThreads) {
            double k;
            int32_t t;
            get(e, k, t);
            if (after(k, t, pk, pi) && better(k, t, bk, bi)) {
                bk = k;
                bi = t;
            }
        }
        wave_best_fast(bk, bi);
        if (lane == 0) {
            xk[r & 1][wave] = bk;
            xi[r & 1][wave] = bi;
        }
        __syncthreads();
        bk = xk[r & 1][0];
        bi = xi[r & 1][0];
#pragma unroll
        for (int w = 1; w < kIterWaves; ++w)
            if (better(xk[r & 1][w], xi[r & 1][w], bk, bi)) {
                bk = xk[r & 1][w];
                bi = xi[r & 1][w];
            }
        pk = bk;
        pi = bi;
        if (tid == 0) {
            ok[r] = bk;
            oi[r] = bi;
        }
    }
    __syncthreads();
}

// Exact top `half` (<= 8) of each side over the block, both sides at once:
// every thread holds NK entries of each side (key, variable; -inf for
// none, every variable at most once per side).  Each wave finds its own
// top half by `half` rounds of a wave-wide best (no block barrier), then
// wave 0 ranks the waves' 4 x 8 entries of each side (lanes 0..31 the up
// side, 32..63 the low side): an entry's rank is the number of entries
// before it in the order of better().  Results to (uk, ui) and (lk, li),
// -inf past the valid entries.  ck / ci: 2 x 32 entries of LDS.
template <int NK>
__device__ __forceinline__ void block_top_half(
    const double (&ku)[NK], const int32_t (&iu)[NK], const double (&kl)[NK],
    const int32_t (&il)[NK], int half, double* uk, int32_t* ui, double* lk,
    int32_t* li, double (*ck)[32], int32_t (*ci)[32])
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double pu = INFINITY, pl = INFINITY;
    int32_t qu = -1, ql = -1;
    for (int r = 0; r < 8; ++r) {
        double bu = -INFINITY, bl = -INFINITY;
        int32_t ju = INT_MAX, jl = INT_MAX;
        if (r < half) {
#pragma unroll
            for (int j = 0; j < NK; ++j) {
                if (after(ku[j], iu[j], pu, qu) &&
                    better(ku[j], iu[j], bu, ju)) {
                    bu = ku[j];
                    ju = iu[j];
                }
                if (after(kl[j], il[j], pl, ql) &&
                    better(kl[j], il[j], bl, jl)) {
                    bl = kl[j];
                    jl = il[j];
                }
            }
            wave_best_pair(bu, ju, bl, jl);
        }
        if (lane == 0) {
            ck[0][8 * wave + r] = bu;
            ci[0][8 * wave + r] = ju;
            ck[1][8 * wave + r] = bl;
            ci[1][8 * wave + r] = jl;
        }
        pu = bu;
        qu = ju;
        pl = bl;
        ql = jl;
    }
    if (tid >= 64 && tid < 64 + kMaxHalf) {
        uk[tid - 64] = lk[tid - 64] = -INFINITY;
        ui[tid - 64] = li[tid - 64] = INT_MAX;
    }
    __syncthreads();
    if (wave == 0) {
        const int side = lane >> 5, e = lane & 31;
        const double me = ck[side][e];
        const int32_t mi = ci[side][e];
        int rank = 0;
#pragma unroll 8
        for (int j = 0; j < 32; ++j)
            rank += better(ck[side][j], ci[side][j], me, mi) ? 1 : 0;
        if (me != -INFINITY && rank < half) {
            (side ? lk : uk)[rank] = me;
            (side ? li : ui)[rank] = mi;
        }
    }
    __syncthreads();
}

template <bool SVR>
__global__ __launch_bounds__(kIterThreads) void k_iter(IterArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    WorkingSet* ws = a.ws;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, nl = lane & 15;
    const int64_t n = a.n;
    const int ldp = (int)a.ldp;
    const int half = a.half;
    const int T = a.tiles, RW = 16 * T;
    const int xstride = rows_xs_stride(ldp);

    __shared__ double upk[kMaxHalf], lok[kMaxHalf];
    __shared__ int32_t upi[kMaxHalf], loi[kMaxHalf];
    __shared__ double xk[2][2][kIterWaves];
    __shared__ int32_t xi[2][2][kIterWaves];
    __shared__ double ck[2][32];
    __shared__ int32_t ci[2][32];
    __shared__ double keepk[2][kMaxHalf];
    __shared__ int32_t keepi[2][kMaxHalf];
    __shared__ int32_t exb[2][kMaxHalf], nex[2], nkeep[2];
    __shared__ int32_t shB[16], shSlot[16], shS[16], shPos[16];
    __shared__ float sl_sq[16];
    __shared__ int32_t sl_smp[16];
    __shared__ double cfS[16];       // coefficient change of each slot
    __shared__ double shDc[16];
    __shared__ uint8_t shStNew[16];  // new state byte of B's variables
    __shared__ float KSS[16][17];
    __shared__ int32_t shNB, shNS, shGo, shDone, shLast;
    __shared__ double shGap, shMx, shMn;

    // ---- (1) the previous launch's candidate records, the done flag and
    // the iteration count ------------------------------------------------
    __shared__ uint64_t tph[7];  // phase times (thread 0), for profiling
    if (tid == 0) tph[0] = wall_clock64();
    const int32_t done0 = ws->done;
    const int64_t iter0 = ws->iter;
    double ku[2 * kIterRecs], kl[2 * kIterRecs];
    int32_t iu[2 * kIterRecs], il[2 * kIterRecs];
#pragma unroll
    for (int j = 0; j < kIterRecs; ++j) {
        const int r = tid + j * kIterThreads;
        double2 k01 = make_double2(-INFINITY, -INFINITY);
        double2 k23 = k01;
        int4 ix = make_int4(INT_MAX, INT_MAX, INT_MAX, INT_MAX);
        if (r < a.nb) {
            const double* rk0 = a.rk_in + 4 * (size_t)r;
            k01 = *reinterpret_cast<const double2*>(rk0);
            k23 = *reinterpret_cast<const double2*>(rk0 + 2);
            ix = *reinterpret_cast<const int4*>(a.ri_in + 4 * (size_t)r);
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
    if (done0) return;  // uniform: the solve has finished

    // top half of each side over the records (ties to the lowest index)
    block_top_half<2 * kIterRecs>(ku, iu, kl, il, half, upk, upi, lok, loi,
                                  ck, ci);
    if (tid == 0) tph[1] = wall_clock64();

    // ---- rescans: a row group (a block of the previous launch) whose two
    // candidates of a side were both taken may hold more of the top half;
    // the keys of its rows are recomputed from the previous responses and
    // ranked with the winners outside such groups
    const int64_t TU = (n + 31) >> 5, NB = a.nb;
    auto group_of = [&](int64_t row) -> int32_t {
        // the largest b with 32 (b TU / NB) <= row, through an fp64
        // quotient corrected to the exact integer
        const int64_t x = ((row >> 5) + 1) * NB - 1;
        int64_t gq = (int64_t)((double)x / (double)TU);
        if (gq * TU > x) --gq;
        else if ((gq + 1) * TU <= x) ++gq;
        return (int32_t)gq;
    };
    auto group_start = [&](int64_t b) -> int64_t { return 32 * (b * TU / NB); };
    if (wave == 0) {
        // lanes [0, 32): the up winners, [32, 64): the low winners
        const int side = lane >> 5, k = lane & 31;
        const double* kk = side ? lok : upk;
        const int32_t* ii = side ? loi : upi;
        const bool valid = k < half && kk[k] != -INFINITY;
        const int32_t b =
            valid ? group_of(iter_sample(SVR, ii[k], n)) : -1 - lane;
        int c = 0;
        bool first = true;
        for (int j = 0; j < half; ++j) {
            const int32_t bu = rl_i32(b, j), bl = rl_i32(b, 32 + j);
            const int32_t bj = side ? bl : bu;
            c += bj == b;
            first &= !(j < k && bj == b);
        }
        const bool ex = valid && c >= kBlockTop && first;
        const unsigned long long m = __ballot(ex);
        const unsigned long long ms = side ? (m >> 32) : (m & 0xffffffffull);
        if (ex) exb[side][__popcll(ms & ((1ull << k) - 1ull))] = b;
        if (k == 0) nex[side] = __popcll(ms);
        // the winners outside the exhausted groups of their side (a group's
        // winners are ranked again with all of its rows)
        bool in_ex = false;
        for (int j = 0; j < half; ++j) {
            // (readlane takes a lane index that is the same on all lanes)
            const int32_t bu = rl_i32(b, j), bl = rl_i32(b, 32 + j);
            const int32_t bj = side ? bl : bu;
            const bool exj = ((side ? (m >> 32) : m) >> j) & 1ull;
            in_ex |= exj && bj == b;
        }
        const bool keep2 = valid && !in_ex;
        const unsigned long long mk2 = __ballot(keep2);
        const unsigned long long mk2s =
            side ? (mk2 >> 32) : (mk2 & 0xffffffffull);
        if (keep2) {
            const int pos = __popcll(mk2s & ((1ull << k) - 1ull));
            keepk[side][pos] = kk[k];
            keepi[side][pos] = ii[k];
        }
        if (k == 0) nkeep[side] = __popcll(mk2s);
    }
    __syncthreads();
    int64_t c_resc = 0;
    if (nex[0] + nex[1] > 0) {
        // every side: its kept winners and the variables of its exhausted
        // groups (a side without such groups: just its winners), ranked
        const uint32_t grows = (uint32_t)a.group_rows;
        const uint32_t per = grows * (SVR ? 2u : 1u);
        const int nk0 = nkeep[0], nk1 = nkeep[1];
        const int64_t tot0 = nk0 + (int64_t)nex[0] * per;
        const int64_t tot1 = nk1 + (int64_t)nex[1] * per;
        // entry e of a side: kept winner e, else variable e - nk of the
        // side's exhausted groups (copy (i,-) of eps-SVR after copy (i,+))
        auto get = [&](int side, int64_t e, double& key, int32_t& t) {
            const int nk = side ? nk1 : nk0;
            key = -INFINITY;
            t = INT_MAX;
            if (e < nk) {
                key = keepk[side][e];
                t = keepi[side][e];
                return;
            }
            const int64_t q = e - nk;
            if (q >= (int64_t)nex[side] * per) return;
            const uint32_t x = (uint32_t)(q / per),
                           o = (uint32_t)(q - (int64_t)x * per);
            const int64_t b = exb[side][x];
            const int64_t row = group_start(b) + (o % grows);
            if (row < min(n, group_start(b + 1))) {
                const int64_t tt = o < grows ? row : n + row;
                const uint8_t st = a.st[tt];
                double rr;
                if (SVR)
                    rr = tt < n ? (double)a.z[row] - a.eps
                                : (double)a.z[row] + a.eps;
                else
                    rr = (st & ST_YPOS) ? 1.0 : -1.0;
                const double v = rr - a.F_in[row];
                key = side ? ((st & ST_LOW) ? -v : -INFINITY)
                           : ((st & ST_UP) ? v : -INFINITY);
                t = (int32_t)tt;
            }
        };
        const int64_t tot = max(tot0, tot1);
        if (tot <= (int64_t)kIterRescanRegs * kIterThreads) {
            // every entry loaded once into registers, then ranked
            double rku[kIterRescanRegs], rkl[kIterRescanRegs];
            int32_t riu[kIterRescanRegs], ril[kIterRescanRegs];
#pragma unroll
            for (int j = 0; j < kIterRescanRegs; ++j) {
                const int64_t e = tid + (int64_t)j * kIterThreads;
                get(0, e, rku[j], riu[j]);
                get(1, e, rkl[j], ril[j]);
            }
            __syncthreads();  // every kept winner read before the lists go
            block_top_half<kIterRescanRegs>(rku, riu, rkl, ril, half, upk,
                                            upi, lok, loi, ck, ci);
        } else {
            // (very large row groups) block-wide rounds, entries fetched
            // again every round
            for (int side = 0; side < 2; ++side) {
                auto gs = [&](int64_t e, double& key, int32_t& t) {
                    get(side, e, key, t);
                };
                iter_rounds(side ? tot1 : tot0, gs, half, side ? lok : upk,
                            side ? loi : upi, xk[side], xi[side]);
            }
        }
        c_resc = 1;
    }
    if (tid == 0) tph[2] = wall_clock64();

    // ---- (2) gap test and working set (wave 0, lane-parallel) -----------
    if (wave == 0) {
        const bool valid = upk[0] != -INFINITY && lok[0] != -INFINITY;
        const double m = upk[0], M = -lok[0];
        const double gap = valid ? m - M : 0.0;
        int go = 1, done = 0;
        if (!valid || gap <= a.tol) {
            done = 1;
            go = 0;
        } else if (iter0 >= a.max_iter) {
            done = 2;
            go = 0;
        }
        int nB = 0, nS = 0;
        if (go) {
            // lanes [0,half): up list, [half,2half): low list; position in
            // the interleaved order U0 L0 U1 L1 ..., repeats dropped
            const bool isU = lane < half;
            const bool inL = lane >= half && lane < 2 * half;
            const int k = isU ? lane : lane - half;
            const double key = isU ? upk[k] : (inL ? lok[k] : -INFINITY);
            const bool ent = (isU || inL) && key != -INFINITY;
            const int32_t idx = ent ? (isU ? upi[k] : loi[k]) : INT_MAX;
            bool keep = ent;
            for (int j = 0; j < half; ++j) {
                const int32_t uj = rl_i32(idx, j), lj = rl_i32(idx, half + j);
                if (isU && j < k && lj == idx) keep = false;
                if (inL && j <= k && uj == idx) keep = false;
            }
            const unsigned long long mk = __ballot(keep);
            const unsigned long long mu = mk & ((1ull << half) - 1ull);
            const unsigned long long ml = (mk >> half) & ((1ull << half) - 1ull);
            const unsigned long long below = (1ull << k) - 1ull;
            int pos = __popcll(mu & below) + __popcll(ml & below);
            if (!isU) pos += (int)((mu >> k) & 1ull);
            if (keep) shB[pos] = idx;
            nB = __popcll(mk);
            __builtin_amdgcn_wave_barrier();
            // slot of each variable: rank of the first occurrence of its
            // sample (eps-SVR: both copies of a sample share one slot); the
            // subproblem takes its variables in increasing index order
            const bool act = lane < nB;
            const int32_t t = act ? shB[lane] : INT_MAX;
            const int32_t s = act ? (int32_t)iter_sample(SVR, t, n) : -1;
            int firstpos = lane;
            if (SVR)
                for (int j = 0; j < nB; ++j) {
                    const int32_t sj = rl_i32(s, j);
                    if (act && j < firstpos && sj == s) firstpos = j;
                }
            const unsigned long long fm = __ballot(act && firstpos == lane);
            const unsigned long long bl =
                firstpos >= 64 ? ~0ull : ((1ull << firstpos) - 1ull);
            const int slot = __popcll(fm & bl);
            int p = 0;
            for (int j = 0; j < nB; ++j) p += rl_i32(t, j) < t ? 1 : 0;
            if (act) {
                shSlot[lane] = slot;
                if (firstpos == lane) shS[slot] = s;
                shPos[p] = lane;
            }
            nS = __popcll(fm);
        }
        if (lane == 0) {
            shGo = go;
            shDone = done;
            shNB = nB;
            shNS = nS;
            shGap = gap;
            shMx = valid ? m : 0.0;
            shMn = valid ? M : 0.0;
        }
    }
    __syncthreads();
    if (tid == 0) tph[3] = wall_clock64();
    const int go = shGo, nB = shNB, nS = shNS;

    // ---- rows of this block: units of 32 rows shared out evenly over the
    // blocks (one candidate record each), the block's tiles over waves 1..3
    const int64_t vb = blockIdx.x;
    const int64_t b0 = 32 * (vb * TU / NB);
    const int64_t b1 = min(32 * ((vb + 1) * TU / NB), n);
    const int tb = (int)((b1 - b0 + 15) >> 4);
    const int rwv = wave > 0 ? wave - 1 : 0;  // row wave index
    const int64_t rw0 = b0 + 16 * (rwv * tb / kIterRowWaves);
    const int nw =
        wave > 0
            ? (int)(min(b0 + 16 * ((rwv + 1) * tb / kIterRowWaves), b1) - rw0)
            : 0;
    const int Tw = (nw + 15) >> 4;
    const int nslab = (ldp + 63) >> 6;

    float* xsl = reinterpret_cast<float*>(smem);
    unsigned char* p0 = smem + (size_t)16 * xstride * sizeof(float);
    float* wbuf = reinterpret_cast<float*>(p0) + rwv * 16 * kSlabStride;
    unsigned char* p1 = p0 + (size_t)kIterRowWaves * 16 * kSlabStride * 4;
    unsigned char* aux = p1 + (size_t)rwv * iter_aux_bytes(T, SVR);
    double* Fw = reinterpret_cast<double*>(aux);
    float* sqw = reinterpret_cast<float*>(aux + 8 * RW);
    float* zw = reinterpret_cast<float*>(aux + 12 * RW);
    uint8_t* stw = aux + (SVR ? 16 : 12) * RW;  // copy (i,-) at stw[RW + r]
    unsigned char* p2 = p1 + (size_t)kIterRowWaves * iter_aux_bytes(T, SVR);
    floatx4* held = reinterpret_cast<floatx4*>(p2) + rwv * (kHeldBytes / 16);
    unsigned char* p3 = p2 + (size_t)kIterRowWaves * kHeldBytes;
    double* brk = reinterpret_cast<double*>(p3);  // [waves][4]
    int32_t* bri = reinterpret_cast<int32_t*>(p3 + kIterWaves * 32);

    const Rsrc rFi = make_rsrc(a.F_in + rw0, (int64_t)nw * 8);
    const Rsrc rFo = make_rsrc(a.F_out + rw0, (int64_t)nw * 8);
    const Rsrc rX = make_rsrc(a.X + rw0 * ldp, (int64_t)nw * ldp * 4);
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
    struct AuxRegs {
        double f[4];
        float q[4], z[4];
        uint8_t s0[4], s1[4];
    };
    auto aux_issue = [&](int k0, AuxRegs& x) {
        const Rsrc rQ = make_rsrc(a.sq + rw0, (int64_t)nw * 4);
        const Rsrc rS0 = make_rsrc(a.st + rw0, nw);
        const Rsrc rS1 = make_rsrc(a.st + n + rw0, SVR ? nw : 0);
        const Rsrc rZ = make_rsrc(a.z + rw0, SVR ? (int64_t)nw * 4 : 0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t r = (uint32_t)(k0 + 64 * j + lane);
            x.f[j] = bld_f64(rFi, 8 * r);
            x.q[j] = bld_f32(rQ, 4 * r);
            x.s0[j] = bld_u8(rS0, r);
            x.s1[j] = SVR ? bld_u8(rS1, r) : 0;
            x.z[j] = SVR ? bld_f32(rZ, 4 * r) : 0.0f;
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

    float4 ring[kRing][4];
    floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
    int pti = 0, psl = 0;  // slab being processed (row waves)
    if (go) {
        // (3) first the working-set rows (every slot, zero past nS and past
        // ldp; they feed K_SS and then the subproblem, the critical path),
        // then the row waves' row data (the previous launch's responses)
        // and their first kRing feature slabs.  The first batch of
        // working-set loads has a fixed count, so the waits below can let
        // the later loads stay in flight.
        const int q4 = (xstride - 4) >> 2;
        const int xs_total = 16 * q4;
        auto xs_load = [&](int e, bool& ok) {
            const int slot = e / q4, c4 = e - slot * q4;
            ok = e < xs_total && slot < nS && 4 * c4 < ldp;
            const int32_t smp = shS[min(slot, 15)];
            const int64_t o = ok ? (int64_t)smp * ldp + 4 * c4 : 0;  // in X
            return ld4(a.X + o);
        };
        auto xs_put = [&](int e, bool ok, float4 v) {
            const int slot = e / q4, c4 = e - slot * q4;
            if (e < xs_total)
                *reinterpret_cast<float4*>(xsl + slot * xstride + 4 * c4) =
                    ok ? v : zero4();
        };
        float4 xv[kIterXsBatch];
        bool xok[kIterXsBatch];
#pragma unroll
        for (int j = 0; j < kIterXsBatch; ++j)
            xv[j] = xs_load(tid + j * kIterThreads, xok[j]);
        float qs = 0.0f;
        if (tid < 16) qs = a.sq[tid < nS ? shS[tid] : 0];
        AuxRegs ar;
        if (wave > 0) {
            aux_issue(0, ar);
#pragma unroll
            for (int j = 0; j < kRing; ++j) fetch(ring[j]);
        }
#pragma unroll
        for (int j = 0; j < kIterXsBatch; ++j)
            xs_put(tid + j * kIterThreads, xok[j], xv[j]);
        if (tid < 16) {
            sl_sq[tid] = tid < nS ? qs : 0.0f;
            sl_smp[tid] = tid < nS ? shS[tid] : -1;
        }
        if (wave > 0) aux_store(0, ar);
        // (many features or rows: the rest, behind uniform branches)
        if (xs_total > kIterXsBatch * kIterThreads) {
            for (int e = tid + kIterXsBatch * kIterThreads; e < xs_total;
                 e += kIterThreads) {
                bool ok;
                const float4 v = xs_load(e, ok);
                xs_put(e, ok, v);
            }
        }
        if (wave > 0 && RW > 256) {
            for (int k0 = 256; k0 < RW; k0 += 256) {
                aux_issue(k0, ar);
                aux_store(k0, ar);
            }
        }
    }
    __syncthreads();
    if (tid == 0) tph[4] = wall_clock64();

    int steps = 0;
    double al = 0.0;      // wave 0: new alpha of the lane's variable
    int bpos = 0;         // wave 0: its position in B
    bool own = false;     // wave 0: the lane writes that variable
    int32_t tvar = 0;     // wave 0: the variable
    if (go && wave == 0) {
        // (4) K_SS on the matrix cores, in the operand order of the row
        // kernels (its values are those of K(x_i, x_s) bit for bit)
        {
            const int ldp16 = (ldp + 15) & ~15;
            floatx4 kacc = floatx4{0.f, 0.f, 0.f, 0.f};
            const bool va = nl < nS;
            for (int cc = 0; cc < ldp16; cc += 16) {
                float4 av = ld4(xsl + nl * xstride + cc + 4 * g);
                float4 bv = av;
                if (!va) av = bv = zero4();
                kacc = mfma_chunk(kacc, av, bv);
            }
            const float sqb = sl_sq[nl];
#pragma unroll
            for (int vv = 0; vv < 4; ++vv) {
                const int ia = 4 * g + vv, ib = nl;
                if (ia < nS && ib < nS)
                    KSS[ia][ib] = (ia == ib && kernel_self_is_one(a.kf))
                                      ? 1.0f
                                      : kernel_from_dot(a.kf, sl_sq[ia], sqb,
                                                        kacc[vv]);
            }
        }
        // (5) the subproblem: maximal-violating-pair steps restricted to B.
        // The variable of rank p by index sits in lane p of rows 0 (its up
        // side) and 1 (its low side), so one row reduction serves both.
        const int p = lane & 15;
        const int prow = lane >> 4;
        const bool act = p < nB && prow < 2;
        own = act && prow == 0;
        bpos = act ? shPos[p] : 0;
        const int32_t t = act ? shB[bpos] : INT_MAX;
        tvar = t;
        const int sl = act ? shSlot[bpos] : 0;
        const int64_t sm = act ? iter_sample(SVR, t, n) : 0;
        al = act ? a.alpha[t] : 0.0;
        double yv = 1.0, rv = 0.0, v = 0.0;
        if (act) {
            if (SVR) {
                yv = t < n ? 1.0 : -1.0;
                rv = t < n ? (double)a.z[sm] - a.eps : (double)a.z[sm] + a.eps;
            } else {
                yv = (a.st[t] & ST_YPOS) ? 1.0 : -1.0;
                rv = yv;
            }
            v = rv - a.F_in[sm];
        }
        __builtin_amdgcn_wave_barrier();
        const double a0 = al;
        const double C = a.C;
        const double itol = fmax(a.inner_ratio * shGap, 0.5 * a.tol);
        for (; steps < a.max_inner; ++steps) {
            const bool up = act && ((yv > 0 && al < C) || (yv < 0 && al > 0));
            const bool lo = act && ((yv > 0 && al > 0) || (yv < 0 && al < C));
            const bool lside = prow == 1;
            const double key =
                lside ? (lo ? -v : -INFINITY) : (up ? v : -INFINITY);
            const int idx = (lside ? lo : up) ? p : INT_MAX;
            const double Mx = row_max_f64(key);
            const unsigned long long hit =
                __ballot(key == Mx && idx != INT_MAX);
            const double bu = rl_f64(Mx, 0);
            const double bl = rl_f64(Mx, 16);
            const int Li = __builtin_ctzll((hit & 0xFFFFull) | 0x10000ull);
            const int Lj =
                __builtin_ctzll(((hit >> 16) & 0xFFFFull) | 0x10000ull);
            if (bu == -INFINITY || bl == -INFINITY) break;
            const double vi = bu, vj = -bl;
            if (!(vi - vj > itol)) break;
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
            if (act && p == Li) {
                al += yi * s;
                if (ci) al = yi > 0 ? C : 0.0;
            }
            if (act && p == Lj) {
                al -= yj * s;
                if (cj) al = yj > 0 ? 0.0 : C;
            }
            if (act) v -= s * (kai - kaj);
        }
        // the change of the coefficient of each slot: the one variable of
        // the slot, or (eps-SVR) the sum of both copies of its sample
        const double dc = own ? yv * (al - a0) : 0.0;
        if (lane < 16) cfS[lane] = 0.0;
        if (own) {
            shDc[p] = dc;
            shStNew[bpos] = state_bits(yv, al, C);
        }
        int partner = -1;
        if (SVR)
            for (int j = 0; j < nB; ++j)
                if (j != p && rl_i32(sl, j) == sl) partner = j;
        __builtin_amdgcn_wave_barrier();
        if (own && (partner < 0 || p < partner))
            cfS[sl] = dc + (partner >= 0 ? shDc[partner] : 0.0);
    } else if (go) {
        // (4') the row waves: the first kRing slabs through the matrix
        // cores while wave 0 solves; a tile completed here waits in LDS for
        // the coefficients, a tile in progress keeps its sums in acc
#pragma unroll
        for (int j = 0; j < kRing; ++j) {
            if (psl == 0) acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                *reinterpret_cast<float4*>(
                    wbuf + (4 * rr + g) * kSlabStride + 4 * nl) = ring[j][rr];
            fetch(ring[j]);  // refill the slot kRing slabs ahead
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int ch = psl * 4 + c;
                if (ch * 16 < ldp) {  // chunk present (uniform)
                    const float4 av =
                        ld4(wbuf + nl * kSlabStride + c * 16 + 4 * g);
                    const float4 bv = ld4(xsl + nl * xstride + ch * 16 + 4 * g);
                    acc = mfma_chunk(acc, av, bv);
                }
            }
            __builtin_amdgcn_wave_barrier();
            if (psl == nslab - 1 && pti < Tw) held[pti * 64 + lane] = acc;
            if (++psl == nslab) {
                psl = 0;
                ++pti;
            }
        }
    }
    __syncthreads();  // the coefficients cfS and the new state bytes
    if (tid == 0) tph[5] = wall_clock64();

    Top2 up, lo;  // this lane's best candidates of each side
    if (go && wave > 0) {
        // the new state of B's variables in this wave's rows (the global
        // bytes are written by the last block, after every block has read)
        if (lane < nB) {
            const int32_t t = shB[lane];
            const int64_t sm = iter_sample(SVR, t, n);
            if (sm >= rw0 && sm < rw0 + nw)
                stw[(t >= n ? RW : 0) + (int)(sm - rw0)] = shStNew[lane];
        }
        __builtin_amdgcn_wave_barrier();
        double cf = cfS[nl];  // slots past nS are 0
        const float ssb = sl_sq[nl];
        const int32_t smb = sl_smp[nl];
        auto push = [&](int lr, double Fn, bool ownr) {
            const int32_t row = (int32_t)(rw0 + lr);
            const uint8_t s0 = stw[lr];
            const double r0 = SVR ? (double)zw[lr] - a.eps
                                  : ((s0 & ST_YPOS) ? 1.0 : -1.0);
            const double v0 = r0 - Fn;
            if (ownr && (s0 & ST_UP)) up.push(v0, row);
            if (ownr && (s0 & ST_LOW)) lo.push(-v0, row);
            if (SVR) {
                const uint8_t s1 = stw[RW + lr];
                const double v1 = ((double)zw[lr] + a.eps) - Fn;
                if (ownr && (s1 & ST_UP)) up.push(v1, (int32_t)(n + row));
                if (ownr && (s1 & ST_LOW)) lo.push(-v1, (int32_t)(n + row));
            }
        };
        // F_i += sum_s cf_s K(x_i, x_s) for the 16 rows of tile ti from the
        // tile's dot products, then the keys (the order of k_rows)
        auto finish_tile = [&](int ti, floatx4 d) {
            const int lr = 16 * ti + 4 * g;
            const float4 q4v = *reinterpret_cast<const float4*>(sqw + lr);
            const float qv[4] = {q4v.x, q4v.y, q4v.z, q4v.w};
            float kv[4];
            if (a.kf.kind == SVM_KERNEL_RBF) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float k = rbf_from_dot(qv[v], ssb, d[v], a.kf.gexp);
                    if (rw0 + lr + v == (int64_t)smb) k = 1.0f;
                    kv[v] = k;
                }
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v) kv[v] = kernel_of_dot(a.kf, d[v]);
            }
            double part[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) part[v] = fma(cf, (double)kv[v], 0.0);
            const int orl = lr + (nl & 3);  // row owned by lanes nl < 4
            double Fn = Fw[orl];
#pragma unroll
            for (int v = 0; v < 4; ++v) part[v] = row_sum_f64(part[v]);
            Fn += pick4(part, nl & 3);
            if (nl < 4) Fw[orl] = Fn;
            push(orl, Fn, nl < 4 && orl < nw);
        };
        // tiles completed before the barrier
        for (int ti = 0; ti < min(pti, Tw); ++ti)
            finish_tile(ti, held[ti * 64 + lane]);
        // the rest of the stream
        for (int s0 = kRing; s0 < Tw * nslab; s0 += kRing) {
#pragma unroll
            for (int j = 0; j < kRing; ++j) {
                if (psl == 0) acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int rr = 0; rr < 4; ++rr)
                    *reinterpret_cast<float4*>(
                        wbuf + (4 * rr + g) * kSlabStride + 4 * nl) =
                        ring[j][rr];
                fetch(ring[j]);
                __builtin_amdgcn_wave_barrier();
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int ch = psl * 4 + c;
                    if (ch * 16 < ldp) {
                        const float4 av =
                            ld4(wbuf + nl * kSlabStride + c * 16 + 4 * g);
                        const float4 bv =
                            ld4(xsl + nl * xstride + ch * 16 + 4 * g);
                        acc = mfma_chunk(acc, av, bv);
                    }
                }
                __builtin_amdgcn_wave_barrier();
                if (psl == nslab - 1 && pti < Tw) finish_tile(pti, acc);
                if (++psl == nslab) {
                    psl = 0;
                    ++pti;
                }
            }
        }
        for (int r = lane; r < nw; r += 64) bst_f64(rFo, 8 * (uint32_t)r, Fw[r]);
    }

    if (tid == 0) tph[6] = tph[5];
    if (go) {
        // (6) this block's candidate record for the next launch: the best
        // two of each side over its rows
        wave_top2_pair(up, lo, brk + 4 * wave, bri + 4 * wave);
        __syncthreads();
        if (tid == 0) tph[6] = wall_clock64();
        if (wave == 0) {
            Top2 u, l;
            if (lane < kIterWaves) {
                u.k1 = brk[4 * lane];
                u.k2 = brk[4 * lane + 1];
                l.k1 = brk[4 * lane + 2];
                l.k2 = brk[4 * lane + 3];
                u.i1 = bri[4 * lane];
                u.i2 = bri[4 * lane + 1];
                l.i1 = bri[4 * lane + 2];
                l.i2 = bri[4 * lane + 3];
            }
            wave_top2_pair(u, l, a.rk_out + (size_t)vb * 2 * kBlockTop,
                           a.ri_out + (size_t)vb * 2 * kBlockTop);
        }
    }

    // ---- (7) ticket: the last block writes what is written once ---------
    __syncthreads();
    if (tid == 0) {
        __threadfence();
        const unsigned int t = atomicAdd(a.ticket, 1u);
        shLast = t == gridDim.x - 1 ? 1 : 0;
    }
    __syncthreads();
    if (!shLast || wave != 0) return;
    if (lane == 0) {
        *a.ticket = 0u;  // for the next launch
        // phase times of this block (wall-clock ticks), summed over launches
        const uint64_t t_end = wall_clock64();
        ws->prof[0] += (int64_t)(tph[1] - tph[0]);
        ws->prof[1] += (int64_t)(tph[2] - tph[1]);
        ws->prof[2] += (int64_t)(tph[3] - tph[2]);
        ws->prof[3] += (int64_t)(tph[4] - tph[3]);
        ws->prof[5] += (int64_t)(tph[5] - tph[4]);
        ws->prof[6] += (int64_t)(tph[6] - tph[5]);
        ws->prof[7] += (int64_t)(t_end - tph[6]);
        ws->prof[4] += 1;
    }
    if (!go) {
        if (lane == 0) {
            ws->done = shDone;
            ws->gap = shGap;
            ws->m = shMx;
            ws->M = shMn;
            ws->rescans += c_resc;
        }
        return;
    }
    if (own) {
        a.alpha[tvar] = al;
        a.st[tvar] = shStNew[bpos];
        ws->alphaB[bpos] = al;
    }
    if (lane < nS) {
        ws->S[lane] = shS[lane];
        ws->sS[lane] = sl_sq[lane];
        ws->coef[lane] = cfS[lane];
        ws->cslot[lane] = -1;
    }
    if (lane < nB) {
        ws->B[lane] = shB[lane];
        ws->slotB[lane] = shSlot[lane];
    }
    if (lane == 0) {
        const int64_t it = iter0 + 1;
        ws->nB = nB;
        ws->nS = nS;
        ws->iter = it;
        ws->rows += nS;
        ws->gap = shGap;
        ws->m = shMx;
        ws->M = shMn;
        ws->steps = steps;
        ws->inner_total += steps;
        ws->rescans += c_resc;
        ws->path = PATH_STREAM;
        ws->path_log[it % kPathLog] = (uint8_t)PATH_STREAM;
        ws->fill_log[it % kPathLog] = 0;
        ws->ns_log[it % kPathLog] = (uint8_t)nS;
    }
}

template <bool SVR>
static void iter_dispatch(const IterArgs& a, int nblocks, hipStream_t s,
                          hipEvent_t e0, hipEvent_t e1)
{
    const size_t lds = iter_lds_bytes(a.ldp, a.tiles, SVR);
    if (!raise_dynamic_lds((const void*)k_iter<SVR>, lds))
        throw Error{SVM_E_UNSUPPORTED,
                    "iteration kernel needs more LDS than the device allows"};
    if (e0)
        hipExtLaunchKernelGGL(k_iter<SVR>, dim3(nblocks), dim3(kIterThreads),
                              (uint32_t)lds, s, e0, e1, 0, a);
    else
        k_iter<SVR><<<nblocks, kIterThreads, lds, s>>>(a);
}

void launch_iter(const IterArgs& a, int nblocks, bool svr, hipStream_t s,
                 hipEvent_t e0, hipEvent_t e1)
{
    if (nblocks <= 0 || nblocks > kIterMaxRecords || a.half > 8)
        throw Error{SVM_E_INTERNAL, "bad iteration kernel launch"};
    if ((int64_t)16 * a.tiles * a.ldp * 4 >= ((int64_t)1 << 31))
        throw Error{SVM_E_UNSUPPORTED, "row group too large for the row kernel"};
    if (svr) iter_dispatch<true>(a, nblocks, s, e0, e1);
    else iter_dispatch<false>(a, nblocks, s, e0, e1);
}

int iter_blocks_per_cu(bool svr, size_t lds)
{
    const void* f = svr ? (const void*)k_iter<true> : (const void*)k_iter<false>;
    return occupancy_memo(f, kIterThreads, lds);
}

}  // namespace msvm
