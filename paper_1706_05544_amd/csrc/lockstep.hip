// Lockstep row/update kernel: several training problems over one stream of
// X (gfx950).
//
// The classes of a one-vs-rest model, the folds of a cross-validation and
// the points of a parameter grid (Section 3's multi-class, cross-validation
// and tuning features) train on the same feature rows.  In lockstep their
// outer iterations advance together: the selections run as the blocks of
// one launch, and one pass over X serves all the working sets.  Each
// 16-row tile of X meets the P x 16 staged working-set samples on the
// matrix cores (one 16x16x4 chain per problem on the same X operand), and
// each problem's epilogue updates its own F and writes its own candidate
// records.  Per problem, the K values, the fp64 order of the F update and
// the candidates are those of k_rows computing the rows from X, so every
// problem takes the iterations it takes alone (without the row cache).  A
// problem that has finished contributes nothing and writes nothing.
#include <hip/hip_ext.h>

#include "common.hpp"
#include "device.hpp"
#include "rowtile.hpp"

namespace msvm {

// Per-wave LDS bytes of the row data of 16 * tiles rows: the norms, then
// per problem F (fp64), for eps-SVR the target, and the state byte of each
// copy.
__host__ __device__ inline int lock_aux_bytes(int P, int tiles, bool svr)
{
    const int RW = 16 * tiles;
    return (RW * 4 + P * RW * (svr ? 8 + 4 + 2 : 8 + 1) + 15) & ~15;
}

__host__ __device__ inline size_t lock_aux_offset(int P, int64_t ldp)
{
    return ((size_t)P * 16 * rows_xs_stride(ldp) +
            (size_t)kRowWaves * 16 * kSlabStride) * sizeof(float);
}

// per problem: the waves' candidate records (4 scores and 4 variables each)
// and the slot table (norm and sample of each of 16 slots)
constexpr int kLockRecBytes = kRowWaves * 4 * (8 + 4) + 16 * (4 + 4);

size_t lock_lds_bytes(int P, int64_t ldp, int tiles, bool svr)
{
    return lock_aux_offset(P, ldp) +
           (size_t)kRowWaves * lock_aux_bytes(P, tiles, svr) +
           (size_t)P * kLockRecBytes;
}

template <bool SVR, int P>
__global__ __launch_bounds__(kRowThreads) void k_lock(LockArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    // each problem's done flag, tested once the first loads are in flight
    bool live[P];
#pragma unroll
    for (int p = 0; p < P; ++p) live[p] = a.ws[p]->done == 0;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, nl = lane & 15;
    const int T = a.tiles, RW = 16 * T;
    const int64_t n = a.n;
    const int ldp = (int)a.ldp;
    const int xstride = rows_xs_stride(ldp);
    float* xsl = reinterpret_cast<float*>(smem);

    // this lane's working-set slot nl of every problem
    double cf[P];
#pragma unroll
    for (int p = 0; p < P; ++p) {
        const int nS = a.ws[p]->nS;
        const double c = a.ws[p]->coef[nl];
        cf[p] = nl < nS ? c : 0.0;
    }

    // rows of this wave, shared out over blocks and waves as in k_rows
    const int64_t TU = (n + 31) >> 5, NB = gridDim.x;
    const int64_t b0 = 32 * ((int64_t)blockIdx.x * TU / NB);
    const int64_t b1 = min(32 * (((int64_t)blockIdx.x + 1) * TU / NB), n);
    const int tb = (int)((b1 - b0 + 15) >> 4);
    const int64_t rw0 = b0 + 16 * (wave * tb / kRowWaves);
    const int nw =
        (int)(min(b0 + 16 * ((wave + 1) * tb / kRowWaves), b1) - rw0);
    const int Tw = (nw + 15) >> 4;

    float* wbuf = xsl + P * 16 * xstride + wave * 16 * kSlabStride;
    unsigned char* aux = smem + lock_aux_offset(P, ldp) +
                         wave * lock_aux_bytes(P, T, SVR);
    double* Fw0 = reinterpret_cast<double*>(aux);  // problem p at p * RW
    float* sqw = reinterpret_cast<float*>(aux + 8 * P * RW);
    float* zw0 = reinterpret_cast<float*>(aux + 8 * P * RW + 4 * RW);
    uint8_t* stw0 = aux + 8 * P * RW + 4 * RW + (SVR ? 4 * P * RW : 0);
    const int stp = SVR ? 2 * RW : RW;  // state bytes per problem
    unsigned char* rec = smem + lock_aux_offset(P, ldp) +
                         kRowWaves * lock_aux_bytes(P, T, SVR);
    double* brk = reinterpret_cast<double*>(rec);  // [P][kRowWaves][4]
    int32_t* bri = reinterpret_cast<int32_t*>(rec + P * kRowWaves * 32);
    float* sl_sq = reinterpret_cast<float*>(rec + P * kRowWaves * 48);
    int32_t* sl_smp =
        reinterpret_cast<int32_t*>(rec + P * kRowWaves * 48 + P * 64);

    // row data of rows k0 .. k0 + 255 of the wave
    struct AuxRegs {
        double f[P][4];
        float q[4], z[P][4];
        uint8_t s0[P][4], s1[P][4];
    };
    auto aux_issue = [&](int k0, AuxRegs& x) {
        const Rsrc rQ = make_rsrc(a.sq + rw0, (int64_t)nw * 4);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            x.q[j] = bld_f32(rQ, 4 * (uint32_t)(k0 + 64 * j + lane));
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const Rsrc rF = make_rsrc(a.F[p] + rw0, (int64_t)nw * 8);
            const Rsrc rS0 = make_rsrc(a.st[p] + rw0, nw);
            const Rsrc rS1 = make_rsrc(a.st[p] + n + rw0, SVR ? nw : 0);
            const Rsrc rZ = make_rsrc(a.z[p] + rw0, SVR ? (int64_t)nw * 4 : 0);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t r = (uint32_t)(k0 + 64 * j + lane);
                x.f[p][j] = bld_f64(rF, 8 * r);
                x.s0[p][j] = bld_u8(rS0, r);
                x.s1[p][j] = SVR ? bld_u8(rS1, r) : 0;
                x.z[p][j] = SVR ? bld_f32(rZ, 4 * r) : 0.0f;
            }
        }
    };
    auto aux_store = [&](int k0, const AuxRegs& x) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = k0 + 64 * j + lane;
            if (r < RW) {
                sqw[r] = x.q[j];
#pragma unroll
                for (int p = 0; p < P; ++p) {
                    Fw0[p * RW + r] = x.f[p][j];
                    stw0[p * stp + r] = x.s0[p][j];
                    if (SVR) {
                        stw0[p * stp + RW + r] = x.s1[p][j];
                        zw0[p * RW + r] = x.z[p][j];
                    }
                }
            }
        }
    };

    Top2 up[P], lo[P];  // this lane's best candidates of each problem
    auto push = [&](int p, int lr, double Fn, bool own) {
        const int32_t row = (int32_t)(rw0 + lr);
        const uint8_t s0 = stw0[p * stp + lr];
        const float z = SVR ? zw0[p * RW + lr] : 0.0f;
        const double r0 = SVR ? (double)z - a.eps[p]
                              : ((s0 & ST_YPOS) ? 1.0 : -1.0);
        const double v0 = r0 - Fn;
        if (own && (s0 & ST_UP)) up[p].push(v0, row);
        if (own && (s0 & ST_LOW)) lo[p].push(-v0, row);
        if (SVR) {
            const uint8_t s1 = stw0[p * stp + RW + lr];
            const double v1 = ((double)z + a.eps[p]) - Fn;
            if (own && (s1 & ST_UP)) up[p].push(v1, (int32_t)(n + row));
            if (own && (s1 & ST_LOW)) lo[p].push(-v1, (int32_t)(n + row));
        }
    };

    // staged working-set rows of all problems (zero-filled to whole
    // 16-feature chunks) and the slot table
    const int q4 = (xstride - 4) >> 2;
    const int xs_total = P * 16 * q4;
    const Rsrc rXs = make_rsrc(a.xS, (int64_t)P * 16 * ldp * 4);
    auto xs_off = [&](int e) -> uint32_t {
        const int slot = e / q4, c4 = e - slot * q4;
        return (e < xs_total && 4 * c4 < ldp)
                   ? (uint32_t)((slot * ldp + 4 * c4) * 4)
                   : kOob;
    };
    const int nslab = (ldp + 63) >> 6;
    const Rsrc rX = make_rsrc(a.X + rw0 * ldp, (int64_t)nw * ldp * 4);
    const uint32_t step4 = (uint32_t)(16 * ldp);  // 4 rows, in bytes
    int fti = 0, fsl = 0;                         // next slab to fetch
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

    float sq0 = 0.0f;
    int32_t smp0 = -1;
#pragma unroll
    for (int p = 0; p < P; ++p) {
        if ((tid >> 4) == p) {
            const int nS = a.ws[p]->nS, s = tid & 15;
            const float q = a.ws[p]->sS[s];
            const int32_t i = a.ws[p]->S[s];
            sq0 = s < nS ? q : 0.0f;
            smp0 = s < nS ? i : -1;
        }
    }
    AuxRegs ar;
    aux_issue(0, ar);
    float4 ring[kRing][4];
    fetch(ring[0]);
    bool any = false;
#pragma unroll
    for (int p = 0; p < P; ++p) any |= live[p];
    if (!any) return;  // uniform over the grid
    // (XB loads in flight per thread; past xs_total they read zero and are
    // not stored)
    constexpr int XB = 8;
    for (int e0 = tid; e0 < xs_total; e0 += XB * kRowThreads) {
        float4 v[XB];
#pragma unroll
        for (int j = 0; j < XB; ++j)
            v[j] = bld_f4(rXs, xs_off(e0 + j * kRowThreads));
#pragma unroll
        for (int j = 0; j < XB; ++j) {
            const int e = e0 + j * kRowThreads;
            const int slot = e / q4, c4 = e - slot * q4;
            if (e < xs_total)
                *reinterpret_cast<float4*>(xsl + slot * xstride + 4 * c4) =
                    v[j];
        }
    }
    aux_store(0, ar);
    if (tid < P * 16) {
        sl_sq[tid] = sq0;
        sl_smp[tid] = smp0;
    }
    for (int k0 = 256; k0 < RW; k0 += 256) {
        aux_issue(k0, ar);
        aux_store(k0, ar);
    }
    // nothing of the staging stays in flight (see k_rows)
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    __syncthreads();
#pragma unroll
    for (int j = 1; j < kRing; ++j) fetch(ring[j]);

    floatx4 acc[P];
    int pti = 0, psl = 0;  // slab being processed
    for (int s0 = 0; s0 < Tw * nslab; s0 += kRing) {
#pragma unroll
        for (int j = 0; j < kRing; ++j) {
            if (psl == 0) {
#pragma unroll
                for (int p = 0; p < P; ++p)
                    acc[p] = floatx4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
                *reinterpret_cast<float4*>(wbuf + (4 * rr + g) * kSlabStride +
                                           4 * nl) = ring[j][rr];
            fetch(ring[j]);  // refill the slot kRing slabs ahead
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int ch = psl * 4 + c;
                if (ch * 16 < ldp) {  // chunk present (uniform)
                    const float4 av =
                        ld4(wbuf + nl * kSlabStride + c * 16 + 4 * g);
                    // the problems' chains interleaved (independent
                    // steps back to back); per problem the order of
                    // mfma_chunk
                    float4 bv[P];
#pragma unroll
                    for (int p = 0; p < P; ++p)
                        bv[p] = ld4(xsl + (p * 16 + nl) * xstride + ch * 16 +
                                    4 * g);
#pragma unroll
                    for (int p = 0; p < P; ++p)
                        acc[p] = mfma4(av.x, bv[p].x, acc[p]);
#pragma unroll
                    for (int p = 0; p < P; ++p)
                        acc[p] = mfma4(av.y, bv[p].y, acc[p]);
#pragma unroll
                    for (int p = 0; p < P; ++p)
                        acc[p] = mfma4(av.z, bv[p].z, acc[p]);
#pragma unroll
                    for (int p = 0; p < P; ++p)
                        acc[p] = mfma4(av.w, bv[p].w, acc[p]);
                }
            }
            __builtin_amdgcn_wave_barrier();
            if (psl == nslab - 1 && pti < Tw) {
                const int lr = 16 * pti + 4 * g;
                const float4 q4v = *reinterpret_cast<const float4*>(sqw + lr);
                const float qv[4] = {q4v.x, q4v.y, q4v.z, q4v.w};
                const int orl = lr + (nl & 3);  // row owned by lanes nl < 4
#pragma unroll
                for (int p = 0; p < P; ++p) {
                    if (!live[p]) continue;  // uniform
                    float kv[4];
                    if (a.kf[p].kind == SVM_KERNEL_RBF) {
                        const float ssb = sl_sq[p * 16 + nl];
                        const int32_t smb = sl_smp[p * 16 + nl];
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            float k = rbf_from_dot(qv[v], ssb, acc[p][v],
                                                   a.kf[p].gexp);
                            if (rw0 + lr + v == (int64_t)smb) k = 1.0f;
                            kv[v] = k;
                        }
                    } else {
#pragma unroll
                        for (int v = 0; v < 4; ++v)
                            kv[v] = kernel_of_dot(a.kf[p], acc[p][v]);
                    }
                    // F_i += sum_s cf_s K(x_i, x_s): the order of k_rows
                    double part[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        part[v] = row_sum_f64(fma(cf[p], (double)kv[v], 0.0));
                    const double Fn = Fw0[p * RW + orl] + pick4(part, nl & 3);
                    if (nl < 4) Fw0[p * RW + orl] = Fn;
                }
            }
            if (++psl == nslab) {
                psl = 0;
                ++pti;
            }
        }
    }
    // the new F back, and the keys of the wave's variables, one row per
    // lane (the candidates do not depend on which lane saw a row)
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int p = 0; p < P; ++p) {
        if (!live[p]) continue;
        const Rsrc rF = make_rsrc(a.F[p] + rw0, (int64_t)nw * 8);
        for (int r0 = 0; r0 < nw; r0 += 64) {
            const int r = r0 + lane;
            const bool own = r < nw;
            const int rr = own ? r : 0;
            const double Fn = Fw0[p * RW + rr];
            if (own) bst_f64(rF, 8 * r, Fn);
            push(p, rr, Fn, own);
        }
    }

    // each problem's best two of each side over the block's rows (as k_rows)
#pragma unroll
    for (int p = 0; p < P; ++p)
        wave_top2_pair(up[p], lo[p], brk + 4 * (p * kRowWaves + wave),
                       bri + 4 * (p * kRowWaves + wave));
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int p = 0; p < P; ++p) {
            if (!live[p]) continue;
            Top2 u, l;
            if (lane < kRowWaves) {
                const int o = 4 * (p * kRowWaves + lane);
                u.k1 = brk[o];
                u.k2 = brk[o + 1];
                l.k1 = brk[o + 2];
                l.k2 = brk[o + 3];
                u.i1 = bri[o];
                u.i2 = bri[o + 1];
                l.i1 = bri[o + 2];
                l.i2 = bri[o + 3];
            }
            wave_top2_pair(u, l,
                           a.cand_key[p] + (size_t)blockIdx.x * 2 * kBlockTop,
                           a.cand_idx[p] + (size_t)blockIdx.x * 2 * kBlockTop);
        }
    }
}

template <bool SVR, int P>
static void lock_dispatch(const LockArgs& a, int nblocks, hipStream_t s,
                          hipEvent_t e0, hipEvent_t e1)
{
    const size_t lds = lock_lds_bytes(P, a.ldp, a.tiles, SVR);
    if (!raise_dynamic_lds((const void*)k_lock<SVR, P>, lds))
        throw Error{SVM_E_UNSUPPORTED,
                    "lockstep row tile needs more LDS than the device allows"};
    if (e0) {
        hipExtLaunchKernelGGL(k_lock<SVR, P>, dim3(nblocks), dim3(kRowThreads),
                              (uint32_t)lds, s, e0, e1, 0, a);
    } else {
        k_lock<SVR, P><<<nblocks, kRowThreads, lds, s>>>(a);
    }
}

template <bool SVR, int P>
static int lock_occupancy(size_t lds)
{
    return occupancy_memo((const void*)k_lock<SVR, P>, kRowThreads, lds);
}

int lock_blocks_per_cu(int P, bool svr, size_t lds)
{
    switch (P * 2 + (svr ? 1 : 0)) {
        case 2: return lock_occupancy<false, 1>(lds);
        case 3: return lock_occupancy<true, 1>(lds);
        case 4: return lock_occupancy<false, 2>(lds);
        case 5: return lock_occupancy<true, 2>(lds);
        case 6: return lock_occupancy<false, 3>(lds);
        case 7: return lock_occupancy<true, 3>(lds);
        case 8: return lock_occupancy<false, 4>(lds);
        case 9: return lock_occupancy<true, 4>(lds);
        default: return 1;
    }
}

void launch_lock(const LockArgs& a, int P, int nblocks, bool svr,
                 hipStream_t s, hipEvent_t e0, hipEvent_t e1)
{
    if (nblocks <= 0) return;
    if ((int64_t)16 * a.tiles * a.ldp * 4 >= ((int64_t)1 << 31))
        throw Error{SVM_E_UNSUPPORTED,
                    "row group too large for the lockstep row kernel"};
    switch (P * 2 + (svr ? 1 : 0)) {
        case 2: lock_dispatch<false, 1>(a, nblocks, s, e0, e1); break;
        case 3: lock_dispatch<true, 1>(a, nblocks, s, e0, e1); break;
        case 4: lock_dispatch<false, 2>(a, nblocks, s, e0, e1); break;
        case 5: lock_dispatch<true, 2>(a, nblocks, s, e0, e1); break;
        case 6: lock_dispatch<false, 3>(a, nblocks, s, e0, e1); break;
        case 7: lock_dispatch<true, 3>(a, nblocks, s, e0, e1); break;
        case 8: lock_dispatch<false, 4>(a, nblocks, s, e0, e1); break;
        case 9: lock_dispatch<true, 4>(a, nblocks, s, e0, e1); break;
        default:
            throw Error{SVM_E_INTERNAL, "bad lockstep problem count"};
    }
}

}  // namespace msvm
