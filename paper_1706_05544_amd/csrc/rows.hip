// Row/update kernel of the working-set dual solve (gfx950).
//
// k_rows runs on the whole grid once per outer iteration (Section 3: the
// responses are updated after the working set has been optimised).  It
// streams X once: for each 16-row tile, the dot products with the (at most
// 16 per column block) working-set samples on the matrix cores (16x16x4
// fp32), the RBF epilogue, F_i += sum_s dc_s K(x_i, x_s) in fp64; then the
// keys v of the variables and per-block candidates of each side for the next
// selection.
#include <hip/hip_ext.h>

#include "common.hpp"
#include "device.hpp"
#include "rowtile.hpp"

namespace msvm {

// ---------------------------------------------------------------------------
// row / update kernel
// ---------------------------------------------------------------------------


// Per-wave LDS bytes for the row data of 16 * tiles rows: F (fp64), the
// squared norm, for eps-SVR the target, and the state byte of each copy
// (dense path only).
__host__ __device__ inline int rows_aux_bytes(int tiles, bool svr, bool csr)
{
    // (the CSR path reads and writes its row data directly, one row per
    // lane)
    return csr ? 0 : ((16 * tiles * (svr ? 18 : 13)) + 15) & ~15;
}

// Floats of the per-wave buffer: a feature slab (dense); the CSR path needs
// none.
__host__ __device__ inline int rows_wave_buf(int nblk_cols, bool csr)
{
    (void)nblk_cols;
    return csr ? 0 : 16 * kSlabStride;
}

// Staged working set.  Dense: nblk_cols * 16 rows of rows_xs_stride floats.
// CSR (csr_cols >= 0): a column map (ldp int32: the compact row of a column
// used by the working set, or -1), then csr_cols + 1 compact rows of
// nblk_cols * 16 floats (the samples' values at one column; the last row is
// zero, for the columns the working set does not use), each padded by 4
// floats: rows then start on 8 different banks, and the 16-byte reads of
// lanes on different rows rarely conflict.
__host__ __device__ inline size_t rows_stage_bytes(int nblk_cols, int64_t ldp,
                                                   int csr_cols)
{
    if (csr_cols < 0)
        return (size_t)nblk_cols * 16 * rows_xs_stride(ldp) * sizeof(float);
    return (((size_t)ldp * 4 + 15) & ~(size_t)15) +
           (size_t)(csr_cols + 1) * (nblk_cols * 16 + 4) * sizeof(float);
}

__host__ __device__ inline size_t rows_aux_offset(int nblk_cols, int64_t ldp,
                                                  int csr_cols)
{
    return rows_stage_bytes(nblk_cols, ldp, csr_cols) +
           (size_t)kRowWaves * rows_wave_buf(nblk_cols, csr_cols >= 0) *
               sizeof(float);
}

// per-block table of the waves' candidate records (see k_rows)
constexpr int kBlockRecBytes = kRowWaves * 4 * (8 + 4);

// per-block table of the working-set slots: norm, sample, cache slot
constexpr int kSlotInfoBytes = kMaxQ * (4 + 4 + 4);

size_t rows_lds_bytes(int nblk_cols, int64_t ldp, int tiles, bool svr,
                      int csr_cols)
{
    return rows_aux_offset(nblk_cols, ldp, csr_cols) +
           (size_t)kRowWaves * rows_aux_bytes(tiles, svr, csr_cols >= 0) +
           kBlockRecBytes +
           kSlotInfoBytes;
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
template <bool SVR, int NBLK, int MODE, bool CSR>
__global__ __launch_bounds__(kRowThreads) void k_rows(RowArgs a)
{
    constexpr bool UPD = (MODE & RU_UPDATE) != 0;
    constexpr bool ROWS = (MODE & RU_ROWS) != 0;
    constexpr bool CAND = (MODE & RU_CAND) != 0;
    constexpr bool XS = UPD || ROWS;  // the working-set samples are needed
    // hot mode (a training iteration): the update and the candidates, with
    // the kernel-row cache
    constexpr bool HOT = UPD && CAND;
    constexpr int kXsEarly = 2;       // staging loads issued with the stream
    extern __shared__ __align__(16) unsigned char smem[];
    const WorkingSet* ws = a.ws;
    // (RU_CHECK_DONE) the test of ws->done waits until the first loads are
    // in flight, so that its round trip overlaps theirs
    const int32_t done = (MODE & RU_CHECK_DONE) ? ws->done : 0;
    if (!XS && done) return;

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
#pragma unroll
    for (int b = 0; b < NBLK; ++b) {
        const int slot = b * 16 + nl;  // < kMaxQ: always inside the arrays
        const double c = ws->coef[slot];
        cf[b] = (slot < nS && UPD) ? c : 0.0;
    }

    // rows of this wave: rw0 .. rw0 + nw - 1, in Tw <= T tiles of 16.  The
    // ceil(n / 32) units of 32 rows are shared out evenly over the blocks
    // (so that no compute unit holds more of them than another, and the
    // part of a block of every per-row fp32 array, norms and cached kernel
    // rows, covers whole 128-byte lines: blocks sit on different L2s), and
    // the block's 16-row tiles evenly over its waves.
    const int64_t TU = (n + 31) >> 5, NB = gridDim.x;
    const int64_t b0 = 32 * ((int64_t)blockIdx.x * TU / NB);
    const int64_t b1 = min(32 * (((int64_t)blockIdx.x + 1) * TU / NB), n);
    const int tb = (int)((b1 - b0 + 15) >> 4);
    const int64_t rw0 = b0 + 16 * (wave * tb / kRowWaves);
    const int nw = (int)(min(b0 + 16 * ((wave + 1) * tb / kRowWaves), b1) - rw0);
    const int Tw = (nw + 15) >> 4;
    unsigned char* aux =
        smem + rows_aux_offset(NBLK, ldp, CSR ? a.csr_cols : -1) +
        wave * rows_aux_bytes(T, SVR, CSR);
    double* Fw = reinterpret_cast<double*>(aux);
    float* sqw = reinterpret_cast<float*>(aux + 8 * RW);
    float* zw = reinterpret_cast<float*>(aux + 12 * RW);
    uint8_t* stw = aux + (SVR ? 16 : 12) * RW;  // copy (i,-) at stw[RW + r]
    unsigned char* brec = smem + rows_aux_offset(NBLK, ldp, CSR ? a.csr_cols : -1) +
                          kRowWaves * rows_aux_bytes(T, SVR, CSR);
    double* brk = reinterpret_cast<double*>(brec);  // [kRowWaves][4]
    int32_t* bri = reinterpret_cast<int32_t*>(brec + kRowWaves * 32);
    // slot table (block-wide): norm, sample and cache slot of every slot
    unsigned char* sinfo = smem + rows_aux_offset(NBLK, ldp, CSR ? a.csr_cols : -1) +
                           kRowWaves * rows_aux_bytes(T, SVR, CSR) + kBlockRecBytes;
    float* sl_sq = reinterpret_cast<float*>(sinfo);
    int32_t* sl_smp = reinterpret_cast<int32_t*>(sinfo + 4 * kMaxQ);
    int32_t* sl_cs = reinterpret_cast<int32_t*>(sinfo + 8 * kMaxQ);

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
    // keys of the variables of row lr (only lanes with own = true hold one)
    auto push_vals = [&](int32_t row, double Fn, uint8_t s0, uint8_t s1,
                         float z, bool own) {
        const double r0 = SVR ? (double)z - a.eps
                              : ((s0 & ST_YPOS) ? 1.0 : -1.0);
        const double v0 = r0 - Fn;
        const bool u0 = own && (s0 & ST_UP), l0 = own && (s0 & ST_LOW);
        if (u0) up.push(v0, row);
        if (l0) lo.push(-v0, row);
        if (SVR) {
            const double v1 = ((double)z + a.eps) - Fn;
            const bool u1 = own && (s1 & ST_UP), l1 = own && (s1 & ST_LOW);
            if (u1) up.push(v1, (int32_t)(n + row));
            if (l1) lo.push(-v1, (int32_t)(n + row));
        }
    };
    auto push = [&](int lr, double Fn, bool own) {
        push_vals((int32_t)(rw0 + lr), Fn, stw[lr], SVR ? stw[RW + lr] : 0,
                  SVR ? zw[lr] : 0.0f, own);
    };
    // Row data of one row per lane for the CSR path (loads past the wave's
    // rows read zero): F, norm, state bytes, target.
    struct RowVals {
        double f;
        float q, z;
        uint8_t s0, s1;
    };
    auto row_vals = [&](int r, RowVals& v) {
        const Rsrc rQ = make_rsrc(a.sq + rw0, (int64_t)nw * 4);
        const Rsrc rS0 = make_rsrc(a.st + rw0, nw);
        const Rsrc rS1 = make_rsrc(a.st + n + rw0, SVR ? nw : 0);
        const Rsrc rZ = make_rsrc(a.z + rw0, SVR ? (int64_t)nw * 4 : 0);
        const uint32_t u = (uint32_t)r;
        v.f = (UPD || CAND) ? bld_f64(rF, 8 * u) : 0.0;
        v.q = XS ? bld_f32(rQ, 4 * u) : 0.0f;
        v.s0 = CAND ? bld_u8(rS0, u) : 0;
        v.s1 = (SVR && CAND) ? bld_u8(rS1, u) : 0;
        v.z = (SVR && CAND) ? bld_f32(rZ, 4 * u) : 0.0f;
    };

    if (XS) {
        // Path of this iteration (hot mode: set by the selection; tests:
        // always computed from X) and the cache slot of this lane's
        // working-set slots.
        const int32_t path = HOT ? ws->path : PATH_STREAM;
        // (dense, hot mode) the cache slot of this lane's working-set slots,
        // requested with the path and waited for with it: issued inside the
        // cached branch, it would be a second round trip after the path's
        int32_t cs_in[NBLK];
#pragma unroll
        for (int b = 0; b < NBLK; ++b) {
            cs_in[b] = (HOT && !CSR) ? ws->cslot[b * 16 + nl] : -1;
            if (HOT && !CSR) asm volatile("" ::"v"(cs_in[b]));
        }

        // F_i += sum_s cf_s K(x_i, x_s) for the 16 rows of tile ti, given
        // this lane's K values kv[b][v] (row lr + v of slot b * 16 + nl),
        // then the keys of the tile's variables.  The same code (and fp64
        // order) whether K was computed or read from the cache.
        auto finish_tile = [&](int ti, const float (&kv)[NBLK][4]) {
            const int lr = 16 * ti + 4 * g;
            double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int b = 0; b < NBLK; ++b) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    part[v] = fma(cf[b], (double)kv[b][v], part[v]);
                    if (ROWS && b * 16 + nl < nS && lr + v < nw)
                        a.rows_out[(int64_t)(b * 16 + nl) * n + rw0 + lr + v] =
                            kv[b][v];
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
            if (CAND) push(orl, Fn, nl < 4 && orl < nw);
        };

        if (CSR) {
            // CSR rows, one row per lane in groups of 64 (its row data read
            // and F written directly).  Computed path: the working set sits
            // by column in LDS: colmap[j] is the float offset e * QT in xsT
            // of the compact row e of column j (-1: no sample has it),
            // xsT[e * QT + s] = x_s[cols[e]] (rows padded to QT floats).
            // Each lane walks its row's nonzeros in column order and, per
            // nonzero, reads the QS samples' values of its column: K(x_i,
            // x_s) sums the products of the common nonzeros in increasing
            // column order (every CSR kernel of the library sums them so;
            // the products with a zero add nothing, exactly).  Cached path:
            // the lane reads K(x_i, x_s) of its row from the cached rows.
            // Either way the same epilogue and fp64 order.
            constexpr int QS = NBLK * 16, QT = QS + 4;
            const int CC = a.csr_cols;
            const bool CACHED = HOT && path == PATH_CACHED;  // uniform
            const bool INS = HOT && path == PATH_INSERT;
            int32_t* colmap = reinterpret_cast<int32_t*>(smem);
            float* xsT =
                reinterpret_cast<float*>(smem + ((ldp * 4 + 15) & ~15));
            float sq0 = 0.0f;
            int32_t smp0 = -1, cs0 = -1;
            if (tid < QS) {
                const float q = ws->sS[tid];
                const int32_t i = ws->S[tid], c = ws->cslot[tid];
                sq0 = tid < nS ? q : 0.0f;
                smp0 = tid < nS ? i : -1;
                cs0 = (HOT && tid < nS) ? c : -1;
            }
            if (done) return;  // uniform over the block
            if (!CACHED)
                for (int e = tid; e < ldp; e += kRowThreads) colmap[e] = -1;
            if (tid < QS) {
                sl_sq[tid] = sq0;
                sl_smp[tid] = smp0;
                sl_cs[tid] = cs0;
            }
            __syncthreads();  // column map cleared, slot table written
            if (!CACHED) {
                // the compact columns and rows, 8 loads in flight per thread
                constexpr int XB = 8;
                for (int e0 = tid; e0 < CC; e0 += XB * kRowThreads) {
                    int32_t c[XB];
#pragma unroll
                    for (int j = 0; j < XB; ++j)
                        c[j] = a.xsc_cols[min(e0 + j * kRowThreads, CC - 1)];
#pragma unroll
                    for (int j = 0; j < XB; ++j)
                        if (e0 + j * kRowThreads < CC && c[j] >= 0)
                            colmap[c[j]] = (e0 + j * kRowThreads) * QT;
                }
                const int n4 = (CC + 1) * QS / 4;
                auto xs_at = [&](int e) {  // float4 e of the table in LDS
                    const int row = e / (QS / 4), j = e - row * (QS / 4);
                    return xsT + row * QT + 4 * j;
                };
                for (int e0 = tid; e0 < n4; e0 += XB * kRowThreads) {
                    float4 v[XB];
#pragma unroll
                    for (int j = 0; j < XB; ++j)
                        v[j] = ld4(a.xsc +
                                   4 * min(e0 + j * kRowThreads, n4 - 1));
#pragma unroll
                    for (int j = 0; j < XB; ++j)
                        if (e0 + j * kRowThreads < n4)
                            *reinterpret_cast<float4*>(
                                xs_at(e0 + j * kRowThreads)) = v[j];
                }
            }
            // nothing stays in flight (a load whose value is unused would
            // make the row loop wait for all loads at every batch)
            __builtin_amdgcn_s_waitcnt(kVmcnt0);
            __syncthreads();

            // every working-set coefficient (uniform over the wave)
            double cfa[QS];
#pragma unroll
            for (int q = 0; q < QS; ++q) {
                const double c = ws->coef[q];
                cfa[q] = uniform_f64((UPD && q < nS) ? c : 0.0);
            }

            // The epilogue of the row of this lane (local row r) from its K
            // values: cache fill (insert path), test rows, F_i += sum_s cf_s
            // K_is in the order of the 16-lane rotation sum of the tiled
            // epilogue (so the dense and CSR kernels order F's update
            // alike), then the keys of its variables.
            auto finish_row = [&](int r, bool rv, const float (&kv)[QS],
                                  const RowVals& rd) {
                if (rv) {
                    if (INS) {
#pragma unroll
                        for (int q = 0; q < QS; ++q) {
                            const int32_t cs = sl_cs[q];
                            if (cs >= 0)
                                a.cache[(int64_t)cs * a.ldc + rw0 + r] = kv[q];
                        }
                    }
                    if (ROWS) {
#pragma unroll
                        for (int q = 0; q < QS; ++q)
                            if (q < nS)
                                a.rows_out[(int64_t)q * n + rw0 + r] = kv[q];
                    }
                }
                double Fn = rd.f;
                if (UPD) {
                    // t_s = sum_b cf K (fma from 0, b ascending); then
                    // ((t_s + t_s+8) + (t_s+4 + t_s+12)) pairwise down to
                    // one sum: the rotation order, term by term
                    auto term = [&](int s) {
                        double t = 0.0;
#pragma unroll
                        for (int b = 0; b < NBLK; ++b)
                            t = fma(cfa[b * 16 + s], (double)kv[b * 16 + s], t);
                        return t;
                    };
                    auto quad = [&](int s) {  // s < 4
                        return (term(s) + term(s + 8)) +
                               (term(s + 4) + term(s + 12));
                    };
                    Fn += (quad(0) + quad(2)) + (quad(1) + quad(3));
                    bst_f64(rF, 8 * (uint32_t)r, Fn);  // dropped past nw
                }
                if (CAND)
                    push_vals((int32_t)(rw0 + r), Fn, rd.s0, rd.s1, rd.z, rv);
            };

            if (CACHED) {
                // K(x_i, x_s) of this lane's row from the cached rows of the
                // slots, the next group's requested while this one is done
                const float* crow[QS];
#pragma unroll
                for (int q = 0; q < QS; ++q) {
                    const int32_t cs = __builtin_amdgcn_readfirstlane(sl_cs[q]);
                    crow[q] = a.cache + (int64_t)(cs >= 0 ? cs : 0) * a.ldc +
                              (cs >= 0 ? rw0 : 0);
                }
                auto cfetch = [&](int p0, float (&kv)[QS], RowVals& rd) {
                    const int r = 16 * p0 + lane;
                    const int rr = r < nw ? r : 0;  // an address in the row
#pragma unroll
                    for (int q = 0; q < QS; ++q) kv[q] = crow[q][rr];
                    row_vals(r, rd);
                };
                float nkv[QS];
                RowVals nrd;
                cfetch(0, nkv, nrd);
                for (int p0 = 0; p0 < Tw; p0 += 4) {
                    const int r = 16 * p0 + lane;
                    const bool rv = r < nw;
                    float kv[QS];
#pragma unroll
                    for (int q = 0; q < QS; ++q)
                        kv[q] = sl_cs[q] >= 0 ? nkv[q] : 0.0f;
                    const RowVals rd = nrd;
                    cfetch(p0 + 4, nkv, nrd);
                    finish_row(r, rv, kv, rd);
                }
            } else {
                // The wave's nonzeros through buffer resources based at its
                // first row: the sliced copy (a.so; nonzero k of a row
                // kSellRows entries after nonzero k - 1, the row padded with
                // zeros to its slice's width; 16-bit columns) or the CSR
                // rows.  Offsets are below 2^31 (16 * tiles * ldp * 4 is,
                // checked at launch), so a 16-bit column's offset (half the
                // value's) is below 2^30, and so is its range: half of kOob
                // still lies past it.  A load past the wave's nonzeros reads
                // zero.
                const bool sell = a.so != nullptr;  // uniform
                int64_t e_beg, e_end;
                if (sell) {
                    const int64_t ns = (n + kSellRows - 1) / kSellRows;
                    e_beg = a.so[rw0 / kSellRows];
                    e_end = a.so[min((rw0 + nw + kSellRows - 1) / kSellRows,
                                     ns)];
                } else {
                    e_beg = a.rp[rw0];
                    e_end = a.rp[rw0 + nw];
                }
                // (values the same on every lane: said so, so that the
                // resources live in scalar registers)
                e_beg = uniform_i64(e_beg);
                e_end = uniform_i64(e_end);
                const Rsrc rCI =
                    sell ? make_rsrc(a.sci + e_beg, 2 * (e_end - e_beg))
                         : make_rsrc(a.ci + e_beg, 4 * (e_end - e_beg));
                const Rsrc rCV = make_rsrc((sell ? a.scv : a.cv) + e_beg,
                                           4 * (e_end - e_beg));
                // byte offset of nonzero 0 and the nonzeros (sliced: the
                // slice width) of this lane's row in the group p0 .. p0 + 3
                auto row_ptrs = [&](int p0, uint32_t& lo, int& nz) {
                    const int r = 16 * p0 + lane;
                    const bool v = r < nw;
                    const int64_t gr = v ? rw0 + r : 0;
                    int64_t k0, k1;
                    if (sell) {
                        const int64_t sl = gr / kSellRows;
                        const int64_t o0 = a.so[sl], o1 = a.so[sl + 1];
                        k0 = o0 + (gr - sl * kSellRows);
                        k1 = k0 + (o1 - o0) / kSellRows;
                    } else {
                        k0 = a.rp[gr];
                        k1 = a.rp[gr + 1];
                    }
                    lo = v ? (uint32_t)(4 * (k0 - e_beg)) : kOob;
                    nz = v ? (int)(k1 - k0) : 0;
                };

                // Per nonzero (column c, value v) of the row: acc[s] += v *
                // x_s[c] from the table row at colmap[c]; a column no sample
                // holds adds exact zeros, so its lanes sit out (the table
                // reads are the LDS cost).  Nonzeros come in batches of KB,
                // two batches in flight (ping-pong registers: a batch is
                // waited for only when it is summed).
                auto run = [&](auto stride_tag) {
                    constexpr uint32_t STR = decltype(stride_tag)::value;
                    constexpr int KB = 8;
                    auto issue = [&](uint32_t vo, int32_t (&cc)[KB],
                                     float (&vv)[KB]) {
#pragma unroll
                        for (int j = 0; j < KB; ++j) {
                            // (sliced copy: 16-bit columns, half the offset)
                            cc[j] = STR == 4 ? bld_i32(rCI, vo + STR * j)
                                             : (int32_t)bld_u16(
                                                   rCI, (vo >> 1) + (STR >> 1) * j);
                            vv[j] = bld_f32(rCV, vo + STR * j);
                        }
                    };
                    auto consume = [&](int kb, int nz, const int32_t (&cc)[KB],
                                       const float (&vv)[KB],
                                       float (&acc)[QS]) {
                        int m[KB];
#pragma unroll
                        for (int j = 0; j < KB; ++j) m[j] = colmap[cc[j]];
#pragma unroll
                        for (int j = 0; j < KB; ++j) {
                            if (kb + j < nz && m[j] >= 0) {
                                const float* xr = xsT + m[j];
#pragma unroll
                                for (int q = 0; q < QS; q += 4) {
                                    const float4 x = ld4(xr + q);
                                    acc[q + 0] = fmaf(vv[j], x.x, acc[q + 0]);
                                    acc[q + 1] = fmaf(vv[j], x.y, acc[q + 1]);
                                    acc[q + 2] = fmaf(vv[j], x.z, acc[q + 2]);
                                    acc[q + 3] = fmaf(vv[j], x.w, acc[q + 3]);
                                }
                            }
                        }
                    };
                    auto wave_max = [&](int v) {
#pragma unroll
                        for (int off = 32; off > 0; off >>= 1)
                            v = max(v, __shfl_xor(v, off));
                        return __builtin_amdgcn_readfirstlane(v);
                    };
                    uint32_t nlo;
                    int nnz_next;
                    RowVals nrd;
                    row_ptrs(0, nlo, nnz_next);
                    row_vals(lane, nrd);
                    // the first batch of the next group, requested before
                    // this group's epilogue (which then covers its latency)
                    int32_t cn[KB];
                    float vn[KB];
                    int mx_next = wave_max(nnz_next);
                    issue(mx_next > 0 ? nlo : kOob, cn, vn);
                    for (int p0 = 0; p0 < Tw; p0 += 4) {
                        const int r = 16 * p0 + lane;  // this lane's row
                        const bool rv = r < nw;
                        const uint32_t lo = nlo;
                        const int nz = nnz_next;
                        const int mx = mx_next;
                        const RowVals rd = nrd;
                        row_ptrs(p0 + 4, nlo, nnz_next);
                        row_vals(r + 64, nrd);
                        float acc[QS];
#pragma unroll
                        for (int q = 0; q < QS; ++q) acc[q] = 0.0f;
                        int32_t ca[KB], cb[KB];
                        float va[KB], vb[KB];
#pragma unroll
                        for (int j = 0; j < KB; ++j) {
                            ca[j] = cn[j];
                            va[j] = vn[j];
                        }
                        for (int kb = 0;;) {
                            issue(kb + KB < mx ? lo + STR * (kb + KB) : kOob,
                                  cb, vb);
                            consume(kb, nz, ca, va, acc);
                            kb += KB;
                            if (kb >= mx) break;
                            issue(kb + KB < mx ? lo + STR * (kb + KB) : kOob,
                                  ca, va);
                            consume(kb, nz, cb, vb, acc);
                            kb += KB;
                            if (kb >= mx) break;
                        }
                        mx_next = p0 + 4 < Tw ? wave_max(nnz_next) : 0;
                        issue(mx_next > 0 ? nlo : kOob, cn, vn);
                        float kv[QS];
                        if (a.kf.kind == SVM_KERNEL_RBF) {
#pragma unroll
                            for (int q = 0; q < QS; ++q) {
                                float k = rbf_from_dot(rd.q, sl_sq[q], acc[q],
                                                       a.kf.gexp);
                                if (rw0 + r == (int64_t)sl_smp[q]) k = 1.0f;
                                kv[q] = k;
                            }
                        } else {
#pragma unroll
                            for (int q = 0; q < QS; ++q)
                                kv[q] = kernel_of_dot(a.kf, acc[q]);
                        }
                        finish_row(r, rv, kv, rd);
                    }
                };
                if (sell)
                    run(std::integral_constant<uint32_t, 4 * kSellRows>{});
                else
                    run(std::integral_constant<uint32_t, 4>{});
            }
        } else         if (HOT && path == PATH_CACHED) {
            // Every working-set sample is cached: lane (g, nl) reads rows
            // lr .. lr + 3 of its slot's row as one float4, kRing tiles
            // ahead.  Unused slots read a valid address and are zeroed.
            int32_t cs[NBLK];
#pragma unroll
            for (int b = 0; b < NBLK; ++b) cs[b] = b * 16 + nl < nS ? cs_in[b] : -1;
            const float* crow[NBLK];
#pragma unroll
            for (int b = 0; b < NBLK; ++b)
                crow[b] = a.cache + (int64_t)(cs[b] >= 0 ? cs[b] : 0) * a.ldc +
                          (nw > 0 ? rw0 : 0);
            auto cfetch = [&](int ti, float4 (&v)[NBLK]) {
                const int t = min(ti, max(Tw - 1, 0));  // a valid tile
#pragma unroll
                for (int b = 0; b < NBLK; ++b)
                    v[b] = ld4(crow[b] + 16 * t + 4 * g);
            };
            float4 ring[kRing][NBLK];
#pragma unroll
            for (int j = 0; j < kRing; ++j) cfetch(j, ring[j]);
            AuxRegs ar;
            aux_issue(0, ar);
            if (done) return;  // uniform over the block
            aux_store(0, ar);
            for (int k0 = 256; k0 < RW; k0 += 256) {
                aux_issue(k0, ar);
                aux_store(k0, ar);
            }
            for (int t0 = 0; t0 < Tw; t0 += kRing) {
#pragma unroll
                for (int j = 0; j < kRing; ++j) {
                    float kv[NBLK][4];
#pragma unroll
                    for (int b = 0; b < NBLK; ++b) {
                        const float4 c = ring[j][b];
                        const bool ok = cs[b] >= 0;
                        kv[b][0] = ok ? c.x : 0.0f;
                        kv[b][1] = ok ? c.y : 0.0f;
                        kv[b][2] = ok ? c.z : 0.0f;
                        kv[b][3] = ok ? c.w : 0.0f;
                    }
                    cfetch(t0 + j + kRing, ring[j]);
                    if (t0 + j < Tw) finish_tile(t0 + j, kv);
                }
            }
        } else {
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
                    *reinterpret_cast<float4*>(xsl + slot * xstride + 4 * c4) =
                        v;
            };

            const int nslab = (ldp + 63) >> 6;
            const Rsrc rX = make_rsrc(a.X + rw0 * ldp, (int64_t)nw * ldp * 4);
            float* wbuf = xsl + NBLK * 16 * xstride +
                          wave * rows_wave_buf(NBLK, false);
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

            // Everything the first slabs need is requested at once: the
            // first staging loads, the slot table, the row data and kRing
            // feature slabs.
            float sq0 = 0.0f;
            int32_t smp0 = -1, cs0 = -1;
            if (tid < NBLK * 16) {
                const float q = ws->sS[tid];
                const int32_t i = ws->S[tid], c = ws->cslot[tid];
                sq0 = tid < nS ? q : 0.0f;
                smp0 = tid < nS ? i : -1;
                cs0 = (HOT && tid < nS) ? c : -1;
            }
            float4 xv[kXsEarly];
#pragma unroll
            for (int i = 0; i < kXsEarly; ++i)
                xv[i] = bld_f4(rXs, xs_off(tid + i * kRowThreads));
            AuxRegs ar;
            aux_issue(0, ar);
            float4 ring[kRing][4];
            fetch(ring[0]);
            if (done) return;  // uniform over the block
#pragma unroll
            for (int i = 0; i < kXsEarly; ++i)
                xs_put(tid + i * kRowThreads, xv[i]);
            aux_store(0, ar);
            if (tid < NBLK * 16) {
                sl_sq[tid] = sq0;
                sl_smp[tid] = smp0;
                sl_cs[tid] = cs0;
            }
            // Row data past the first 256 rows and staged rows past the
            // early loads (large tiles or many features), behind a uniform
            // branch: their loads wait for everything in flight, the slabs
            // included, so the common shapes do not pass through them.
            if (RW > 256 || xs_total > kXsEarly * kRowThreads) {
                for (int k0 = 256; k0 < RW; k0 += 256) {
                    aux_issue(k0, ar);
                    aux_store(k0, ar);
                }
                for (int e = tid + kXsEarly * kRowThreads; e < xs_total;
                     e += kRowThreads)
                    xs_put(e, bld_f4(rXs, xs_off(e)));
                // nothing of these loops stays in flight (a load whose value
                // is unused would otherwise make the slab loop wait for all
                // loads at every slab)
                __builtin_amdgcn_s_waitcnt(kVmcnt0);
            }
            __syncthreads();
#pragma unroll
            for (int j = 1; j < kRing; ++j) fetch(ring[j]);

            // The slab loop; on the insert path the rows of the samples
            // missing from the cache also go to their new cache slots.
            {
                const bool INS = HOT && path == PATH_INSERT;
                floatx4 acc[NBLK];
                int pti = 0, psl = 0;  // slab being processed
                for (int s0 = 0; s0 < Tw * nslab; s0 += kRing) {
                    // all kRing slots every trip (slabs past the end are
                    // zeros and touch no memory), so the loads in flight
                    // are countable
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
                                const float4 av = ld4(wbuf + nl * kSlabStride +
                                                      c * 16 + 4 * g);
#pragma unroll
                                for (int b = 0; b < NBLK; ++b) {
                                    const float4 bv =
                                        ld4(xsl + (b * 16 + nl) * xstride +
                                            ch * 16 + 4 * g);
                                    acc[b] = mfma_chunk(acc[b], av, bv);
                                }
                            }
                        }
                        __builtin_amdgcn_wave_barrier();
                        if (psl == nslab - 1 && pti < Tw) {
                            const int lr = 16 * pti + 4 * g;
                            const float4 q4v =
                                *reinterpret_cast<const float4*>(sqw + lr);
                            const float qv[4] = {q4v.x, q4v.y, q4v.z, q4v.w};
                            float kv[NBLK][4];
                            if (a.kf.kind == SVM_KERNEL_RBF) {
#pragma unroll
                                for (int b = 0; b < NBLK; ++b) {
                                    const float ssb = sl_sq[b * 16 + nl];
                                    const int32_t smb = sl_smp[b * 16 + nl];
#pragma unroll
                                    for (int v = 0; v < 4; ++v) {
                                        float k = rbf_from_dot(qv[v], ssb,
                                                               acc[b][v],
                                                               a.kf.gexp);
                                        if (rw0 + lr + v == (int64_t)smb)
                                            k = 1.0f;
                                        kv[b][v] = k;
                                    }
                                }
                            } else {
#pragma unroll
                                for (int b = 0; b < NBLK; ++b)
#pragma unroll
                                    for (int v = 0; v < 4; ++v)
                                        kv[b][v] = kernel_of_dot(a.kf,
                                                                 acc[b][v]);
                            }
#pragma unroll
                            for (int b = 0; b < NBLK; ++b) {
                                // rows lr .. lr+3 of a row stored padded to
                                // ldc (a multiple of 4): in bounds when row
                                // lr is
                                const int32_t csb = INS ? sl_cs[b * 16 + nl] : -1;
                                if (csb >= 0 && rw0 + lr < n)
                                    *reinterpret_cast<float4*>(
                                        a.cache + (int64_t)csb * a.ldc + rw0 +
                                        lr) = make_float4(kv[b][0], kv[b][1],
                                                          kv[b][2], kv[b][3]);
                            }
                            finish_tile(pti, kv);
                        }
                        if (++psl == nslab) {
                            psl = 0;
                            ++pti;
                        }
                    }
                }
            }
        }
        if (UPD && !CSR)
            for (int r = lane; r < nw; r += 64) bst_f64(rF, 8 * r, Fw[r]);
    } else if (CAND) {
        if (CSR) {
            // keys of the wave's variables, one row per lane, read directly
            for (int r0 = 0; r0 < nw; r0 += 64) {
                const int r = r0 + lane;
                RowVals rd;
                row_vals(r, rd);
                push_vals((int32_t)(rw0 + r), rd.f, rd.s0, rd.s1, rd.z, r < nw);
            }
        } else {
            AuxRegs ar;
            for (int k0 = 0; k0 < RW; k0 += 256) {
                aux_issue(k0, ar);
                aux_store(k0, ar);
            }
            // keys of the wave's variables, one row per lane
            for (int r0 = 0; r0 < nw; r0 += 64) {
                const int r = r0 + lane;
                const bool own = r < nw;
                const int rr = own ? r : 0;
                push(rr, Fw[rr], own);
            }
        }
    }

    if (!CAND) return;
    // The best two of each side over the block's rows: every wave's best
    // two go to the block table, then wave 0 takes the best two of those.
    // A variable outside the global top q/2 never needs more (k_select
    // rescans a row group whose two candidates were both taken).
    wave_top2_pair(up, lo, brk + 4 * wave, bri + 4 * wave);
    __syncthreads();
    if (wave == 0) {
        Top2 u, l;
        if (lane < kRowWaves) {
            u.k1 = brk[4 * lane];
            u.k2 = brk[4 * lane + 1];
            l.k1 = brk[4 * lane + 2];
            l.k2 = brk[4 * lane + 3];
            u.i1 = bri[4 * lane];
            u.i2 = bri[4 * lane + 1];
            l.i1 = bri[4 * lane + 2];
            l.i2 = bri[4 * lane + 3];
        }
        wave_top2_pair(u, l, a.cand_key + (size_t)blockIdx.x * 2 * kBlockTop,
                       a.cand_idx + (size_t)blockIdx.x * 2 * kBlockTop);
    }
}

template <bool SVR, int NBLK, int MODE, bool CSR>
static void rows_dispatch(const RowArgs& a, int nblocks, hipStream_t s,
                          hipEvent_t e0, hipEvent_t e1)
{
    const size_t lds = rows_lds_bytes(NBLK, a.ldp, a.tiles, SVR,
                                      CSR ? a.csr_cols : -1);
    if (!raise_dynamic_lds((const void*)k_rows<SVR, NBLK, MODE, CSR>, lds))
        throw Error{SVM_E_UNSUPPORTED,
                    "row tile needs more LDS than the device allows"};
    if (e0) {
        hipExtLaunchKernelGGL(k_rows<SVR, NBLK, MODE, CSR>, dim3(nblocks),
                              dim3(kRowThreads), (uint32_t)lds, s, e0, e1, 0,
                              a);
    } else {
        k_rows<SVR, NBLK, MODE, CSR><<<nblocks, kRowThreads, lds, s>>>(a);
    }
}

constexpr int kModeHot = RU_UPDATE | RU_CAND | RU_CHECK_DONE;

template <bool SVR, int NBLK, bool CSR>
static void rows_mode(const RowArgs& a, int nblocks, hipStream_t s,
                      hipEvent_t e0, hipEvent_t e1)
{
    switch (a.mode) {
        case kModeHot:
            rows_dispatch<SVR, NBLK, kModeHot, CSR>(a, nblocks, s, e0, e1);
            break;
        case RU_CAND:
            rows_dispatch<SVR, NBLK, RU_CAND, CSR>(a, nblocks, s, e0, e1);
            break;
        case RU_ROWS:
            rows_dispatch<SVR, NBLK, RU_ROWS, CSR>(a, nblocks, s, e0, e1);
            break;
        case RU_UPDATE:
            rows_dispatch<SVR, NBLK, RU_UPDATE, CSR>(a, nblocks, s, e0, e1);
            break;
        default: throw Error{SVM_E_INTERNAL, "bad row kernel mode"};
    }
}

template <bool SVR, int NBLK, bool CSR>
static int rows_occupancy(size_t lds)
{
    return occupancy_memo(
        (const void*)k_rows<SVR, NBLK, kModeHot, CSR>, kRowThreads, lds);
}

// The CSR row kernel covers up to 32 working-set slots (its per-lane
// accumulators); q = 64 with CSR input is refused by the solver.
int rows_blocks_per_cu(int nblk_cols, bool svr, size_t lds, bool csr)
{
    switch (nblk_cols * 4 + (svr ? 2 : 0) + (csr ? 1 : 0)) {
        case 4: return rows_occupancy<false, 1, false>(lds);
        case 5: return rows_occupancy<false, 1, true>(lds);
        case 6: return rows_occupancy<true, 1, false>(lds);
        case 7: return rows_occupancy<true, 1, true>(lds);
        case 8: return rows_occupancy<false, 2, false>(lds);
        case 9: return rows_occupancy<false, 2, true>(lds);
        case 10: return rows_occupancy<true, 2, false>(lds);
        case 11: return rows_occupancy<true, 2, true>(lds);
        case 16: return rows_occupancy<false, 4, false>(lds);
        case 18: return rows_occupancy<true, 4, false>(lds);
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
    const bool csr = a.rp != nullptr;
    switch (nblk_cols * 4 + (svr ? 2 : 0) + (csr ? 1 : 0)) {
        case 4: rows_mode<false, 1, false>(a, nblocks, s, e0, e1); break;
        case 5: rows_mode<false, 1, true>(a, nblocks, s, e0, e1); break;
        case 6: rows_mode<true, 1, false>(a, nblocks, s, e0, e1); break;
        case 7: rows_mode<true, 1, true>(a, nblocks, s, e0, e1); break;
        case 8: rows_mode<false, 2, false>(a, nblocks, s, e0, e1); break;
        case 9: rows_mode<false, 2, true>(a, nblocks, s, e0, e1); break;
        case 10: rows_mode<true, 2, false>(a, nblocks, s, e0, e1); break;
        case 11: rows_mode<true, 2, true>(a, nblocks, s, e0, e1); break;
        case 16: rows_mode<false, 4, false>(a, nblocks, s, e0, e1); break;
        case 18: rows_mode<true, 4, false>(a, nblocks, s, e0, e1); break;
        default:
            throw Error{SVM_E_UNSUPPORTED,
                        "CSR input supports working sets of at most 32"};
    }
}

}  // namespace msvm
