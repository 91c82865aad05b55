// Batched decision function D(x) = sum_j c_j K(sv_j, x) + b (gfx950).
//
// The paper times training together with prediction (Section 5, Fig. 1);
// the same kernel recomputes the responses F_i = sum_j c_j K(x_j, x_i) from
// scratch once the incremental solve has converged.
//
// Tiling: a block of 4 waves owns 64 test rows (16 per wave, the MFMA row
// tile) and one range of the support rows (up to 8 ranges of whole 64-row
// tiles, set by the number of support rows), which it walks 64 rows at a
// time.  Each wave accumulates its 16 x 64 dot products on the matrix cores
// in the feature order shared with the training kernels, applies the RBF
// epilogue and accumulates c_j K in fp64 per lane; the per-lane partial sums
// are reduced across the 16 support columns at the end of the range.  With
// one range that is the output (+ b); with several, each range's sums go to
// a buffer that k_predict_sum adds in range order, so each output is
// written once, without atomics, and the same bits whatever the batch.
// k_predict stages both operand tiles in LDS by 64-feature chunks (row
// stride padded by 4 floats against bank conflicts); for rows of at most
// 128 features k_predict_ra keeps the query rows in registers and loads
// each support tile straight into LDS.
#include <algorithm>

#include "common.hpp"
#include "device.hpp"

namespace msvm {

constexpr int kPredDK = 64;            // features per LDS chunk
constexpr int kPredLS = kPredDK + 4;   // padded LDS row stride

// Support rows [lo, hi) of range r of nrange: whole 64-row tiles, split as
// evenly as the tiles allow.
__device__ __forceinline__ void predict_range_of(int64_t nsv, int nrange,
                                                 int r, int64_t& lo,
                                                 int64_t& hi)
{
    const int64_t tiles = (nsv + 63) / 64;
    lo = 64 * (tiles * r / nrange);
    hi = min(nsv, 64 * (tiles * (r + 1) / nrange));
}

// A row's sums: the decision values (one range), or the range's partial
// sums (several ranges; k_predict_sum adds them with b).
template <int NOUT>
__device__ __forceinline__ void predict_store(const PredictArgs& a,
                                              int64_t row,
                                              const double (&part)[NOUT][4],
                                              int nl)
{
    const int n_out = a.n_out;
#pragma unroll
    for (int o = 0; o < NOUT; ++o) {
        if (o >= n_out) continue;
        const double v = pick4(part[o], nl);
        if (a.nrange <= 1)
            a.out[row * n_out + o] = v + (a.b ? a.b[o] : 0.0);
        else
            a.part[((int64_t)blockIdx.y * a.m + row) * n_out + o] = v;
    }
}

template <int NOUT>
__global__ __launch_bounds__(256) void k_predict(PredictArgs a)
{
    __shared__ __align__(16) float As[64 * kPredLS];
    __shared__ __align__(16) float Bs[64 * kPredLS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, nl = lane & 15;
    const int64_t m = a.m, ldp = a.ldp, nsv = a.nsv;
    const int64_t row0 = (int64_t)blockIdx.x * 64;
    const int n_out = a.n_out;

    float sqr[4];
    int64_t rid[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        rid[v] = row0 + wave * 16 + 4 * g + v;
        sqr[v] = rid[v] < m ? a.sqt[rid[v]] : 0.0f;
    }
    double part[NOUT][4];
#pragma unroll
    for (int o = 0; o < NOUT; ++o)
#pragma unroll
        for (int v = 0; v < 4; ++v) part[o][v] = 0.0;

    const int q4c = kPredDK / 4;
    int64_t sv_lo, sv_hi;
    predict_range_of(nsv, a.nrange, (int)blockIdx.y, sv_lo, sv_hi);
    for (int64_t sv0 = sv_lo; sv0 < sv_hi; sv0 += 64) {
        floatx4 acc[4];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
        // the epilogue's data of the tile's support rows, requested now so
        // that it lands during the tile's matrix-core work (buffer loads:
        // a row past the end reads 0, and so does the index table when
        // self_match is off)
        float ssv[4];
        int64_t stn[4];
        double cf[4][NOUT];
        {
            const Rsrc rQ = make_rsrc(a.sqsv + sv0, (nsv - sv0) * 4);
            const Rsrc rT =
                make_rsrc(a.sv_train_idx + (a.self_match ? sv0 : 0),
                          a.self_match ? (nsv - sv0) * 4 : 0);
            const Rsrc rC = make_rsrc(a.coef + sv0 * n_out,
                                      (nsv - sv0) * n_out * 8);
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const uint32_t j = (uint32_t)(cb * 16 + nl);
                ssv[cb] = bld_f32(rQ, 4 * j);
                const int32_t t = bld_i32(rT, 4 * j);
                stn[cb] = (a.self_match && sv0 + j < nsv) ? t : -1;
#pragma unroll
                for (int o = 0; o < NOUT; ++o)
                    cf[cb][o] = o < n_out
                                    ? bld_f64(rC, 8 * (j * (uint32_t)n_out +
                                                       (uint32_t)o))
                                    : 0.0;
            }
        }
        for (int64_t c0 = 0; c0 < ldp; c0 += kPredDK) {
            __syncthreads();
            for (int e = tid; e < 64 * q4c; e += 256) {
                int r = e / q4c, c4 = e - r * q4c;
                int64_t col = c0 + 4 * c4;
                int64_t gr = row0 + r, gs = sv0 + r;
                float4 va = (gr < m && col < ldp) ? ld4(a.Xt + gr * ldp + col)
                                                  : zero4();
                float4 vb = (gs < nsv && col < ldp)
                                ? ld4(a.SV + gs * ldp + col)
                                : zero4();
                *reinterpret_cast<float4*>(As + r * kPredLS + 4 * c4) = va;
                *reinterpret_cast<float4*>(Bs + r * kPredLS + 4 * c4) = vb;
            }
            __syncthreads();
            for (int kk = 0; kk < kPredDK && c0 + kk < ldp; kk += 16) {
                float4 av = ld4(As + (wave * 16 + nl) * kPredLS + kk + 4 * g);
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    float4 bv = ld4(Bs + (cb * 16 + nl) * kPredLS + kk + 4 * g);
                    acc[cb] = mfma_chunk(acc[cb], av, bv);
                }
            }
        }
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
            float kv[4];
            if (a.kf.kind == SVM_KERNEL_RBF) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    kv[v] = rbf_from_dot(sqr[v], ssv[cb], acc[cb][v],
                                         a.kf.gexp);
                    if (stn[cb] == rid[v] + a.row_base) kv[v] = 1.0f;
                }
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    kv[v] = kernel_of_dot(a.kf, acc[cb][v]);
            }
#pragma unroll
            for (int v = 0; v < 4; ++v) {
#pragma unroll
                for (int o = 0; o < NOUT; ++o)
                    part[o][v] = fma(cf[cb][o], (double)kv[v], part[o][v]);
            }
        }
    }

#pragma unroll
    for (int o = 0; o < NOUT; ++o)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int off = 8; off > 0; off >>= 1)
                part[o][v] += __shfl_xor(part[o][v], off, 16);

    if (nl < 4) {
        const int64_t row = row0 + wave * 16 + 4 * g + nl;
        if (row < m) predict_store<NOUT>(a, row, part, nl);
    }
}

// The same decision sums for rows of at most kRaMaxLdp features: each wave's
// 16 test rows stay in registers, in the matrix-core operand layout, for the
// whole kernel, and only the support tiles pass through LDS, whole (64
// support rows x ldp features a step): half the staging of k_predict and
// all of a tile's matrix-core work between one pair of barriers.  Same
// chunk order, so the same K bits.
constexpr int kRaMaxLdp = 128;
constexpr int kRaLS = kRaMaxLdp + 4;  // padded LDS row stride
// The support tile goes from memory straight into LDS (buffer loads to LDS:
// lane l of a wave's load writes 16 bytes at the wave's base + 16 l), in
// float4 slots of the padded layout: slot S holds row S / 33, float4
// S % 33 (the 33rd of a row is padding).  4 waves x 9 loads x 64 lanes
// cover the 64 x 33 slots; slots past the tile, past ldp or past the last
// support row are written with zeros (range-checked offsets).
constexpr int kRaSlotsRow = kRaLS / 4;                 // 33
constexpr int kRaLoads = 9;                            // per wave
constexpr int kRaSlots = 4 * kRaLoads * 64;            // 2304 >= 64 x 33
static_assert(kRaSlots >= 64 * kRaSlotsRow, "support tile slots");
typedef __attribute__((address_space(3))) void* LdsPtr;

template <int NOUT>
__device__ __forceinline__ void predict_ra_body(const PredictArgs& a)
{
    __shared__ __align__(16) float Bs[kRaSlots * 4];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, nl = lane & 15;
    const int64_t m = a.m, ldp = a.ldp, nsv = a.nsv;
    const int64_t row0 = (int64_t)blockIdx.x * 64;
    const int n_out = a.n_out;
    const int kch = (int)((ldp + 15) / 16);  // 16-feature chunks (<= 8)

    float sqr[4];
    int32_t rself[4];  // training index of the row (self_match), int32
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int64_t r = row0 + wave * 16 + 4 * g + v;
        sqr[v] = r < m ? a.sqt[r] : 0.0f;
        rself[v] = (int32_t)(r + a.row_base);
    }
    // this lane's A operand: row wave*16 + nl, features 16c + 4g .. + 3
    float4 ar[kRaMaxLdp / 16];
    {
        const int64_t r = row0 + wave * 16 + nl;
        const Rsrc rA = make_rsrc(a.Xt + (r < m ? r : 0) * ldp,
                                  r < m ? ldp * 4 : 0);
#pragma unroll
        for (int c = 0; c < kRaMaxLdp / 16; ++c) {
            const int col = 16 * c + 4 * g;
            ar[c] = bld_f4(rA, col < ldp ? (uint32_t)(4 * col) : kOob);
        }
    }
    double part[NOUT][4];
#pragma unroll
    for (int o = 0; o < NOUT; ++o)
#pragma unroll
        for (int v = 0; v < 4; ++v) part[o][v] = 0.0;

    const int q4 = (int)(ldp / 4);  // float4 per support row
    int64_t sv_lo, sv_hi;
    predict_range_of(nsv, a.nrange, (int)blockIdx.y, sv_lo, sv_hi);
    for (int64_t sv0 = sv_lo; sv0 < sv_hi; sv0 += 64) {
        // the tile's epilogue data (it lands during the work below)
        float ssv[4];
        int32_t stn[4];
        double cf[4][NOUT];
        {
            const Rsrc rQ = make_rsrc(a.sqsv + sv0, (nsv - sv0) * 4);
            const Rsrc rT =
                make_rsrc(a.sv_train_idx + (a.self_match ? sv0 : 0),
                          a.self_match ? (nsv - sv0) * 4 : 0);
            const Rsrc rC = make_rsrc(a.coef + sv0 * n_out,
                                      (nsv - sv0) * n_out * 8);
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                const uint32_t j = (uint32_t)(cb * 16 + nl);
                ssv[cb] = bld_f32(rQ, 4 * j);
                const int32_t t = bld_i32(rT, 4 * j);
                stn[cb] = (a.self_match && sv0 + j < nsv) ? t : -1;
#pragma unroll
                for (int o = 0; o < NOUT; ++o)
                    cf[cb][o] = o < n_out
                                    ? bld_f64(rC, 8 * (j * (uint32_t)n_out +
                                                       (uint32_t)o))
                                    : 0.0;
            }
        }
        const Rsrc rB = make_rsrc(a.SV + sv0 * ldp,
                                  min((int64_t)64, nsv - sv0) * ldp * 4);
        __syncthreads();  // the previous tile's reads are done
#pragma unroll
        for (int j = 0; j < kRaLoads; ++j) {
            // this lane's slot of the load, and its offset (kOob: a zero)
            const int S = (wave * kRaLoads + j) * 64 + lane;
            const int r = S / kRaSlotsRow, c4 = S - r * kRaSlotsRow;
            const uint32_t off = (r < 64 && c4 < q4)
                                     ? (uint32_t)((r * (int)ldp + 4 * c4) * 4)
                                     : kOob;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rB, (LdsPtr)(Bs + (wave * kRaLoads + j) * 64 * 4), 16,
                (int)off, 0, 0, 0);
        }
        // the loads write LDS behind the compiler's back: wait for all of
        // them (and the epilogue data above) before the barrier
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        floatx4 acc[4];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < kRaMaxLdp / 16; ++c) {
            if (c < kch) {  // uniform
#pragma unroll
                for (int cb = 0; cb < 4; ++cb) {
                    const float4 bv =
                        ld4(Bs + (cb * 16 + nl) * kRaLS + 16 * c + 4 * g);
                    acc[cb] = mfma_chunk(acc[cb], ar[c], bv);
                }
            }
        }
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
            float kv[4];
            if (a.kf.kind == SVM_KERNEL_RBF) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    kv[v] = rbf_from_dot(sqr[v], ssv[cb], acc[cb][v],
                                         a.kf.gexp);
                    if (stn[cb] == rself[v]) kv[v] = 1.0f;
                }
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    kv[v] = kernel_of_dot(a.kf, acc[cb][v]);
            }
#pragma unroll
            for (int v = 0; v < 4; ++v) {
#pragma unroll
                for (int o = 0; o < NOUT; ++o)
                    part[o][v] = fma(cf[cb][o], (double)kv[v], part[o][v]);
            }
        }
    }

#pragma unroll
    for (int o = 0; o < NOUT; ++o)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int off = 8; off > 0; off >>= 1)
                part[o][v] += __shfl_xor(part[o][v], off, 16);

    if (nl < 4) {
        const int64_t row = row0 + wave * 16 + 4 * g + nl;
        if (row < m) predict_store<NOUT>(a, row, part, nl);
    }
}

// One output: 120 VGPRs, so four waves a SIMD fit (the 64 x 33-slot tile
// takes 36 KB of LDS, four blocks a CU).  Four outputs keep the default
// (asking them for four waves spills).
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
void k_predict_ra1(PredictArgs a)
{
    predict_ra_body<1>(a);
}

__global__ __launch_bounds__(256) void k_predict_ra4(PredictArgs a)
{
    predict_ra_body<4>(a);
}

// out = the ranges' partial sums added in range order, + b
__global__ void k_predict_sum(const double* part, int nrange, int64_t mn,
                              int n_out, const double* b, double* out)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < mn;
         e += (int64_t)gridDim.x * blockDim.x) {
        double v = 0.0;
        for (int r = 0; r < nrange; ++r) v += part[(int64_t)r * mn + e];
        out[e] = v + (b ? b[e % n_out] : 0.0);
    }
}

int32_t predict_ranges(int64_t nsv)
{
    // about 1600 support rows a range: 64-row work items of 25 tiles, which
    // fill the chip's block slots in whole rounds for a wide range of m
    const int64_t r = (nsv + 1599) / 1600;
    return (int32_t)std::max<int64_t>(1, std::min<int64_t>(8, r));
}

int64_t predict_part_doubles(int64_t nsv, int64_t m, int32_t n_out)
{
    const int32_t r = predict_ranges(nsv);
    return r > 1 ? (int64_t)r * m * n_out : 0;
}

void launch_predict(const PredictArgs& a, hipStream_t s)
{
    if (a.m <= 0) return;
    if (a.nrange < 1 || a.nrange > 8 || (a.nrange > 1 && !a.part))
        throw Error{SVM_E_INTERNAL, "decision ranges"};
    const dim3 grid((unsigned)((a.m + 63) / 64), (unsigned)a.nrange);
    if (a.ldp <= kRaMaxLdp && a.n_out <= 4) {
        if (a.n_out <= 1)
            k_predict_ra1<<<grid, 256, 0, s>>>(a);
        else
            k_predict_ra4<<<grid, 256, 0, s>>>(a);
    } else if (a.n_out <= 1) {
        k_predict<1><<<grid, 256, 0, s>>>(a);
    } else if (a.n_out <= 4) {
        k_predict<4><<<grid, 256, 0, s>>>(a);
    } else if (a.n_out <= 16) {
        k_predict<16><<<grid, 256, 0, s>>>(a);
    } else {
        throw Error{SVM_E_UNSUPPORTED, "more than 16 outputs"};
    }
    if (a.nrange > 1) {
        const int64_t mn = a.m * a.n_out;
        const unsigned blocks =
            (unsigned)std::min<int64_t>((mn + 255) / 256, 4096);
        k_predict_sum<<<blocks, 256, 0, s>>>(a.part, a.nrange, mn, a.n_out,
                                             a.b, a.out);
    }
}

}  // namespace msvm

namespace msvm {

// ---------------------------------------------------------------------------
// Sparse decision path: CSR query rows against the support rows by column.
//
// With a few nonzeros per row nearly every product of the dense path is a
// product with a zero.  The support rows are grouped in chunks of 16 and
// stored by column (the columns some row of the chunk holds, increasing,
// each with the 16 values).  A block owns 256 query rows, one per lane, with
// the first kSpRegNz nonzeros of each in registers, and walks over all
// chunks: while it sums chunk k it writes chunk k + 1 into LDS (a map
// column -> (chunk, table row), the table, the chunk's norms and
// coefficients) from registers and loads chunk k + 2 into them, one barrier
// per chunk.  Per query nonzero at column c the lane looks c up
// and, if the chunk holds it, adds v * x_s[c] to its 16 dot products: the
// sum over the common nonzeros in the query row's column order, as every
// CSR kernel of the library sums it (the skipped products are products with
// a zero, which change nothing), so the K values are bitwise those of the
// training kernels.  Per output, c_s K is accumulated in fp64 in chunk and
// slot order: no atomics, the result does not depend on scheduling.

constexpr int kSpThreads = 256;
constexpr int kSpRegNz = 32;  // query nonzeros held in registers
constexpr int kSpOutMax = 16;
constexpr int kSpTabMax = 512;  // columns of a chunk (fits the registers)
// LDS table rows: 16 values padded to 20 floats, so that rows start on 8
// different banks and the 16-byte reads of lanes on different rows rarely
// conflict
constexpr int kSpTS = 20;

// one LDS buffer: map (int2 per column), table (cap x 16 floats), 16 norms,
// 16 training indices, 16 x kSpOutMax coefficients
__host__ __device__ inline size_t sp_buf_bytes(int64_t ldp, int cap)
{
    return (size_t)ldp * 8 + (size_t)(cap + 1) * kSpTS * 4 + 64 + 64 +
           16 * kSpOutMax * 8;
}

size_t predict_sparse_lds_bytes(int64_t ldp, int cap)
{
    return 2 * sp_buf_bytes(ldp, cap);
}

bool predict_sparse_fits(int64_t ldp, int cap)
{
    // two blocks per compute unit; a chunk's columns fit the prefetch
    return cap > 0 && cap <= kSpTabMax &&
           predict_sparse_lds_bytes(ldp, cap) <= 80 * 1024;
}

template <int NOUT>
__global__ __launch_bounds__(kSpThreads) void k_predict_sparse(PredictArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x;
    const int64_t ldp = a.ldp, nsv = a.nsv;
    const int cap = a.ch_cap, n_out = a.n_out;
    const int64_t nchunk = (nsv + 15) / 16;
    const size_t per = sp_buf_bytes(ldp, cap);
    auto map_of = [&](int p) {
        return reinterpret_cast<int2*>(smem + p * per);
    };
    auto tab_of = [&](int p) {
        return reinterpret_cast<float*>(smem + p * per + ldp * 8);
    };
    const size_t tb_bytes = (size_t)(cap + 1) * kSpTS * 4;
    auto sq_of = [&](int p) {
        return reinterpret_cast<float*>(smem + p * per + ldp * 8 + tb_bytes);
    };
    auto tix_of = [&](int p) {
        return reinterpret_cast<int32_t*>(smem + p * per + ldp * 8 +
                                          tb_bytes + 64);
    };
    auto coef_of = [&](int p) {
        return reinterpret_cast<double*>(smem + p * per + ldp * 8 +
                                         tb_bytes + 128);
    };

    for (int64_t c = tid; c < 2 * ldp; c += kSpThreads) {
        const int p = c >= ldp;
        map_of(p)[c - p * ldp] = make_int2(-1, 0);
    }
    if (tid < 2 * kSpTS) tab_of(tid / kSpTS)[cap * kSpTS + tid % kSpTS] = 0.0f;
    __syncthreads();

    // Chunk k + 2 is loaded into registers while chunk k is summed, and
    // written to LDS (buffer of chunk k + 2) in the next iteration, so that
    // no barrier waits for a global load.
    constexpr int kPF = kSpTabMax * 4 / kSpThreads;  // float4 per thread
    constexpr int kPC = kSpTabMax / kSpThreads;      // columns per thread
    struct Pre {
        float4 t[kPF];
        int32_t c[kPC];
        int E;
        float sq;
        int32_t tix;
        double cf;
    };
    auto fetch = [&](int64_t k, Pre& q) {
        q.E = a.ch_ncol[k];
        const float* src = a.ch_tab + k * cap * 16;
#pragma unroll
        for (int i = 0; i < kPF; ++i) {
            const int e = tid + i * kSpThreads;
            q.t[i] = e < q.E * 4 ? ld4(src + 4 * e) : make_float4(0, 0, 0, 0);
        }
        const int32_t* cols = a.ch_cols + k * cap;
#pragma unroll
        for (int i = 0; i < kPC; ++i) {
            const int e = tid + i * kSpThreads;
            q.c[i] = e < q.E ? cols[e] : 0;
        }
        const int64_t j = k * 16 + (tid & 15);
        const bool ok = tid < 16 && j < nsv;
        q.sq = ok ? a.sqsv[j] : 0.0f;
        q.tix = (ok && a.self_match) ? a.sv_train_idx[j] : -1;
        const int s = tid / NOUT, o = tid - s * NOUT;
        const int64_t jc = k * 16 + s;
        q.cf = (tid < 16 * NOUT && jc < nsv && o < n_out)
                   ? a.coef[jc * n_out + o]
                   : 0.0;
    };
    auto put = [&](int64_t k, int p, const Pre& q) {
        int2* mp = map_of(p);
#pragma unroll
        for (int i = 0; i < kPC; ++i) {
            const int e = tid + i * kSpThreads;
            if (e < q.E) mp[q.c[i]] = make_int2((int)k, e);
        }
        float* dst = tab_of(p);
#pragma unroll
        for (int i = 0; i < kPF; ++i) {
            const int e = tid + i * kSpThreads;
            if (e < q.E * 4)
                *reinterpret_cast<float4*>(dst + (e >> 2) * kSpTS +
                                           4 * (e & 3)) = q.t[i];
        }
        if (tid < 16) {
            sq_of(p)[tid] = q.sq;
            tix_of(p)[tid] = q.tix;
        }
        if (tid < 16 * NOUT) coef_of(p)[tid] = q.cf;
    };
    Pre pre;
    if (nchunk > 0) {
        fetch(0, pre);
        put(0, 0, pre);
    }
    if (nchunk > 1) fetch(1, pre);

    // this lane's query row
    const int64_t r = (int64_t)blockIdx.x * kSpThreads + tid;
    const bool rv = r < a.m;
    const int64_t k0 = rv ? a.rpt[r] : 0, k1 = rv ? a.rpt[r + 1] : 0;
    const int nz = (int)(k1 - k0);
    int32_t qc[kSpRegNz];
    float qv[kSpRegNz];
#pragma unroll
    for (int i = 0; i < kSpRegNz; ++i) {
        const bool ok = i < nz;
        qc[i] = ok ? a.cit[k0 + i] : 0;
        qv[i] = ok ? a.cvt[k0 + i] : 0.0f;
    }
    int mxall = nz;  // the longest row of the wave
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        mxall = max(mxall, __shfl_xor(mxall, off));
    const int mx = min(mxall, kSpRegNz);  // its part held in registers
    const int zrow = cap * kSpTS;         // the zero row of a table
    const float sqr = rv ? a.sqt[r] : 0.0f;
    const int64_t self = r + a.row_base;
    double outv[NOUT];
#pragma unroll
    for (int o = 0; o < NOUT; ++o) outv[o] = 0.0;
    // the query nonzeros (and chunk 1) have arrived: no wait on them inside
    // the chunk loop
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    __syncthreads();

    for (int64_t k = 0; k < nchunk; ++k) {
        const int p = (int)(k & 1);
        if (k + 1 < nchunk) put(k + 1, p ^ 1, pre);
        if (k + 2 < nchunk) fetch(k + 2, pre);
        const int2* mp = map_of(p);
        const float* tb = tab_of(p);
        float acc[16];
#pragma unroll
        for (int s = 0; s < 16; ++s) acc[s] = 0.0f;
        // four nonzeros at a time: the four lookups, then the four table
        // rows (a miss reads the zero row; a product with zero changes
        // nothing), no branch on the lookups
        auto rows4 = [&](const int32_t (&c)[4], const float (&v)[4]) {
            int off[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int2 t = mp[c[j]];
                off[j] = t.x == (int)k ? t.y * kSpTS : zrow;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float* xr = tb + off[j];
#pragma unroll
                for (int s = 0; s < 16; s += 4) {
                    const float4 x = ld4(xr + s);
                    acc[s + 0] = fmaf(v[j], x.x, acc[s + 0]);
                    acc[s + 1] = fmaf(v[j], x.y, acc[s + 1]);
                    acc[s + 2] = fmaf(v[j], x.z, acc[s + 2]);
                    acc[s + 3] = fmaf(v[j], x.w, acc[s + 3]);
                }
            }
        };
#pragma unroll
        for (int g = 0; g < kSpRegNz / 4; ++g) {
            if (4 * g < mx) {  // uniform over the wave
                const int32_t c[4] = {qc[4 * g], qc[4 * g + 1], qc[4 * g + 2],
                                      qc[4 * g + 3]};
                const float v[4] = {qv[4 * g], qv[4 * g + 1], qv[4 * g + 2],
                                    qv[4 * g + 3]};
                rows4(c, v);
            }
        }
        if (mxall > kSpRegNz) {  // uniform: a row of the wave is longer
            for (int i = kSpRegNz; i < mxall; i += 4) {
                int32_t c[4];
                float v[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const bool ok = i + j < nz;
                    c[j] = ok ? a.cit[k0 + i + j] : 0;
                    v[j] = ok ? a.cvt[k0 + i + j] : 0.0f;
                }
                rows4(c, v);
            }
        }
        const float* sq = sq_of(p);
        const int32_t* tix = tix_of(p);
        const double* cf = coef_of(p);
        float kv[16];
        if (a.kf.kind == SVM_KERNEL_RBF) {
#pragma unroll
            for (int s = 0; s < 16; ++s) {
                kv[s] = rbf_from_dot(sqr, sq[s], acc[s], a.kf.gexp);
                if ((int64_t)tix[s] == self) kv[s] = 1.0f;
            }
        } else {
#pragma unroll
            for (int s = 0; s < 16; ++s) kv[s] = kernel_of_dot(a.kf, acc[s]);
        }
#pragma unroll
        for (int s = 0; s < 16; ++s) {
#pragma unroll
            for (int o = 0; o < NOUT; ++o)
                outv[o] = fma(cf[s * NOUT + o], (double)kv[s], outv[o]);
        }
        __syncthreads();
    }

    if (rv) {
#pragma unroll
        for (int o = 0; o < NOUT; ++o)
            if (o < n_out)
                a.out[r * n_out + o] = outv[o] + (a.b ? a.b[o] : 0.0);
    }
}

void launch_predict_sparse(const PredictArgs& a, hipStream_t s)
{
    if (a.m <= 0) return;
    if (!predict_sparse_fits(a.ldp, a.ch_cap))
        throw Error{SVM_E_INTERNAL, "sparse decision tables exceed LDS"};
    const unsigned blocks = (unsigned)((a.m + kSpThreads - 1) / kSpThreads);
    const size_t lds = predict_sparse_lds_bytes(a.ldp, a.ch_cap);
    if (a.n_out <= 1)
        k_predict_sparse<1><<<blocks, kSpThreads, lds, s>>>(a);
    else if (a.n_out <= 4)
        k_predict_sparse<4><<<blocks, kSpThreads, lds, s>>>(a);
    else if (a.n_out <= kSpOutMax)
        k_predict_sparse<16><<<blocks, kSpThreads, lds, s>>>(a);
    else
        throw Error{SVM_E_UNSUPPORTED, "more than 16 outputs"};
}

// One block per chunk of 16 support rows: flag the columns the rows hold,
// number them in increasing order (block scan), scatter the values into an
// LDS table and write it out with the columns.
__global__ __launch_bounds__(256) void k_sv_chunks(ChunkArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int wsum[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t ldp = a.ldp, k = blockIdx.x;
    const int cap = a.cap;
    int* fl = reinterpret_cast<int*>(smem);
    float* tl = reinterpret_cast<float*>(smem + ((ldp * 4 + 15) & ~15));
    for (int64_t c = tid; c < ldp; c += 256) fl[c] = 0;
    for (int e = tid; e < cap * 16; e += 256) tl[e] = 0.0f;
    __syncthreads();
    // the nonzeros of the chunk's rows: wave w takes slots w, w + 4, ...
    auto each = [&](auto fn) {
        for (int s = wave; s < 16; s += 4) {
            const int64_t j = k * 16 + s;
            if (j >= a.nsv) break;
            const int64_t row = a.idx ? (int64_t)a.idx[j] : j;
            const int64_t p0 = a.rp[row], p1 = a.rp[row + 1];
            for (int64_t q = p0 + lane; q < p1; q += 64)
                fn(s, a.ci[q], a.cv[q]);
        }
    };
    each([&](int, int32_t c, float) { fl[c] = 1; });
    __syncthreads();
    const int E = block_exclusive_scan<256>(fl, ldp, wsum);
    each([&](int s, int32_t c, float v) {
        const int e = fl[c];
        if (e < cap) tl[e * 16 + s] = v;
    });
    for (int64_t c = tid; c < ldp; c += 256) {
        const int e = fl[c];
        const bool used = (c + 1 < ldp ? fl[c + 1] : E) > e;
        if (used && e < cap) a.cols[k * cap + e] = (int32_t)c;
    }
    if (a.sq_out && tid < 16 && k * 16 + tid < a.nsv) {
        const int64_t j = k * 16 + tid;
        a.sq_out[j] = a.sq[a.idx ? (int64_t)a.idx[j] : j];
    }
    __syncthreads();
    const int Ec = min(E, cap);
    float* dst = a.tab + k * cap * 16;
    for (int e = tid; e < Ec * 4; e += 256)
        *reinterpret_cast<float4*>(dst + 4 * e) = ld4(tl + 4 * e);
    if (tid == 0) a.ncol[k] = Ec;
}

void launch_sv_chunks(const ChunkArgs& a, hipStream_t s)
{
    const int64_t nchunk = (a.nsv + 15) / 16;
    if (nchunk <= 0) return;
    const size_t lds = (size_t)((a.ldp * 4 + 15) & ~15) + (size_t)a.cap * 64;
    k_sv_chunks<<<(unsigned)nchunk, 256, lds, s>>>(a);
}

}  // namespace msvm
