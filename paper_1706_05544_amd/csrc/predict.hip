// Batched decision function D(x) = sum_j c_j K(sv_j, x) + b (gfx950).
//
// The paper times training together with prediction (Section 5, Fig. 1);
// the same kernel recomputes the responses F_i = sum_j c_j K(x_j, x_i) from
// scratch once the incremental solve has converged.
//
// Tiling: a block of 4 waves owns 64 test rows (16 per wave, the MFMA row
// tile) and walks over the support rows 64 at a time.  For every 64-feature
// chunk both operand tiles are staged in LDS (row stride padded by 4 floats
// against bank conflicts); each wave accumulates its 16 x 64 dot products on
// the matrix cores in the feature order shared with the training kernels,
// applies the RBF epilogue and accumulates c_j K in fp64 per lane.  The
// per-lane partial sums are reduced across the 16 support columns at the
// end, so each output is written once, without atomics.
#include "common.hpp"
#include "device.hpp"

namespace msvm {

constexpr int kPredDK = 64;            // features per LDS chunk
constexpr int kPredLS = kPredDK + 4;   // padded LDS row stride

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
    for (int64_t sv0 = 0; sv0 < nsv; sv0 += 64) {
        floatx4 acc[4];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
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
            const int64_t sv = sv0 + cb * 16 + nl;
            const bool ok = sv < nsv;
            const float ssv = ok ? a.sqsv[sv] : 0.0f;
            const int64_t st = (ok && a.self_match) ? a.sv_train_idx[sv] : -1;
            double cf[NOUT];
#pragma unroll
            for (int o = 0; o < NOUT; ++o)
                cf[o] = (ok && o < n_out) ? a.coef[sv * n_out + o] : 0.0;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float kv = rbf_from_dot(sqr[v], ssv, acc[cb][v], a.gexp);
                if (st == rid[v] + a.row_base) kv = 1.0f;
#pragma unroll
                for (int o = 0; o < NOUT; ++o)
                    part[o][v] = fma(cf[o], (double)kv, part[o][v]);
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
        if (row < m) {
#pragma unroll
            for (int o = 0; o < NOUT; ++o) {
                if (o < n_out) {
                    double bias = a.b ? a.b[o] : 0.0;
                    a.out[row * n_out + o] = pick4(part[o], nl) + bias;
                }
            }
        }
    }
}

void launch_predict(const PredictArgs& a, hipStream_t s)
{
    if (a.m <= 0) return;
    unsigned blocks = (unsigned)((a.m + 63) / 64);
    if (a.n_out <= 1)
        k_predict<1><<<blocks, 256, 0, s>>>(a);
    else if (a.n_out <= 4)
        k_predict<4><<<blocks, 256, 0, s>>>(a);
    else if (a.n_out <= 16)
        k_predict<16><<<blocks, 256, 0, s>>>(a);
    else
        throw Error{SVM_E_UNSUPPORTED, "more than 16 outputs"};
}

}  // namespace msvm
