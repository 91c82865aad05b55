// Device helpers shared by the HIP kernels of the library (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>

namespace msvm {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// s_waitcnt immediate (gfx9 encoding): vmcnt 0, expcnt and lgkmcnt not
// waited.  Where the compiler cannot count the loads in flight (a load in
// a loop or behind a branch) it waits for all of them at the next use of
// any loaded value; an explicit wait once they are all needed anyway keeps
// that wait out of the loops that follow.
constexpr int kVmcnt0 = 0x0f70;

// One 16x16x4 fp32 matrix-core step.  Lane l supplies A[l%16][l/16] and
// B[l/16][l%16]; lane l, register v of the result holds D[4(l/16)+v][l%16].
__device__ __forceinline__ floatx4 mfma4(float a, float b, floatx4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Accumulate the dot products of 16 A rows with 16 B rows over ldp features
// in the fixed order used by every kernel of the library: 16-feature chunks
// in increasing order, lane group g = lane/16 covering features
// c0 + 4g .. c0 + 4g + 3 of each chunk, one MFMA per component.  Using one
// order everywhere makes every K value computed for a pair bitwise equal,
// whichever kernel computes it.
__device__ __forceinline__ floatx4 mfma_chunk(floatx4 acc, float4 a, float4 b)
{
    acc = mfma4(a.x, b.x, acc);
    acc = mfma4(a.y, b.y, acc);
    acc = mfma4(a.z, b.z, acc);
    acc = mfma4(a.w, b.w, acc);
    return acc;
}

// RBF kernel value from the expansion |a|^2 + |b|^2 - 2 a.b, clamped at 0
// (fp32 cancellation can make it slightly negative), as 2^(-gexp * d2)
// with gexp = gamma * log2(e).
__device__ __forceinline__ float rbf_from_dot(float sa, float sb, float dot,
                                              float gexp)
{
    float d2 = fmaf(-2.0f, dot, sa + sb);
    d2 = fmaxf(d2, 0.0f);
    return __builtin_amdgcn_exp2f(-gexp * d2);
}

// b^e for an integer e >= 1 by binary exponentiation (the same product
// order wherever a kernel value is computed)
__device__ __forceinline__ float powi_f32(float b, int e)
{
    float r = 1.0f;
    while (e > 0) {
        if (e & 1) r *= b;
        b *= b;
        e >>= 1;
    }
    return r;
}

// Kernel value of a pair from its dot product for the kernels other than
// RBF (linear, polynomial, sigmoid).
__device__ __forceinline__ float kernel_of_dot(const KernelFn& kf, float dot)
{
    if (kf.kind == SVM_KERNEL_LINEAR) return dot;
    const float t = fmaf(kf.gamma, dot, kf.coef0);
    if (kf.kind == SVM_KERNEL_POLY) return powi_f32(t, kf.degree);
    return tanhf(t);
}

// Kernel value of a pair from its dot product and squared norms (the norms
// enter the RBF kernel only).  kf.kind is uniform over a launch; the hot
// loops test it once around a whole tile (kf.kind == SVM_KERNEL_RBF ?
// rbf_from_dot : kernel_of_dot) instead of per value.
__device__ __forceinline__ float kernel_from_dot(const KernelFn& kf, float sa,
                                                 float sb, float dot)
{
    if (kf.kind == SVM_KERNEL_RBF) return rbf_from_dot(sa, sb, dot, kf.gexp);
    return kernel_of_dot(kf, dot);
}

// K(x, x) := 1 exactly for the RBF kernel when both sides are the same
// training row (its expansion |x|^2 + |x|^2 - 2 x.x cancels in fp32 to a
// small non-zero); the other kernels have no cancellation there.
__device__ __forceinline__ bool kernel_self_is_one(const KernelFn& kf)
{
    return kf.kind == SVM_KERNEL_RBF;
}

// Order "largest key first, lowest index on ties".
__device__ __forceinline__ bool better(double k1, int32_t i1, double k2,
                                       int32_t i2)
{
    return k1 > k2 || (k1 == k2 && i1 < i2);
}

// (k1,i1) comes strictly after (k2,i2) in that order.
__device__ __forceinline__ bool after(double k1, int32_t i1, double k2,
                                      int32_t i2)
{
    return k1 < k2 || (k1 == k2 && i1 > i2);
}

// Wave-wide best (key, index); every lane ends with the result.
__device__ __forceinline__ void wave_best(double& k, int32_t& i)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        double ok = __shfl_xor(k, off);
        int32_t oi = __shfl_xor(i, off);
        if (better(ok, oi, k, i)) {
            k = ok;
            i = oi;
        }
    }
}

// ---- fast cross-lane reductions (DPP row rotates + readlane) ----

constexpr int kDppRor1 = 0x121, kDppRor2 = 0x122, kDppRor4 = 0x124,
              kDppRor8 = 0x128;

// (a row rotate has a source lane for every lane, so no lane keeps the old
// value, and the result needs no copy of the source first)
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v)
{
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, false);
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v)
{
    int lo = dpp_i32<CTRL>(__double2loint(v));
    int hi = dpp_i32<CTRL>(__double2hiint(v));
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double rl_f64(double v, int lane)
{
    int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
    int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ int rl_i32(int v, int lane)
{
    return __builtin_amdgcn_readlane(v, lane);
}

// every lane of each 16-lane row receives the row maximum / minimum
__device__ __forceinline__ double row_max_f64(double v)
{
    v = fmax(v, dpp_f64<kDppRor8>(v));
    v = fmax(v, dpp_f64<kDppRor4>(v));
    v = fmax(v, dpp_f64<kDppRor2>(v));
    v = fmax(v, dpp_f64<kDppRor1>(v));
    return v;
}

__device__ __forceinline__ int row_min_i32(int v)
{
    v = min(v, dpp_i32<kDppRor8>(v));
    v = min(v, dpp_i32<kDppRor4>(v));
    v = min(v, dpp_i32<kDppRor2>(v));
    v = min(v, dpp_i32<kDppRor1>(v));
    return v;
}

// every lane of each 16-lane row receives the row sum (fixed order)
__device__ __forceinline__ double row_sum_f64(double v)
{
    v += dpp_f64<kDppRor8>(v);
    v += dpp_f64<kDppRor4>(v);
    v += dpp_f64<kDppRor2>(v);
    v += dpp_f64<kDppRor1>(v);
    return v;
}

// every lane of each 16-lane row receives the row sum
__device__ __forceinline__ int row_sum_i32(int v)
{
    v += dpp_i32<kDppRor8>(v);
    v += dpp_i32<kDppRor4>(v);
    v += dpp_i32<kDppRor2>(v);
    v += dpp_i32<kDppRor1>(v);
    return v;
}

// Best (key, index) of a 16-lane row, in the order of better(); every lane
// of the row receives its row's result.
__device__ __forceinline__ void row_best(double& k, int32_t& i)
{
    const double M = row_max_f64(k);
    i = row_min_i32(k == M ? i : INT_MAX);
    k = M;
}

// Best (key, index) of the wave; the result is wave-uniform.
__device__ __forceinline__ void wave_best_fast(double& k, int32_t& i)
{
    double M = row_max_f64(k);
    M = fmax(fmax(rl_f64(M, 0), rl_f64(M, 16)),
             fmax(rl_f64(M, 32), rl_f64(M, 48)));
    int c = row_min_i32(k == M ? i : INT_MAX);
    c = min(min(rl_i32(c, 0), rl_i32(c, 16)), min(rl_i32(c, 32), rl_i32(c, 48)));
    k = M;
    i = c;
}

// Two independent wave-wide best searches, interleaved.
__device__ __forceinline__ void wave_best_pair(double& k0, int32_t& i0,
                                               double& k1, int32_t& i1)
{
    double M0 = row_max_f64(k0), M1 = row_max_f64(k1);
    M0 = fmax(fmax(rl_f64(M0, 0), rl_f64(M0, 16)),
              fmax(rl_f64(M0, 32), rl_f64(M0, 48)));
    M1 = fmax(fmax(rl_f64(M1, 0), rl_f64(M1, 16)),
              fmax(rl_f64(M1, 32), rl_f64(M1, 48)));
    int c0 = row_min_i32(k0 == M0 ? i0 : INT_MAX);
    int c1 = row_min_i32(k1 == M1 ? i1 : INT_MAX);
    c0 = min(min(rl_i32(c0, 0), rl_i32(c0, 16)),
             min(rl_i32(c0, 32), rl_i32(c0, 48)));
    c1 = min(min(rl_i32(c1, 0), rl_i32(c1, 16)),
             min(rl_i32(c1, 32), rl_i32(c1, 48)));
    k0 = M0;
    i0 = c0;
    k1 = M1;
    i1 = c1;
}

// The working set by column (CSR input): every column c in [0, ldp) where
// some of the nS slots holds a nonzero gets one compact row e (in no
// particular order): cols[e] = c, vals[e * qs + s] = x_s[c] (0 for slots
// past nS).  The rows after the last used one, up to csr_cols, are zero
// with cols = -1 (row csr_cols included).  csr_cols bounds the columns used
// (at most qs times the longest row, and ldp).  val(s, c) reads the dense
// working-set rows.  Run by the whole block; cnt is a zeroed LDS counter.
template <class Val>
__device__ void compact_by_column(Val val, int nS, int64_t ldp, int qs,
                                  int csr_cols, int32_t* cols, float* vals,
                                  int* cnt)
{
    for (int64_t c = threadIdx.x; c < ldp; c += blockDim.x) {
        bool any = false;
        for (int s = 0; s < nS; ++s) any |= val(s, c) != 0.0f;
        if (any) {
            const int e = atomicAdd(cnt, 1);
            if (e < csr_cols) {
                cols[e] = (int32_t)c;
                for (int s = 0; s < qs; s += 4)
                    *reinterpret_cast<float4*>(vals + (int64_t)e * qs + s) =
                        make_float4(s + 0 < nS ? val(s + 0, c) : 0.0f,
                                    s + 1 < nS ? val(s + 1, c) : 0.0f,
                                    s + 2 < nS ? val(s + 2, c) : 0.0f,
                                    s + 3 < nS ? val(s + 3, c) : 0.0f);
            }
        }
    }
    __syncthreads();
    const int E = min(*cnt, csr_cols);
    for (int64_t k = (int64_t)E * qs + threadIdx.x;
         k < (int64_t)(csr_cols + 1) * qs; k += blockDim.x)
        vals[k] = 0.0f;
    for (int e = E + (int)threadIdx.x; e < csr_cols; e += (int)blockDim.x)
        cols[e] = -1;
}

// In-place exclusive prefix sum of v[0..L) (non-negative ints) by a block
// of NT threads; returns the total.  Thread t sums a contiguous chunk;
// wsum holds NT / 64 ints of LDS.
template <int NT>
__device__ int block_exclusive_scan(int* v, int64_t L, int* wsum)
{
    constexpr int NW = NT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t K = (L + NT - 1) / NT;
    const int64_t b0 = min((int64_t)tid * K, L), b1 = min(b0 + K, L);
    int loc = 0;
    for (int64_t i = b0; i < b1; ++i) loc += v[i];
    int inc = loc;  // inclusive over the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(inc, o);
        if (lane >= o) inc += u;
    }
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int off = 0, tot = 0;
    for (int w = 0; w < NW; ++w) {
        const int x = wsum[w];
        off += w < wave ? x : 0;
        tot += x;
    }
    int run = off + inc - loc;
    for (int64_t i = b0; i < b1; ++i) {
        const int x = v[i];
        v[i] = run;
        run += x;
    }
    __syncthreads();
    return tot;
}

// number of set bits of m below this lane
__device__ __forceinline__ int lanes_below(unsigned long long m)
{
    return __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((unsigned)m, 0));
}

__device__ __forceinline__ float4 ld4(const float* p)
{
    return *reinterpret_cast<const float4*>(p);
}

// ---- raw buffer accesses ----
// A buffer resource covers `bytes` bytes from a base address.  A load at an
// offset at or past the end returns zero without touching memory and a store
// there is dropped, so ragged tails need no branch around the access (a
// branch around a load also keeps the compiler from counting the loads in
// flight).  Offsets are byte offsets below 2^31; kOob lies past every range.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcRaw32 = 0x00020000;  // word 3: 32-bit data format
constexpr uint32_t kOob = 0x80000000u;

__device__ __forceinline__ Rsrc make_rsrc(const void* p, int64_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0,
                                             (int)bytes, kRsrcRaw32);
}

__device__ __forceinline__ float4 bld_f4(Rsrc r, uint32_t off)
{
    const floatx4 v = __builtin_bit_cast(
        floatx4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
    return make_float4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ float bld_f32(Rsrc r, uint32_t off)
{
    return __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}

// A 64-bit value that is the same on every active lane, in scalar registers.
__device__ __forceinline__ int64_t uniform_i64(int64_t v)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ double uniform_f64(double v)
{
    return __builtin_bit_cast(double,
                              uniform_i64(__builtin_bit_cast(int64_t, v)));
}

__device__ __forceinline__ int32_t bld_i32(Rsrc r, uint32_t off)
{
    return __builtin_bit_cast(
        int32_t, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}

__device__ __forceinline__ double bld_f64(Rsrc r, uint32_t off)
{
    return __builtin_bit_cast(
        double, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
}

__device__ __forceinline__ uint8_t bld_u8(Rsrc r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
}

__device__ __forceinline__ uint16_t bld_u16(Rsrc r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}

__device__ __forceinline__ void bst_f64(Rsrc r, uint32_t off, double v)
{
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), r,
                                          (int)off, 0, 0);
}

__device__ __forceinline__ float4 zero4()
{
    return make_float4(0.0f, 0.0f, 0.0f, 0.0f);
}

__device__ __forceinline__ double pick4(const double (&v)[4], int k)
{
    return k == 0 ? v[0] : k == 1 ? v[1] : k == 2 ? v[2] : v[3];
}

__device__ __forceinline__ uint8_t state_bits(double y, double a, double C)
{
    uint8_t s = y > 0 ? 1 : 0;
    bool up = (y > 0 && a < C) || (y < 0 && a > 0);
    bool lo = (y > 0 && a > 0) || (y < 0 && a < C);
    return (uint8_t)(s | (up ? 2 : 0) | (lo ? 4 : 0));
}

}  // namespace msvm
