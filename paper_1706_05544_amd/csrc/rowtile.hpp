// Layout and candidate helpers shared by the row/update kernels (k_rows,
// one problem; k_lock, several problems in lockstep).
#pragma once

#include "common.hpp"
#include "device.hpp"

namespace msvm {

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

}  // namespace msvm
