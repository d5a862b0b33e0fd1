// tail.h -- the normal upper tail Q(z) = erfc(z / sqrt 2) / 2 as a table of
// linear cells, shared by the screening kernels of libqlm.
//
// 1024 cells cover z in [-6, 6] (beyond, Q is within 1e-9 of 0 or 1).  A kernel
// forms t = 1536 - (1024 / 12) z in single precision and clamps it to
// [1024, 2048): there every float has exponent 10, so the ten leading mantissa
// bits are the cell.  Cell k holds the line that best fits Q over its width
// (the chord, moved by half its largest deviation), as (a, b) with
// Q ~ a + b t; the two end cells are the constants 0 and 1.  The largest
// error of the lines is below 2.2e-6.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace qlm_tail {

constexpr int kCells = 1024;
constexpr double kZ = 6.0;
constexpr double kScale = kCells / (2.0 * kZ);                  // cells per unit z
constexpr float kMid = 1536.0f;
constexpr float kLo = 1024.0f;
constexpr float kHi = 2047.9998779296875f;                      // 2048 - 2^-13
constexpr uint32_t kCellBits = 0x7FE000u;                       // mantissa bits 22..13
// Variances multiplied by this make the reciprocal square root of their sum
// come out in cells per unit of margin.
constexpr double kVarScale = 1.0 / (kScale * kScale);

// Fills the table; a workgroup of kThreads threads calls it, every thread with
// the same fixed trip count (no exit that depends on the thread).
template <int kThreads>
__device__ inline void build(float2 *tab)
{
    static_assert(kCells % kThreads == 0, "tail cells per thread");
#pragma unroll
    for (int k0 = 0; k0 < kCells; k0 += kThreads) {
        const int k = k0 + (int)threadIdx.x;
        const double r2 = 0.70710678118654752440;
        const double p0 = 0.5 * erfc((512.0 - k) / kScale * r2);
        const double p1 = 0.5 * erfc((511.0 - k) / kScale * r2);
        const double pm = 0.5 * erfc((511.5 - k) / kScale * r2);
        double c1 = p1 - p0;
        double c0 = p0 + 0.5 * (pm - 0.5 * (p0 + p1));
        // the end cells are flat at exactly 0 and 1 (their Q is within 2e-9 of it),
        // so that clamped margins give exact zero and one terms
        if (k == 0 || k == kCells - 1) {
            c0 = k == 0 ? 0.0 : 1.0;
            c1 = 0.0;
        }
        // the line in t itself (c0 - c1 (1024 + k) + c1 t): no fraction to form
        // in the kernel; the constant is at most 9.6 in size, so its rounding adds
        // below 6e-7
        tab[k] = make_float2((float)(c0 - c1 * (kLo + k)), (float)c1);
    }
}

// Q at the margin num (seconds, slo - E[W]) for the scaled variance vz
// (variance in s^2 times kVarScale): rsq(vz) is in cells per second of margin.
// vz = 0 gives 0 or 1 by the sign of num (0 for num = 0).
__device__ inline float q_of(const float2 *tab, float num, float vz)
{
    const float rs = __builtin_amdgcn_rsqf(vz);
    float t = fmaf(-num, rs, kMid);
    t = __builtin_amdgcn_fmed3f(t, kLo, kHi);         // NaN (0 * inf) -> low end
    const float2 c = tab[(__float_as_uint(t) & kCellBits) >> 13];
    return fmaf(c.y, t, c.x);
}

}  // namespace qlm_tail
