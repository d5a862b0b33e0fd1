// ripple.h -- wavefront helpers shared by the exact walks of libqlm's kernels
// (not part of the public interface).
//
// An exact walk gives each of the 64 lanes of a wavefront one position of a
// queue.  A running sum ripples from lane to lane (at each of up to 63 steps
// every lane takes its left neighbour's sum and adds its left neighbour's
// input), so that each lane ends with the sum of the inputs to its left,
// formed in position order with the same additions as a serial walk.
#pragma once

#include <hip/hip_runtime.h>

namespace qlm_ripple {

constexpr int kWave = 64;

// Lane l receives lane l - 1's value (DPP wave_shr:1); lane 0 keeps its own.
__device__ inline double from_left(double v)
{
    const int lo = __double2loint(v), hi = __double2hiint(v);
    return __hiloint2double(__builtin_amdgcn_update_dpp(hi, hi, 0x138, 0xF, 0xF, false),
                            __builtin_amdgcn_update_dpp(lo, lo, 0x138, 0xF, 0xF, false));
}

// The same, with zero in lane 0.
__device__ inline double from_left0(double v)
{
    const int lo = __double2loint(v), hi = __double2hiint(v);
    return __hiloint2double(__builtin_amdgcn_update_dpp(0, hi, 0x138, 0xF, 0xF, false),
                            __builtin_amdgcn_update_dpp(0, lo, 0x138, 0xF, 0xF, false));
}

// Lane j's value (j the same in every lane).
__device__ inline double lane_value(double v, int j)
{
    const int hi = __builtin_amdgcn_readlane(__double2hiint(v), j);
    const int lo = __builtin_amdgcn_readlane(__double2loint(v), j);
    return __hiloint2double(hi, lo);
}

// This thread's wavefront within its workgroup, as a value the compiler
// knows to be the same in every lane (loops over it stay scalar).
__device__ inline int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave)); }

}  // namespace qlm_ripple
