// internal.h -- host helpers shared by the translation units of libqlm
// (not part of the public interface).
#pragma once

#include <hip/hip_runtime.h>

#include <string>

#include "qlm.h"

namespace qlm_internal {

// Records the message as this host thread's last error and returns `code`.
int fail(int code, const std::string &msg);
// QLM_ERR_HIP with the HIP error text.
int hip_fail(hipError_t e, const char *what);
// Argument checks of the problem and plan structs (sizes, required pointers).
int check_problem(const qlm_problem *pr);
int check_plans(const qlm_problem *pr, const qlm_plans *pl);

// Launch timing (qlm_timing_enable): a launch bracketed by two HIP events on
// its stream when timing is on; the pair is queued for qlm_timing_read.
struct TimedLaunch {
    hipEvent_t e0, e1;
};
int timing_begin(hipStream_t stream, TimedLaunch *t);
void timing_end(hipStream_t stream, TimedLaunch *t);

}  // namespace qlm_internal
