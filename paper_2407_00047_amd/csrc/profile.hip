// profile.hip -- problem tables from a hardware profile (qlm_apply_profile in
// include/qlm.h): the prefill, drain and throughput terms of the estimator
// folded into the tables the scoring kernels read, so that their cost is
// unchanged.
//
// A request's completion is its wait, its prefill and its decode (Sec. 6,
// Eq. total_completion_time), the decode its output tokens at eps * d seconds
// each (Eq. total_decode_time, the largest output taken), a group's completion
// its last request's (Eq. group_completion_time):
//
//   SLO       The SLO bounds the time to the first token, the wait plus the
//             request's own prefill: slo - P[m].
//   swap      Before an instance of class c changes from model a to model b,
//             the running requests finish, the last admitted needing its
//             prefill and up to O_max[a] decode steps: the completion time
//             Eq. completion_time charges at each transition.
//             S'[c][a][b] = S[c][a][b] + (P[a] + O_max[a] eps[c][a] d[c][a]).
//   Theta     The batch the GPU's token memory holds over the time of one
//             decode step (Appendix): B = GPU[c][m] / E[I + O][m],
//             Theta = B / (d[c][m] eps[c][m]).
//
// Each value is formed in double precision in the order written and stored in
// single precision.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"
#include "qlm.h"

namespace {

using qlm_internal::check_problem;
using qlm_internal::fail;
using qlm_internal::hip_fail;

constexpr int kThreads = 256;

struct ProfArgs {
    int32_t G, I, M, C;
    const int32_t *grp_count, *grp_model, *inst_class, *inst_model;
    const float *grp_slo, *inst_tput, *swap_cost;
    qlm_profile pf;
    float *swap_out, *slo_out, *tput_out;
    const float *req_slo;
    int64_t n_req;
    float *req_out;
};

__device__ inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

#pragma clang fp contract(off)

// One thread per entry of the swap table, then of the SLOs, then of the
// throughputs (grid-stride).
__global__ __launch_bounds__(kThreads) void k_profile(ProfArgs a)
{
    const int64_t nsw = (int64_t)a.C * a.M * a.M;
    const int64_t total = nsw + a.G + a.I;
    const bool drain = a.pf.prefill && a.pf.decode_time && a.pf.ineff && a.pf.max_tokens;
    const bool thr = a.pf.kv_tokens && a.pf.decode_time && a.pf.ineff && a.pf.mean_tokens &&
                     a.inst_model;
    for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < total;
         k += (int64_t)gridDim.x * kThreads) {
        if (k < nsw) {
            const int b = (int)(k % a.M);
            const int ab = (int)(k / a.M);
            const int am = ab % a.M;
            const int c = ab / a.M;
            double S = a.swap_cost ? (double)a.swap_cost[k] : 0.0;
            if (drain && am != b) {
                const int64_t ca = (int64_t)c * a.M + am;
                const double D = (double)a.pf.max_tokens[am] * (double)a.pf.ineff[ca] *
                                 (double)a.pf.decode_time[ca];
                S = S + ((double)a.pf.prefill[am] + D);
            }
            a.swap_out[k] = (float)S;
        } else if (k < nsw + a.G) {
            const int i = (int)(k - nsw);
            double slo = (double)a.grp_slo[i];
            if (a.pf.prefill) slo = slo - (double)a.pf.prefill[clampi(a.grp_model[i], 0, a.M - 1)];
            a.slo_out[i] = (float)slo;
        } else {
            const int g = (int)(k - nsw - a.G);
            double theta = (double)a.inst_tput[g];
            const int m = a.inst_model ? a.inst_model[g] : -1;
            if (thr && m >= 0 && m < a.M) {
                const int64_t cm = (int64_t)clampi(a.inst_class[g], 0, a.C - 1) * a.M + m;
                const double B = (double)a.pf.kv_tokens[cm] / (double)a.pf.mean_tokens[m];
                theta = B / ((double)a.pf.decode_time[cm] * (double)a.pf.ineff[cm]);
            }
            a.tput_out[g] = (float)theta;
        }
    }
}

// Per-request SLOs less their group's prefill.  One workgroup: the request
// offsets of the groups by a scan, then each thread its range of groups.
__global__ __launch_bounds__(kThreads) void k_profile_req(ProfArgs a)
{
    __shared__ int64_t part[kThreads];
    const int t = threadIdx.x;
    const int per = (a.G + kThreads - 1) / kThreads;
    const int b = t * per, e = min(a.G, b + per);
    int64_t s = 0;
    for (int i = b; i < e; ++i) s += a.grp_count[i] > 0 ? a.grp_count[i] : 0;
    part[t] = s;
    __syncthreads();
    if (t == 0) {
        int64_t run = 0;
        for (int k = 0; k < kThreads; ++k) {
            const int64_t v = part[k];
            part[k] = run;
            run += v;
        }
    }
    __syncthreads();
    int64_t r = part[t];
    for (int i = b; i < e && r < a.n_req; ++i) {
        const int n = a.grp_count[i] > 0 ? a.grp_count[i] : 0;
        const double P = a.pf.prefill ? (double)a.pf.prefill[clampi(a.grp_model[i], 0, a.M - 1)]
                                      : 0.0;
        for (int k = 0; k < n && r < a.n_req; ++k, ++r) {
            double slo = (double)a.req_slo[r];
            if (a.pf.prefill) slo = slo - P;
            a.req_out[r] = (float)slo;
        }
    }
}

}  // namespace

extern "C" {

int qlm_apply_profile(const qlm_problem *problem, const qlm_profile *profile,
                      const int32_t *inst_model, float *swap_out, float *slo_out, float *tput_out,
                      const float *req_slo, int64_t n_requests, float *req_slo_out,
                      qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    int rc = check_problem(problem);
    if (rc) return rc;
    if (!profile) return fail(QLM_ERR_ARG, "profile is NULL");
    if (!swap_out || !slo_out || !tput_out)
        return fail(QLM_ERR_ARG, "swap_out, slo_out and tput_out are required");
    if (n_requests < 0) return fail(QLM_ERR_ARG, "n_requests must be >= 0");
    if ((req_slo == nullptr) != (req_slo_out == nullptr))
        return fail(QLM_ERR_ARG, "req_slo and req_slo_out go together");
    if (req_slo && n_requests == 0) req_slo = nullptr;
    ProfArgs a{};
    a.G = problem->n_groups;
    a.I = problem->n_instances;
    a.M = problem->n_models;
    a.C = problem->n_classes;
    a.grp_count = problem->grp_count;
    a.grp_model = problem->grp_model;
    a.inst_class = problem->inst_class;
    a.inst_model = inst_model;
    a.grp_slo = problem->grp_slo;
    a.inst_tput = problem->inst_tput;
    a.swap_cost = problem->swap_cost;
    a.pf = *profile;
    a.swap_out = swap_out;
    a.slo_out = slo_out;
    a.tput_out = tput_out;
    a.req_slo = req_slo;
    a.n_req = n_requests;
    a.req_out = req_slo_out;
    const int64_t total = (int64_t)a.C * a.M * a.M + a.G + a.I;
    int64_t blocks = (total + kThreads - 1) / kThreads;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(k_profile, dim3((unsigned)blocks), dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_profile launch");
    if (req_slo) {
        hipLaunchKernelGGL(k_profile_req, dim3(1), dim3(kThreads), 0, stream, a);
        e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "k_profile_req launch");
    }
    return QLM_OK;
}

}  // extern "C"
