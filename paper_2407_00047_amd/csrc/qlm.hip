// qlm.hip -- HIP kernels and C interface of libqlm (gfx950 / MI355X).
//
// Batched request waiting time (RWT) estimation and SLO-violation scoring of
// candidate virtual-queue plans, after QLM (arXiv 2407.00047), Secs. 6-7.  The
// interface and the model are documented in include/qlm.h.
//
// Kernels
//   k_score   one plan per lane.  Plans are stored slot-major, so the 64 lanes of
//             a wavefront read one slot of 64 consecutive plans as one 256-byte
//             row.  Each lane walks its plan's slots in order, so the segmented
//             prefix sums of Eq. base_equation / Eq. output_token_dist are plain
//             running sums in registers (no scan), reset at each queue head.
//             Group statistics, the swap/eviction cost table and the instance
//             table are staged once per workgroup in LDS; each slot gathers its
//             group's 16-byte record with one ds_read_b128.  Waits accumulate in
//             double, variances in single precision within blocks of 32 slots on
//             top of a double sum; the violation probability is read from a
//             linear-cell table of the normal tail in LDS.  LDS reads are
//             software-pipelined one slot ahead of their use.
//   k_gselect the plans whose screened score is within the screening error
//             bound of the minimum (the candidates of qlm_best_plan)
//   k_gexact  exact double-precision re-score of the candidates (same
//             definition as the oracle, summed per queue then over queues): one
//             wavefront per (candidate, queue), the running sums rippling from
//             lane to lane in position order
//   k_gpick   lowest exact score, lowest index on ties.
//   k_exact   exact re-score of a list of plans (qlm_rwt_score_exact), one
//             workgroup per plan, its wavefronts over the plan's queues.
//   k_validate_plans / k_validate_problem   structural checks.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "internal.h"
#include "qlm.h"
#include "ripple.h"
#include "tail.h"

namespace {

using qlm_ripple::from_left;
using qlm_ripple::from_left0;
using qlm_ripple::lane_value;
using qlm_ripple::wave_id;

constexpr int kWave = 64;
constexpr int kScoreThreads = 1024;     // 16 wavefronts per workgroup, 4 per SIMD
constexpr int kExactThreads = 1024;     // qlm_rwt_score_exact: 16 wavefronts per plan
constexpr int kExactPass = 1024;        // queue sums a workgroup holds in LDS at once
constexpr int kSelThreads = 256;
constexpr int kSelBlocks = 1024;
constexpr int kGexThreads = 256;
constexpr int kGexBlocks = 512;
// Per-(candidate, queue) sums of qlm_best_plan's workspace by default (the
// candidates beyond them are re-scored a workgroup each).
constexpr size_t kCandSumBytes = size_t(32) << 20;
constexpr int kMaxScoreBlocks = 4096;
// Row offsets of a block's prefetch (up to 67 rows of 4 * plan_stride bytes)
// are 32-bit register operands.
constexpr int64_t kMaxPlanStride = 1 << 22;
// Request counts are 21-bit (the interface's limit).
constexpr uint32_t kCountMask = (1u << 21) - 1u;
// Compact group records of the scoring kernel's fast path (see stage_compact):
// counts up to 2048 ride as half-precision numbers in the low 16 bits of the
// double n mu, models below 64 in the low 6 bits of the single-precision
// variance.
constexpr uint32_t kCompactCountMax = 2048u;
constexpr int kCompactModels = 64;
constexpr uint32_t kModelBits = 63u;
// The fast path finds a cost entry's eviction twin 2^10 doubles (8 KiB) on.
constexpr int kTwinShift = 10;
constexpr uint32_t kTwinEntries = 1u << kTwinShift;
// General records (the exact walk): the count above the model's 8 bits.
constexpr int kGenCountShift = 8;

// Screening error bound per request: the tabulated tail (below 2.2e-6),
// single-precision rounding of the standardised margin and of the block-wise
// variance (below 1e-6) and of the block-wise sums of n P (32 terms at most:
// below 1.9e-6 of their total), with margin.
constexpr double kEpsP = 8e-6;

// Normal upper tail as a table of linear cells (tail.h).
constexpr int kTailCells = qlm_tail::kCells;
constexpr double kTailScale = qlm_tail::kScale;
constexpr float kTailMid = qlm_tail::kMid;
constexpr float kTailLo = qlm_tail::kLo;
constexpr float kTailHi = qlm_tail::kHi;
constexpr uint32_t kTailCellBits = qlm_tail::kCellBits;
// Variances are staged multiplied by 1 / kTailScale^2, so that the reciprocal
// square root of the running sum is already in cells per unit of margin.
constexpr double kVarScale = qlm_tail::kVarScale;

struct ScoreArgs {
    int32_t G, I, M, C;
    int32_t col_shift;        // log2(entries per cost-table row)
    int32_t ev_shift;         // log2(bytes from a cost entry to its evicted twin)
    int32_t fast_ok;          // the fast path's shape conditions hold (M <= 64, twin at 8 KiB)
    uint32_t lut_bytes;       // bytes of the cost table (both halves), multiple of 16
    const int32_t *grp_count;
    const float *grp_mu, *grp_var, *grp_slo;
    const int32_t *grp_model;
    const float *inst_tput;
    const int32_t *inst_class, *inst_model0;
    const float *swap_cost;
    float evict_cost;
    int64_t P, ld;
    const int32_t *perm, *qoff;
    const uint32_t *evict;
    int32_t nparts;           // wavefronts per tile: 1, 2 or 4
    int32_t bound[3];         // slots where parts 1, 2, 3 of every plan start (multiples of 32)
    double *score, *penalty;
    int64_t d_begin, d_count;
    float *d_mean, *d_sd, *d_prob;
    double *wg_min;           // best_plan: per-workgroup minimum score, or null
    double *wg_nsum;          // best_plan: total requests (written by block 0)
    int32_t *ncand;           // best_plan: candidate count, zeroed by block 0
};

__device__ inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// LDS of the scoring kernel.  The normal-tail table is a static array (8 KiB at
// the start of LDS).  Dynamic part, byte addresses from `base`:
//   group table   16 (G + 1) bytes, one record per group, in one of two forms
//                 (the same for every workgroup of a launch):
//                   compact (fast path): {n mu as a double whose low 16 bits
//                   hold n, slo, n var / kTailScale^2 as a float whose low 6
//                   bits hold the model}
//                   general (exact walk): {mu, var, slo, (n << 8) | model}
//                 Entry G is an all-zero record (clamped out-of-range ids land
//                 there).
//   cost table    lut_bytes of doubles.  Row r = c (M + 1) + previous model
//                 (previous = M: none loaded) starts at byte r << (col_shift + 3);
//                 its entry at + model * 8 holds the seconds of swapping to
//                 `model` on class c (0 for the same model or none loaded).  The
//                 twin at + (1 << ev_shift) adds the eviction cost.
//   instances     16 bytes each: theta (double), the cost-table row base of its
//                 class, the row of its head (initial model, or none)
//   scratch       16 doubles for workgroup reductions
struct Lds {
    uint32_t grp, lut, inst, red;
};

// LDS byte address of a pointer into LDS (a cast to the local address space:
// no generic-pointer null check, so the address folds to a constant)
__device__ inline uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char *)p;
}

__device__ inline Lds lds_layout(const ScoreArgs &a, const unsigned char *base)
{
    Lds l;
    l.grp = lds_addr(base);
    l.lut = l.grp + 16u * (uint32_t)(a.G + 1);
    l.inst = l.lut + a.lut_bytes;
    l.red = l.inst + 16u * (uint32_t)a.I;
    return l;
}

// Generic pointer to LDS byte address `addr` (an address-space cast from the
// local address space, so loads and stores through it stay ds_* instructions).
template <typename T>
__device__ inline T *lds_ptr(uint32_t addr)
{
    return (T *)((__attribute__((address_space(3))) T *)(uintptr_t)addr);
}

// Bit b of w moved to bit kTwinShift (other bits arbitrary): for b >= 10 a
// right shift of the word, below that a left shift of its low half (16-bit
// shifts keep the short issue form; b is a constant in the unrolled blocks).
__device__ inline uint32_t twin_bit(uint32_t w, uint32_t b)
{
    if (b >= (uint32_t)kTwinShift) return w >> (b - kTwinShift);
    return (uint32_t)(uint16_t)((uint16_t)w << (kTwinShift - b));
}

// Fields of a compact group record (stage_compact).
__device__ inline double rec_nmu(const uint4 r)
{
    return __longlong_as_double((long long)(((uint64_t)r.y << 32) | r.x));
}
__device__ inline float rec_slo(const uint4 r) { return __uint_as_float(r.z); }
__device__ inline float rec_nv(const uint4 r) { return __uint_as_float(r.w); }
__device__ inline uint32_t rec_model(uint32_t w) { return w & kModelBits; }
// S + n * p, n the record's count (the half-precision low half of x); the
// compiler forms it as one v_fma_mix_f32, which widens the half on the way in.
__device__ inline float fma_count(uint32_t x, float p, float S)
{
    return fmaf((float)__builtin_bit_cast(_Float16, (uint16_t)(x & 0xFFFFu)), p, S);
}

// Makes v opaque to the optimizer, in a vector register (no instruction): keeps
// a uniform value out of scalar operands, and a sum from being regrouped.
template <typename T>
__device__ inline T in_vgpr(T v)
{
    asm volatile("" : "+v"(v));
    return v;
}

// Entry w of the cost table (swap seconds, plus the eviction cost in the twin
// half), 0 for the diagonal, no model loaded, padding and no swap table.
__device__ inline double cost_entry(const ScoreArgs &a, int w)
{
    const int Mp = 1 << a.col_shift;
    const int rows = a.M + 1;
    const int half = a.C * rows * Mp;
    const int twin = 1 << (a.ev_shift - 3);
    const int ev = w >= twin;
    const int k = ev ? w - twin : w;
    double v = 0.0;
    if (k < half) {
        const int col = k % Mp;
        const int row = (k / Mp) % rows;
        const int c = k / (Mp * rows);
        if (a.swap_cost && row < a.M && col < a.M && row != col)
            v = (double)a.swap_cost[((int64_t)c * a.M + row) * a.M + col];
        if (ev) v += (double)a.evict_cost;
    }
    return v;
}

// The fast path's conditions.  A cost entry: at most 29 significant bits (the
// low 24 bits of its mantissa clear), so that its product with any
// single-precision throughput is exact in double precision (the fast path
// needs that at queue heads, where SD = 0).  A group: 0 < n <= 2048 and a
// scaled variance that is a normal single-precision number (so every position
// after a queue head has SD > 0).
__device__ inline bool cost_fits(double v)
{
    return ((uint64_t)__double_as_longlong(v) & 0xFFFFFFull) == 0;
}
__device__ inline uint32_t group_count(const ScoreArgs &a, int i)
{
    return (uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
}
__device__ inline float group_scaled_var(const ScoreArgs &a, int i, uint32_t n)
{
    return (float)((double)n * (double)a.grp_var[i] * kVarScale);
}
__device__ inline bool group_fits(uint32_t n, float nv)
{
    return n >= 1u && n <= kCompactCountMax && nv >= 1.17549435e-38f && nv <= 3.4028235e38f;
}

// Cost table and instance records.  Returns whether every cost entry this
// thread staged fits the fast path.
__device__ bool stage_costs(const ScoreArgs &a, const Lds &l)
{
    bool ok = true;
    double *lut = lds_ptr<double>(l.lut);
    const int rows = a.M + 1;
    const int entries = (int)(a.lut_bytes / 8u);
    for (int w = threadIdx.x; w < entries; w += blockDim.x) {
        const double v = cost_entry(a, w);
        lut[w] = v;
        ok = ok && cost_fits(v);
    }
    const uint32_t row_bytes = 8u << a.col_shift;
    for (int g = threadIdx.x; g < a.I; g += blockDim.x) {
        const int c = clampi(a.inst_class[g], 0, a.C - 1);
        const int m0 = a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
        const uint32_t cb = l.lut + (uint32_t)(c * rows) * row_bytes;
        const double th = (double)a.inst_tput[g];
        uint4 r;
        r.x = (uint32_t)__double_as_longlong(th);
        r.y = (uint32_t)((uint64_t)__double_as_longlong(th) >> 32);
        r.z = cb;
        r.w = cb + (uint32_t)(m0 >= 0 ? m0 : a.M) * row_bytes;
        lds_ptr<uint4>(l.inst)[g] = r;
    }
    return ok;
}

// Compact group records of the fast path.  n mu is exact in double precision
// and, for n <= 2048, fills at most 36 of its 53 significand bits, so the low
// 16 bits are free and carry n as a half-precision number (exact up to 2048):
// the value read back differs from n mu by less than 2^-36 of it.  The scaled
// variance is rounded to single precision and its low 6 mantissa bits carry
// the model, which moves it by less than 2^-17 of itself.  Returns whether this
// thread's groups fit the form: 0 < n <= 2048, a variance that is a normal
// single-precision number (so every position after a queue head has SD > 0),
// and a model below 64.
__device__ bool stage_compact(const ScoreArgs &a, const Lds &l)
{
    bool ok = a.fast_ok != 0;
    uint4 *grp = lds_ptr<uint4>(l.grp);
    for (int i = threadIdx.x; i <= a.G; i += blockDim.x) {
        uint4 r = make_uint4(0u, 0u, 0u, 0u);
        if (i < a.G) {
            const uint32_t n = group_count(a, i);
            const uint32_t m = (uint32_t)clampi(a.grp_model[i], 0, a.M - 1);
            const uint64_t nm = (uint64_t)__double_as_longlong((double)n * (double)a.grp_mu[i]);
            const float nv = group_scaled_var(a, i, n);
            ok = ok && group_fits(n, nv);
            const uint32_t nh = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)(float)min(n, kCompactCountMax));
            r.x = ((uint32_t)nm & 0xFFFF0000u) | nh;
            r.y = (uint32_t)(nm >> 32);
            r.z = __float_as_uint(a.grp_slo[i]);
            r.w = (__float_as_uint(nv) & ~kModelBits) | (m & kModelBits);
        }
        grp[i] = r;
    }
    return ok;
}

// General group records of the exact walk: {mu, var, slo, (n << 8) | model}.
__device__ void stage_general(const ScoreArgs &a, const Lds &l)
{
    uint4 *grp = lds_ptr<uint4>(l.grp);
    for (int i = threadIdx.x; i <= a.G; i += blockDim.x) {
        uint4 r = make_uint4(0u, 0u, 0u, 0u);
        if (i < a.G) {
            const uint32_t n = (uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
            const uint32_t m = (uint32_t)clampi(a.grp_model[i], 0, a.M - 1);
            r.x = __float_as_uint(a.grp_mu[i]);
            r.y = __float_as_uint(a.grp_var[i]);
            r.z = __float_as_uint(a.grp_slo[i]);
            r.w = (n << kGenCountShift) | m;
        }
        grp[i] = r;
    }
}

// The normal-tail table: cell k covers t in [1024 + k, 1025 + k), i.e. z from
// (512 - k) / kTailScale down to (511 - k) / kTailScale, and holds the line
// that fits Q best there (the chord, moved by half its deviation at the middle
// of the cell).
__device__ void stage_tail(float2 *tab)
{
    // a fixed trip count (the kernel runs kScoreThreads threads): no loop whose
    // exit depends on the thread, after which uniform values would turn divergent
    qlm_tail::build<kScoreThreads>(tab);
}

__device__ inline double wave_min(double v)
{
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

// Bitwise or of v over the 64 lanes (every lane active), as a scalar: within
// quads, half rows and rows by DPP, then the four rows' results read out.
__device__ inline uint32_t wave_or(uint32_t v)
{
    v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);    // quad_perm 1,0,3,2
    v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);    // quad_perm 2,3,0,1
    v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, false);   // row_half_mirror
    v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, false);   // row_mirror
    return (uint32_t)(__builtin_amdgcn_readlane((int)v, 0) | __builtin_amdgcn_readlane((int)v, 16) |
                      __builtin_amdgcn_readlane((int)v, 32) | __builtin_amdgcn_readlane((int)v, 48));
}

// qlm_score_form: 1 when the scoring kernel takes its fast path for this
// problem (the conditions above, evaluated as its staging evaluates them),
// else 0.  One workgroup.
__global__ __launch_bounds__(1024) void k_score_form(ScoreArgs a, int32_t *form)
{
    bool ok = a.fast_ok != 0;
    const int entries = (int)(a.lut_bytes / 8u);
    for (int w = threadIdx.x; w < entries; w += blockDim.x) ok = ok && cost_fits(cost_entry(a, w));
    for (int i = threadIdx.x; i < a.G; i += blockDim.x) {
        const uint32_t n = group_count(a, i);
        ok = ok && group_fits(n, group_scaled_var(a, i, n));
    }
    const int all = __syncthreads_and((int)ok);
    if (threadIdx.x == 0) *form = all ? 1 : 0;
}

#pragma clang fp contract(off)
// The exact walk of the scoring kernel, taken when the group records are in
// the general form (a group with no requests or no variance, a count of 2^13
// or more, 65 models or more, or a cost whose product with a throughput may
// round).  One lane walks its plan's slots in order and forms the running sums
// as the definition reads them: the tokens and the variance ahead as exact
// products n mu and n var added in position order, the swap and then the
// eviction seconds added one by one.  At a position whose variance ahead is
// zero, P compares A / theta + K with the SLO in exactly that arithmetic, so
// the indicator is the one the definition gives; where the scaled variance is
// too small for single precision, P is the double-precision erfc; elsewhere
// it comes from the tail table as in the fast path.
template <bool EVICT, bool PEN, bool DETAIL>
__device__ void walk_general(const ScoreArgs &a, const Lds &L, uint32_t tail0, int64_t tb, int lp,
                             bool det, int64_t dq, double &S_out, double &PE_out)
{
    const int G = a.G;
    const int I1 = a.I - 1;
    const int64_t ld4 = a.ld * 4;
    const uint32_t lpb = (uint32_t)lp * 4u;
    const uint32_t row_bytes = 8u << a.col_shift;
    auto at = [&](const void *base, int row) __attribute__((always_inline)) {
        const unsigned char *rp =
            reinterpret_cast<const unsigned char *>(base) + (int64_t)row * ld4 + tb * 4;
        return *reinterpret_cast<const uint32_t *>(rp + lpb);
    };
    const double ecost = (double)a.evict_cost;
    double A = 0.0, K = 0.0, V = 0.0, S = 0.0, PE = 0.0;
    double theta = 1.0, inv_theta = 1.0;
    uint32_t cbase = 0u, rowb = 0u;   // class row base; cost row of the slot before
    int g = -1, nb = 0;               // current queue, the slot where the next starts
    for (int s0 = 0; s0 < G; s0 += 8) {
        uint32_t id[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) id[k] = at(a.perm, min(s0 + k, G - 1));
        const uint32_t evw = EVICT ? at(a.evict, s0 >> 5) : 0u;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int s = s0 + k;
            if (s >= G) break;
            if (s == nb) {
                // the queue holding slot s: the next one not empty
                int h = g, e_nb;
                do {
                    ++h;
                    e_nb = h >= I1 ? INT_MAX : (int)at(a.qoff, h + 1);
                } while (e_nb <= s && h < I1);
                g = h;
                nb = e_nb;
                const uint4 ir = *lds_ptr<const uint4>(L.inst + 16u * (uint32_t)g);
                theta = __longlong_as_double((long long)(((uint64_t)ir.y << 32) | ir.x));
                inv_theta = 1.0 / theta;
                cbase = ir.z;
                rowb = ir.w;
                A = 0.0;
                K = 0.0;
                V = 0.0;
            }
            const uint4 r = *lds_ptr<const uint4>((min(id[k], (uint32_t)G) << 4) + L.grp);
            const double mu = (double)__uint_as_float(r.x);
            const double var = (double)__uint_as_float(r.y);
            const float slo = __uint_as_float(r.z);
            const double n = (double)(r.w >> kGenCountShift);
            const uint32_t m = r.w & 255u;
            K = K + *lds_ptr<const double>(rowb + (m << 3));    // swap (0 when none)
            if (EVICT && ((evw >> (s & 31)) & 1u)) K = K + ecost;
            const double Yg = fma(K, theta, A);                  // theta E[W]
            const double num = fma((double)slo, theta, -Yg);     // theta (slo - E[W])
            const float vz = (float)(V * kVarScale);
            float prob;
            if (vz >= 1.17549435e-38f) {
                const float rs = __builtin_amdgcn_rsqf(vz);
                float tt = fmaf(-(float)num, rs, kTailMid);
                tt = __builtin_amdgcn_fmed3f(tt, kTailLo, kTailHi);
                const float2 c =
                    *lds_ptr<const float2>(tail0 + ((__float_as_uint(tt) & kTailCellBits) >> 10));
                prob = fmaf(c.y, tt, c.x);
            } else {
                const double EW = A / theta + K;
                if (V > 0.0) {
                    const double SD = sqrt(V) / theta;
                    prob = (float)(0.5 * erfc(((double)slo - EW) / (SD * 1.4142135623730951)));
                } else {
                    prob = EW > (double)slo ? 1.0f : 0.0f;
                }
            }
            S = fma(n, (double)prob, S);
            if (PEN) PE = fma(-num, inv_theta, PE);
            if (DETAIL && det) {
                const int64_t o = (int64_t)s * a.d_count + dq;
                if (a.d_mean) a.d_mean[o] = (float)(Yg * inv_theta);
                if (a.d_sd) a.d_sd[o] = (float)(sqrt(V) * inv_theta);
                if (a.d_prob) a.d_prob[o] = prob;
            }
            A = A + n * mu;
            V = V + n * var;
            rowb = cbase + m * row_bytes;
        }
    }
    S_out = S;
    PE_out = PE;
}
#pragma clang fp contract(on)

// Screening score of every plan.  One lane = one plan; the slots of a plan are
// walked in order, so every prefix sum is a running sum.  Per slot: the
// group's record (one LDS gather), the tokens ahead and the swap/eviction
// seconds in double (Y = tokens + theta * seconds), the variance ahead in
// single precision within a block of 32 slots on top of a double sum of the
// earlier blocks, the standardised margin, and the violation probability from
// the tail table.
template <bool EVICT, bool PEN, bool DETAIL>
__global__ __launch_bounds__(kScoreThreads) __attribute__((amdgpu_waves_per_eu(4, 4))) void k_score(ScoreArgs a)
{
    __shared__ __align__(16) float2 s_tail[kTailCells];
    extern __shared__ __align__(16) unsigned char lds[];
    const Lds L = lds_layout(a, lds);
    stage_tail(s_tail);
    // The form of the group records: compact when every group, model and cost
    // fits it, else general (and every plan takes the exact walk).  Every
    // workgroup stages the same tables, so all take the same decision.  (The
    // flag goes through LDS and readfirstlane, so that the compiler knows it is
    // uniform: the fast path's scalar row addressing depends on that.)
    __shared__ int s_compact;
    if (threadIdx.x == 0) s_compact = 1;
    __syncthreads();
    // (both tables are staged whatever the first one's answer)
    const bool costs_fit = stage_costs(a, L);
    const bool groups_fit = stage_compact(a, L);
    const bool fits = costs_fit && groups_fit;
    if (!fits) s_compact = 0;
    __syncthreads();
    const bool compact = __builtin_amdgcn_readfirstlane(s_compact) != 0;
    if (!compact) stage_general(a, L);
    double *red = lds_ptr<double>(L.red);
    if (a.wg_nsum && blockIdx.x == 0) {
        if (threadIdx.x == 0 && a.ncand) *a.ncand = 0;
        double t = 0.0;
        for (int i = threadIdx.x; i < a.G; i += blockDim.x)
            t += (double)(uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
        for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o, kWave);
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = t;
        __syncthreads();
        if (threadIdx.x == 0) {
            double s = 0.0;
            for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += red[w];
            *a.wg_nsum = s;
        }
    }
    __syncthreads();

    const uint32_t grp0 = L.grp;
    const uint32_t inst0 = L.inst;
    const uint32_t tail0 = lds_addr(s_tail);

    const int lane = threadIdx.x & (kWave - 1);
    // the wavefront index is uniform within a wavefront; say so, so that the
    // tile, its row addresses and the buffer resources live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wpb = blockDim.x / kWave;
    const int64_t ntiles = (a.P + kWave - 1) / kWave;
    const int G = a.G;
    // G held in a vector register (a scalar operand would cost the gather's
    // clamp its short issue form)
    const uint32_t Gv = in_vgpr((uint32_t)G);
    const int I1 = a.I - 1;
    const int64_t ld = a.ld;
    const int ev_shift = a.ev_shift;
    const int cs3 = a.col_shift + 3;          // log2(bytes per cost-table row)
    double lane_min = INFINITY;

    // With a.nparts = 2 or 4 every tile (64 plans) is scored by that many
    // wavefronts of the workgroup: part k takes slots [bound[k-1], bound[k])
    // (bound[-1] = 0, bound[nparts-1] = G), each part after the first after a
    // warm-up that rebuilds the running sums of the queue holding its first
    // slot.  The partial sums pass through the outputs from the last part to
    // the first, one barrier apart; the first part adds its own last.  Tiles
    // are taken in rounds, the same number for every wavefront of the
    // workgroup.
    const int np = a.nparts;
    const bool halves = np > 1;
    const int per_round = wpb / np;
    const int in_round = wave / np;
    const int part = wave & (np - 1);
    const bool back = part > 0;
    const int s_begin = back ? a.bound[part - 1] : 0;
    const int s_end = part < np - 1 ? a.bound[part] : G;
    if (!compact) {
      // General records: the front wavefront of each tile walks the whole plan
      // exactly (walk_general); the back one, if any, idles.
      for (int64_t r0 = (int64_t)blockIdx.x * per_round; r0 < ntiles;
           r0 += (int64_t)gridDim.x * per_round) {
        const int64_t t = r0 + in_round;
        if (back || t >= ntiles) continue;
        const int64_t tb = t * kWave;
        const bool live = tb + lane < a.P;
        const int lp = live ? lane : (int)(a.P - 1 - tb);
        const int64_t p = tb + lp;
        const bool det = DETAIL && live && p >= a.d_begin && p < a.d_begin + a.d_count;
        double S = 0.0, PE = 0.0;
        walk_general<EVICT, PEN, DETAIL>(a, L, tail0, tb, lp, det, p - a.d_begin, S, PE);
        if (live) {
          a.score[p] = S;
          if (PEN) a.penalty[p] = PE;
          lane_min = fmin(lane_min, S);
        }
      }
    } else
    for (int64_t r0 = (int64_t)blockIdx.x * per_round; r0 < ntiles; r0 += (int64_t)gridDim.x * per_round) {
      const int64_t t = r0 + in_round;
      double S_out = 0.0, PE_out = 0.0;
      int64_t p_out = -1;                           // the lane's plan when live
      if (t < ntiles) {
        const int64_t tb = t * kWave;               // first plan of the tile (uniform)
        const bool live = tb + lane < a.P;
        const int lp = live ? lane : (int)(a.P - 1 - tb);   // lane's plan, relative to tb
        const uint32_t lpb = (uint32_t)lp * 4u;     // its byte offset within a row
        const int64_t p = tb + lp;
        const bool det = DETAIL && live && p >= a.d_begin && p < a.d_begin + a.d_count;
        const int64_t dq = p - a.d_begin;
        // Row r of a slot-major array, lane's column: a plain global load (queue
        // offsets, rare), and buffer loads from a resource based at a block's
        // first row (group ids, eviction words), whose row offset is a scalar
        // operand: no per-load vector arithmetic.
        const int64_t ld4 = ld * 4;
        auto at = [&](const void *base, int row) __attribute__((always_inline)) {
            const unsigned char *rp =
                reinterpret_cast<const unsigned char *>(base) + (int64_t)row * ld4 + tb * 4;
            return *reinterpret_cast<const uint32_t *>(rp + lpb);
        };
        auto rsrc_at = [&](const void *base, int row) __attribute__((always_inline)) {
            const unsigned char *rp =
                reinterpret_cast<const unsigned char *>(base) + (int64_t)row * ld4 + tb * 4;
            return __builtin_amdgcn_make_buffer_rsrc((void *)rp, (short)0, 0x7FFFFFFF, 0x00020000);
        };
        // (non-temporal: every plan row is read once, and streaming it past the
        // caches leaves them to the queue offsets and tables that are reused)
        auto ld_rel = [&](__amdgpu_buffer_rsrc_t r, int rel_row) __attribute__((always_inline)) {
            return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)lpb, rel_row * (int)ld4, 2);
        };

        double Y = 0.0;        // tokens ahead + theta * (swap and eviction seconds so far)
        double V = 0.0;        // scaled variance ahead, through the previous block
        float vb = 0.0f;       // V rounded to single precision
        float vblk = 0.0f;     // scaled variance ahead added within the current block
        // rsqrt of the next slot's scaled variance ahead, formed one slot early
        // (the reciprocal square root has a long latency; inf at a queue head,
        // where the variance ahead is 0)
        float rsn = INFINITY;
        double S = 0.0;        // sum of n * P, through the previous block
        float S32 = 0.0f;      // sum of n * P within the current block
        double PE = 0.0;       // sum of (E[W] - slo)
        double theta = 1.0, inv_theta = 1.0;
        uint32_t cbase = 0u;   // cost-table row base of the current queue's class
        // Queue bookkeeping.  g is the queue of the current slot and nb the slot
        // where the next queue starts.  Parameters of upcoming queues reach a
        // queue head through a prefetch at the start of every block of 32 slots:
        //   f1, f2   queues q0+1 and q0+2, q0 = g at the start of the block
        //   x        at the start of a block, the next queue's parameters from the
        //            previous block's f1 or f2 (by how many queues that block
        //            entered); `fast` marks lanes for which x is valid and the
        //            queue not empty.  A block's first head uses x; a second one
        //            uses this block's f2; anything else loads on the spot.
        struct QP {
            int nb;               // end boundary of the queue (INT_MAX for the last)
            double theta, inv;
            uint32_t cbase, head;
        };
        int g = -1, nb = 0, q0 = -1;
        int base = 0, nbr = 0;    // current block start, nb - base
        // In a fast block: bit k set when some lane's next queue starts at slot
        // base + k + 1 (the or over the wavefront of each lane's one head)
        uint32_t hm = 0u;
        QP x{0, 1.0, 1.0, 0u, 0u}, f1 = x, f2 = x;
        bool fast = false;

        // Issued for every lane, never under a per-lane condition (clamped
        // index), so that the compiler counts the outstanding loads exactly.
        // (the lane's queue-offset column: one 32 x 32 -> 64-bit multiply-add
        // per row; plan_stride <= 2^22 keeps the row pitch within 32 bits)
        const unsigned char *qcol = reinterpret_cast<const unsigned char *>(a.qoff) + tb * 4 + lpb;
        const uint32_t ld4u = (uint32_t)ld4;
        auto load_qp = [&](int h) __attribute__((always_inline)) {
            h = min(h, I1);                   // g >= 0 wherever this is called
            QP q;
            q.nb = (int)*reinterpret_cast<const uint32_t *>(qcol + (uint64_t)(uint32_t)(h + 1) * ld4u);
            const uint4 r = *lds_ptr<const uint4>(inst0 + 16u * (uint32_t)h);
            q.theta = __longlong_as_double((long long)(((uint64_t)r.y << 32) | r.x));
            q.inv = 1.0;
            q.cbase = r.z;
            q.head = r.w;
            return q;
        };
        int c_in = 0;                 // queues entered in the block before
        uint32_t ev_nx = 0u;          // eviction word of the next block
        auto block_start = [&]() __attribute__((always_inline)) {
            const int c = g - q0;     // queues entered since the previous start
            x.nb = c == 0 ? f1.nb : f2.nb;
            x.theta = c == 0 ? f1.theta : f2.theta;
            x.cbase = c == 0 ? f1.cbase : f2.cbase;
            x.head = c == 0 ? f1.head : f2.head;
            if (g + 1 >= I1) x.nb = INT_MAX;
            if (PEN || DETAIL) x.inv = 1.0 / x.theta;
            fast = c <= 1 && g < I1 && x.nb > nb;
            q0 = g;
            c_in = c;
        };
        // The reads for the next block (queue parameters, eviction word), issued
        // at the start of either path of a block, not before the choice: where
        // the two paths join, a read issued before the choice looks just issued
        // on the path that consumed it long ago, and the wait for it there
        // waited for every later read too (memory reads complete in order), the
        // fast path's ring of group ids included.
        auto prefetch = [&](int sb) __attribute__((always_inline)) {
            __builtin_amdgcn_sched_barrier(0);        // select before the reload
            // queue g + 1 is x itself when every lane entered at most one queue
            // in the block before: only queue g + 2 is loaded then
            if (__builtin_amdgcn_ballot_w64(c_in > 1) == 0)
                f1 = x;
            else
                f1 = load_qp(g + 1);
            f2 = load_qp(g + 2);
            if (EVICT) ev_nx = ld_rel(rsrc_at(a.evict, min((sb >> 5) + 1, (G - 1) >> 5)), 0);
        };
        // Enter queue g + 1 (or the first non-empty queue after it) at slot s,
        // loading its parameters on the spot and waiting for them.
        auto enter_slow = [&](int s, uint32_t &rowb) __attribute__((always_inline)) {
            int h = g + 1;
            int e_nb = (int)at(a.qoff, h + 1);
            uint4 r = *lds_ptr<const uint4>(inst0 + 16u * (uint32_t)h);
            __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0)
            g = h;
            // empty queues: skip them.  The loop runs while any lane needs it (a
            // wavefront-uniform exit), the lanes that are done idle in it.
            bool more = e_nb <= s && g < I1;
            while (__builtin_amdgcn_ballot_w64(more)) {
                if (more) {
                    h = g + 1;
                    e_nb = (int)at(a.qoff, h + 1);
                    r = *lds_ptr<const uint4>(inst0 + 16u * (uint32_t)h);
                    __builtin_amdgcn_s_waitcnt(0x0070);
                    g = h;
                    more = e_nb <= s && g < I1;
                }
            }
            nb = g >= I1 ? INT_MAX : e_nb;
            theta = __longlong_as_double((long long)(((uint64_t)r.y << 32) | r.x));
            if (PEN || DETAIL) inv_theta = 1.0 / theta;
            cbase = r.z;
            rowb = r.w;
        };
        // Slot s is the head of the next queue: switch to it and reset the sums.
        // enter_fast is the common case, where the next queue is x (prefetched a
        // block ago, not empty); enter_any takes every case.
        auto reset_sums = [&]() __attribute__((always_inline)) {
            Y = 0.0;
            V = 0.0;
            vb = 0.0f;
            vblk = 0.0f;
        };
        // (In a fast block g, nb and the double variance sum are brought up to
        // date at the end of the block, from whether the block held the head nbr
        // names; nbr itself stays, as no second head can follow in the block.)
        auto enter_fast = [&](uint32_t &rowb) __attribute__((always_inline)) {
            theta = x.theta;
            if (PEN || DETAIL) inv_theta = x.inv;
            cbase = x.cbase;
            rowb = x.head;
            Y = 0.0;
            if (DETAIL) V = 0.0;
            vb = 0.0f;
            vblk = 0.0f;
        };
        auto enter_any = [&](int s, uint32_t &rowb) __attribute__((always_inline)) {
            if (fast) {
                g += 1;
                nb = x.nb;
                theta = x.theta;
                if (PEN || DETAIL) inv_theta = x.inv;
                cbase = x.cbase;
                rowb = x.head;
                fast = false;
            } else if (g == q0 + 1 && q0 + 2 <= I1 && (q0 + 2 >= I1 || f2.nb > s)) {
                g = q0 + 2;
                nb = g >= I1 ? INT_MAX : f2.nb;
                theta = f2.theta;
                if (PEN || DETAIL) inv_theta = 1.0 / theta;
                cbase = f2.cbase;
                rowb = f2.head;
            } else {
                enter_slow(s, rowb);
            }
            nbr = nb - base;
            reset_sums();
        };

        // Software pipeline over the slots of the plan:
        //   ring[8]   group ids of the next 8 slots (buffer loads, 8 slots ahead: with
        //             four wavefronts per SIMD that covers the memory latency, and
        //             leaves the kernel within 128 registers without spills)
        //   rec[4]    LDS records of slots s..s+2 (gathered D = 2 slots ahead)
        //   cost      swap/eviction seconds of slot s, read during slot s-1
        //   rsn       rsqrt of slot s's variance ahead, formed at the end of slot s-1
        //   tc, tcp   tail-table cells of slots s-1 and s-2 (with tf, tfp, tnx, tnxp)
        // Slot s: (0) the probability of slot s-2, (1) the cost of s+1 read on the
        // current queue's row, (2) waits and variances of slot s, (3) its tail
        // position, (4) if s+1 starts a queue: switch, and read the cost of s+1
        // again on the head row, (5) the rsqrt of s+1's variance ahead and the
        // tail cell of slot s.  A cost is used one
        // slot after its read, a tail cell two.
        // At the start of a block at slot sb: ring[j] holds the group id of slot
        // sb + j (j >= D) or sb + R + j (j < D), rec[k] the record of slot sb + k
        // (k < D), cost and colc those of slot sb.
        constexpr int D = 2;
        constexpr int R = 8;
        int32_t ring[R];
        uint4 rec[4];                 // rec[s % 4] holds slot s's record
        // (ids clamped to G in 16 bits: G < 2^16, and an id of 2^16 or more
        // lands on some group, in bounds)
        auto gather = [&](int32_t gid) __attribute__((always_inline)) {
            const uint32_t c = (uint32_t)min((uint16_t)gid, (uint16_t)Gv);
            return *lds_ptr<const uint4>((c << 4) + grp0);
        };
        // Back half: the state of the plan at slot s_begin (a multiple of 32,
        // > 0).  The queue holding it is the last one starting at or before it
        // (found from a scan of the queue offsets); its running sums are rebuilt
        // from its first slot qs over the rows [min qs, s_begin), read in
        // lockstep (a lane skips the rows before its own qs).  rowb: the
        // cost-table row of slot s_begin.
        auto warm_up = [&](uint32_t &rowb) __attribute__((always_inline)) {
            const int Gs = s_begin;
            int c = 0, qs = 0, nxt = INT_MAX;
            for (int h0 = 0; h0 <= I1 + 1; h0 += 8) {
                uint32_t qv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) qv[u] = at(a.qoff, min(h0 + u, I1 + 1));
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int q = (int)qv[u];
                    const bool in = h0 + u <= I1 + 1;
                    if (in && q <= Gs) {
                        c = h0 + u + 1;
                        qs = q;
                    }
                    if (in && q > Gs) nxt = min(nxt, q);
                }
            }
            g = clampi(c - 1, 0, I1);
            nb = g >= I1 ? INT_MAX : nxt;
            const uint4 ir = *lds_ptr<const uint4>(inst0 + 16u * (uint32_t)g);
            theta = __longlong_as_double((long long)(((uint64_t)ir.y << 32) | ir.x));
            if (PEN || DETAIL) inv_theta = 1.0 / theta;
            cbase = ir.z;
            qs = clampi(qs, 0, Gs);
            int qmin = qs;
            for (int o = 32; o > 0; o >>= 1) qmin = min(qmin, __shfl_xor(qmin, o, kWave));
            const int s0 = __builtin_amdgcn_readfirstlane(qmin) & ~15;
            double Yw = 0.0, Vw = 0.0;
            uint32_t colp = 0u;
            for (int c0 = s0; c0 < Gs; c0 += 16) {      // Gs - s0 is a multiple of 16
                const __amdgpu_buffer_rsrc_t rw = rsrc_at(a.perm, c0);
                uint32_t id[16];
#pragma unroll
                for (int k = 0; k < 16; ++k) id[k] = ld_rel(rw, k);
                const uint32_t evw = EVICT ? at(a.evict, c0 >> 5) : 0u;
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    const int s = c0 + k;
                    const uint4 r = gather((int32_t)id[k]);
                    const uint32_t col = rec_model(r.w);
                    if (s >= qs) {
                        const uint32_t evb =
                            EVICT ? __builtin_amdgcn_ubfe(evw, (uint32_t)(s & 31), 1u) << ev_shift : 0u;
                        const uint32_t rb = s == qs ? ir.w : cbase + (colp << cs3);
                        const double cst = *lds_ptr<const double>(rb + (col << 3) + evb);
                        Yw = fma(cst, theta, Yw);
                        Yw = Yw + rec_nmu(r);
                        Vw += (double)rec_nv(r);
                    }
                    colp = col;
                }
            }
            Y = Yw;
            V = Vw;
            vb = (float)V;
            vblk = 0.0f;
            rsn = __builtin_amdgcn_rsqf(vb);
            rowb = qs == Gs ? ir.w : cbase + (colp << cs3);
            // prefetch as if queue g had been entered during the block before
            q0 = g - 1;
            f1 = load_qp(g);
            f2 = load_qp(g + 1);
        };
        uint32_t rowb0 = 0u;          // cost-table row of slot s_begin
        if (!back) {
            // prefetch relative to q0 = -1 (queues 0 and 1), issued before the
            // entry into queue 0, whose full wait leaves nothing pending
            q0 = -1;
            f1 = load_qp(0);
            f2 = load_qp(1);
            enter_slow(0, rowb0);
        } else {
            warm_up(rowb0);
        }
        // the pipeline at s_begin (a multiple of 32)
        __amdgpu_buffer_rsrc_t rp = rsrc_at(a.perm, s_begin);
#pragma unroll
        for (int k = 0; k < R; ++k) ring[k] = (int32_t)ld_rel(rp, min(s_begin + k, G - 1) - s_begin);
#pragma unroll
        for (int k = 0; k < D; ++k) {
            rec[k] = gather(ring[k]);
            ring[k] = (int32_t)ld_rel(rp, min(s_begin + k + R, G - 1) - s_begin);
        }
        rec[D] = rec[0];
        uint32_t ev = EVICT ? ld_rel(rsrc_at(a.evict, s_begin >> 5), 0) : 0u;   // word of the block
        uint32_t colc = rec_model(rec[0].w);    // cost-table column (model) of the current slot
        double cost = *lds_ptr<const double>(rowb0 + (colc << 3) + (EVICT ? (ev & 1u) << ev_shift : 0u));
        // Tail cells in flight: slot s's cell is read at the end of slot s, after
        // the cost entries (so that waiting for a cost, or rereading it at a
        // queue head, does not wait for the tail read) and used at the start of
        // slot s + 2.  (tc, tf, tnx): slot s - 1's cell, t and record word x
        // (count in the low half); (tcp, tfp, tnxp): slot s - 2's.
        float2 tc = make_float2(0.0f, 0.0f), tcp = tc;
        float tf = 0.0f, tfp = 0.0f;
        uint32_t tnx = 0u, tnxp = 0u;

        // The probability of the previous slot from its tail cell.
        auto finish = [&](int s_prev) __attribute__((always_inline)) {
            const float prob = fmaf(tcp.y, tfp, tcp.x);
            S32 = fma_count(tnxp, prob, S32);
            // settled here: sunk to the end of the block, the sums of all 32 slots
            // would keep their tail cells live in registers
            asm volatile("" : "+v"(S32));
            if (DETAIL && det && a.d_prob && s_prev >= s_begin)
                a.d_prob[(int64_t)s_prev * a.d_count + dq] = prob;
        };

        // One slot.  w1: record word of slot s + 1; evw, b1: its eviction word and
        // bit.  fast_block (std::true_type / false_type): only the common queue
        // switch can happen here.
        auto step = [&](auto fast_block, int s, const uint4 r, uint32_t w1, uint32_t evw,
                        uint32_t b1) __attribute__((always_inline)) {
            // (0) the probability of slot s-2
            finish(s - 2);
            tcp = tc;
            tfp = tf;
            tnxp = tnx;
            // (1) cost of slot s+1 if it stays in this queue
            const uint32_t col1 = rec_model(w1);
            // entry of the row, in doubles, the eviction twin included (bit b1 of
            // the eviction word moved to bit kTwinShift: a right shift, or a
            // 16-bit left shift for the low bits)
            const uint32_t off1 = EVICT ? (col1 | (twin_bit(evw, b1) & kTwinEntries)) : col1;
            const uint32_t rb = in_vgpr(cbase + (colc << cs3));
            double cost1 = *lds_ptr<const double>(rb + (off1 << 3));

            // (2) slot s
            const double nmu = rec_nmu(r);
            const float nv = rec_nv(r);
            const float slo = rec_slo(r);
            Y = fma(cost, theta, Y);
            const double nnum = fma(-(double)slo, theta, Y);  // theta (E[W] - slo)
            if (DETAIL && det) {
                const int64_t o = (int64_t)s * a.d_count + dq;
                if (a.d_mean) a.d_mean[o] = (float)(Y * inv_theta);
                if (a.d_sd) a.d_sd[o] = (float)(sqrt(V + (double)vblk) * kTailScale * inv_theta);
            }
            vblk += nv;
            const float rs = rsn;                 // cells per unit margin; inf if V = 0
            if (PEN) {
                PE = fma(nnum, inv_theta, PE);
                asm volatile("" : "+v"(PE));     // not sunk to the end of the block
            }
            Y = Y + nmu;

            // (3) tail cell of slot s
            tf = __builtin_amdgcn_fmed3f(fmaf((float)nnum, rs, kTailMid), kTailLo, kTailHi);
            tnx = r.x;
            // settled before the branch: nothing of slot s may sink into it
            asm volatile("" : "+v"(tf), "+v"(vblk));
            const uint32_t cell = (__float_as_uint(tf) & kTailCellBits) >> 10;   // cell * 8

            // (4) queue head at s+1?  In a fast block only where the block's head
            // mask says so: a scalar test, the comparison of every lane made in
            // those slots alone.
            if (!decltype(fast_block)::value || ((hm >> (uint32_t)(s - base)) & 1u)) {
                // (a branch of its own: the comparison is not to be merged into
                // the scalar test and made in every slot)
                asm volatile("");
                if (s + 1 - base == nbr) {       // s + 1 == nb, compared block-relative
                    uint32_t rowb;
                    if constexpr (decltype(fast_block)::value)
                        enter_fast(rowb);
                    else
                        enter_any(s + 1, rowb);
                    // (its own shift: one v_lshl_add_u32 here and one above, not a
                    // shared shift and two adds)
                    cost1 = *lds_ptr<const double>(rowb + (in_vgpr(off1) << 3));
                }
            }
            // (5) the variance ahead of slot s+1 (0 after a queue head, where its
            // reciprocal square root is inf) and the tail cell of slot s, read last
            rsn = __builtin_amdgcn_rsqf(vb + vblk);
            tc = *lds_ptr<const float2>(tail0 + cell);
            cost = cost1;
            colc = col1;
        };

        // Full 32-slot blocks.  A block runs unrolled and pipelined when every
        // lane enters at most the one queue x in it; otherwise (a second queue
        // head in the block, an empty queue, a queue not prefetched) the whole
        // wavefront takes the generic path for that block, slot by slot with
        // plain loads, and then refills the pipeline for the next block.
        const int G32 = G & ~31;
        const int s_full = s_end & ~31;       // the part bounds are multiples of 32
        for (int sb0 = s_begin; sb0 < s_full; sb0 += 32) {
            // uniform by construction; said explicitly so that the row offsets and
            // buffer resources below stay scalar
            const int sb = __builtin_amdgcn_readfirstlane(sb0);
            block_start();
            base = sb;
            nbr = nb - sb;
            const bool odd = nbr >= 1 && nbr <= 32 && (!fast || x.nb <= sb + 32);
            if (__builtin_amdgcn_ballot_w64(odd) == 0) {
                prefetch(sb);
                hm = wave_or(nbr >= 1 && nbr <= 32 ? 1u << (uint32_t)(nbr - 1) : 0u);
                rp = rsrc_at(a.perm, sb);
                const int lim = G - 1 - sb;           // last row, relative to the block
#pragma unroll
                for (int k = 0; k < 32; ++k) {
                    const int s = sb + k;
                    // ring entry of slot s+D: turned into its LDS record, then
                    // refilled with slot s+D+R (rows past the end clamp to the
                    // last row), so both share one register
                    const int j = (k + D) & (R - 1);
                    rec[(k + D) & 3] = gather(ring[j]);
                    __builtin_amdgcn_sched_barrier(0);    // consume before the refill
                    ring[j] = (int32_t)ld_rel(rp, min(k + D + R, lim));
                    step(std::true_type{}, s, rec[k & 3], rec[(k + 1) & 3].w,
                         k == 31 ? ev_nx : ev, (uint32_t)((k + 1) & 31));
                }
                // at most one queue entered in this block: bring g, nb and the
                // double variance sum up to date
                const bool moved = nbr >= 1 && nbr <= 32;
                g += moved ? 1 : 0;
                nb = moved ? x.nb : nb;
                if (!DETAIL) V = moved ? 0.0 : V;
            } else {
                prefetch(sb);
                uint4 r = rec[0];                     // slot sb (sb % 4 == 0)
                for (int k = 0; k < 32; ++k) {
                    const int s = sb + k;
                    const uint4 rn = gather((int32_t)at(a.perm, min(s + 1, G - 1)));
                    step(std::false_type{}, s, r, rn.w, k == 31 ? ev_nx : ev,
                         (uint32_t)((k + 1) & 31));
                    r = rn;
                }
                // refill the pipeline for the block at nx = sb + 32 (nx may be G:
                // every row is clamped to the last one, G - 1, and the resource is
                // based at a row that exists)
                const int nx = sb + 32;
                const int rb = min(nx, G - 1);
                const __amdgpu_buffer_rsrc_t rn = rsrc_at(a.perm, rb);
#pragma unroll
                for (int j = 0; j < R; ++j)
                    ring[j] = (int32_t)ld_rel(rn, min(nx + (j < D ? j + R : j), G - 1) - rb);
#pragma unroll
                for (int k = 0; k < D; ++k)
                    rec[k] = gather((int32_t)at(a.perm, min(nx + k, G - 1)));
            }
            if (EVICT) ev = ev_nx;
            V += (double)vblk;        // fold the block into the double sums
            vb = (float)V;
            vblk = 0.0f;
            S += (double)S32;
            S32 = 0.0f;
        }
        // Remaining G % 32 slots, one at a time (plain loads).  The pipeline has
        // already resolved the head and the cost of slot G32, whose record is
        // rec[0] (G32 is a multiple of 4).
        if (s_end == G) {
            uint4 r = rec[0];
            base = G32;
            nbr = nb - G32;
            for (int s = G32; s < G; ++s) {
                const uint4 rn = gather((int32_t)at(a.perm, min(s + 1, G - 1)));
                step(std::false_type{}, s, r, rn.w, ev, (uint32_t)((s + 1) & 31));
                r = rn;
            }
        }
        finish(s_end - 2);
        tcp = tc;
        tfp = tf;
        tnxp = tnx;
        finish(s_end - 1);
        S += (double)S32;
        if (live) {
            S_out = S;
            PE_out = PE;
            p_out = p;
        }
      }
      if (halves) {
          // the later parts' sums go through the outputs to the first part
          for (int k = np - 1; k >= 1; --k) {
              if (part == k && p_out >= 0) {
                  if (k < np - 1) {
                      S_out += a.score[p_out];
                      if (PEN) PE_out += a.penalty[p_out];
                  }
                  a.score[p_out] = S_out;
                  if (PEN) a.penalty[p_out] = PE_out;
              }
              __syncthreads();
          }
          if (!back && p_out >= 0) {
              S_out += a.score[p_out];
              if (PEN) PE_out += a.penalty[p_out];
          }
      }
      if (!back && p_out >= 0) {
          a.score[p_out] = S_out;
          if (PEN) a.penalty[p_out] = PE_out;
          lane_min = fmin(lane_min, S_out);
      }
    }
    if (a.wg_min) {
        const double m = wave_min(lane_min);
        __syncthreads();
        if (lane == 0) red[wave] = m;
        __syncthreads();
        if (threadIdx.x == 0) {
            double b = INFINITY;
            for (int w = 0; w < wpb; ++w) b = fmin(b, red[w]);
            a.wg_min[blockIdx.x] = b;
        }
    }
}

// ---------------------------------------------------------------------------
// Exact double-precision scoring: the definition written out as the oracle
// reads it (tokens and variance ahead summed in position order, E[W] = A/Theta
// + K, SD = sqrt(V)/Theta, P = erfc((slo - E)/(SD sqrt 2))/2), summed per queue
// and then over queues in order.  No contraction into fused multiply-adds.

struct ExactArgs {
    int32_t G, I, M, C;
    const int32_t *grp_count;
    const float *grp_mu, *grp_var, *grp_slo;
    const int32_t *grp_model;
    const float *inst_tput;
    const int32_t *inst_class, *inst_model0;
    const float *swap_cost;
    float evict_cost;
    int64_t P, ld;
    const int32_t *perm, *qoff;
    const uint32_t *evict;
};

#pragma clang fp contract(off)
// Exact score of queue g of plan p by one wavefront.  Each round takes the
// next 64 positions, one per lane; the running sums (tokens n mu and variance
// n var ahead, costs K) ripple from lane to lane in position order, so every
// lane holds the same sums a serial walk forms at its position.  Each lane
// then forms its position's E[W], SD and term n P, and the terms ripple into
// the queue's sum the same way.  A ripple takes the round's positions less
// one steps, rounded up to blocks of 8 (a step past the last position leaves
// every position's sums unchanged), with the count in a scalar register so
// that only a block ends in a branch.  Loads run ahead: the next round's group
// fields and swap costs, and the group ids of the round after.  Returns the
// queue's score in every lane.  Group ids are clamped to [0, G), offsets to
// [0, G] (malformed plans never read out of bounds).
struct RoundIn {
    int m;                    // model (0 where the lane holds no position)
    uint32_t n;               // requests (0 where none)
    float mu, var, slo;
    uint32_t ev;              // eviction word of the lane's position
};

__device__ double wave_queue_exact(const ExactArgs &a, int64_t p, int g)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int G = a.G;
    const int64_t ld = a.ld;
    const int bq = clampi(a.qoff[(int64_t)g * ld + p], 0, G);
    const int eq = clampi(a.qoff[(int64_t)(g + 1) * ld + p], bq, G);
    const double theta = (double)a.inst_tput[g];
    const int64_t swap_row = (int64_t)clampi(a.inst_class[g], 0, a.C - 1) * a.M;
    int prev = a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
    const double ecost = (double)a.evict_cost;
    // group id at position v0 + lane, -1 beyond the queue
    auto ids = [&](int v0) -> int {
        const int s = v0 + lane;
        return s < eq ? (int)min((uint32_t)a.perm[(int64_t)s * ld + p], (uint32_t)(G - 1)) : -1;
    };
    auto fields = [&](int i, int v0) -> RoundIn {
        RoundIn f{0, 0u, 0.f, 0.f, 0.f, 0u};
        if (i >= 0) {
            f.m = clampi(a.grp_model[i], 0, a.M - 1);
            f.n = (uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
            f.mu = a.grp_mu[i];
            f.var = a.grp_var[i];
            f.slo = a.grp_slo[i];
            if (a.evict) f.ev = a.evict[(int64_t)((v0 + lane) >> 5) * ld + p];
        }
        return f;
    };
    // swap cost into this lane's position from the one before (prev for lane 0)
    auto swap_in = [&](const RoundIn &f, bool on) -> float {
        int pm = __shfl_up(f.m, 1, kWave);
        if (lane == 0) pm = prev;
        return (on && pm >= 0 && pm != f.m && a.swap_cost)
                   ? a.swap_cost[(swap_row + pm) * a.M + f.m] : 0.f;
    };
    int i0 = ids(bq);
    RoundIn f = fields(i0, bq);
    int i2 = ids(bq + kWave);
    float sw = swap_in(f, i0 >= 0);
    double rA = 0.0, rV = 0.0, rK = 0.0, rC = 0.0;
    for (int v0 = bq; v0 < eq; v0 += kWave) {
        const int cnt = min(kWave, eq - v0);
        const bool on = lane < cnt;
        const int i1 = i2;
        const RoundIn f1 = fields(i1, v0 + kWave);
        i2 = ids(v0 + 2 * kWave);
        const double n = (double)f.n;
        const double xa = n * (double)f.mu;
        const double xb = n * (double)f.var;
        const double c1 = (double)sw;
        const double c2 = (on && ((f.ev >> ((v0 + lane) & 31)) & 1u)) ? ecost : 0.0;
        const double la = from_left0(xa), lb = from_left0(xb);
        const double l1 = from_left0(c1), l2 = from_left0(c2);
        double A = rA, V = rV, K = rK;
        const int steps = __builtin_amdgcn_readfirstlane(cnt - 1);
        for (int j = 0; j < steps; j += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                A = from_left(A) + la;
                V = from_left(V) + lb;
                K = (from_left(K) + l1) + l2;
            }
        }
        K = K + c1;
        K = K + c2;
        const double EW = A / theta + K;
        const double SD = sqrt(V) / theta;
        const double slo = (double)f.slo;
        double P;
        if (SD > 0.0)
            P = 0.5 * erfc((slo - EW) / (SD * 1.4142135623730951));
        else
            P = (EW > slo) ? 1.0 : 0.0;
        const double term = on ? n * P : 0.0;
        const double lt = from_left0(term);
        double C = rC;
        for (int j = 0; j < steps; j += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) C = from_left(C) + lt;
        }
        const int last = cnt - 1;
        rA = lane_value(A, last) + lane_value(xa, last);
        rV = lane_value(V, last) + lane_value(xb, last);
        rK = lane_value(K, last);
        rC = lane_value(C, last) + lane_value(term, last);
        prev = __builtin_amdgcn_readlane(f.m, last);
        f = f1;
        sw = swap_in(f, i1 >= 0);
    }
    return rC;
}

// Exact score of plan p by a whole workgroup: its wavefronts take queues, the
// queue sums go to LDS, and thread 0 adds them in queue order.
__device__ double block_plan_exact(const ExactArgs &a, int64_t p, double *qpart)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int nw = blockDim.x / kWave;
    double total = 0.0;
    for (int g0 = 0; g0 < a.I; g0 += kExactPass) {
        const int n = min(kExactPass, a.I - g0);
        for (int j = wave_id(); j < n; j += nw) {
            const double sc = wave_queue_exact(a, p, g0 + j);
            if (lane == 0) qpart[j] = sc;
        }
        __syncthreads();
        if (threadIdx.x == 0)
            for (int k = 0; k < n; ++k) total += qpart[k];
        __syncthreads();
    }
    return total;   // valid in thread 0
}
#pragma clang fp contract(on)

__global__ __launch_bounds__(kExactThreads) void k_exact(ExactArgs a, const int64_t *idx,
                                                         int64_t n, double *out)
{
    __shared__ double qpart[kExactPass];
    for (int64_t k = blockIdx.x; k < n; k += gridDim.x) {
        int64_t p = idx[k];
        const bool ok = p >= 0 && p < a.P;
        p = ok ? p : 0;
        const double s = block_plan_exact(a, p, qpart);
        if (threadIdx.x == 0) out[k] = ok ? s : NAN;
    }
}

// (score, index) minimum over a workgroup: lowest score, then lowest index;
// index -1 marks "none".  Result valid in every thread.
__device__ void block_argmin(double &s, int64_t &i, double *ls, int64_t *li)
{
    for (int o = 32; o > 0; o >>= 1) {
        const double s2 = __shfl_xor(s, o, kWave);
        const int64_t i2 = __shfl_xor(i, o, kWave);
        const bool take = i2 >= 0 && (i < 0 || s2 < s || (s2 == s && i2 < i));
        s = take ? s2 : s;
        i = take ? i2 : i;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    __syncthreads();
    if (lane == 0) {
        ls[wave] = s;
        li[wave] = i;
    }
    __syncthreads();
    s = INFINITY;
    i = -1;
    for (int w = 0; w < nw; ++w) {
        const bool take = li[w] >= 0 && (i < 0 || ls[w] < s || (ls[w] == s && li[w] < i));
        s = take ? ls[w] : s;
        i = take ? li[w] : i;
    }
    __syncthreads();
}

__device__ double block_min(double v, double *ls)
{
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    __syncthreads();
    if (lane == 0) ls[wave] = v;
    __syncthreads();
    double b = INFINITY;
    for (int w = 0; w < (int)(blockDim.x / kWave); ++w) b = fmin(b, ls[w]);
    __syncthreads();
    return b;
}

// Candidate selection: every workgroup reduces the per-workgroup minima of the
// screened scores, then appends the plans of its share whose screened score is
// within twice the screening error bound of the minimum (the exact minimum is
// always among them) to the candidate list, one atomic per wavefront.  The
// scoring kernel zeroed the count.
__global__ __launch_bounds__(kSelThreads) void k_gselect(const double *fast, const double *wg_min,
                                                         int n_wg, const double *nsum, int64_t P,
                                                         int64_t *cand, int32_t *ncand)
{
    __shared__ double ls[kSelThreads / kWave];
    double m = INFINITY;
    for (int k = threadIdx.x; k < n_wg; k += blockDim.x) m = fmin(m, wg_min[k]);
    m = block_min(m, ls);
    // |screened - exact| <= eps * (total requests), plus the rounding of both sums
    const double delta = kEpsP * (*nsum) * (1.0 + 1e-9) + 1e-300;
    const double thr = m + 2.0 * delta;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t stride = (int64_t)gridDim.x * kSelThreads;
    for (int64_t base = (int64_t)blockIdx.x * kSelThreads + (threadIdx.x - lane); base < P;
         base += stride) {
        const int64_t p = base + lane;
        const bool c = p < P && fast[p] <= thr;
        const uint64_t bal = __ballot(c);
        if (bal) {
            int off = 0;
            if (lane == 0) off = atomicAdd(ncand, __popcll(bal));
            off = __shfl(off, 0, kWave);
            if (c) cand[off + __popcll(bal & ((1ull << lane) - 1ull))] = p;
        }
    }
}

// Exact scores of the candidates.  When the per-(candidate, queue) sums fit
// (count <= cap), one wavefront per (candidate, queue) writes its queue's
// score to Q; else every workgroup scores whole candidates and writes the
// plan's score over its screened score in X.
__global__ __launch_bounds__(kGexThreads) void k_gexact(ExactArgs a, const int64_t *cand,
                                                        const int32_t *ncand, int64_t cap,
                                                        double *Q, double *X)
{
    __shared__ double qpart[kExactPass];
    const int64_t n = __builtin_amdgcn_readfirstlane(ncand[0]);
    if (n <= cap) {
        constexpr int nwv = kGexThreads / kWave;
        const int64_t tasks = n * a.I;
        for (int64_t t = (int64_t)blockIdx.x * nwv + wave_id(); t < tasks;
             t += (int64_t)gridDim.x * nwv) {
            const int64_t k = t / a.I;
            const int g = (int)(t - k * a.I);
            int64_t p = cand[k];
            p = p < 0 ? 0 : (p >= a.P ? a.P - 1 : p);
            const double sc = wave_queue_exact(a, p, g);
            if ((threadIdx.x & (kWave - 1)) == 0) Q[k * a.I + g] = sc;
        }
    } else {
        for (int64_t k = blockIdx.x; k < n; k += gridDim.x) {
            int64_t p = cand[k];
            p = p < 0 ? 0 : (p >= a.P ? a.P - 1 : p);
            const double s = block_plan_exact(a, p, qpart);
            if (threadIdx.x == 0) X[p] = s;
        }
    }
}

// The candidate with the lowest exact score, the lowest index on ties; a NaN
// score never wins.  Plan scores are the queue sums added in queue order (or
// the whole-plan scores of k_gexact's second form).  No candidates: index -1,
// score +inf.
__global__ __launch_bounds__(256) void k_gpick(const int64_t *cand, const int32_t *ncand,
                                               int64_t cap, int I, const double *Q,
                                               const double *X, int64_t *out_i, double *out_s)
{
    __shared__ double ls[256 / kWave];
    __shared__ int64_t li[256 / kWave];
    const int64_t n = ncand ? (int64_t)ncand[0] : 0;
    double s = INFINITY;
    int64_t i = -1;
    // one wavefront per candidate: the lanes load its queue sums, which are
    // added in queue order
    const int lane = threadIdx.x & (kWave - 1);
    const int nw = blockDim.x / kWave;
    for (int64_t k = wave_id(); k < n; k += nw) {
        const int64_t p = cand[k];
        double t = 0.0;
        if (n <= cap) {
            for (int g0 = 0; g0 < I; g0 += kWave) {
                const double q = g0 + lane < I ? Q[k * I + g0 + lane] : 0.0;
                const int c = min(kWave, I - g0);
                for (int j = 0; j < c; ++j) t += lane_value(q, j);
            }
        } else {
            t = X[p];
        }
        const bool take = lane == 0 && t == t && (i < 0 || t < s || (t == s && p < i));
        s = take ? t : s;
        i = take ? p : i;
    }
    block_argmin(s, i, ls, li);
    if (threadIdx.x == 0) {
        *out_i = i;
        *out_s = i >= 0 ? s : INFINITY;
    }
}

// ---------------------------------------------------------------------------
// Validation

__global__ void k_zero_i64(int64_t *p)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) *p = 0;
}

// One workgroup per plan: a bitmap of seen group ids in LDS.
__global__ __launch_bounds__(256) void k_validate_plans(ExactArgs a, int64_t *n_invalid,
                                                       int32_t *status)
{
    extern __shared__ unsigned int seen[];
    __shared__ int s_bad;
    const int W = (a.G + 31) / 32;
    for (int64_t p = blockIdx.x; p < a.P; p += gridDim.x) {
        for (int w = threadIdx.x; w < W; w += blockDim.x) seen[w] = 0u;
        if (threadIdx.x == 0) s_bad = 0;
        __syncthreads();
        int bad = 0;
        for (int g = threadIdx.x; g <= a.I; g += blockDim.x) {
            const int32_t q = a.qoff[(int64_t)g * a.ld + p];
            if (g == 0 && q != 0) bad |= 1;
            if (g == a.I && q != a.G) bad |= 1;
            if (g < a.I && q > a.qoff[(int64_t)(g + 1) * a.ld + p]) bad |= 1;
            if (q < 0 || q > a.G) bad |= 1;
        }
        for (int s = threadIdx.x; s < a.G; s += blockDim.x) {
            const int32_t i = a.perm[(int64_t)s * a.ld + p];
            if (i < 0 || i >= a.G) {
                bad |= 2;
            } else {
                const unsigned int bit = 1u << (i & 31);
                if (atomicOr(&seen[i >> 5], bit) & bit) bad |= 2;
            }
        }
        if (a.evict && (a.G & 31)) {
            if (threadIdx.x == 0) {
                const uint32_t w = a.evict[(int64_t)(W - 1) * a.ld + p];
                if (w >> (a.G & 31)) bad |= 4;
            }
        }
        if (bad) atomicOr(&s_bad, bad);
        __syncthreads();
        if (threadIdx.x == 0) {
            if (status) status[p] = s_bad;
            if (s_bad) atomicAdd((unsigned long long *)n_invalid, 1ull);
        }
        __syncthreads();
    }
}

__global__ void k_validate_problem(ExactArgs a, int64_t *n_invalid)
{
    long long bad = 0;
    const int tid = blockIdx.x * blockDim.x + threadIdx.x;
    const int nth = gridDim.x * blockDim.x;
    for (int i = tid; i < a.G; i += nth) {
        const int32_t n = a.grp_count[i];
        const float var = a.grp_var[i];
        const int32_t m = a.grp_model[i];
        if (n < 0 || (uint32_t)n > kCountMask) ++bad;
        if (!(var >= 0.0f)) ++bad;
        if (m < 0 || m >= a.M) ++bad;
        if (!isfinite(a.grp_mu[i]) || !isfinite(var) || isnan(a.grp_slo[i])) ++bad;
    }
    for (int g = tid; g < a.I; g += nth) {
        const float t = a.inst_tput[g];
        if (!(t > 0.0f) || !isfinite(t)) ++bad;
        const int32_t c = a.inst_class[g];
        if (c < 0 || c >= a.C) ++bad;
        if (a.inst_model0) {
            const int32_t m0 = a.inst_model0[g];
            if (m0 < -1 || m0 >= a.M) ++bad;
        }
    }
    if (bad) atomicAdd((unsigned long long *)n_invalid, (unsigned long long)bad);
}

}  // namespace

// ---------------------------------------------------------------------------
// Host side

namespace qlm_internal {

thread_local std::string t_err;

int fail(int code, const std::string &msg)
{
    t_err = msg;
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(QLM_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

int check_problem(const qlm_problem *pr)
{
    if (!pr) return fail(QLM_ERR_ARG, "problem is NULL");
    if (pr->n_groups < 1 || pr->n_instances < 1 || pr->n_models < 1 || pr->n_classes < 1)
        return fail(QLM_ERR_ARG, "n_groups, n_instances, n_models and n_classes must be >= 1");
    if (pr->n_models > 255) return fail(QLM_ERR_ARG, "n_models must be <= 255");
    if (pr->n_groups > (1 << 24)) return fail(QLM_ERR_ARG, "n_groups too large");
    if (!pr->grp_count || !pr->grp_mu || !pr->grp_var || !pr->grp_model || !pr->grp_slo ||
        !pr->inst_tput || !pr->inst_class)
        return fail(QLM_ERR_ARG, "a required problem array is NULL");
    return QLM_OK;
}

int check_plans(const qlm_problem *pr, const qlm_plans *pl)
{
    if (!pl) return fail(QLM_ERR_ARG, "plans is NULL");
    if (pl->n_plans < 0) return fail(QLM_ERR_ARG, "n_plans must be >= 0");
    if (pl->plan_stride < pl->n_plans || pl->plan_stride < 1)
        return fail(QLM_ERR_ARG, "plan_stride must be >= max(n_plans, 1)");
    if (pl->plan_stride > kMaxPlanStride)
        return fail(QLM_ERR_ARG, "plan_stride must be <= 4194304");
    if (pl->n_plans > 0 && (!pl->perm || !pl->qoff))
        return fail(QLM_ERR_ARG, "perm and qoff are required");
    (void)pr;
    return QLM_OK;
}

// Launch timing (benchmarks only)
std::atomic<bool> g_timing{false};
std::mutex g_timing_mu;
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_events;

int timing_begin(hipStream_t stream, TimedLaunch *t)
{
    t->e0 = t->e1 = nullptr;
    if (!g_timing.load()) return QLM_OK;
    if (hipEventCreate(&t->e0) != hipSuccess || hipEventCreate(&t->e1) != hipSuccess)
        return fail(QLM_ERR_HIP, "hipEventCreate");
    (void)hipEventRecord(t->e0, stream);
    return QLM_OK;
}

void timing_end(hipStream_t stream, TimedLaunch *t)
{
    if (!t->e0) return;
    (void)hipEventRecord(t->e1, stream);
    std::lock_guard<std::mutex> lk(g_timing_mu);
    g_events.emplace_back(t->e0, t->e1);
}

}  // namespace qlm_internal

namespace {

using qlm_internal::check_plans;
using qlm_internal::check_problem;
using qlm_internal::fail;
using qlm_internal::hip_fail;

constexpr size_t kLdsLimit = 160 * 1024;   // gfx950 LDS per workgroup

// Dynamic LDS of the scoring kernel: everything but its static tail table.
constexpr size_t kScoreLdsLimit = kLdsLimit - sizeof(float) * 2 * kTailCells;

struct Geometry {
    int col_shift, ev_shift;
    uint32_t lut_bytes;
    size_t lds_bytes;         // dynamic LDS of the scoring kernel
};

int ceil_log2(uint32_t v)
{
    int s = 0;
    while ((1u << s) < v) ++s;
    return s;
}

Geometry geometry(int G, int I, int M, int C, bool evict)
{
    Geometry g;
    g.col_shift = ceil_log2((uint32_t)M);
    const uint32_t half = (uint32_t)(C * (M + 1)) << (g.col_shift + 3);   // bytes of one half
    // the twin at 8 KiB (where the fast path expects it) when a half fits there
    g.ev_shift = half <= (kTwinEntries << 3) ? kTwinShift + 3 : ceil_log2(half);
    const uint32_t bytes = evict ? (1u << g.ev_shift) + half : half;
    g.lut_bytes = (bytes + 15u) / 16u * 16u;
    // group table, cost table, instances, scratch
    g.lds_bytes = 16 * (size_t)(G + 1) + g.lut_bytes + 16 * (size_t)I + 128;
    return g;
}

ScoreArgs score_args(const qlm_problem *pr, const qlm_plans *pl, const Geometry &geo)
{
    ScoreArgs a{};
    a.G = pr->n_groups;
    a.I = pr->n_instances;
    a.M = pr->n_models;
    a.C = pr->n_classes;
    a.col_shift = geo.col_shift;
    a.ev_shift = geo.ev_shift;
    a.fast_ok = pr->n_models <= kCompactModels &&
                (pl->evict_bits == nullptr || geo.ev_shift == kTwinShift + 3);
    a.lut_bytes = geo.lut_bytes;
    a.grp_count = pr->grp_count;
    a.grp_mu = pr->grp_mu;
    a.grp_var = pr->grp_var;
    a.grp_slo = pr->grp_slo;
    a.grp_model = pr->grp_model;
    a.inst_tput = pr->inst_tput;
    a.inst_class = pr->inst_class;
    a.inst_model0 = pr->inst_model0;
    a.swap_cost = pr->swap_cost;
    a.evict_cost = pr->evict_cost;
    a.P = pl->n_plans;
    a.ld = pl->plan_stride;
    a.perm = pl->perm;
    a.qoff = pl->qoff;
    a.evict = pl->evict_bits;
    return a;
}

ExactArgs exact_args(const qlm_problem *pr, const qlm_plans *pl)
{
    ExactArgs a{};
    a.G = pr->n_groups;
    a.I = pr->n_instances;
    a.M = pr->n_models;
    a.C = pr->n_classes;
    a.grp_count = pr->grp_count;
    a.grp_mu = pr->grp_mu;
    a.grp_var = pr->grp_var;
    a.grp_slo = pr->grp_slo;
    a.grp_model = pr->grp_model;
    a.inst_tput = pr->inst_tput;
    a.inst_class = pr->inst_class;
    a.inst_model0 = pr->inst_model0;
    a.swap_cost = pr->swap_cost;
    a.evict_cost = pr->evict_cost;
    if (pl) {
        a.P = pl->n_plans;
        a.ld = pl->plan_stride;
        a.perm = pl->perm;
        a.qoff = pl->qoff;
        a.evict = pl->evict_bits;
    }
    return a;
}


using ScoreKernel = void (*)(ScoreArgs);

template <bool E, bool P, bool D>
ScoreKernel pick3() { return &k_score<E, P, D>; }

ScoreKernel pick_kernel(bool ev, bool pen, bool det)
{
    if (ev) {
        if (pen) return det ? pick3<true, true, true>() : pick3<true, true, false>();
        return det ? pick3<true, false, true>() : pick3<true, false, false>();
    }
    if (pen) return det ? pick3<false, true, true>() : pick3<false, true, false>();
    return det ? pick3<false, false, true>() : pick3<false, false, false>();
}

int device_cus(int *cus)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    e = hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    return QLM_OK;
}

struct OccKey {
    int dev;
    ScoreKernel k;
    size_t lds;
};
std::mutex g_occ_mu;
std::vector<std::pair<OccKey, std::pair<int, int>>> g_occ;   // -> (CUs, blocks per CU)

// CU count and resident workgroups per CU for kernel k with lds bytes, cached.
int occupancy(ScoreKernel k, size_t lds, int *cus, int *per_cu)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    {
        std::lock_guard<std::mutex> lk(g_occ_mu);
        for (auto &it : g_occ)
            if (it.first.dev == dev && it.first.k == k && it.first.lds == lds) {
                *cus = it.second.first;
                *per_cu = it.second.second;
                return QLM_OK;
            }
    }
    int rc = device_cus(cus);
    if (rc) return rc;
    e = hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return hip_fail(e, "hipFuncSetAttribute");
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, (const void *)k, kScoreThreads, lds);
    if (e != hipSuccess) return hip_fail(e, "hipOccupancyMaxActiveBlocksPerMultiprocessor");
    if (*per_cu < 1) *per_cu = 1;
    std::lock_guard<std::mutex> lk(g_occ_mu);
    g_occ.push_back({OccKey{dev, k, lds}, {*cus, *per_cu}});
    return QLM_OK;
}

// Slots where parts 1 .. n-1 of every plan start when each plan is split
// into n parts: multiples of 32, each part at least 64 slots.  A part after
// the first also rebuilds about one queue's running sums (w slots), so it is
// given that much less: the first part takes (G + (n - 1) w) / n slots.
// Returns false when no such split exists.
bool part_bounds(int G, int I, int n, int32_t *bound)
{
    const int w = G / I;
    const int first = (G + (n - 1) * w) / n;
    int prev = 0;
    for (int k = 1; k < n; ++k) {
        const int b = (first + (k - 1) * (first - w)) & ~31;
        if (b - prev < 64) return false;
        bound[k - 1] = b;
        prev = b;
    }
    return G - prev >= 64;
}

// Grid of the scoring kernel: persistent, at most as many workgroups as fit.
// When the tiles (64 plans each) fill at most a quarter (or half) of the
// wavefronts the chip holds at once, every tile is split between four (or
// two) wavefronts (part_bounds); four only where the queues are short against
// a part (a part's warm-up rebuilds one queue's sums).
int score_grid(ScoreKernel k, size_t lds, int64_t P, int G, int I, int *grid, int *nparts,
               int32_t *bound)
{
    int cus = 0, per_cu = 0;
    int rc = occupancy(k, lds, &cus, &per_cu);
    if (rc) return rc;
    const int wpb = kScoreThreads / kWave;
    const int64_t tiles = (P + kWave - 1) / kWave;
    const int64_t resident = (int64_t)per_cu * cus * wpb;
    int np = 1;
    if (G >= 512 && 8 * (G / I) <= G && 4 * tiles <= resident && part_bounds(G, I, 4, bound))
        np = 4;
    else if (G >= 256 && 2 * tiles <= resident && part_bounds(G, I, 2, bound))
        np = 2;
    for (int k = np - 1; k < 3; ++k) bound[k] = G;
    *nparts = np;
    const int per_round = wpb / np;
    const int64_t need = (tiles + per_round - 1) / per_round;
    int64_t g = (int64_t)per_cu * cus;
    if (g > need) g = need;
    if (g > kMaxScoreBlocks) g = kMaxScoreBlocks;
    if (g < 1) g = 1;
    *grid = (int)g;
    return QLM_OK;
}

int launch_score(const qlm_problem *pr, const qlm_plans *pl, double *score, double *penalty,
                 const qlm_detail *det, double *wg_min, double *wg_nsum, int32_t *ncand,
                 int *grid_out, hipStream_t stream, bool timed = true)
{
    const bool ev = pl->evict_bits != nullptr;
    const Geometry geo = geometry(pr->n_groups, pr->n_instances, pr->n_models, pr->n_classes, ev);
    if (geo.lds_bytes > kScoreLdsLimit)
        return fail(QLM_ERR_CAPACITY, "group, cost and instance tables need " +
                                          std::to_string(geo.lds_bytes) +
                                          " bytes of LDS; the limit is " +
                                          std::to_string(kScoreLdsLimit));
    ScoreArgs a = score_args(pr, pl, geo);
    a.score = score;
    a.penalty = penalty;
    a.wg_min = wg_min;
    a.wg_nsum = wg_nsum;
    a.ncand = ncand;
    if (det) {
        a.d_begin = det->plan_begin;
        a.d_count = det->plan_count;
        a.d_mean = det->wait_mean;
        a.d_sd = det->wait_sd;
        a.d_prob = det->prob;
    }
    const bool use_det = det && det->plan_count > 0 &&
                         (det->wait_mean || det->wait_sd || det->prob);
    ScoreKernel k = pick_kernel(ev, penalty != nullptr, use_det);
    int grid = 1;
    int rc = score_grid(k, geo.lds_bytes, pl->n_plans, pr->n_groups, pr->n_instances, &grid,
                        &a.nparts, a.bound);
    if (rc) return rc;
    if (grid_out) *grid_out = grid;

    qlm_internal::TimedLaunch tl{nullptr, nullptr};
    if (timed) {
        rc = qlm_internal::timing_begin(stream, &tl);
        if (rc) return rc;
    }
    hipLaunchKernelGGL(k, dim3(grid), dim3(kScoreThreads), geo.lds_bytes, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_score launch");
    if (timed) qlm_internal::timing_end(stream, &tl);
    return QLM_OK;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// qlm_best_plan's workspace before the per-(candidate, queue) sums: screened
// scores [P], per-workgroup minima, total requests and candidate count,
// candidates [P].
size_t best_plan_fixed_bytes(int64_t P)
{
    return align256(8 * (size_t)P) + align256(8 * (size_t)kMaxScoreBlocks) + 256 +
           align256(8 * (size_t)P);
}

int best_plan_impl(const qlm_problem *problem, const qlm_plans *plans, void *ws, size_t ws_bytes,
                   int64_t *best_index, double *best_score, hipStream_t stream, bool timed);

// Scratch of qlm_best_plan_static, for callers that cannot allocate: a
// file-scope device array (each GPU the library runs on holds its own copy
// until the process ends).  Host code never passes the array's name to a
// kernel or a copy: its device address comes from hipGetSymbolAddress, taken
// once per device with that device current and kept per device.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

std::mutex g_scratch_mu;
std::vector<void *> g_scratch_ptr;   // by device ordinal; null until taken

int static_scratch(void **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if ((size_t)dev >= g_scratch_ptr.size()) g_scratch_ptr.resize((size_t)dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(QLM_ERR_HIP, "hipGetSymbolAddress(scratch) gave no address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return QLM_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C interface

extern "C" {

int qlm_rwt_score(const qlm_problem *problem, const qlm_plans *plans, double *score,
                  double *penalty, const qlm_detail *detail, qlm_stream stream)
{
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    if (plans->n_plans == 0) return QLM_OK;
    if (!score) return fail(QLM_ERR_ARG, "score is NULL");
    if (detail) {
        if (detail->plan_begin < 0 || detail->plan_count < 0 ||
            detail->plan_begin + detail->plan_count > plans->n_plans)
            return fail(QLM_ERR_ARG, "detail plan range outside [0, n_plans)");
    }
    return launch_score(problem, plans, score, penalty, detail, nullptr, nullptr, nullptr, nullptr,
                        (hipStream_t)stream);
}

int qlm_rwt_score_exact(const qlm_problem *problem, const qlm_plans *plans,
                        const int64_t *plan_index, int64_t n, double *score, qlm_stream stream)
{
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    if (n < 0) return fail(QLM_ERR_ARG, "n must be >= 0");
    if (n == 0) return QLM_OK;
    if (!plan_index || !score) return fail(QLM_ERR_ARG, "plan_index and score are required");
    if (plans->n_plans == 0) return fail(QLM_ERR_ARG, "no plans to index");
    ExactArgs a = exact_args(problem, plans);
    const int grid = (int)(n < 65535 ? n : 65535);
    hipLaunchKernelGGL(k_exact, dim3(grid), dim3(kExactThreads), 0, (hipStream_t)stream, a,
                       plan_index, n, score);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_exact launch");
    return QLM_OK;
}

size_t qlm_best_plan_workspace_bytes(const qlm_problem *problem, int64_t n_plans)
{
    if (!problem || problem->n_instances < 1) return 0;
    if (n_plans < 0) n_plans = 0;
    const size_t I = (size_t)problem->n_instances;
    size_t rows = kCandSumBytes / (8 * I);
    if (rows < 256) rows = 256;
    if (rows > (size_t)n_plans) rows = (size_t)n_plans;
    return best_plan_fixed_bytes(n_plans) + align256(8 * rows * I);
}

int qlm_best_plan(const qlm_problem *problem, const qlm_plans *plans, void *ws, size_t ws_bytes,
                  int64_t *best_index, double *best_score, qlm_stream stream_)
{
    return best_plan_impl(problem, plans, ws, ws_bytes, best_index, best_score,
                          (hipStream_t)stream_, true);
}

int qlm_best_plan_static(const qlm_problem *problem, const qlm_plans *plans,
                         int64_t *best_index, double *best_score, qlm_stream stream_)
{
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    if (!best_index || !best_score) return fail(QLM_ERR_ARG, "best_index and best_score are required");
    const size_t need = qlm_best_plan_workspace_bytes(problem, plans->n_plans);
    if (need > kStaticScratchBytes)
        return fail(QLM_ERR_CAPACITY, "qlm_best_plan_static: " + std::to_string(plans->n_plans) +
                                          " plans need " + std::to_string(need) +
                                          " bytes of scratch; the static scratch holds " +
                                          std::to_string(kStaticScratchBytes));
    void *ws = nullptr;
    rc = static_scratch(&ws);
    if (rc) return rc;
    // the same workspace size qlm_best_plan is given for these plans, so that
    // both take the same path; no timing events are created
    return best_plan_impl(problem, plans, ws, need, best_index, best_score, (hipStream_t)stream_,
                          false);
}

}  // extern "C"

namespace {

int best_plan_impl(const qlm_problem *problem, const qlm_plans *plans, void *ws, size_t ws_bytes,
                   int64_t *best_index, double *best_score, hipStream_t stream, bool timed)
{
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    if (!best_index || !best_score) return fail(QLM_ERR_ARG, "best_index and best_score are required");
    const int64_t P = plans->n_plans;
    const int I = problem->n_instances;
    if (!ws || ((uintptr_t)ws & 255u))
        return fail(QLM_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    const size_t fixed = best_plan_fixed_bytes(P);
    if (ws_bytes < qlm_best_plan_workspace_bytes(problem, P))
        return fail(QLM_ERR_WORKSPACE, "workspace too small");
    hipError_t e;
    if (P == 0) {
        hipLaunchKernelGGL(k_gpick, dim3(1), dim3(256), 0, stream, nullptr, nullptr, (int64_t)0, I,
                           nullptr, nullptr, best_index, best_score);
        e = hipGetLastError();
        return e == hipSuccess ? QLM_OK : hip_fail(e, "k_gpick launch");
    }
    unsigned char *w = (unsigned char *)ws;
    double *fast = (double *)w;
    w += align256(8 * (size_t)P);
    double *wg_min = (double *)w;
    w += align256(8 * (size_t)kMaxScoreBlocks);
    double *nsum = (double *)w;
    int32_t *ncand = (int32_t *)(w + 128);
    w += 256;
    int64_t *cand = (int64_t *)w;
    w += align256(8 * (size_t)P);
    double *Q = (double *)w;
    // candidates whose per-queue sums fit in the rest of the workspace
    int64_t cap = (int64_t)((ws_bytes - fixed) / (8 * (size_t)I));
    if (cap > P) cap = P;
    int grid = 0;
    rc = launch_score(problem, plans, fast, nullptr, nullptr, wg_min, nsum, ncand, &grid, stream,
                      timed);
    if (rc) return rc;
    int sgrid = (int)((P + kSelThreads - 1) / kSelThreads);
    if (sgrid > kSelBlocks) sgrid = kSelBlocks;
    hipLaunchKernelGGL(k_gselect, dim3(sgrid), dim3(kSelThreads), 0, stream, fast, wg_min, grid,
                       nsum, P, cand, ncand);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_gselect launch");
    ExactArgs a = exact_args(problem, plans);
    hipLaunchKernelGGL(k_gexact, dim3(kGexBlocks), dim3(kGexThreads), 0, stream, a,
                       (const int64_t *)cand, (const int32_t *)ncand, cap, Q, fast);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_gexact launch");
    hipLaunchKernelGGL(k_gpick, dim3(1), dim3(256), 0, stream, (const int64_t *)cand,
                       (const int32_t *)ncand, cap, I, (const double *)Q, (const double *)fast,
                       best_index, best_score);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_gpick launch");
    return QLM_OK;
}

}  // namespace

extern "C" {

int qlm_validate_plans(const qlm_problem *problem, const qlm_plans *plans, int64_t *n_invalid,
                       int32_t *plan_status, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    if (!n_invalid) return fail(QLM_ERR_ARG, "n_invalid is NULL");
    hipLaunchKernelGGL(k_zero_i64, dim3(1), dim3(64), 0, stream, n_invalid);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_zero launch");
    if (plans->n_plans == 0) return QLM_OK;
    ExactArgs a = exact_args(problem, plans);
    const size_t lds = 4 * (size_t)((problem->n_groups + 31) / 32);
    if (lds > kLdsLimit) return fail(QLM_ERR_CAPACITY, "too many groups to validate");
    e = hipFuncSetAttribute((const void *)k_validate_plans,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return hip_fail(e, "hipFuncSetAttribute");
    const int grid = (int)(plans->n_plans < 8192 ? plans->n_plans : 8192);
    hipLaunchKernelGGL(k_validate_plans, dim3(grid), dim3(256), lds, stream, a, n_invalid,
                       plan_status);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_validate_plans launch");
    return QLM_OK;
}

int qlm_validate_problem(const qlm_problem *problem, int64_t *n_invalid, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    int rc = check_problem(problem);
    if (rc) return rc;
    if (!n_invalid) return fail(QLM_ERR_ARG, "n_invalid is NULL");
    hipLaunchKernelGGL(k_zero_i64, dim3(1), dim3(64), 0, stream, n_invalid);
    ExactArgs a = exact_args(problem, nullptr);
    const int n = problem->n_groups > problem->n_instances ? problem->n_groups : problem->n_instances;
    int grid = (n + 255) / 256;
    if (grid > 1024) grid = 1024;
    hipLaunchKernelGGL(k_validate_problem, dim3(grid), dim3(256), 0, stream, a, n_invalid);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_validate_problem launch");
    return QLM_OK;
}

int32_t qlm_max_groups(int32_t n_models, int32_t n_classes, int32_t n_instances,
                       int32_t with_eviction)
{
    if (n_models < 1 || n_models > 255 || n_classes < 1 || n_instances < 1) return 0;
    const Geometry g0 = geometry(0, n_instances, n_models, n_classes, with_eviction != 0);
    if (g0.lds_bytes > kScoreLdsLimit) return 0;
    return (int32_t)((kScoreLdsLimit - g0.lds_bytes) / 16);
}

int qlm_score_form(const qlm_problem *problem, int32_t with_eviction, int32_t *form,
                   qlm_stream stream)
{
    int rc = check_problem(problem);
    if (rc) return rc;
    if (!form) return fail(QLM_ERR_ARG, "form is NULL");
    const bool ev = with_eviction != 0;
    const Geometry geo = geometry(problem->n_groups, problem->n_instances, problem->n_models,
                                  problem->n_classes, ev);
    qlm_plans none{};
    none.evict_bits = ev ? reinterpret_cast<const uint32_t *>(form) : nullptr;   // only tested for NULL
    ScoreArgs a = score_args(problem, &none, geo);
    hipLaunchKernelGGL(k_score_form, dim3(1), dim3(1024), 0, (hipStream_t)stream, a, form);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_score_form launch");
    return QLM_OK;
}

const char *qlm_status_string(int status)
{
    switch (status) {
    case QLM_OK: return "ok";
    case QLM_ERR_ARG: return "invalid argument";
    case QLM_ERR_CAPACITY: return "tables exceed the LDS budget";
    case QLM_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case QLM_ERR_HIP: return "HIP error";
    default: return "unknown status";
    }
}

const char *qlm_last_error(void) { return qlm_internal::t_err.c_str(); }

int qlm_timing_enable(int on)
{
    qlm_internal::g_timing.store(on != 0);
    return QLM_OK;
}

int qlm_timing_read(int64_t *launches, double *total_ms)
{
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
    {
        std::lock_guard<std::mutex> lk(qlm_internal::g_timing_mu);
        ev.swap(qlm_internal::g_events);
    }
    double tot = 0.0;
    int rc = QLM_OK;
    for (auto &pr : ev) {
        hipError_t e = hipEventSynchronize(pr.second);
        float ms = 0.0f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, pr.first, pr.second);
        if (e != hipSuccess) rc = hip_fail(e, "timing event");
        tot += ms;
        (void)hipEventDestroy(pr.first);
        (void)hipEventDestroy(pr.second);
    }
    if (launches) *launches = (int64_t)ev.size();
    if (total_ms) *total_ms = tot;
    return rc;
}

}  // extern "C"
