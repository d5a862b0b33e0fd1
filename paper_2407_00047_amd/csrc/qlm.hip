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
//             group's 16-byte record with one ds_read_b128.  The violation
//             probability is a fused single-precision normal tail (Abramowitz &
//             Stegun 26.2.19); waits and variances accumulate in double.
//   k_refine  exact double-precision re-score (same definition as the oracle,
//             summed per queue then over queues) of every plan whose screened
//             score is within the screening error bound of the minimum.
//   k_final   lowest exact score, lowest index on ties.
//   k_exact   exact re-score of a list of plans (qlm_rwt_score_exact).
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

#include "qlm.h"

namespace {

constexpr int kWave = 64;
constexpr int kScoreThreads = 512;      // 8 wavefronts per workgroup
constexpr int kRefineThreads = 256;
constexpr int kMaxScoreBlocks = 4096;
constexpr int kRefineBlocks = 1024;
constexpr uint32_t kCountMask = 0xFFFFFFu;  // counts are 24-bit in the LDS record

// Screening error bound per slot of the single-precision probability: the
// approximation error of A&S 26.2.19 (1.5e-7) plus single-precision rounding of
// the standardised margin and of the evaluation (below 4e-6), with margin.
constexpr double kEpsP = 8e-6;

// A&S 26.2.19: Q(x) ~ 1/2 (1 + d1 x + ... + d6 x^6)^-16 for x >= 0, |error| <
// 1.5e-7.  Every coefficient is scaled by 2^(1/16) so that the sixteenth power
// carries the factor 2 and Q = 1 / y^16.
constexpr double kRoot16of2 = 1.0442737824274138403;
constexpr float kQ0 = (float)(kRoot16of2);
constexpr float kQ1 = (float)(kRoot16of2 * 0.0498673470);
constexpr float kQ2 = (float)(kRoot16of2 * 0.0211410061);
constexpr float kQ3 = (float)(kRoot16of2 * 0.0032776263);
constexpr float kQ4 = (float)(kRoot16of2 * 0.0000380036);
constexpr float kQ5 = (float)(kRoot16of2 * 0.0000488906);
constexpr float kQ6 = (float)(kRoot16of2 * 0.0000053830);

struct ScoreArgs {
    int32_t G, I, M, C;
    int32_t row_shift;        // log2(bytes per cost-table row)
    int32_t ev_shift;         // log2(bytes from a cost entry to its evicted twin)
    uint32_t lut_align;       // alignment of the cost table in LDS (power of two)
    uint32_t lut_region;      // bytes of the cost table (both halves)
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
    double *score, *penalty;
    int64_t d_begin, d_count;
    float *d_mean, *d_sd, *d_prob;
    double *wg_min;           // best_plan: per-workgroup minimum score, or null
    double *wg_nsum;          // best_plan: total requests (written by block 0)
};

__device__ inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// LDS layout of the scoring kernel (byte addresses; `base` = the dynamic LDS
// pointer):
//   group table   base, 16 (G + 1) bytes: group i -> {mu, var, slo, (n << 8) | model};
//                 entry G is an all-zero record (clamped out-of-range ids land there)
//   cost table    at `lut`, the first multiple of lut_align after the group table:
//                 byte (row << row_shift) | (col << 2) holds the seconds of swapping
//                 from model `row` to model `col` on class c, where row = c (M + 1) +
//                 previous model (previous model = M: none loaded; diagonal 0).  The
//                 twin at + (1 << ev_shift) adds the eviction cost.  Both shifts are
//                 powers of two and the table is aligned, so the address of a slot's
//                 cost is a bitwise OR of its row, its column and its eviction bit.
//   instances     theta (double) [I], class row base [I], head row [I] (LDS addresses)
//   scratch       8 doubles for workgroup reductions
struct Lds {
    uint32_t grp, lut, inst, red;
};

__device__ inline Lds lds_layout(const ScoreArgs &a, const unsigned char *base)
{
    Lds l;
    l.grp = (uint32_t)(uintptr_t)base;
    l.lut = (l.grp + 16u * (uint32_t)(a.G + 1) + a.lut_align - 1u) & ~(a.lut_align - 1u);
    l.inst = l.lut + a.lut_region;
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

__device__ void stage_tables(const ScoreArgs &a, const Lds &l)
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
            r.w = (n << 8) | m;
        }
        grp[i] = r;
    }
    float *lut = lds_ptr<float>(l.lut);
    const int Mp = 1 << (a.row_shift - 2);
    const int rows = a.M + 1;
    const int half_words = a.C * rows * Mp;
    const int twin_words = 1 << (a.ev_shift - 2);
    const int words = (int)(a.lut_region / 4u);
    for (int w = threadIdx.x; w < words; w += blockDim.x) {
        const int ev = w >= twin_words;
        const int k = ev ? w - twin_words : w;
        float v = 0.0f;
        if (k < half_words) {
            const int col = k % Mp;
            const int row = (k / Mp) % rows;
            const int c = k / (Mp * rows);
            if (a.swap_cost && row < a.M && col < a.M && row != col)
                v = a.swap_cost[((int64_t)c * a.M + row) * a.M + col];
            if (ev) v += a.evict_cost;
        }
        lut[w] = v;
    }
    double *theta = lds_ptr<double>(l.inst);
    uint32_t *cbase = reinterpret_cast<uint32_t *>(theta + a.I);
    uint32_t *head = cbase + a.I;
    for (int g = threadIdx.x; g < a.I; g += blockDim.x) {
        const int c = clampi(a.inst_class[g], 0, a.C - 1);
        const int m0 = a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
        theta[g] = (double)a.inst_tput[g];
        const uint32_t cb = l.lut + ((uint32_t)(c * rows) << a.row_shift);
        cbase[g] = cb;
        head[g] = cb + ((uint32_t)(m0 >= 0 ? m0 : a.M) << a.row_shift);
    }
}

__device__ inline double wave_min(double v)
{
    for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

// Screening score of every plan.  One lane = one plan; the slots of a plan are
// walked in order, so every prefix sum is a running sum.
template <bool EVICT, bool PEN, bool DETAIL>
__global__ __launch_bounds__(kScoreThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_score(ScoreArgs a)
{
    extern __shared__ __align__(16) unsigned char lds[];
    const Lds L = lds_layout(a, lds);
    stage_tables(a, L);
    double *red = lds_ptr<double>(L.red);
    if (a.wg_nsum && blockIdx.x == 0) {
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

    const double *s_theta = lds_ptr<double>(L.inst);
    const uint32_t *s_cbase = reinterpret_cast<const uint32_t *>(s_theta + a.I);
    const uint32_t *s_head = s_cbase + a.I;
    const uint32_t grp0 = L.grp;

    const int lane = threadIdx.x & (kWave - 1);
    // the wavefront index is uniform within a wavefront; say so, so that the
    // tile, its row addresses and the buffer resources live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int wpb = blockDim.x / kWave;
    const int64_t ntiles = (a.P + kWave - 1) / kWave;
    const int G = a.G;
    const int I1 = a.I - 1;
    const int64_t ld = a.ld;
    const int ev_shift = a.ev_shift;
    const int row_shift = a.row_shift;
    double lane_min = INFINITY;

    for (int64_t t = (int64_t)blockIdx.x * wpb + wave; t < ntiles; t += (int64_t)gridDim.x * wpb) {
        const int64_t tb = t * kWave;               // first plan of the tile (uniform)
        const bool live = tb + lane < a.P;
        const int lp = live ? lane : (int)(a.P - 1 - tb);   // lane's plan, relative to tb
        const uint32_t lpb = (uint32_t)lp * 4u;     // its byte offset within a row
        const int32_t *qrow = a.qoff + tb;
        const int64_t p = tb + lp;
        const bool det = DETAIL && live && p >= a.d_begin && p < a.d_begin + a.d_count;
        const int64_t dq = p - a.d_begin;
        // Row r of a slot-major array, lane's column: a plain global load (used
        // for the queue offsets, once per block), and buffer loads from a
        // resource based at a block's first row (group ids, eviction words),
        // whose row offset is a scalar operand: no per-load vector arithmetic.
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
        auto ld_rel = [&](__amdgpu_buffer_rsrc_t r, int rel_row) __attribute__((always_inline)) {
            return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)lpb, rel_row * (int)ld4, 0);
        };

        double Y = 0.0;        // tokens ahead + theta * (swap and eviction seconds so far)
        double V = 0.0;        // variance of the tokens ahead
        double S = 0.0;        // sum of n * P
        double PE = 0.0;       // sum of (E[W] - slo)
        double theta = 1.0, inv_theta = 1.0;
        uint32_t cbase = 0, rowb = 0;
        // Queue bookkeeping.  g is the queue of the current slot and nb the slot
        // where the next queue starts.  Parameters of upcoming queues reach a
        // queue head through a two-stage prefetch, so that a head never waits for
        // a load younger than one block (32 slots):
        //   f1, f2   queues q0+1 and q0+2, q0 = g at the start of the previous
        //            block; loaded at that start
        //   x_*      the next queue's parameters for the current block, chosen at
        //            its start from f1 or f2 by how many queues the previous block
        //            entered (two or more: not available, `need`)
        struct QP {
            int nb;               // end boundary of the queue
            double theta;
            uint32_t cbase, head;
        };
        int g = -1, nb = 0;
        QP x{0, 1.0, 0u, 0u}, f1{0, 1.0, 0u, 0u}, f2{0, 1.0, 0u, 0u};
        int q0 = -1;
        bool need = true;             // x belongs to a queue already entered

        // Issued for every lane, never under a per-lane condition (clamped
        // index), so that the compiler counts the outstanding loads exactly.
        auto load_qp = [&](int h) __attribute__((always_inline)) {
            h = min(max(h, 0), I1);
            QP q;
            q.nb = (int)at(a.qoff, h + 1);
            q.theta = s_theta[h];
            q.cbase = s_cbase[h];
            q.head = s_head[h];
            return q;
        };
        auto block_start = [&]() __attribute__((always_inline)) {
            const int c = g - q0;     // queues entered since the previous start
            x.nb = c == 0 ? f1.nb : f2.nb;
            x.theta = c == 0 ? f1.theta : f2.theta;
            x.cbase = c == 0 ? f1.cbase : f2.cbase;
            x.head = c == 0 ? f1.head : f2.head;
            need = c > 1;
            q0 = g;
            __builtin_amdgcn_sched_barrier(0);        // select before the reload
            f1 = load_qp(g + 1);
            f2 = load_qp(g + 2);
        };

        // Enter the queue that owns slot s (called when s == nb).  The common
        // case uses x_*, fetched at the start of the block; a second head in one
        // block, or an empty queue, loads what it needs and waits for it on the
        // spot, so that no wait on the common path covers a load issued after
        // the block's group-id refills.
        auto enter = [&](int s) __attribute__((always_inline)) {
            int e_nb;
            double e_theta;
            uint32_t e_cbase, e_head;
            if (!need) {
                e_nb = x.nb;
                e_theta = x.theta;
                e_cbase = x.cbase;
                e_head = x.head;
            } else {
                const int h = g + 1;
                e_nb = (int)at(a.qoff, h + 1);
                e_theta = s_theta[h];
                e_cbase = s_cbase[h];
                e_head = s_head[h];
                __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0)
            }
            ++g;
            nb = e_nb;
            theta = e_theta;
            cbase = e_cbase;
            rowb = e_head;
            need = true;
            while (nb <= s && g < I1) {   // empty queues: skip them (rare)
                const int h = g + 1;
                nb = (int)at(a.qoff, h + 1);
                theta = s_theta[h];
                cbase = s_cbase[h];
                rowb = s_head[h];
                __builtin_amdgcn_s_waitcnt(0x0070);
                ++g;
            }
            if (g >= I1) nb = INT_MAX;    // last queue: no further head
            inv_theta = 1.0 / theta;
            Y = 0.0;
            V = 0.0;
        };

        // Software pipeline over the slots of the plan:
        //   ring[32]  group ids of the next 32 slots (global loads, 32 slots ahead)
        //   rec[4]    LDS records of slots s..s+3 (gathered 4 slots ahead)
        //   cost      swap/eviction seconds of slot s (looked up one slot ahead)
        // Slot s: (A) waits and variances with its cost, (B) resolve whether s+1
        // starts a queue and look up the cost of s+1, (C) the normal tail of s,
        // which overlaps that lookup.
        constexpr int D = 3;          // records gathered D slots ahead
        int32_t ring[32];
        uint4 rec[4];                 // rec[s % 4] holds slot s's record
        __amdgpu_buffer_rsrc_t rp = rsrc_at(a.perm, 0);
#pragma unroll
        for (int k = 0; k < 32; ++k) ring[k] = (int32_t)ld_rel(rp, min(k, G - 1));
        auto gather = [&](int32_t gid) __attribute__((always_inline)) {
            return *lds_ptr<const uint4>((min((uint32_t)gid, (uint32_t)G) << 4) + grp0);
        };
        // prologue: records of slots 0..D-1 (their ring entries refilled with
        // slots 32..32+D-1), the head of slot 0 and its cost
#pragma unroll
        for (int k = 0; k < D; ++k) {
            rec[k] = gather(ring[k]);
            ring[k] = (int32_t)ld_rel(rp, min(k + 32, G - 1));
        }
        rec[D] = rec[0];
        uint32_t ev = EVICT ? ld_rel(rsrc_at(a.evict, 0), 0) : 0u;   // word of the block
        uint32_t ev_nx = 0u;                              // word of the next block
        // prefetch relative to q0 = -1 (queues 0 and 1), issued before enter(0),
        // whose full wait leaves no load of the prologue pending at the loop
        q0 = -1;
        f1 = load_qp(0);
        f2 = load_qp(1);
        enter(0);                     // need: loads and waits (once per tile)
        float cost = *lds_ptr<const float>(rowb | ((rec[0].w & 0xFFu) << 2) |
                                           (EVICT ? (ev & 1u) << ev_shift : 0u));

        // Full 32-slot blocks: no per-slot guard, so every refill is unconditional
        // and the compiler's counting of outstanding loads stays exact.
        const int G32 = G & ~31;
        const int Gx = __builtin_amdgcn_readfirstlane(G);
        for (int sb = 0; sb < G32; sb += 32) {
            block_start();
            if (EVICT) ev_nx = ld_rel(rsrc_at(a.evict, min((sb >> 5) + 1, (G - 1) >> 5)), 0);
            rp = rsrc_at(a.perm, sb);
#pragma unroll
            for (int k = 0; k < 32; ++k) {
                const int s = sb + k;
                // ring entry of slot s+D: turned into its LDS address, then refilled
                // with slot s+D+32 (unconditionally: rows past the end clamp to the
                // last row), so both share one register and every wait on the ring
                // counts loads exactly
                const int j = (k + D) & 31;
                rec[(k + D) & 3] = gather(ring[j]);   // record of slot s+D
                __builtin_amdgcn_sched_barrier(0);    // consume before the refill
                ring[j] = (int32_t)ld_rel(rp, min(s + D + 32, G - 1) - sb);
                // always true here; an opaque bound keeps each slot a region of its
                // own, which keeps the record pipeline in fixed registers
                if (s >= Gx) continue;
                const uint4 r = rec[k & 3];
                const float mu = __uint_as_float(r.x);
                const float var = __uint_as_float(r.y);
                const float slo = __uint_as_float(r.z);
                const uint32_t m = r.w & 0xFFu;
                const double n = (double)(r.w >> 8);

                // (A) waits of slot s
                Y = fma((double)cost, theta, Y);                  // its swap / eviction
                const double num = fma((double)slo, theta, -Y);   // theta (slo - E[W])
                const float rs = __builtin_amdgcn_rsqf((float)V); // 1/sqrt(V); inf if V = 0
                // |z|; a zero margin with zero variance gives +inf (no violation)
                const float x = fmaxf(fabsf((float)num), 1e-38f) * rs;
                if (PEN) PE = fma(-num, inv_theta, PE);
                if (DETAIL && det) {
                    const int64_t o = (int64_t)s * a.d_count + dq;
                    if (a.d_mean) a.d_mean[o] = (float)(Y * inv_theta);
                    if (a.d_sd) a.d_sd[o] = (float)(sqrt(V) * inv_theta);
                }
                Y = fma(n, (double)mu, Y);
                V = fma(n, (double)var, V);
                rowb = cbase + (m << row_shift);

                // (B) queue head at s+1?  Then the cost of slot s+1
                if (s + 1 == nb) enter(s + 1);
                {
                    const uint32_t m1 = rec[(k + 1) & 3].w & 0xFFu;
                    uint32_t idx = rowb | (m1 << 2);
                    if (EVICT) {
                        const uint32_t w = k == 31 ? ev_nx : ev;
                        idx |= __builtin_amdgcn_ubfe(w, (uint32_t)((k + 1) & 31), 1u) << ev_shift;
                    }
                    cost = *lds_ptr<const float>(idx);
                }

                // (C) normal tail of slot s (A&S 26.2.19)
                float y = fmaf(x, kQ6, kQ5);
                y = fmaf(y, x, kQ4);
                y = fmaf(y, x, kQ3);
                y = fmaf(y, x, kQ2);
                y = fmaf(y, x, kQ1);
                y = fmaf(y, x, kQ0);
                y = y * y;
                y = y * y;
                y = y * y;
                y = y * y;
                const float q = __builtin_amdgcn_rcpf(y);         // Q(|z|)
                const float prob = num < 0.0 ? 1.0f - q : q;
                S = fma(n, (double)prob, S);
                if (DETAIL && det && a.d_prob) a.d_prob[(int64_t)s * a.d_count + dq] = prob;
            }
            if (EVICT) ev = ev_nx;
        }
        // Remaining G % 32 slots, one at a time (plain loads; small G only).  The
        // pipeline has already resolved the head and the cost of slot G32.
        for (int s = G32; s < G; ++s) {
            const uint4 r = gather((int32_t)at(a.perm, s));
            const uint32_t m = r.w & 0xFFu;
            if (s > G32) {
                if (s == nb) enter(s);
                uint32_t idx = rowb | (m << 2);
                if (EVICT) idx |= __builtin_amdgcn_ubfe(ev, (uint32_t)(s & 31), 1u) << ev_shift;
                cost = *lds_ptr<const float>(idx);
            }
            const float mu = __uint_as_float(r.x);
            const float var = __uint_as_float(r.y);
            const float slo = __uint_as_float(r.z);
            const double n = (double)(r.w >> 8);
            Y = fma((double)cost, theta, Y);
            const double num = fma((double)slo, theta, -Y);
            const float rs = __builtin_amdgcn_rsqf((float)V);
            const float x = fmaxf(fabsf((float)num), 1e-38f) * rs;
            if (PEN) PE = fma(-num, inv_theta, PE);
            if (DETAIL && det) {
                const int64_t o = (int64_t)s * a.d_count + dq;
                if (a.d_mean) a.d_mean[o] = (float)(Y * inv_theta);
                if (a.d_sd) a.d_sd[o] = (float)(sqrt(V) * inv_theta);
            }
            Y = fma(n, (double)mu, Y);
            V = fma(n, (double)var, V);
            rowb = cbase + (m << row_shift);
            float y = fmaf(x, kQ6, kQ5);
            y = fmaf(y, x, kQ4);
            y = fmaf(y, x, kQ3);
            y = fmaf(y, x, kQ2);
            y = fmaf(y, x, kQ1);
            y = fmaf(y, x, kQ0);
            y = y * y;
            y = y * y;
            y = y * y;
            y = y * y;
            const float q = __builtin_amdgcn_rcpf(y);
            const float prob = num < 0.0 ? 1.0f - q : q;
            S = fma(n, (double)prob, S);
            if (DETAIL && det && a.d_prob) a.d_prob[(int64_t)s * a.d_count + dq] = prob;
        }
        if (live) {
            a.score[p] = S;
            if (PEN) a.penalty[p] = PE;
            lane_min = fmin(lane_min, S);
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
__device__ double exact_queue(const ExactArgs &a, int64_t p, int g)
{
    int32_t b = a.qoff[(int64_t)g * a.ld + p];
    int32_t e = a.qoff[(int64_t)(g + 1) * a.ld + p];
    b = clampi(b, 0, a.G);
    e = clampi(e, b, a.G);
    const double theta = (double)a.inst_tput[g];
    const int cls = clampi(a.inst_class[g], 0, a.C - 1);
    int m_prev = a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
    double A = 0.0, V = 0.0, K = 0.0, sc = 0.0;
    for (int s = b; s < e; ++s) {
        const int i = (int)min((uint32_t)a.perm[(int64_t)s * a.ld + p], (uint32_t)(a.G - 1));
        const int m = clampi(a.grp_model[i], 0, a.M - 1);
        const double n = (double)(uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
        const double mu = (double)a.grp_mu[i];
        const double var = (double)a.grp_var[i];
        const double slo = (double)a.grp_slo[i];
        if (m_prev >= 0 && m_prev != m && a.swap_cost)
            K += (double)a.swap_cost[((int64_t)cls * a.M + m_prev) * a.M + m];
        if (a.evict && ((a.evict[(int64_t)(s >> 5) * a.ld + p] >> (s & 31)) & 1u))
            K += (double)a.evict_cost;
        const double EW = A / theta + K;
        const double SD = sqrt(V) / theta;
        double P;
        if (SD > 0.0)
            P = 0.5 * erfc((slo - EW) / (SD * 1.4142135623730951));
        else
            P = (EW > slo) ? 1.0 : 0.0;
        sc += n * P;
        A += n * mu;
        V += n * var;
        m_prev = m;
    }
    return sc;
}

// Exact score of plan p by a whole workgroup, serial per queue (threads take
// queues, thread 0 adds the per-queue sums in queue order).  Used when the
// slot-parallel form below does not fit in LDS.
__device__ double exact_plan_serial(const ExactArgs &a, int64_t p, double *part)
{
    double total = 0.0;
    for (int g0 = 0; g0 < a.I; g0 += blockDim.x) {
        const int g = g0 + threadIdx.x;
        if (g < a.I) part[threadIdx.x] = exact_queue(a, p, g);
        __syncthreads();
        if (threadIdx.x == 0) {
            const int n = min((int)blockDim.x, a.I - g0);
            for (int k = 0; k < n; ++k) total += part[k];
        }
        __syncthreads();
    }
    return total;   // valid in thread 0
}

// The same exact score, slot-parallel, with the same arithmetic and the same
// summation order.  Inputs are first gathered into LDS by independent loads
// (no chains of dependent global loads):
//   0. every thread takes slots: a = n mu and b = n var (exact products) and
//      the model of the slot's group; the eviction words; the swap table
//   1. per queue (one thread each), the running sums in position order give
//      every slot's E[W] = A/Theta + K and SD = sqrt(V)/Theta (in place of a, b)
//   2. every thread takes slots: P and the term n P (in place of E[W])
//   3. per queue, the terms are added in position order; thread 0 adds the
//      queue sums in queue order.
struct ExactLds {
    double *x, *y;            // [G] each
    uint32_t *evw;            // [ceil(G/32)]
    float *swap;              // [C M M] or null (then read from global memory)
    unsigned char *mdl;       // [G]
};

__device__ double exact_plan(const ExactArgs &a, int64_t p, const ExactLds &L, double *part)
{
    const int G = a.G;
    const int W = (G + 31) >> 5;
    const int64_t ld = a.ld;
    // 0. gather (8 independent slots per thread per step)
    for (int s0 = threadIdx.x; s0 < G; s0 += 8 * blockDim.x) {
        int i[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int s = s0 + u * blockDim.x;
            i[u] = s < G ? (int)min((uint32_t)a.perm[(int64_t)s * ld + p], (uint32_t)(G - 1)) : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int s = s0 + u * blockDim.x;
            if (s < G) {
                const double n = (double)(uint32_t)clampi(a.grp_count[i[u]], 0, (int)kCountMask);
                L.x[s] = n * (double)a.grp_mu[i[u]];
                L.y[s] = n * (double)a.grp_var[i[u]];
                L.mdl[s] = (unsigned char)clampi(a.grp_model[i[u]], 0, a.M - 1);
            }
        }
    }
    for (int w = threadIdx.x; w < W; w += blockDim.x)
        L.evw[w] = a.evict ? a.evict[(int64_t)w * ld + p] : 0u;
    if (L.swap && a.swap_cost)
        for (int k = threadIdx.x; k < a.C * a.M * a.M; k += blockDim.x) L.swap[k] = a.swap_cost[k];
    __syncthreads();
    // 1. running sums per queue
    for (int g = threadIdx.x; g < a.I; g += blockDim.x) {
        const int32_t b = clampi(a.qoff[(int64_t)g * ld + p], 0, G);
        const int32_t e = clampi(a.qoff[(int64_t)(g + 1) * ld + p], b, G);
        const double theta = (double)a.inst_tput[g];
        const int cls = clampi(a.inst_class[g], 0, a.C - 1);
        int m_prev = a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
        const double ecost = (double)a.evict_cost;
        double A = 0.0, V = 0.0, K = 0.0;
        for (int s = b; s < e; ++s) {
            const int m = L.mdl[s];
            if (m_prev >= 0 && m_prev != m && a.swap_cost) {
                const int64_t k = ((int64_t)cls * a.M + m_prev) * a.M + m;
                K += (double)(L.swap ? L.swap[k] : a.swap_cost[k]);
            }
            if ((L.evw[s >> 5] >> (s & 31)) & 1u) K += ecost;
            const double xa = L.x[s], yb = L.y[s];
            L.x[s] = A / theta + K;            // E[W]
            L.y[s] = sqrt(V) / theta;          // SD[W]
            A += xa;
            V += yb;
            m_prev = m;
        }
    }
    __syncthreads();
    // 2. probability and term per slot
    for (int s0 = threadIdx.x; s0 < G; s0 += 8 * blockDim.x) {
        int i[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int s = s0 + u * blockDim.x;
            i[u] = s < G ? (int)min((uint32_t)a.perm[(int64_t)s * ld + p], (uint32_t)(G - 1)) : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int s = s0 + u * blockDim.x;
            if (s < G) {
                const double n = (double)(uint32_t)clampi(a.grp_count[i[u]], 0, (int)kCountMask);
                const double slo = (double)a.grp_slo[i[u]];
                const double EW = L.x[s], SD = L.y[s];
                double P;
                if (SD > 0.0)
                    P = 0.5 * erfc((slo - EW) / (SD * 1.4142135623730951));
                else
                    P = (EW > slo) ? 1.0 : 0.0;
                L.x[s] = n * P;
            }
        }
    }
    __syncthreads();
    // 3. sums per queue, then over queues
    double total = 0.0;
    for (int g0 = 0; g0 < a.I; g0 += blockDim.x) {
        const int g = g0 + threadIdx.x;
        if (g < a.I) {
            const int32_t b = clampi(a.qoff[(int64_t)g * ld + p], 0, G);
            const int32_t e = clampi(a.qoff[(int64_t)(g + 1) * ld + p], b, G);
            double sc = 0.0;
            for (int s = b; s < e; ++s) sc += L.x[s];
            part[threadIdx.x] = sc;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            const int n = min((int)blockDim.x, a.I - g0);
            for (int k = 0; k < n; ++k) total += part[k];
        }
        __syncthreads();
    }
    return total;   // valid in thread 0
}

// Exact score with whichever form fits: `big` = 1 the kernel got the LDS of
// the staged form, 2 the same plus room for the swap table.
__device__ double exact_score(const ExactArgs &a, int64_t p, unsigned char *dyn, int big,
                              double *part)
{
    if (big) {
        ExactLds L;
        L.x = reinterpret_cast<double *>(dyn);
        L.y = L.x + a.G;
        L.evw = reinterpret_cast<uint32_t *>(L.y + a.G);
        float *after = reinterpret_cast<float *>(L.evw + ((a.G + 31) >> 5));
        L.swap = big == 2 ? after : nullptr;
        L.mdl = reinterpret_cast<unsigned char *>(after + (big == 2 ? a.C * a.M * a.M : 0));
        return exact_plan(a, p, L, part);
    }
    return exact_plan_serial(a, p, part);
}
#pragma clang fp contract(on)

__global__ __launch_bounds__(kRefineThreads) void k_exact(ExactArgs a, const int64_t *idx,
                                                          int64_t n, double *out, int big)
{
    extern __shared__ __align__(16) unsigned char dyn[];
    __shared__ double part[kRefineThreads];
    for (int64_t k = blockIdx.x; k < n; k += gridDim.x) {
        int64_t p = idx[k];
        const bool ok = p >= 0 && p < a.P;
        p = ok ? p : 0;
        const double s = exact_score(a, p, dyn, big, part);
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

// Candidate selection and exact re-score.  Every workgroup first reduces the
// per-workgroup minima of the screening scores, then walks its own contiguous
// range of plans in index order and re-scores exactly every plan whose
// screening score is within twice the screening error bound of the minimum
// (the exact minimum is always among them).
__global__ __launch_bounds__(kRefineThreads) void k_refine(ExactArgs a, const double *fast,
                                                           const double *wg_min, int n_wg,
                                                           const double *nsum,
                                                           double *best_s, int64_t *best_i,
                                                           int big)
{
    extern __shared__ __align__(16) unsigned char dyn[];
    __shared__ double part[kRefineThreads];
    __shared__ double ls[kRefineThreads / kWave];
    __shared__ int64_t li[kRefineThreads / kWave];
    double m = INFINITY;
    for (int k = threadIdx.x; k < n_wg; k += blockDim.x) m = fmin(m, wg_min[k]);
    m = block_min(m, ls);
    // |screened - exact| <= eps * (total requests), plus the rounding of both sums
    const double delta = kEpsP * (*nsum) * (1.0 + 1e-9) + 1e-300;
    const double thr = m + 2.0 * delta;

    const int64_t per = (a.P + gridDim.x - 1) / gridDim.x;
    const int64_t lo = (int64_t)blockIdx.x * per;
    const int64_t hi = min(a.P, lo + per);
    double bs = INFINITY;
    int64_t bi = -1;
    for (int64_t base = lo; base < hi; base += blockDim.x) {
        const int64_t p = base + threadIdx.x;
        const bool cand = p < hi && fast[p] <= thr;
        if (!__syncthreads_or(cand)) continue;
        // candidates of this chunk, one at a time in index order
        int64_t next = cand ? p : INT64_MAX;
        while (true) {
            int64_t q = next;
            // lowest remaining candidate index in the block
            for (int o = 32; o > 0; o >>= 1) {
                const int64_t q2 = __shfl_xor(q, o, kWave);
                q = q2 < q ? q2 : q;
            }
            __syncthreads();
            if ((threadIdx.x & (kWave - 1)) == 0) li[threadIdx.x / kWave] = q;
            __syncthreads();
            q = INT64_MAX;
            for (int w = 0; w < (int)(blockDim.x / kWave); ++w) q = li[w] < q ? li[w] : q;
            __syncthreads();
            if (q == INT64_MAX) break;
            const double e = exact_score(a, q, dyn, big, part);
            if (threadIdx.x == 0 && e < bs) {     // ascending index: the first minimum wins
                bs = e;
                bi = q;
            }
            if (next == q) next = INT64_MAX;
        }
    }
    if (threadIdx.x == 0) {
        best_s[blockIdx.x] = bs;
        best_i[blockIdx.x] = bi;
    }
}

__global__ __launch_bounds__(256) void k_final(const double *best_s, const int64_t *best_i, int n,
                                               int64_t *out_i, double *out_s)
{
    __shared__ double ls[256 / kWave];
    __shared__ int64_t li[256 / kWave];
    double s = INFINITY;
    int64_t i = -1;
    for (int k = threadIdx.x; k < n; k += blockDim.x) {
        const double s2 = best_s[k];
        const int64_t i2 = best_i[k];
        const bool take = i2 >= 0 && (i < 0 || s2 < s || (s2 == s && i2 < i));
        s = take ? s2 : s;
        i = take ? i2 : i;
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

// ---------------------------------------------------------------------------
// Host side

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

constexpr size_t kLdsLimit = 160 * 1024;   // gfx950 LDS per workgroup

struct Geometry {
    int row_shift, ev_shift;
    uint32_t lut_align, lut_region;
    size_t lds_bytes;
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
    const uint32_t Mp = 1u << ceil_log2((uint32_t)M);
    g.row_shift = ceil_log2(Mp) + 2;
    const uint32_t half = (uint32_t)(C * (M + 1)) << g.row_shift;   // bytes of one half
    g.ev_shift = ceil_log2(half < 16u ? 16u : half);
    if (evict) {
        g.lut_region = 2u << g.ev_shift;
        g.lut_align = 2u << g.ev_shift;
    } else {
        g.lut_region = (half + 15u) / 16u * 16u;
        g.lut_align = (1u << g.row_shift) < 16u ? 16u : (1u << g.row_shift);
    }
    // group table, worst-case alignment padding, cost table, instances, scratch
    g.lds_bytes = 16 * (size_t)(G + 1) + (g.lut_align - 1) + g.lut_region + 16 * (size_t)I + 64;
    g.lds_bytes = (g.lds_bytes + 15) / 16 * 16;
    return g;
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
    if (pl->n_plans > 0 && (!pl->perm || !pl->qoff))
        return fail(QLM_ERR_ARG, "perm and qoff are required");
    (void)pr;
    return QLM_OK;
}

ScoreArgs score_args(const qlm_problem *pr, const qlm_plans *pl, const Geometry &geo)
{
    ScoreArgs a{};
    a.G = pr->n_groups;
    a.I = pr->n_instances;
    a.M = pr->n_models;
    a.C = pr->n_classes;
    a.row_shift = geo.row_shift;
    a.ev_shift = geo.ev_shift;
    a.lut_align = geo.lut_align;
    a.lut_region = geo.lut_region;
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

// Launch timing (benchmarks only)
std::atomic<bool> g_timing{false};
std::mutex g_timing_mu;
std::vector<std::pair<hipEvent_t, hipEvent_t>> g_events;

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

// Grid of the scoring kernel: persistent, at most as many workgroups as fit.
int score_grid(ScoreKernel k, size_t lds, int64_t P, int *grid)
{
    int cus = 0, per_cu = 0;
    int rc = occupancy(k, lds, &cus, &per_cu);
    if (rc) return rc;
    const int64_t tiles = (P + kWave - 1) / kWave;
    const int64_t need = (tiles + kScoreThreads / kWave - 1) / (kScoreThreads / kWave);
    int64_t g = (int64_t)per_cu * cus;
    if (g > need) g = need;
    if (g > kMaxScoreBlocks) g = kMaxScoreBlocks;
    if (g < 1) g = 1;
    *grid = (int)g;
    return QLM_OK;
}

int launch_score(const qlm_problem *pr, const qlm_plans *pl, double *score, double *penalty,
                 const qlm_detail *det, double *wg_min, double *wg_nsum, int *grid_out,
                 hipStream_t stream)
{
    const bool ev = pl->evict_bits != nullptr;
    const Geometry geo = geometry(pr->n_groups, pr->n_instances, pr->n_models, pr->n_classes, ev);
    if (geo.lds_bytes > kLdsLimit)
        return fail(QLM_ERR_CAPACITY, "group, cost and instance tables need " +
                                          std::to_string(geo.lds_bytes) +
                                          " bytes of LDS; the limit is 163840");
    ScoreArgs a = score_args(pr, pl, geo);
    a.score = score;
    a.penalty = penalty;
    a.wg_min = wg_min;
    a.wg_nsum = wg_nsum;
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
    int rc = score_grid(k, geo.lds_bytes, pl->n_plans, &grid);
    if (rc) return rc;
    if (grid_out) *grid_out = grid;

    hipEvent_t e0 = nullptr, e1 = nullptr;
    const bool timing = g_timing.load();
    if (timing) {
        if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess)
            return fail(QLM_ERR_HIP, "hipEventCreate");
        (void)hipEventRecord(e0, stream);
    }
    hipLaunchKernelGGL(k, dim3(grid), dim3(kScoreThreads), geo.lds_bytes, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_score launch");
    if (timing) {
        (void)hipEventRecord(e1, stream);
        std::lock_guard<std::mutex> lk(g_timing_mu);
        g_events.emplace_back(e0, e1);
    }
    return QLM_OK;
}

// Dynamic LDS of the exact re-score: the staged form when it fits (with the
// swap table when that fits too), else none (serial form).
int exact_lds(const void *kernel, const qlm_problem *pr, size_t *lds, int *big)
{
    const size_t G = (size_t)pr->n_groups;
    const size_t base = 16 * G + 4 * ((G + 31) / 32) + G;
    const size_t swap = 4 * (size_t)pr->n_classes * pr->n_models * pr->n_models;
    const size_t static_lds = 8 * (size_t)kRefineThreads + 256;
    size_t want = (base + 15) / 16 * 16;
    int kind = 1;
    if (pr->swap_cost && ((base + swap + 15) / 16 * 16) + static_lds <= kLdsLimit) {
        want = (base + swap + 15) / 16 * 16;
        kind = 2;
    }
    if (want + static_lds <= kLdsLimit) {
        hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)want);
        if (e != hipSuccess) return hip_fail(e, "hipFuncSetAttribute");
        *lds = want;
        *big = kind;
    } else {
        *lds = 0;
        *big = 0;
    }
    return QLM_OK;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

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
    return launch_score(problem, plans, score, penalty, detail, nullptr, nullptr, nullptr,
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
    size_t lds = 0;
    int big = 0;
    rc = exact_lds((const void *)k_exact, problem, &lds, &big);
    if (rc) return rc;
    hipLaunchKernelGGL(k_exact, dim3(grid), dim3(kRefineThreads), lds, (hipStream_t)stream, a,
                       plan_index, n, score, big);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_exact launch");
    return QLM_OK;
}

size_t qlm_best_plan_workspace_bytes(const qlm_problem *problem, int64_t n_plans)
{
    (void)problem;
    if (n_plans < 0) n_plans = 0;
    return align256(8 * (size_t)n_plans) + align256(8 * (size_t)kMaxScoreBlocks) + 256 +
           align256(8 * (size_t)kRefineBlocks) + align256(8 * (size_t)kRefineBlocks);
}

int qlm_best_plan(const qlm_problem *problem, const qlm_plans *plans, void *ws, size_t ws_bytes,
                  int64_t *best_index, double *best_score, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    if (!best_index || !best_score) return fail(QLM_ERR_ARG, "best_index and best_score are required");
    const int64_t P = plans->n_plans;
    if (!ws || ((uintptr_t)ws & 255u))
        return fail(QLM_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    if (ws_bytes < qlm_best_plan_workspace_bytes(problem, P))
        return fail(QLM_ERR_WORKSPACE, "workspace too small");
    unsigned char *w = (unsigned char *)ws;
    double *fast = (double *)w;
    w += align256(8 * (size_t)P);
    double *wg_min = (double *)w;
    w += align256(8 * (size_t)kMaxScoreBlocks);
    double *nsum = (double *)w;
    w += 256;
    double *bs = (double *)w;
    w += align256(8 * (size_t)kRefineBlocks);
    int64_t *bi = (int64_t *)w;
    if (P == 0) {
        hipLaunchKernelGGL(k_final, dim3(1), dim3(256), 0, stream, bs, bi, 0, best_index,
                           best_score);
        hipError_t e = hipGetLastError();
        return e == hipSuccess ? QLM_OK : hip_fail(e, "k_final launch");
    }
    int grid = 0;
    rc = launch_score(problem, plans, fast, nullptr, nullptr, wg_min, nsum, &grid, stream);
    if (rc) return rc;
    ExactArgs a = exact_args(problem, plans);
    int rgrid = (int)((P + kRefineThreads - 1) / kRefineThreads);
    if (rgrid > kRefineBlocks) rgrid = kRefineBlocks;
    size_t lds = 0;
    int big = 0;
    rc = exact_lds((const void *)k_refine, problem, &lds, &big);
    if (rc) return rc;
    hipLaunchKernelGGL(k_refine, dim3(rgrid), dim3(kRefineThreads), lds, stream, a, fast, wg_min,
                       grid, nsum, bs, bi, big);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_refine launch");
    hipLaunchKernelGGL(k_final, dim3(1), dim3(256), 0, stream, bs, bi, rgrid, best_index,
                       best_score);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "k_final launch");
    return QLM_OK;
}

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
    if (g0.lds_bytes > kLdsLimit) return 0;
    return (int32_t)((kLdsLimit - g0.lds_bytes) / 16);
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

const char *qlm_last_error(void) { return t_err.c_str(); }

int qlm_timing_enable(int on)
{
    g_timing.store(on != 0);
    return QLM_OK;
}

int qlm_timing_read(int64_t *launches, double *total_ms)
{
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
    {
        std::lock_guard<std::mutex> lk(g_timing_mu);
        ev.swap(g_events);
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
