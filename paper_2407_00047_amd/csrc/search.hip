// search.hip -- plan search on the GPU: steepest-descent local search over
// virtual-queue plans, every move scored exactly (double precision) and
// incrementally.  Interface: qlm_search_* and qlm_local_search in include/qlm.h.
//
// Moves are the scheduler's actions on virtual queues (reordering within a
// queue, reassignment to another instance: Sec. 5); the paper itself places
// groups with an LP (Sec. 7) and compares with EDF and same-model grouping.
//   SWAP(s, d)  k = s*W + d - 1     the groups at slots s and s + d (one queue)
//                                   trade places
//   MOVE(s, h)  k = G*W + s*I + h   the group at slot s joins queue h != its
//                                   own, before the first group of h whose SLO
//                                   is strictly later (else at the end)
// A moved group keeps its eviction flag.
//
// Incremental scoring.  A move changes at most two queues, each from one
// position on.  For every chain (a plan being improved) k_sstate caches, per
// slot, the running sums ahead of it (tokens A, variance V, fixed costs K up
// to the previous slot, and the score C of the slots ahead in its queue), and
// the score of every queue.  A move restarts the sums at its first changed
// position and walks the rest of the queue; the operations and their order are
// those of scoring the moved plan from its first slot (positions in order,
// then queues in order), so a move's score is exactly the plan score of the
// moved plan.
//
// Kernels
//   k_sprep    once per call: 32-byte group records; the groups ranked by SLO
//   k_sload    the start plans, slot-major -> chain-major working copies
//   k_sstate   one workgroup per chain: the cache above, per-queue scores and
//              their running sum over queues (= the plan score)
//   k_sswap    one lane per (chain, slot s, d = 0..W): d = 0 scores the queue
//              of s without s (a MOVE's source queue), d >= 1 SWAP(s, d)
//   k_smove    one lane per (chain, target queue h, group rank r by SLO):
//              MOVE(slot of that group, h).  Adjacent lanes hold groups of
//              adjacent SLOs, so their insertion points and walks are alike.
//   k_spick    one workgroup per chain: lowest (score, k) over all moves;
//              applied when strictly below the plan's score, else the chain
//              has converged and every later kernel skips it
//   k_sout     final plans back to the caller's slot-major layout
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <string>

#include "internal.h"
#include "qlm.h"

namespace {

using qlm_internal::fail;
using qlm_internal::hip_fail;

constexpr int kWave = 64;
constexpr int kStateThreads = 1024;
constexpr int kTaskThreads = 256;
constexpr int kPickThreads = 256;
constexpr int kPrepThreads = 256;
constexpr int kRankTile = 1024;
constexpr int32_t kMaxSearchGroups = 1 << 16;
constexpr int32_t kMaxSearchInstances = 4096;
constexpr int32_t kMaxWindow = 1024;
constexpr uint32_t kCountMask = (1u << 21) - 1u;
constexpr uint32_t kFlagBit = 1u << 8;
constexpr int kCountShift = 9;

// Group record: n mu and n sigma^2 (exact products of the fp32 inputs in
// double), SLO, and n << 9 | model.
struct GRec {
    double a, b;
    float slo;
    uint32_t nm;
    uint32_t pad[2];
};

// A chain's slot record, in slot order: the group's record with its eviction
// flag in bit 8, the running maximum of the SLOs of the queue up to this slot,
// and the slot's queue.
struct SRec {
    double a, b;
    float slo;
    uint32_t nmf;
    float pmax;
    uint32_t q;
};

// Running sums ahead of a slot: tokens and variance of the groups before it in
// its queue, fixed costs up to and including the slot itself, and the score of
// the slots before it in its queue.
struct SSt {
    double A, V, K, C;
};

struct SearchArgs {
    int32_t G, I, M, C, W;
    int64_t B;                    // chains
    const int32_t *grp_count;
    const float *grp_mu, *grp_var, *grp_slo;
    const int32_t *grp_model;
    const float *inst_tput;
    const int32_t *inst_class, *inst_model0;
    const float *swap_cost;
    float evict_cost;
    GRec *grec;                   // [G]
    int32_t *by_slo;              // [G] groups in SLO order
    // per chain, chain b at b * (per-chain size)
    int32_t *perm;                // [G]
    uint8_t *flag;                // [G]
    int32_t *qof;                 // [I + 1]
    int32_t *inv;                 // [G] slot of each group
    SRec *srec;                   // [G]
    SSt *sst;                     // [G]
    double *R;                    // [G] score of the queue of s without s
    double *Q;                    // [I] queue scores
    double *T;                    // [I + 1] running sum of queue scores
    double *cur;                  // [1] plan score
    int32_t *done, *steps;        // [1] each
    double *wmin_s;               // [nwg] workgroup minima of the move scores
    int64_t *wmin_i;              // [nwg] and their move numbers
    int32_t *scratch;             // [2 G] shifts of k_spick
    int32_t nwg_a, nwg_b, nwg;    // per chain: k_sswap, k_smove (per queue), total
    int64_t n_moves;
    double *move_score;           // [B][n_moves] or null
    int64_t *trace;               // [B][max_steps] or null
    int32_t max_steps;
};

__device__ inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

__device__ inline int model0_of(const SearchArgs &a, int g)
{
    return a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
}

// Total order on floats (the sign-magnitude bits made monotone).
__device__ inline uint32_t order_key(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

#pragma clang fp contract(off)

// The running sums of one queue walk, and one position of it: the definition
// in the order of the exact plan score (costs, then E[W] = A/Theta + K,
// SD = sqrt(V)/Theta, P = erfc((slo - E)/(SD sqrt 2))/2 or [E > slo] at SD = 0,
// then the term n P and the sums ahead of the next position).
struct Run {
    double A, V, K, sc;
    int prev;
};

__device__ inline void visit(Run &r, const SRec &x, double theta, int cls, const SearchArgs &a)
{
    const int m = (int)(x.nmf & 0xFFu);
    if (r.prev >= 0 && r.prev != m && a.swap_cost)
        r.K += (double)a.swap_cost[((int64_t)cls * a.M + r.prev) * a.M + m];
    if (x.nmf & kFlagBit) r.K += (double)a.evict_cost;
    const double EW = r.A / theta + r.K;
    const double SD = sqrt(r.V) / theta;
    const double slo = (double)x.slo;
    double P;
    if (SD > 0.0)
        P = 0.5 * erfc((slo - EW) / (SD * 1.4142135623730951));
    else
        P = (EW > slo) ? 1.0 : 0.0;
    r.sc += (double)(x.nmf >> kCountShift) * P;
    r.A += x.a;
    r.V += x.b;
    r.prev = m;
}

// The sums ahead of slot st of queue g (which starts at slot bq).
__device__ inline Run start_at(const SearchArgs &a, const SRec *sr, const SSt *ss, int st, int bq,
                               int g)
{
    const SSt x = ss[st];
    Run r;
    r.A = x.A;
    r.V = x.V;
    r.sc = x.C;
    if (st > bq) {
        r.K = ss[st - 1].K;
        r.prev = (int)(sr[st - 1].nmf & 0xFFu);
    } else {
        r.K = 0.0;
        r.prev = model0_of(a, g);
    }
    return r;
}

// First slot of [bq, eq) whose group's SLO is strictly later than slo (eq if
// none): the running maxima are non-decreasing, and the first one above slo
// is at the first SLO above it.
__device__ inline int insertion_point(const SRec *sr, int bq, int eq, float slo)
{
    int lo = bq, hi = eq;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (sr[mid].pmax > slo)
            hi = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

// (score, k) is better than (s2, k2): lower score, then lower k.  A NaN score
// is never better.
__device__ inline bool better(double s, int64_t k, double s2, int64_t k2)
{
    return s < s2 || (s == s2 && k < k2);
}

// Workgroup minimum of (score, k); the result is valid in thread 0.
template <int kThreads>
__device__ void block_best(double &s, int64_t &k, double *ls, int64_t *lk)
{
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const double s2 = __shfl_xor(s, o, kWave);
        const int64_t k2 = __shfl_xor(k, o, kWave);
        if (better(s2, k2, s, k)) {
            s = s2;
            k = k2;
        }
    }
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    if (lane == 0) {
        ls[wave] = s;
        lk[wave] = k;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kThreads / kWave; ++w)
            if (better(ls[w], lk[w], s, k)) {
                s = ls[w];
                k = lk[w];
            }
    }
}

// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kPrepThreads) void k_sprep(SearchArgs a)
{
    __shared__ uint32_t keys[kRankTile];
    const int G = a.G;
    const int i = blockIdx.x * kPrepThreads + threadIdx.x;
    uint32_t mine = 0;
    if (i < G) {
        const uint32_t n = (uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
        const double dn = (double)n;
        GRec r;
        r.a = dn * (double)a.grp_mu[i];
        r.b = dn * (double)a.grp_var[i];
        r.slo = a.grp_slo[i];
        r.nm = (n << kCountShift) | (uint32_t)clampi(a.grp_model[i], 0, a.M - 1);
        r.pad[0] = r.pad[1] = 0u;
        a.grec[i] = r;
        mine = order_key(r.slo);
    }
    // rank = groups ordered before i by (SLO, id)
    int rank = 0;
    for (int t0 = 0; t0 < G; t0 += kRankTile) {
        __syncthreads();
        for (int k = threadIdx.x; k < kRankTile; k += kPrepThreads)
            keys[k] = t0 + k < G ? order_key(a.grp_slo[t0 + k]) : 0xFFFFFFFFu;
        __syncthreads();
        const int n = min(kRankTile, G - t0);
        for (int k = 0; k < n; ++k) {
            const uint32_t o = keys[k];
            rank += (o < mine || (o == mine && t0 + k < i)) ? 1 : 0;
        }
    }
    if (i < G) a.by_slo[rank] = i;
}

// Start plans into the working copies; qoff is forced to a monotone split of
// [0, G] and group ids to [0, G) so that every later access stays in bounds.
__global__ __launch_bounds__(kPrepThreads) void k_sload(SearchArgs a, qlm_plans pl)
{
    const int G = a.G, I = a.I;
    const int nblk = (G + kPrepThreads - 1) / kPrepThreads;
    const int64_t b = blockIdx.x / nblk;
    const int s = (blockIdx.x % nblk) * kPrepThreads + threadIdx.x;
    if (s < G) {
        const int64_t e = (int64_t)s * pl.plan_stride + b;
        a.perm[b * G + s] = clampi(pl.perm[e], 0, G - 1);
        uint8_t f = 0;
        if (pl.evict_bits)
            f = (uint8_t)((pl.evict_bits[(int64_t)(s >> 5) * pl.plan_stride + b] >> (s & 31)) & 1u);
        a.flag[b * G + s] = f;
    }
    if (blockIdx.x % nblk == 0 && threadIdx.x == 0) {
        int32_t *q = a.qof + b * (I + 1);
        int prev = 0;
        q[0] = 0;
        for (int g = 1; g < I; ++g) {
            prev = clampi(pl.qoff[(int64_t)g * pl.plan_stride + b], prev, G);
            q[g] = prev;
        }
        q[I] = G;
        a.done[b] = 0;
        a.steps[b] = 0;
        if (a.trace)
            for (int t = 0; t < a.max_steps; ++t) a.trace[b * a.max_steps + t] = -1;
    }
}

// The cache of one chain's plan (one workgroup per chain).
__global__ __launch_bounds__(kStateThreads) void k_sstate(SearchArgs a, int force)
{
    __shared__ int32_t qo[kMaxSearchInstances + 1];
    const int64_t b = blockIdx.x;
    if (!force && a.done[b]) return;
    const int G = a.G, I = a.I;
    const int32_t *__restrict__ perm = a.perm + b * G;
    const uint8_t *__restrict__ flag = a.flag + b * G;
    SRec *__restrict__ sr = a.srec + b * G;
    SSt *__restrict__ ss = a.sst + b * G;
    int32_t *__restrict__ inv = a.inv + b * G;
    double *__restrict__ Q = a.Q + b * I;
    for (int g = threadIdx.x; g <= I; g += kStateThreads) qo[g] = a.qof[b * (I + 1) + g];
    __syncthreads();
    // 0. slot records in slot order
    for (int s = threadIdx.x; s < G; s += kStateThreads) {
        int lo = 0, hi = I;                     // last g with qo[g] <= s
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (qo[mid] <= s)
                lo = mid;
            else
                hi = mid;
        }
        const int i = perm[s];
        const GRec r = a.grec[i];
        SRec x;
        x.a = r.a;
        x.b = r.b;
        x.slo = r.slo;
        x.nmf = r.nm | (flag[s] ? kFlagBit : 0u);
        x.pmax = 0.0f;
        x.q = (uint32_t)lo;
        sr[s] = x;
        inv[i] = s;
    }
    __syncthreads();
    // 1. running sums per queue, in position order (8 records fetched ahead)
    for (int g = threadIdx.x; g < I; g += kStateThreads) {
        const int bq = qo[g], eq = qo[g + 1];
        const int cls = clampi(a.inst_class[g], 0, a.C - 1);
        Run r{0.0, 0.0, 0.0, 0.0, model0_of(a, g)};
        float pm = -INFINITY;
        for (int s0 = bq; s0 < eq; s0 += 8) {
            SRec x[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (s0 + u < eq) x[u] = sr[s0 + u];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (s0 + u >= eq) break;
                const int m = (int)(x[u].nmf & 0xFFu);
                if (r.prev >= 0 && r.prev != m && a.swap_cost)
                    r.K += (double)a.swap_cost[((int64_t)cls * a.M + r.prev) * a.M + m];
                if (x[u].nmf & kFlagBit) r.K += (double)a.evict_cost;
                pm = x[u].slo > pm ? x[u].slo : pm;
                ss[s0 + u] = SSt{r.A, r.V, r.K, 0.0};
                sr[s0 + u].pmax = pm;
                r.A += x[u].a;
                r.V += x[u].b;
                r.prev = m;
            }
        }
    }
    __syncthreads();
    // 2. each slot's term n P
    for (int s = threadIdx.x; s < G; s += kStateThreads) {
        const SRec x = sr[s];
        const SSt t = ss[s];
        const double theta = (double)a.inst_tput[x.q];
        const double EW = t.A / theta + t.K;
        const double SD = sqrt(t.V) / theta;
        const double slo = (double)x.slo;
        double P;
        if (SD > 0.0)
            P = 0.5 * erfc((slo - EW) / (SD * 1.4142135623730951));
        else
            P = (EW > slo) ? 1.0 : 0.0;
        ss[s].C = (double)(x.nmf >> kCountShift) * P;
    }
    __syncthreads();
    // 3. scores ahead of each slot, and per queue, in position order
    for (int g = threadIdx.x; g < I; g += kStateThreads) {
        const int bq = qo[g], eq = qo[g + 1];
        double c = 0.0;
        for (int s0 = bq; s0 < eq; s0 += 8) {
            double t[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (s0 + u < eq) t[u] = ss[s0 + u].C;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (s0 + u >= eq) break;
                ss[s0 + u].C = c;
                c += t[u];
            }
        }
        Q[g] = c;
    }
    __syncthreads();
    // 4. queue scores summed in queue order
    if (threadIdx.x == 0) {
        double *T = a.T + b * (I + 1);
        double t = 0.0;
        T[0] = 0.0;
        for (int g = 0; g < I; ++g) {
            t += Q[g];
            T[g + 1] = t;
        }
        a.cur[b] = t;
    }
}

// Plan score with queue g's score replaced by qg (queues summed in order).
__device__ inline double total_with(const double *T, const double *Q, int I, int g, double qg)
{
    double t = T[g] + qg;
    for (int q = g + 1; q < I; ++q) t += Q[q];
    return t;
}

__global__ __launch_bounds__(kTaskThreads) void k_sswap(SearchArgs a)
{
    __shared__ double ls[kTaskThreads / kWave];
    __shared__ int64_t lk[kTaskThreads / kWave];
    const int64_t b = blockIdx.x / a.nwg_a;
    const int wg = blockIdx.x % a.nwg_a;
    if (a.done[b]) return;
    const int G = a.G, I = a.I, W = a.W;
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int t = wg * kTaskThreads + threadIdx.x;
    const int s = t / (W + 1);
    const int d = t - s * (W + 1);
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    if (s < G) {
        const int g = (int)sr[s].q;
        const int bq = qof[g], eq = qof[g + 1];
        const double theta = (double)a.inst_tput[g];
        const int cls = clampi(a.inst_class[g], 0, a.C - 1);
        if (d == 0) {
            Run r = start_at(a, sr, ss, s, bq, g);
            for (int u = s + 1; u < eq; ++u) visit(r, sr[u], theta, cls, a);
            a.R[b * G + s] = r.sc;
        } else {
            const int64_t k = (int64_t)s * W + (d - 1);
            double score = INFINITY;
            if (s + d < eq) {
                Run r = start_at(a, sr, ss, s, bq, g);
                for (int u = s; u < eq; ++u) {
                    const int v = u == s ? s + d : (u == s + d ? s : u);
                    visit(r, sr[v], theta, cls, a);
                }
                score = total_with(a.T + b * (I + 1), a.Q + b * I, I, g, r.sc);
                if (better(score, k, best, bk)) {
                    best = score;
                    bk = k;
                }
            }
            if (a.move_score) a.move_score[b * a.n_moves + k] = score;
        }
    }
    block_best<kTaskThreads>(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        a.wmin_s[b * a.nwg + wg] = best;
        a.wmin_i[b * a.nwg + wg] = bk;
    }
}

__global__ __launch_bounds__(kTaskThreads) void k_smove(SearchArgs a)
{
    __shared__ double ls[kTaskThreads / kWave];
    __shared__ int64_t lk[kTaskThreads / kWave];
    const int G = a.G, I = a.I;
    const int per_chain = I * a.nwg_b;
    const int64_t b = blockIdx.x / per_chain;
    const int h = (blockIdx.x % per_chain) / a.nwg_b;
    const int wg = blockIdx.x % a.nwg_b;
    if (a.done[b]) return;
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int r = wg * kTaskThreads + threadIdx.x;
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    if (r < G) {
        const int i = a.by_slo[r];
        const int s = clampi(a.inv[b * G + i], 0, G - 1);
        const SRec x = sr[s];
        const int g = (int)x.q;
        const int64_t k = (int64_t)G * a.W + (int64_t)s * I + h;
        double score = INFINITY;
        if (g != h) {
            const int bq = qof[h], eq = qof[h + 1];
            const double theta = (double)a.inst_tput[h];
            const int cls = clampi(a.inst_class[h], 0, a.C - 1);
            Run w;
            if (bq == eq) {
                w = Run{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
                visit(w, x, theta, cls, a);
            } else {
                const int p = insertion_point(sr, bq, eq, x.slo);
                if (p == eq) {
                    w = start_at(a, sr, ss, eq - 1, bq, h);
                    visit(w, sr[eq - 1], theta, cls, a);
                    visit(w, x, theta, cls, a);
                } else {
                    w = start_at(a, sr, ss, p, bq, h);
                    visit(w, x, theta, cls, a);
                    for (int u = p; u < eq; ++u) visit(w, sr[u], theta, cls, a);
                }
            }
            const double *T = a.T + b * (I + 1);
            const double *Q = a.Q + b * I;
            const double Rs = a.R[b * G + s];
            const int lo = g < h ? g : h;
            double t = T[lo];
            for (int q = lo; q < I; ++q) t += q == g ? Rs : (q == h ? w.sc : Q[q]);
            score = t;
            if (better(score, k, best, bk)) {
                best = score;
                bk = k;
            }
        }
        if (a.move_score) a.move_score[b * a.n_moves + k] = score;
    }
    block_best<kTaskThreads>(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        const int64_t o = b * a.nwg + a.nwg_a + (int64_t)h * a.nwg_b + wg;
        a.wmin_s[o] = best;
        a.wmin_i[o] = bk;
    }
}

#pragma clang fp contract(on)

// Best move of each chain; applied when it improves on the plan.
__global__ __launch_bounds__(kPickThreads) void k_spick(SearchArgs a, int step)
{
    __shared__ double ls[kPickThreads / kWave];
    __shared__ int64_t lk[kPickThreads / kWave];
    __shared__ int apply;
    __shared__ int64_t kk;
    const int64_t b = blockIdx.x;
    if (a.done[b]) return;
    const int G = a.G, I = a.I, W = a.W;
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    for (int w = threadIdx.x; w < a.nwg; w += kPickThreads) {
        const double s = a.wmin_s[b * a.nwg + w];
        const int64_t k = a.wmin_i[b * a.nwg + w];
        if (better(s, k, best, bk)) {
            best = s;
            bk = k;
        }
    }
    block_best<kPickThreads>(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        apply = (best < a.cur[b] && bk >= 0 && bk < a.n_moves) ? 1 : 0;
        kk = bk;
        if (apply) {
            a.cur[b] = best;
            a.steps[b] += 1;
            if (a.trace) a.trace[b * a.max_steps + step] = bk;
        } else {
            a.done[b] = 1;
        }
    }
    __syncthreads();
    if (!apply) return;
    int32_t *perm = a.perm + b * G;
    uint8_t *flag = a.flag + b * G;
    int32_t *qof = a.qof + b * (I + 1);
    const int64_t k = kk;
    if (k < (int64_t)G * W) {
        if (threadIdx.x == 0) {
            const int s = (int)(k / W), t = s + (int)(k % W) + 1;
            const int32_t pi = perm[s];
            const uint8_t fi = flag[s];
            perm[s] = perm[t];
            flag[s] = flag[t];
            perm[t] = pi;
            flag[t] = fi;
        }
        return;
    }
    const int64_t r = k - (int64_t)G * W;
    const int s = (int)(r / I), h = (int)(r % I);
    const SRec *sr = a.srec + b * G;
    const int g = (int)sr[s].q;
    const int p = insertion_point(sr, qof[h], qof[h + 1], sr[s].slo);
    // the slots from s to the insertion point rotate by one
    const int lo = h > g ? s : p;
    const int hi = h > g ? p - 1 : s;
    int32_t *sp = a.scratch + b * 2 * G;
    int32_t *sf = sp + G;
    for (int u = lo + threadIdx.x; u <= hi; u += kPickThreads) {
        sp[u] = perm[u];
        sf[u] = flag[u];
    }
    __syncthreads();
    for (int u = lo + threadIdx.x; u <= hi; u += kPickThreads) {
        int v;
        if (h > g)
            v = u == hi ? s : u + 1;          // left by one, the group at the end
        else
            v = u == lo ? s : u - 1;          // right by one, the group at the front
        perm[u] = sp[v];
        flag[u] = (uint8_t)sf[v];
    }
    if (h > g) {
        for (int q = g + 1 + threadIdx.x; q <= h; q += kPickThreads) qof[q] -= 1;
    } else {
        for (int q = h + 1 + threadIdx.x; q <= g; q += kPickThreads) qof[q] += 1;
    }
}

// Final plans to the caller's slot-major arrays, with their scores and steps.
__global__ __launch_bounds__(kPrepThreads) void k_sout(SearchArgs a, qlm_plans_out out,
                                                       double *score, int32_t *steps)
{
    const int G = a.G, I = a.I;
    const int64_t B = a.B;
    const int nw = (G + 31) >> 5;
    const int64_t rows = (int64_t)G + (I + 1) + (out.evict_bits ? nw : 0) + 1;
    for (int64_t x = (int64_t)blockIdx.x * kPrepThreads + threadIdx.x; x < rows * B;
         x += (int64_t)gridDim.x * kPrepThreads) {
        const int64_t row = x / B, b = x % B;
        if (row < G) {
            out.perm[row * out.plan_stride + b] = a.perm[b * G + row];
        } else if (row < G + I + 1) {
            const int64_t g = row - G;
            out.qoff[g * out.plan_stride + b] = a.qof[b * (I + 1) + g];
        } else if (row < rows - 1) {
            const int w = (int)(row - G - I - 1);
            uint32_t word = 0;
            for (int j = 0; j < 32 && 32 * w + j < G; ++j)
                word |= (uint32_t)(a.flag[b * G + 32 * w + j] & 1u) << j;
            out.evict_bits[(int64_t)w * out.plan_stride + b] = word;
        } else {
            if (score) score[b] = a.cur[b];
            if (steps) steps[b] = a.steps[b];
        }
    }
}

// ---------------------------------------------------------------------------
// Host side

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

struct Layout {
    int nwg_a, nwg_b, nwg;
    size_t grec, by_slo, perm, flag, qof, inv, srec, sst, R, Q, T, cur, done, steps, wmin_s,
        wmin_i, scratch, total;
};

Layout layout(int G, int I, int W, int64_t B)
{
    Layout L{};
    L.nwg_a = (int)(((int64_t)G * (W + 1) + kTaskThreads - 1) / kTaskThreads);
    L.nwg_b = (G + kTaskThreads - 1) / kTaskThreads;
    L.nwg = L.nwg_a + I * L.nwg_b;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align256(bytes);
        return at;
    };
    const size_t b = (size_t)B;
    L.grec = take(sizeof(GRec) * G);
    L.by_slo = take(4 * (size_t)G);
    L.perm = take(4 * (size_t)G * b);
    L.flag = take((size_t)G * b);
    L.qof = take(4 * (size_t)(I + 1) * b);
    L.inv = take(4 * (size_t)G * b);
    L.srec = take(sizeof(SRec) * G * b);
    L.sst = take(sizeof(SSt) * G * b);
    L.R = take(8 * (size_t)G * b);
    L.Q = take(8 * (size_t)I * b);
    L.T = take(8 * (size_t)(I + 1) * b);
    L.cur = take(8 * b);
    L.done = take(4 * b);
    L.steps = take(4 * b);
    L.wmin_s = take(8 * (size_t)L.nwg * b);
    L.wmin_i = take(8 * (size_t)L.nwg * b);
    L.scratch = take(8 * (size_t)G * b);
    L.total = o;
    return L;
}

int check_search(const qlm_problem *pr, int64_t B, int32_t W)
{
    int rc = qlm_internal::check_problem(pr);
    if (rc) return rc;
    if (pr->n_groups > kMaxSearchGroups) return fail(QLM_ERR_ARG, "search: n_groups must be <= 65536");
    if (pr->n_instances > kMaxSearchInstances)
        return fail(QLM_ERR_ARG, "search: n_instances must be <= 4096");
    if (W < 0 || W > kMaxWindow) return fail(QLM_ERR_ARG, "search: window must be in [0, 1024]");
    if (B < 0) return fail(QLM_ERR_ARG, "search: n_plans must be >= 0");
    const Layout L = layout(pr->n_groups, pr->n_instances, W, B > 0 ? B : 1);
    if ((int64_t)L.nwg * B > INT_MAX || (int64_t)pr->n_instances * L.nwg_b * B > INT_MAX ||
        (int64_t)L.nwg_a * B > INT_MAX)
        return fail(QLM_ERR_ARG, "search: too many plans for one launch");
    return QLM_OK;
}

SearchArgs search_args(const qlm_problem *pr, int64_t B, int32_t W, unsigned char *ws,
                       const Layout &L)
{
    SearchArgs a{};
    a.G = pr->n_groups;
    a.I = pr->n_instances;
    a.M = pr->n_models;
    a.C = pr->n_classes;
    a.W = W;
    a.B = B;
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
    a.grec = (GRec *)(ws + L.grec);
    a.by_slo = (int32_t *)(ws + L.by_slo);
    a.perm = (int32_t *)(ws + L.perm);
    a.flag = ws + L.flag;
    a.qof = (int32_t *)(ws + L.qof);
    a.inv = (int32_t *)(ws + L.inv);
    a.srec = (SRec *)(ws + L.srec);
    a.sst = (SSt *)(ws + L.sst);
    a.R = (double *)(ws + L.R);
    a.Q = (double *)(ws + L.Q);
    a.T = (double *)(ws + L.T);
    a.cur = (double *)(ws + L.cur);
    a.done = (int32_t *)(ws + L.done);
    a.steps = (int32_t *)(ws + L.steps);
    a.wmin_s = (double *)(ws + L.wmin_s);
    a.wmin_i = (int64_t *)(ws + L.wmin_i);
    a.scratch = (int32_t *)(ws + L.scratch);
    a.nwg_a = L.nwg_a;
    a.nwg_b = L.nwg_b;
    a.nwg = L.nwg;
    a.n_moves = (int64_t)a.G * W + (int64_t)a.G * a.I;
    return a;
}

int launched(const char *what)
{
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? QLM_OK : hip_fail(e, what);
}

// Set-up shared by both entry points: checks, the group records and ranks, the
// start plans, and the cache of every chain.
int search_begin(const qlm_problem *pr, const qlm_plans *pl, int32_t W, void *ws, size_t ws_bytes,
                 SearchArgs *out, hipStream_t stream)
{
    int rc = check_search(pr, pl ? pl->n_plans : 0, W);
    if (rc) return rc;
    rc = qlm_internal::check_plans(pr, pl);
    if (rc) return rc;
    const int64_t B = pl->n_plans;
    const Layout L = layout(pr->n_groups, pr->n_instances, W, B);
    if (!ws || ((uintptr_t)ws & 255u))
        return fail(QLM_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    if (ws_bytes < L.total) return fail(QLM_ERR_WORKSPACE, "workspace too small");
    SearchArgs a = search_args(pr, B, W, (unsigned char *)ws, L);
    *out = a;
    if (B == 0) return QLM_OK;
    const int G = a.G;
    hipLaunchKernelGGL(k_sprep, dim3((G + kPrepThreads - 1) / kPrepThreads), dim3(kPrepThreads), 0,
                       stream, a);
    return launched("k_sprep launch");
}

int load_and_state(SearchArgs &a, const qlm_plans *pl, hipStream_t stream)
{
    const int nblk = (a.G + kPrepThreads - 1) / kPrepThreads;
    hipLaunchKernelGGL(k_sload, dim3((unsigned)(nblk * a.B)), dim3(kPrepThreads), 0, stream, a, *pl);
    int rc = launched("k_sload launch");
    if (rc) return rc;
    hipLaunchKernelGGL(k_sstate, dim3((unsigned)a.B), dim3(kStateThreads), 0, stream, a, 1);
    return launched("k_sstate launch");
}

int score_moves(SearchArgs &a, hipStream_t stream)
{
    hipLaunchKernelGGL(k_sswap, dim3((unsigned)(a.nwg_a * a.B)), dim3(kTaskThreads), 0, stream, a);
    int rc = launched("k_sswap launch");
    if (rc) return rc;
    qlm_internal::TimedLaunch tl;
    if ((rc = qlm_internal::timing_begin(stream, &tl))) return rc;
    hipLaunchKernelGGL(k_smove, dim3((unsigned)((int64_t)a.I * a.nwg_b * a.B)), dim3(kTaskThreads),
                       0, stream, a);
    if ((rc = launched("k_smove launch"))) return rc;
    qlm_internal::timing_end(stream, &tl);
    return QLM_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C interface

extern "C" {

int64_t qlm_search_n_moves(int32_t n_groups, int32_t n_instances, int32_t window)
{
    if (n_groups < 1 || n_instances < 1 || window < 0) return 0;
    return (int64_t)n_groups * window + (int64_t)n_groups * n_instances;
}

size_t qlm_search_workspace_bytes(const qlm_problem *problem, int64_t n_plans, int32_t window)
{
    if (!problem || problem->n_groups < 1 || problem->n_instances < 1 || window < 0 ||
        n_plans < 0)
        return 0;
    return layout(problem->n_groups, problem->n_instances, window, n_plans > 0 ? n_plans : 1).total;
}

int qlm_search_moves(const qlm_problem *problem, const qlm_plans *plans, int32_t window, void *ws,
                     size_t ws_bytes, double *move_score, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!move_score) return fail(QLM_ERR_ARG, "move_score is NULL");
    SearchArgs a;
    int rc = search_begin(problem, plans, window, ws, ws_bytes, &a, stream);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    a.move_score = move_score;
    rc = load_and_state(a, plans, stream);
    if (rc) return rc;
    return score_moves(a, stream);
}

int qlm_local_search(const qlm_problem *problem, const qlm_plans *start, const qlm_plans_out *out,
                     int32_t window, int32_t max_steps, void *ws, size_t ws_bytes, double *score,
                     int32_t *steps, int64_t *trace, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!out) return fail(QLM_ERR_ARG, "out is NULL");
    if (max_steps < 0) return fail(QLM_ERR_ARG, "max_steps must be >= 0");
    if (start && start->n_plans > 0) {
        if (!out->perm || !out->qoff) return fail(QLM_ERR_ARG, "out perm and qoff are required");
        if (out->plan_stride < start->n_plans)
            return fail(QLM_ERR_ARG, "out plan_stride must be >= n_plans");
        if (start->evict_bits && !out->evict_bits)
            return fail(QLM_ERR_ARG, "out evict_bits is required when the plans have eviction bits");
    }
    SearchArgs a;
    int rc = search_begin(problem, start, window, ws, ws_bytes, &a, stream);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    a.trace = trace;
    a.max_steps = max_steps;
    rc = load_and_state(a, start, stream);
    if (rc) return rc;
    for (int t = 0; t < max_steps; ++t) {
        if (t > 0) {
            hipLaunchKernelGGL(k_sstate, dim3((unsigned)a.B), dim3(kStateThreads), 0, stream, a, 0);
            if ((rc = launched("k_sstate launch"))) return rc;
        }
        if ((rc = score_moves(a, stream))) return rc;
        hipLaunchKernelGGL(k_spick, dim3((unsigned)a.B), dim3(kPickThreads), 0, stream, a, t);
        if ((rc = launched("k_spick launch"))) return rc;
    }
    if (max_steps > 0) {
        hipLaunchKernelGGL(k_sstate, dim3((unsigned)a.B), dim3(kStateThreads), 0, stream, a, 1);
        if ((rc = launched("k_sstate launch"))) return rc;
    }
    qlm_plans_out o = *out;
    if (!start->evict_bits) o.evict_bits = nullptr;
    const int64_t rows = (int64_t)a.G + a.I + 1 + (o.evict_bits ? (a.G + 31) / 32 : 0) + 1;
    int64_t grid = (rows * a.B + kPrepThreads - 1) / kPrepThreads;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(k_sout, dim3((unsigned)grid), dim3(kPrepThreads), 0, stream, a, o, score,
                       steps);
    return launched("k_sout launch");
}

}  // extern "C"
