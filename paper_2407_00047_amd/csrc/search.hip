// search.hip -- plan search on the GPU: steepest-descent local search over
// virtual-queue plans.  Interface: qlm_search_* and qlm_local_search in
// include/qlm.h.
//
// Moves are the scheduler's actions on virtual queues (reordering within a
// queue, reassignment to another instance, eviction: Sec. 5); the paper
// itself places groups with an LP (Sec. 7) and compares with EDF and
// same-model grouping.  The first slot of a non-empty queue holds the group
// its instance is running: no move takes it, and only RELOCATE passes it.
//   SWAP(s, d)      k = s*W + d - 1         the groups at slots s and s + d
//                                           (one queue) trade places
//   MOVE(s, h)      k = G*W + s*I + h       the group at slot s joins queue
//                                           h != its own, before the first
//                                           group after h's head whose SLO is
//                                           strictly later (else at the end;
//                                           the head of an empty h)
//   RELOCATE(s, h)  k = G*W + G*I + s*I + h the group at slot s becomes the
//                                           head of the non-empty queue h (its
//                                           own or another), its eviction flag
//                                           set
// Any other moved group keeps its eviction flag.
//
// Exact scores.  A move changes at most two queues, each from one position
// on.  For every chain (a plan being improved) k_sstate caches, per slot, the
// running sums ahead of it (tokens A, variance V, fixed costs K, the score C
// of the slots ahead in its queue) and the score of every queue.  An exact
// move score restarts the sums at the first changed position and walks the
// rest of the queue with the operations, in the order, of scoring the moved
// plan from its first slot (positions in order, then queues in order): it is
// the plan score of the moved plan, bit for bit.
//
// Screened steps.  A search step needs the exact score of the best move only.
// Every move is first screened: past the positions it changes, a queue is the
// old queue shifted by constants (the moved group's tokens and variance, the
// change of fixed costs), so each later position costs one subtraction from
// its cached margin slo - E[W] and one lookup in the linear-cell table of the
// normal tail (tail.h).  The screened score F has a proven bound D on its
// distance to the exact score (below); the moves whose exact score can still
// be the lowest, F - D <= min(F + D), and can still improve on the plan, are
// re-scored exactly, one wavefront per move, and the lowest exact score (the
// lowest k on ties) decides.  The search takes the same steps as one that
// scores every move exactly.
//
// Screening bound, per request of the queue the screen walks: the table is
// within 2.2e-6 of Q; single-precision rounding of the margin, the scaled
// variance, the cell coordinate and n P adds below 1.5e-6; so D = 8e-6 times
// the requests of that queue, plus 1e-12 of the scores for double rounding.
// The margin itself is formed in double precision from cached sums, which may
// differ from the exact score's own sums in their last bits; a move whose
// smallest spread is so small that this could move z by more than 1e-7 gets
// D = infinity (re-scored exactly), as does one whose walk meets a variance
// that single precision cannot hold.  A queue that loses the moved group is
// screened with its variance ahead in double precision (no cancellation), and
// a MOVE's or another queue's RELOCATE's bound adds the bounds of both its
// queues.  A RELOCATE within one queue walks two shifted stretches (the
// groups it passes gain its tokens and variance; past its old slot only the
// costs change) and forms the position after its old slot afresh; where
// nothing ahead of that position has variance its indicator would not be
// formed from the exact score's sums, so the move is re-scored exactly.
// Exact scores (of the candidates) walk both queues exactly.
//
// Kernels
//   k_srank    once per call: the groups ranked by SLO (partial counts per
//              tile of 1024 groups; k_srankout sums them, places each group
//              at its rank and writes the group records)
//   k_stail    once per call: the normal-tail table, which the screens copy
//              into LDS
//   k_sload    start plans, slot-major -> chain-major working copies
//   k_sstate   one wavefront per queue: slot records, the exact running sums,
//              the cached margins, the queue score (k_stotal: their sum)
//   k_fswap    one lane per task: the screened score of the queue of each slot
//              s without s (for the MOVEs of s), and screened SWAP(s, d); the
//              positions past the changes are walked in step by the wavefront
//   k_fmove    one wavefront per (target queue h, 64 groups adjacent in SLO
//              order), each lane both moves of its group into h: screened
//              MOVE and screened RELOCATE into another queue; the positions
//              past the insertion points are walked in step by the whole
//              wavefront (one record read per position for all 128 moves); in
//              the same launch, one lane per slot: screened RELOCATE within
//              the slot's queue
//   k_sbound / k_sselect / k_sexact   the bound min(F + D), the candidates,
//              their exact scores
//   k_spick    lowest (exact score, k) of the candidates; applied when it
//              improves on the plan, else the chain has converged
//   k_sout     final plans back to the caller's slot-major layout
//   k_sswap / k_smove / k_sreloc   exact scores of every move, one lane per
//              move (qlm_search_moves)
//   k_place_eval / k_place_pick   placement of one group (qlm_place_group):
//              one wavefront per (plan, place) scores the group placed there
//              (the EDF position after a queue's head, or a queue's head with
//              eviction) exactly; the lowest score is applied
//   k_seedrank / k_seedassign / k_seedwrite   seed plans (qlm_seed_plans):
//              EDF or same-model order, each group to the queue with the
//              smallest drain time after it (one wavefront per seed)
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <string>

#include "internal.h"
#include "qlm.h"
#include "ripple.h"
#include "tail.h"

namespace {

using qlm_internal::fail;
using qlm_internal::hip_fail;
using qlm_ripple::from_left;
using qlm_ripple::from_left0;
using qlm_ripple::lane_value;
using qlm_ripple::wave_id;

constexpr int kWave = 64;
constexpr int kThreads = 256;              // every search kernel: 4 wavefronts
constexpr int kWaves = kThreads / kWave;
constexpr int kRankTile = 1024;
constexpr int kSwapStage = 512;              // tail records the removal/swap screen stages
constexpr int kSwapStageBytes = kSwapStage * 24;   // 16-byte records and 8-byte variances
constexpr int kSwapRecs = kSwapStageBytes / 32;    // or that many 32-byte slot records
constexpr int kSwapCostStage = 1024;         // swap-cost entries it stages
constexpr int kExactBlocks = 64;           // per chain, for the exact re-scores
constexpr int kStage = 256;                // tail records k_fmove stages in LDS at a time
constexpr int kRelStage = 128;             // tail records each wavefront of the
                                           // own-queue relocation screen stages
constexpr int32_t kMaxSearchGroups = 1 << 16;
constexpr int32_t kMaxSearchInstances = 4096;
constexpr int32_t kMaxWindow = 1024;
constexpr int kStageSlots = 8192;            // slots a placement moves through LDS
constexpr uint32_t kCountMask = (1u << 21) - 1u;
constexpr uint32_t kFlagBit = 1u << 8;
constexpr int kCountShift = 9;
constexpr double kEpsP = 8e-6;             // screening bound per request
constexpr double kZErr = 1e-7;             // largest z error from the margin's rounding

// Group record: n mu and n sigma^2 (exact products of the fp32 inputs in
// double), SLO, and n << 9 | model.
struct GRec {
    double a, b;
    float slo;
    uint32_t nm;
    uint32_t pad[2];
};

// A chain's slot record, in slot order: the group's record with its eviction
// flag in bit 8, the running maximum of the SLOs of the queue's groups after
// its head up to this slot (-inf at the head), and the slot's queue.
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

// What a screen reads at a position past the change: the margin slo - E[W]
// (seconds), the variance ahead scaled for the tail table (V / Theta^2 times
// kVarScale, single precision), and the request count.
struct TRec {
    double m;
    float vz;
    float n;
};
static_assert(sizeof(SRec) == 32 && sizeof(TRec) == 16, "the screens' LDS staging sizes");

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
    int32_t *rank_part;           // [ceil(G / kRankTile)][G] partial ranks
    float2 *tail;                 // [kCells] the normal-tail table (tail.h)
    // per chain, chain b at b * (per-chain size)
    int32_t *perm;                // [G]
    uint8_t *flag;                // [G]
    int32_t *qof;                 // [I + 1]
    int32_t *inv;                 // [G] slot of each group
    SRec *srec;                   // [G]
    SSt *sst;                     // [G]
    TRec *trec;                   // [G]
    double *R;                    // [G] score of the queue of s without s (exact in
                                  // the exact kernels, screened in the screens)
    double *RD;                   // [G] bound of the screened one
    double *Q;                    // [I] queue scores
    double *Nq;                   // [I] requests per queue
    double *Es;                   // [I] largest |E[W]| + |slo| in the queue
    double *T;                    // [I + 1] running sum of queue scores
    double *cur;                  // [1] plan score
    int32_t *done, *steps;        // [1] each
    double *wmin_s;               // [nwg] exact kernels: workgroup minima
    int64_t *wmin_i;              // [nwg] and their move numbers
    double *smin;                 // [nws] screens: workgroup minima of F + D
    double *F, *D;                // [n_moves] screened scores and their bounds
    int32_t *cand;                // [n_moves] candidate moves
    double *cex;                  // [n_moves] their exact scores
    int32_t *ncand;               // [1]
    double *U;                    // [1] min(F + D)
    int32_t *scratch;             // [2 G] shifts of k_spick
    int32_t *dq;                  // [4] placement: the group's slot and queue, and
                                  // whether it is running (stays)
    int32_t nwg_a, nwg_b, nwg;    // per chain: k_sswap, k_smove and k_sreloc (per
                                  // queue), total
    int32_t nwg_f, nwg_r, nws;    // per chain: k_fswap (d = 0..W), k_fmove's own-queue
                                  // relocations, all screen workgroups
    int64_t n_moves;
    double *move_score;           // [B][n_moves] or null (exact kernels)
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

__device__ inline double wave_min(double v)
{
    for (int o = kWave / 2; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline double wave_max(double v)
{
    for (int o = kWave / 2; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline double wave_sum(double v)
{
    for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// Workgroup minimum; the result is valid in thread 0.
__device__ inline double block_min(double v, double *lmin)
{
    v = wave_min(v);
    if ((threadIdx.x & (kWave - 1)) == 0) lmin[threadIdx.x / kWave] = v;
    __syncthreads();
    if (threadIdx.x == 0)
        for (int w = 1; w < kWaves; ++w) v = fmin(v, lmin[w]);
    return v;
}

// Workgroup minimum of an int, valid in every thread.
__device__ inline int block_min_int(int v, int *lint)
{
    for (int o = kWave / 2; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, kWave));
    __syncthreads();
    if ((threadIdx.x & (kWave - 1)) == 0) lint[threadIdx.x / kWave] = v;
    __syncthreads();
    for (int w = 0; w < kWaves; ++w) v = min(v, lint[w]);
    return v;
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

// The same over the running maxima of [bq, eq) staged in LDS (pm[u - bq]).
__device__ inline int insertion_point_lds(const float *pm, int bq, int eq, float slo)
{
    int lo = bq, hi = eq;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (pm[mid - bq] > slo)
            hi = mid;
        else
            lo = mid + 1;
    }
    return lo;
}

// The same, by the wavefront: 64 positions a read, the first whose running
// maximum is later by a ballot (long queues take the binary search).
__device__ inline int insertion_point_wave(const SRec *sr, int bq, int eq, float slo)
{
    if (eq - bq > 8 * kWave) return insertion_point(sr, bq, eq, slo);
    const int lane = threadIdx.x & (kWave - 1);
    for (int u0 = bq; u0 < eq; u0 += kWave) {
        const int u = u0 + lane;
        const bool later = u < eq && sr[u].pmax > slo;
        const uint64_t m = __builtin_amdgcn_ballot_w64(later);
        if (m) return u0 + (int)__builtin_ctzll(m);
    }
    return eq;
}

// The EDF position of queue [bq, eq) for a group with SLO slo: the insertion
// point among the groups after the head (the running maxima leave the head
// out), or the head of an empty queue.
__device__ inline int edf_point(const SRec *sr, int bq, int eq, float slo)
{
    return bq == eq ? bq : insertion_point(sr, bq + 1, eq, slo);
}

// (score, k) is better than (s2, k2): lower score, then lower k.  A NaN score
// is never better.
__device__ inline bool better(double s, int64_t k, double s2, int64_t k2)
{
    return s < s2 || (s == s2 && k < k2);
}

// Workgroup minimum of (score, k); the result is valid in thread 0.
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
        for (int w = 1; w < kWaves; ++w)
            if (better(ls[w], lk[w], s, k)) {
                s = ls[w];
                k = lk[w];
            }
    }
}

// The exact walk of nv positions by one wavefront (visit() in effect for each
// position in turn, with the same operations in the same order).  Position v
// holds the record rec(v); the sums start from r, which every lane holds, and
// end there.  64 positions at a time, one per lane: the running sums ripple
// from lane to lane (at each of up to 63 steps every lane takes its left
// neighbour's sum and adds its left neighbour's input), which forms each
// lane's sums in position order exactly as a serial walk does; then each lane
// forms its probability, and the terms ripple the same way.  A lane adds its
// own model-change and eviction costs to the costs it receives (adding a zero
// cost leaves a sum unchanged).  out(v, x, A, V, K, C, E) receives each
// position's sums on entry, its score ahead C and its E[W] (in the lane that
// holds the position).
// wave_walk_rounds takes each round's records from load(v0, on), called in
// every lane (on: the lane holds position v0 + lane), so that a loader can
// form them with wavefront operations.
template <class LoadRound, class Out>
__device__ void wave_walk_rounds(Run &r, int nv, const LoadRound &load, double theta, int cls,
                                 const SearchArgs &a, const Out &out)
{
    const int lane = threadIdx.x & (kWave - 1);
    const double ecost = (double)a.evict_cost;
    for (int v0 = 0; v0 < nv; v0 += kWave) {
        const int cnt = min(kWave, nv - v0);
        const bool on = lane < cnt;
        const SRec x = load(v0, on);
        const int m = (int)(x.nmf & 0xFFu);
        int pm = __shfl_up(m, 1, kWave);
        if (lane == 0) pm = r.prev;
        double c1 = 0.0;
        if (on && pm >= 0 && pm != m && a.swap_cost)
            c1 = (double)a.swap_cost[((int64_t)cls * a.M + pm) * a.M + m];
        const double c2 = (on && (x.nmf & kFlagBit)) ? ecost : 0.0;
        // inputs of the left neighbour (zero in lane 0, whose sums stay at r)
        const double la = from_left0(x.a);
        const double lb = from_left0(x.b);
        const double l1 = from_left0(c1);
        const double l2 = from_left0(c2);
        double A = r.A, V = r.V, K0 = r.K;     // K0: costs before this position's own
        // cnt - 1 steps, rounded up to blocks of 8 (a step past the last
        // position leaves every position's sums unchanged), the count in a
        // scalar register so that only a block ends in a branch
        const int steps = __builtin_amdgcn_readfirstlane(cnt - 1);
        for (int j = 0; j < steps; j += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                A = from_left(A) + la;
                V = from_left(V) + lb;
                K0 = (from_left(K0) + l1) + l2;
            }
        }
        double K = K0 + c1;
        K = K + c2;
        double term = 0.0, E = 0.0;
        if (on) {
            E = A / theta + K;
            const double SD = sqrt(V) / theta;
            const double slo = (double)x.slo;
            double P;
            if (SD > 0.0)
                P = 0.5 * erfc((slo - E) / (SD * 1.4142135623730951));
            else
                P = (E > slo) ? 1.0 : 0.0;
            term = (double)(x.nmf >> kCountShift) * P;
        }
        const double lt = from_left0(term);
        double C = r.sc;
        for (int j = 0; j < steps; j += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) C = from_left(C) + lt;
        }
        const int last = cnt - 1;
        r.A = lane_value(A, last) + lane_value(x.a, last);
        r.V = lane_value(V, last) + lane_value(x.b, last);
        r.K = lane_value(K, last);
        r.sc = lane_value(C, last) + lane_value(term, last);
        r.prev = __builtin_amdgcn_readlane(m, last);
        if (on) out(v0 + lane, x, A, V, K, C, E);
    }
}

// wave_walk takes position v's record from rec(v); the next round's records
// are read while a round ripples.
template <class RecOf, class Out>
__device__ void wave_walk(Run &r, int nv, const RecOf &rec, double theta, int cls,
                          const SearchArgs &a, const Out &out)
{
    const int lane = threadIdx.x & (kWave - 1);
    SRec nxt{};
    if (lane < nv) nxt = rec(lane);
    wave_walk_rounds(r, nv, [&](int v0, bool) {
        const SRec x = nxt;
        const int v1 = v0 + kWave + lane;
        nxt = SRec{};
        if (v1 < nv) nxt = rec(v1);
        return x;
    }, theta, cls, a, out);
}

struct NoOut {
    __device__ void operator()(int, const SRec &, double, double, double, double, double) const {}
};

// Plan score with queue g's score replaced by qg (queues summed in order).
__device__ inline double total_with(const double *T, const double *Q, int I, int g, double qg)
{
    double t = T[g] + qg;
    for (int q = g + 1; q < I; ++q) t += Q[q];
    return t;
}

// Plan score with queues g and h (g != h) replaced by rg and nh.
__device__ inline double total_with2(const double *T, const double *Q, int I, int g, double rg,
                                     int h, double nh)
{
    const int lo = g < h ? g : h;
    double t = T[lo];
    for (int q = lo; q < I; ++q) t += q == g ? rg : (q == h ? nh : Q[q]);
    return t;
}

// ---------------------------------------------------------------------------
// Set-up

// Group records, and each group's rank in (SLO, id) order.  A workgroup takes
// 64 groups; its four wavefronts count a quarter of the keys each.
// Group i's record: n mu and n var (exact products in double), SLO, and the
// request count with the model.
__device__ inline GRec group_record(const SearchArgs &a, int i)
{
    const uint32_t n = (uint32_t)clampi(a.grp_count[i], 0, (int)kCountMask);
    const double dn = (double)n;
    GRec r;
    r.a = dn * (double)a.grp_mu[i];
    r.b = dn * (double)a.grp_var[i];
    r.slo = a.grp_slo[i];
    r.nm = (n << kCountShift) | (uint32_t)clampi(a.grp_model[i], 0, a.M - 1);
    r.pad[0] = r.pad[1] = 0u;
    return r;
}

// Ranks in (SLO, id) order, counted: workgroup (tile t, block of 64 groups)
// counts, for each of its groups, the groups of tile t (kRankTile ids) that
// order before it, its four wavefronts a quarter of the tile each, and leaves
// the partial counts in rank_part[t][i].
__global__ __launch_bounds__(kThreads) void k_srank(SearchArgs a)
{
    __shared__ __align__(16) uint32_t keys[kRankTile];
    __shared__ int part[kThreads];
    const int G = a.G;
    const int nb = (G + kWave - 1) / kWave;
    const int gb = blockIdx.x % nb, tile = blockIdx.x / nb;
    const int li = threadIdx.x & (kWave - 1), quarter = threadIdx.x / kWave;
    const int i = gb * kWave + li;
    const uint32_t mine = i < G ? order_key(a.grp_slo[i]) : 0u;
    const int t0 = tile * kRankTile;
    for (int k = threadIdx.x; k < kRankTile; k += kThreads)
        keys[k] = t0 + k < G ? order_key(a.grp_slo[t0 + k]) : 0xFFFFFFFFu;
    __syncthreads();
    int cnt = 0;
    const int base = quarter * (kRankTile / kWaves);
#pragma unroll 4
    for (int k = 0; k < kRankTile / kWaves; k += 4) {
        const uint4 o = *reinterpret_cast<const uint4 *>(&keys[base + k]);
        const int id = t0 + base + k;          // ids past G hold the largest key
        cnt += (o.x < mine || (o.x == mine && id < i)) ? 1 : 0;
        cnt += (o.y < mine || (o.y == mine && id + 1 < i)) ? 1 : 0;
        cnt += (o.z < mine || (o.z == mine && id + 2 < i)) ? 1 : 0;
        cnt += (o.w < mine || (o.w == mine && id + 3 < i)) ? 1 : 0;
    }
    part[threadIdx.x] = cnt;
    __syncthreads();
    if (quarter == 0 && i < G)
        a.rank_part[(int64_t)tile * G + i] =
            part[li] + part[li + kWave] + part[li + 2 * kWave] + part[li + 3 * kWave];
}

// Group records, and each group at its rank (the sum of its partial counts)
// in the SLO order.
__global__ __launch_bounds__(kThreads) void k_srankout(SearchArgs a, int ntiles)
{
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= a.G) return;
    int r = 0;
    for (int t = 0; t < ntiles; ++t) r += a.rank_part[(int64_t)t * a.G + i];
    a.by_slo[r] = i;
    a.grec[i] = group_record(a, i);
}

// Group records only (when no screen runs).
__global__ __launch_bounds__(kThreads) void k_sgrec(SearchArgs a)
{
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= a.G) return;
    a.grec[i] = group_record(a, i);
}

// The normal-tail table, once per call, for the screens to copy into LDS.
__global__ __launch_bounds__(kThreads) void k_stail(SearchArgs a)
{
    __shared__ float2 tab[qlm_tail::kCells];
    qlm_tail::build<kThreads>(tab);
    __syncthreads();
    for (int k = threadIdx.x; k < qlm_tail::kCells; k += kThreads) a.tail[k] = tab[k];
}

// Start plans into the working copies; qoff is forced to a monotone split of
// [0, G] and group ids to [0, G) so that every later access stays in bounds.
__global__ __launch_bounds__(kThreads) void k_sload(SearchArgs a, qlm_plans pl)
{
    const int G = a.G, I = a.I;
    const int nblk = (G + kThreads - 1) / kThreads;
    const int64_t b = blockIdx.x / nblk;
    const int s = (blockIdx.x % nblk) * kThreads + threadIdx.x;
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

// The cache of one queue of one chain (one wavefront per queue).
__global__ __launch_bounds__(kThreads) void k_sstate(SearchArgs a, int force)
{
    const int I = a.I, G = a.G;
    const int nblk = (I + kWaves - 1) / kWaves;
    const int64_t b = blockIdx.x / nblk;
    const int g = (blockIdx.x % nblk) * kWaves + wave_id();
    const int lane = threadIdx.x & (kWave - 1);
    if (g >= I || (!force && a.done[b])) return;
    const int32_t *__restrict__ perm = a.perm + b * G;
    const uint8_t *__restrict__ flag = a.flag + b * G;
    SRec *__restrict__ sr = a.srec + b * G;
    SSt *__restrict__ ss = a.sst + b * G;
    TRec *__restrict__ tr = a.trec + b * G;
    int32_t *__restrict__ inv = a.inv + b * G;
    const int bq = a.qof[b * (I + 1) + g], eq = a.qof[b * (I + 1) + g + 1];
    const double theta = (double)a.inst_tput[g];
    const int cls = clampi(a.inst_class[g], 0, a.C - 1);
    const double vscale = qlm_tail::kVarScale / (theta * theta);
    // each round's slot records (with the running maximum of the SLOs) are
    // formed, stored, and walked at once: the exact running sums and the
    // screens' margins
    float pm = -INFINITY;
    auto load = [&](int v0, bool on) {
        const int u = bq + v0 + lane;
        SRec x{};
        float mx = -INFINITY;
        if (on) {
            const int i = perm[u];
            const GRec gr = a.grec[i];
            x.a = gr.a;
            x.b = gr.b;
            x.slo = gr.slo;
            x.nmf = gr.nm | (flag[u] ? kFlagBit : 0u);
            x.q = (uint32_t)g;
            mx = u == bq ? -INFINITY : gr.slo;     // the running head is never passed
            inv[i] = u;
        }
        for (int o = 1; o < kWave; o <<= 1) {
            const float y = __shfl_up(mx, o, kWave);
            if (lane >= o) mx = y > mx ? y : mx;
        }
        mx = pm > mx ? pm : mx;
        x.pmax = mx;
        if (on) sr[u] = x;
        pm = __shfl(mx, kWave - 1, kWave);
        return x;
    };
    Run r{0.0, 0.0, 0.0, 0.0, model0_of(a, g)};
    double nsum = 0.0, emax = 0.0;
    wave_walk_rounds(r, eq - bq, load, theta, cls, a,
              [&](int v, const SRec &x, double A, double V, double K, double C, double E) {
                  const int u = bq + v;
                  ss[u] = SSt{A, V, K, C};
                  const double slo = (double)x.slo;
                  TRec t;
                  t.m = slo - E;
                  t.vz = (float)(V * vscale);
                  t.n = (float)(x.nmf >> kCountShift);
                  tr[u] = t;
                  nsum += (double)(x.nmf >> kCountShift);
                  emax = fmax(emax, fabs(E) + fabs(slo));
              });
    nsum = wave_sum(nsum);
    emax = wave_max(emax);
    if (lane == 0) {
        a.Q[b * I + g] = r.sc;
        a.Nq[b * I + g] = nsum;
        a.Es[b * I + g] = emax;
    }
}

// Queue scores summed in queue order: the plan score (the scores are staged
// in LDS by all threads, then added in order by one).
__global__ __launch_bounds__(kThreads) void k_stotal(SearchArgs a, int force)
{
    __shared__ double q[kThreads];
    const int64_t b = blockIdx.x;
    if (!force && a.done[b]) return;
    const int I = a.I;
    const double *Q = a.Q + b * I;
    double *T = a.T + b * (I + 1);
    double t = 0.0;
    if (threadIdx.x == 0) T[0] = 0.0;
    for (int g0 = 0; g0 < I; g0 += kThreads) {
        if (g0 + (int)threadIdx.x < I) q[threadIdx.x] = Q[g0 + threadIdx.x];
        __syncthreads();
        if (threadIdx.x == 0) {
            const int n = min(kThreads, I - g0);
            for (int k = 0; k < n; ++k) {
                t += q[k];
                T[g0 + k + 1] = t;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) a.cur[b] = t;
}

// ---------------------------------------------------------------------------
// Exact scores of every move, one lane per move (qlm_search_moves)

__global__ __launch_bounds__(kThreads) void k_sswap(SearchArgs a)
{
    __shared__ double ls[kWaves];
    __shared__ int64_t lk[kWaves];
    const int64_t b = blockIdx.x / a.nwg_a;
    const int wg = blockIdx.x % a.nwg_a;
    if (a.done[b]) return;
    const int G = a.G, I = a.I, W = a.W;
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int t = wg * kThreads + threadIdx.x;
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
            if (s + d < eq && s != bq) {
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
    block_best(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        a.wmin_s[b * a.nwg + wg] = best;
        a.wmin_i[b * a.nwg + wg] = bk;
    }
}

__global__ __launch_bounds__(kThreads) void k_smove(SearchArgs a)
{
    __shared__ double ls[kWaves];
    __shared__ int64_t lk[kWaves];
    const int G = a.G, I = a.I;
    const int per_chain = I * a.nwg_b;
    const int64_t b = blockIdx.x / per_chain;
    const int h = (blockIdx.x % per_chain) / a.nwg_b;
    const int wg = blockIdx.x % a.nwg_b;
    if (a.done[b]) return;
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int r = wg * kThreads + threadIdx.x;
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    if (r < G) {
        const int i = a.by_slo[r];
        const int s = clampi(a.inv[b * G + i], 0, G - 1);
        const SRec x = sr[s];
        const int g = (int)x.q;
        const int64_t k = (int64_t)G * a.W + (int64_t)s * I + h;
        double score = INFINITY;
        if (g != h && s != qof[g]) {
            const int bq = qof[h], eq = qof[h + 1];
            const double theta = (double)a.inst_tput[h];
            const int cls = clampi(a.inst_class[h], 0, a.C - 1);
            Run w;
            if (bq == eq) {
                w = Run{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
                visit(w, x, theta, cls, a);
            } else {
                const int p = edf_point(sr, bq, eq, x.slo);
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
            score = total_with2(a.T + b * (I + 1), a.Q + b * I, I, g, a.R[b * G + s], h, w.sc);
            if (better(score, k, best, bk)) {
                best = score;
                bk = k;
            }
        }
        if (a.move_score) a.move_score[b * a.n_moves + k] = score;
    }
    block_best(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        const int64_t o = b * a.nwg + a.nwg_a + (int64_t)h * a.nwg_b + wg;
        a.wmin_s[o] = best;
        a.wmin_i[o] = bk;
    }
}

// RELOCATE(s, h): one lane per (slot s, queue h); the group goes first in h,
// flagged, and h's groups follow it in order (its own slot left out when h is
// its own queue).
__global__ __launch_bounds__(kThreads) void k_sreloc(SearchArgs a)
{
    __shared__ double ls[kWaves];
    __shared__ int64_t lk[kWaves];
    const int G = a.G, I = a.I;
    const int per_chain = I * a.nwg_b;
    const int64_t b = blockIdx.x / per_chain;
    const int h = (blockIdx.x % per_chain) / a.nwg_b;
    const int wg = blockIdx.x % a.nwg_b;
    if (a.done[b]) return;
    const SRec *__restrict__ sr = a.srec + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int s = wg * kThreads + threadIdx.x;
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    if (s < G) {
        SRec x = sr[s];
        const int g = (int)x.q;
        const int64_t k = (int64_t)G * a.W + (int64_t)G * I + (int64_t)s * I + h;
        const int bq = qof[h], eq = qof[h + 1];
        double score = INFINITY;
        if (s != qof[g] && bq < eq) {
            x.nmf |= kFlagBit;
            const double theta = (double)a.inst_tput[h];
            const int cls = clampi(a.inst_class[h], 0, a.C - 1);
            Run w{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
            visit(w, x, theta, cls, a);
            for (int u = bq; u < eq; ++u)
                if (u != s) visit(w, sr[u], theta, cls, a);
            score = g == h ? total_with(a.T + b * (I + 1), a.Q + b * I, I, g, w.sc)
                           : total_with2(a.T + b * (I + 1), a.Q + b * I, I, g, a.R[b * G + s], h,
                                         w.sc);
            if (better(score, k, best, bk)) {
                best = score;
                bk = k;
            }
        }
        if (a.move_score) a.move_score[b * a.n_moves + k] = score;
    }
    block_best(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        const int64_t o = b * a.nwg + a.nwg_a + (int64_t)(I + h) * a.nwg_b + wg;
        a.wmin_s[o] = best;
        a.wmin_i[o] = bk;
    }
}

// ---------------------------------------------------------------------------
// Screened steps

// The z error a margin error of eps_rel * scale may cause stays below kZErr
// when the scaled variance is at least the returned value (rsq of the scaled
// variance is in cells per second of margin).
__device__ inline double vz_floor(double eps_rel, double scale)
{
    // (a product with the constant's reciprocal: a quotient costs a dozen fp64
    // instructions, and the floor only needs to be right to an ulp)
    constexpr double kInvZ = 1.0 / (kZErr * qlm_tail::kScale);
    const double t = eps_rel * scale * kInvZ;
    return fmax(t * t, 1.1754943508222875e-38);
}

// Relative rounding of a margin formed from sums over a queue of L positions.
__device__ inline double margin_eps(int L) { return (8.0 + 2.0 * L) * 2.220446049250313e-16; }

// One position of a screened walk: the running sums as in visit(), then P from
// the tail table (or exactly [E > slo] where nothing ahead has variance, with
// E formed as the exact score forms it).  A position whose spread is too small
// for the rounding of its margin sets `force`.
__device__ inline void screen_visit(Run &r, const SRec &x, double theta, double inv_theta, int cls,
                                    double vscale, double eps_rel, const float2 *tab,
                                    const SearchArgs &a, bool &force, const float *swc = nullptr)
{
    const int m = (int)(x.nmf & 0xFFu);
    if (r.prev >= 0 && r.prev != m && a.swap_cost)
        r.K += (double)(swc ? swc : a.swap_cost)[((int64_t)cls * a.M + r.prev) * a.M + m];
    if (x.nmf & kFlagBit) r.K += (double)a.evict_cost;
    const double slo = (double)x.slo;
    double P;
    if (r.V == 0.0) {
        const double EW = r.A / theta + r.K;
        P = (EW > slo) ? 1.0 : 0.0;
    } else {
        const double EW = fma(r.A, inv_theta, r.K);
        const float vz = (float)(r.V * vscale);
        force = force || !((double)vz >= vz_floor(eps_rel, fabs(EW) + fabs(slo)));
        P = (double)qlm_tail::q_of(tab, (float)(slo - EW), vz);
    }
    r.sc += (double)(x.nmf >> kCountShift) * P;
    r.A += x.a;
    r.V += x.b;
    r.prev = m;
}

// The in-step walks read one tail record per position for a whole wavefront,
// at an address every lane shares, through the scalar cache (the records are
// not written while the screens run).
typedef const __attribute__((address_space(4))) TRec CTRec;
typedef const __attribute__((address_space(4))) SSt CSSt;

template <class T>
__device__ inline const __attribute__((address_space(4))) T *as_const(const T *p)
{
    return reinterpret_cast<const __attribute__((address_space(4))) T *>(
        reinterpret_cast<uintptr_t>(p));
}

// Sum over the positions u in [lo, hi) of each lane of n_u Q(z), the margin
// m_u - dE and the scaled variance either the cached one plus dvz or, with
// `exactv`, (V_u - db) vscale from the double-precision variances (which a
// removal needs: no cancellation).  The wavefront walks the union of its
// lanes' ranges in step.  Lanes with on = false add nothing.
template <class TrAt, class VAt>
__device__ inline double tail_walk(const TrAt &tr_at, const VAt &v_at, const float2 *tab, bool on,
                                   int lo, int hi, double dE, float dvz, double db, double vscale,
                                   bool exactv)
{
    const int ulo = __builtin_amdgcn_readfirstlane((int)wave_min(on ? (double)lo : 1e9));
    const int uhi = __builtin_amdgcn_readfirstlane((int)wave_max(on ? (double)hi : -1.0));
    double acc = 0.0;
    int u = ulo;
    if (exactv) {
        for (; u < uhi; u += 8) {
            float s32 = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int uu = min(u + j, uhi - 1);
                const TRec x = tr_at(uu);
                const double v = v_at(uu);
                const float q = qlm_tail::q_of(tab, (float)(x.m - dE), (float)((v - db) * vscale));
                const float w = (on && u + j >= lo && u + j < hi) ? x.n : 0.0f;
                s32 = fmaf(w, q, s32);
            }
            acc += (double)s32;
        }
    } else {
        for (; u < uhi; u += 8) {
            float s32 = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int uu = min(u + j, uhi - 1);
                const TRec x = tr_at(uu);
                const float q = qlm_tail::q_of(tab, (float)(x.m - dE), x.vz + dvz);
                const float w = (on && u + j >= lo && u + j < hi) ? x.n : 0.0f;
                s32 = fmaf(w, q, s32);
            }
            acc += (double)s32;
        }
    }
    return acc;
}

// Screened removals and SWAPs, one lane per task: tasks [0, G) are the
// queues of each slot s without s (which the MOVE screens of s take up),
// tasks G + s*W + d - 1 the moves SWAP(s, d).
__global__ __launch_bounds__(kThreads) void k_fswap(SearchArgs a)
{
    __shared__ float2 tab[qlm_tail::kCells];
    __shared__ double lmin[kWaves];
    __shared__ int lint_lo[kWaves], lint_hi[kWaves];
    // one buffer: first the slot records the lanes visit, then their tails
    // (records and variances ahead)
    __shared__ __align__(16) unsigned char stbuf[kSwapStageBytes];
    __shared__ float st_c[kSwapCostStage];
    SRec *st_r = reinterpret_cast<SRec *>(stbuf);
    TRec *st_t = reinterpret_cast<TRec *>(stbuf);
    double *st_v = reinterpret_cast<double *>(stbuf + kSwapStage * sizeof(TRec));
    const int64_t b = blockIdx.x / a.nwg_f;
    const int wg = blockIdx.x % a.nwg_f;
    if (a.done[b]) return;                    // the same in the whole workgroup
    const int G = a.G, I = a.I, W = a.W;
    const SRec *__restrict__ sr = a.srec + b * G;
    // the slots this workgroup's tasks visit, [vlo, vhi): removals t < G visit
    // t and t + 1, swaps s = (t - G) / W up to W + 1 past s; a workgroup can
    // hold both kinds
    const int t0 = wg * kThreads, t1 = min(t0 + kThreads, G + G * W) - 1;
    int vlo = G, vhi = 0;
    if (t0 < G) {
        vlo = t0;
        vhi = min(t1, G - 1) + 2;
    }
    if (t1 >= G) {
        vlo = min(vlo, (max(t0, G) - G) / W);
        vhi = max(vhi, (t1 - G) / W + W + 2);
    }
    vhi = min(vhi, G);
    const bool rec_lds = vhi - vlo <= kSwapRecs;
    const int ncost = a.swap_cost ? a.C * a.M * a.M : 0;
    const bool cost_lds = ncost <= kSwapCostStage;
    for (int k = threadIdx.x; k < qlm_tail::kCells; k += kThreads) tab[k] = a.tail[k];
    if (rec_lds)
        for (int u = vlo + (int)threadIdx.x; u < vhi; u += kThreads) st_r[u - vlo] = sr[u];
    if (cost_lds)
        for (int k = threadIdx.x; k < ncost; k += kThreads) st_c[k] = a.swap_cost[k];
    __syncthreads();
    auto rec = [&](int u) { return rec_lds ? st_r[u - vlo] : sr[u]; };
    const float *swc = cost_lds ? st_c : nullptr;
    const SSt *__restrict__ ss = a.sst + b * G;
    const TRec *__restrict__ tr = a.trec + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int t = wg * kThreads + threadIdx.x;
    const bool removal = t < G;
    const bool swap = !removal && t < G + G * W;
    const int s = removal ? t : (swap ? (t - G) / W : 0);
    const int d = swap ? (t - G) - s * W + 1 : 0;
    int g = 0, eq = 0, lo = 0;
    bool on = false, force = false, valid = false;
    double q = 0.0, dE = 0.0, db = 0.0, vscale = 0.0;
    if (removal || swap) {
        g = (int)min(rec(s).q, (uint32_t)(I - 1));
        const int bq = qof[g];
        eq = qof[g + 1];
        const double theta = (double)a.inst_tput[g];
        const double inv_theta = 1.0 / theta;
        vscale = qlm_tail::kVarScale / (theta * theta);
        const int cls = clampi(a.inst_class[g], 0, a.C - 1);
        const double eps = margin_eps(eq - bq);
        Run r = start_at(a, sr, ss, s, bq, g);
        if (removal) {
            // without s: the group after it moves up one position; past that the
            // queue is the old one less s's tokens and variance, with its costs
            // shifted
            valid = true;
            q = r.sc;
            if (s + 1 < eq) {
                screen_visit(r, rec(s + 1), theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
                q = r.sc;
                lo = s + 2;
                if (lo < eq) {
                    const SRec xs = rec(s);
                    dE = (r.K - ss[s + 1].K) - xs.a * inv_theta;
                    db = xs.b;
                    // the variance left ahead keeps most of its bits and a spread wide
                    // enough for the margin's rounding (both grow along the queue)
                    const double v0 = ss[lo].V, v1 = v0 - db;
                    force = force || !(v1 >= 0x1p-20 * v0) ||
                            !((double)(float)(v1 * vscale) >=
                              vz_floor(eps, a.Es[b * I + g] + fabs(dE)));
                    on = true;
                }
            }
        } else if (s + d < eq && s != bq) {
            valid = true;
            screen_visit(r, rec(s + d), theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
            for (int u = s + 1; u < s + d; ++u)
                screen_visit(r, rec(u), theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
            screen_visit(r, rec(s), theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
            q = r.sc;
            const int u1 = s + d + 1;
            if (u1 < eq) {
                screen_visit(r, rec(u1), theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
                q = r.sc;
                lo = u1 + 1;
                if (lo < eq) {
                    // past u1 the queue is the old one with its costs shifted by dK
                    const double dK = r.K - ss[u1].K;
                    force = force || !((double)tr[lo].vz >=
                                       vz_floor(eps, a.Es[b * I + g] + fabs(dK)));
                    if (dK == 0.0)
                        q += a.Q[b * I + g] - ss[lo].C;
                    else {
                        dE = dK;
                        on = true;
                    }
                }
            }
        }
    }
    const bool exactv = __ballot(on && removal) != 0;
    // the tails of the workgroup's lanes lie in one range of slots: staged in
    // LDS (records and variances ahead) when it fits, so that the walks read
    // no global memory
    const int wlo = block_min_int(on ? lo : INT_MAX, lint_lo);
    const int whi = -block_min_int(on ? -eq : 0, lint_hi);
    const bool staged = wlo < whi && whi - wlo <= kSwapStage;
    if (staged)
        for (int u = wlo + (int)threadIdx.x; u < whi; u += kThreads) {
            st_t[u - wlo] = tr[u];
            st_v[u - wlo] = ss[u].V;
        }
    __syncthreads();
    if (staged)
        q += tail_walk([&](int u) { return st_t[u - wlo]; }, [&](int u) { return st_v[u - wlo]; },
                       tab, on, lo, eq, dE, 0.0f, db, vscale, exactv);
    else
        q += tail_walk([&](int u) { return tr[u]; }, [&](int u) { return ss[u].V; }, tab, on, lo,
                       eq, dE, 0.0f, db, vscale, exactv);
    double F = INFINITY, D = 0.0;
    if (valid) {
        const double nq = a.Nq[b * I + g];
        if (removal) {
            a.R[b * G + s] = q;
            a.RD[b * G + s] = force ? INFINITY : kEpsP * nq + 1e-12 * (fabs(a.Q[b * I + g]) + nq);
        } else {
            const double cur = a.cur[b];
            F = cur - a.Q[b * I + g] + q;
            D = force ? INFINITY : kEpsP * nq + 1e-12 * (fabs(cur) + nq);
        }
    }
    if (swap) {
        const int64_t k = (int64_t)s * W + (d - 1);
        a.F[b * a.n_moves + k] = F;
        a.D[b * a.n_moves + k] = D;
    }
    const double m = block_min(F + D, lmin);
    if (threadIdx.x == 0) a.smin[b * a.nws + wg] = m;
}

// Screened MOVE and RELOCATE into another queue h: one workgroup per (target
// queue h, 256 groups adjacent in SLO order), each lane one group and both of
// its moves into h.  MOVE puts the group at its insertion point in h;
// RELOCATE puts it, flagged, at the head of h, ahead of the running group.
// Each lane scores each move's position and the position after it with
// running sums; past that, the queue is the old one shifted by the group's
// tokens, variance and the change of costs.  The whole wavefront walks those
// positions in step from the earliest of its lanes' tails, forming both
// moves' terms at each position (a lane's MOVE term only past its insertion
// point).
__device__ inline void fmove_body(const SearchArgs &a, int bid, float2 *tab, float *st_c,
                                  double *lmin, int *lint, TRec *stage)
{
    const int G = a.G, I = a.I;
    const int per_chain = I * a.nwg_b;
    const int64_t b = bid / per_chain;
    const int h = (bid % per_chain) / a.nwg_b;
    const int wg = bid % a.nwg_b;
    if (a.done[b]) return;                    // the same in the whole workgroup
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const TRec *__restrict__ tr = a.trec + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int bq = qof[h], eq = qof[h + 1];
    // the target queue's running SLO maxima, for the insertion points, share
    // the tail records' staging buffer (the tails are staged after a barrier)
    float *pmax = reinterpret_cast<float *>(stage);
    constexpr int kPmaxSlots = (int)(kStage * sizeof(TRec) / sizeof(float));
    const bool pm_lds = eq - bq <= kPmaxSlots;
    const int ncost = a.swap_cost ? a.C * a.M * a.M : 0;
    const bool cost_lds = ncost <= kSwapCostStage;
    for (int k = threadIdx.x; k < qlm_tail::kCells; k += kThreads) tab[k] = a.tail[k];
    if (pm_lds)
        for (int u = bq + (int)threadIdx.x; u < eq; u += kThreads) pmax[u - bq] = sr[u].pmax;
    if (cost_lds)
        for (int k = threadIdx.x; k < ncost; k += kThreads) st_c[k] = a.swap_cost[k];
    __syncthreads();
    const float *swc = cost_lds ? st_c : nullptr;
    const double theta = (double)a.inst_tput[h];
    const double inv_theta = 1.0 / theta;
    const double vscale = qlm_tail::kVarScale / (theta * theta);
    const int cls = clampi(a.inst_class[h], 0, a.C - 1);
    const double eps = margin_eps(eq - bq + 1);
    const double Qh = a.Q[b * I + h];
    const int r = wg * kThreads + threadIdx.x;
    bool valid_m = false, valid_r = false, tail_m = false, tail_r = false;
    bool force_m = false, force_r = false;
    int s = 0, g = 0, p = eq;
    double N_m = 0.0, N_r = 0.0, dE_m = 0.0, dE_r = 0.0;
    float dvz = 0.0f;
    if (r < G) {
        const int i = a.by_slo[r];
        s = clampi(a.inv[b * G + i], 0, G - 1);
        const SRec x = sr[s];
        g = (int)x.q;
        // a running group never moves; RELOCATE needs a group to evict
        valid_m = g != h && s != qof[g];
        valid_r = valid_m && bq < eq;
        dvz = (float)(x.b * vscale);
        if (valid_m) {
            Run w;
            if (bq == eq) {
                w = Run{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
                screen_visit(w, x, theta, inv_theta, cls, vscale, eps, tab, a, force_m, swc);
            } else {
                p = pm_lds ? insertion_point_lds(pmax + 1, bq + 1, eq, x.slo)   // pmax from bq
                           : insertion_point(sr, bq + 1, eq, x.slo);
                if (p == eq) {
                    const SSt t = ss[eq - 1];
                    const SRec y = sr[eq - 1];
                    w = Run{t.A + y.a, t.V + y.b, t.K, Qh, (int)(y.nmf & 0xFFu)};
                    screen_visit(w, x, theta, inv_theta, cls, vscale, eps, tab, a, force_m, swc);
                } else {
                    w = start_at(a, sr, ss, p, bq, h);
                    screen_visit(w, x, theta, inv_theta, cls, vscale, eps, tab, a, force_m, swc);
                    screen_visit(w, sr[p], theta, inv_theta, cls, vscale, eps, tab, a, force_m, swc);
                    const double dK = w.K - ss[p].K;
                    dE_m = x.a * inv_theta + dK;
                    tail_m = p + 1 < eq;
                    if (tail_m) {
                        const double floor = vz_floor(eps, a.Es[b * I + h] + fabs(dE_m));
                        force_m = force_m || !((double)(tr[p + 1].vz + dvz) >= floor);
                    }
                }
            }
            N_m = w.sc;
        }
        if (valid_r) {
            SRec xr = x;
            xr.nmf |= kFlagBit;
            Run w = start_at(a, sr, ss, bq, bq, h);
            screen_visit(w, xr, theta, inv_theta, cls, vscale, eps, tab, a, force_r, swc);
            screen_visit(w, sr[bq], theta, inv_theta, cls, vscale, eps, tab, a, force_r, swc);
            const double dK = w.K - ss[bq].K;
            dE_r = xr.a * inv_theta + dK;
            tail_r = bq + 1 < eq;
            if (tail_r) {
                const double floor = vz_floor(eps, a.Es[b * I + h] + fabs(dE_r));
                force_r = force_r || !((double)(tr[bq + 1].vz + dvz) >= floor);
            }
            N_r = w.sc;
        }
    }
    // the shifted tails: queue h's tail records pass through LDS in chunks
    // (every wavefront of the workgroup targets h); each wavefront walks its
    // lanes' tails in step from the earliest, a lane's MOVE terms masked
    // until its insertion point is passed (a RELOCATE's tail starts at the
    // first position after the head, where the walk starts)
    {
        const int lo_m = tail_m ? p + 1 : eq;
        const int lo = min(lo_m, tail_r ? bq + 1 : eq);
        const int ulo = __builtin_amdgcn_readfirstlane((int)wave_min((double)lo));
        const int umask = __builtin_amdgcn_readfirstlane(
            (int)wave_max(tail_m ? (double)lo_m : -1.0));        // from here no MOVE lane waits
        const int wlo = __builtin_amdgcn_readfirstlane(block_min_int(ulo, lint));   // the workgroup's earliest
        double acc_m = 0.0, acc_r = 0.0;
        for (int c0 = wlo; c0 < eq; c0 += kStage) {
            const int c1 = min(c0 + kStage, eq);
            __syncthreads();
            for (int u = c0 + (int)threadIdx.x; u < c1; u += kThreads) stage[u - c0] = tr[u];
            // seven blank records past the chunk (no requests, a finite margin
            // and variance): the unrolled walk reads up to seven past its end
            if (threadIdx.x < 7) stage[c1 - c0 + threadIdx.x] = TRec{0.0, 1.0f, 0.0f};
            __syncthreads();
            int u = max(c0, ulo);
            // masked part: some lanes' MOVE tails start later
            for (; u < c1 && u <= umask; ++u) {
                const TRec x = stage[u - c0];
                const float q_m = qlm_tail::q_of(tab, (float)(x.m - dE_m), x.vz + dvz);
                const float q_r = qlm_tail::q_of(tab, (float)(x.m - dE_r), x.vz + dvz);
                acc_m += (double)((tail_m && u > p) ? x.n * q_m : 0.0f);
                acc_r += (double)(x.n * q_r);
            }
            // every lane with a tail is in it now: blocks of eight records at
            // one address and fixed offsets
            for (; u < c1; u += 8) {
                const TRec *xs = stage + (u - c0);
                float s_m = 0.0f, s_r = 0.0f;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const TRec x = xs[j];
                    const float q_m = qlm_tail::q_of(tab, (float)(x.m - dE_m), x.vz + dvz);
                    const float q_r = qlm_tail::q_of(tab, (float)(x.m - dE_r), x.vz + dvz);
                    s_m = fmaf(x.n, q_m, s_m);
                    s_r = fmaf(x.n, q_r, s_r);
                }
                acc_m += (double)s_m;
                acc_r += (double)s_r;
            }
        }
        N_m += tail_m ? acc_m : 0.0;
        N_r += tail_r ? acc_r : 0.0;
    }
    double F_m = INFINITY, D_m = 0.0, F_r = INFINITY, D_r = 0.0;
    if (valid_m) {
        const double cur = a.cur[b];
        const double nq = a.Nq[b * I + h];
        const double base = a.R[b * G + s] - a.Q[b * I + g];
        const double rd = a.RD[b * G + s] + kEpsP * nq + 1e-12 * (fabs(cur) + nq);
        F_m = cur + base + (N_m - Qh);
        D_m = force_m ? INFINITY : rd;
        if (valid_r) {
            F_r = cur + base + (N_r - Qh);
            D_r = force_r ? INFINITY : rd;
        }
    }
    if (r < G) {
        const int64_t k = (int64_t)G * a.W + (int64_t)s * I + h;
        a.F[b * a.n_moves + k] = F_m;
        a.D[b * a.n_moves + k] = D_m;
        if (g != h) {                         // frel_body screens RELOCATE into the own queue
            a.F[b * a.n_moves + k + (int64_t)G * I] = F_r;
            a.D[b * a.n_moves + k + (int64_t)G * I] = D_r;
        }
    }
    const double m = block_min(fmin(F_m + D_m, F_r + D_r), lmin);
    if (threadIdx.x == 0) a.smin[b * a.nws + a.nwg_f + (int64_t)h * a.nwg_b + wg] = m;
}

// Screened RELOCATE within the group's own queue, one lane per slot s: the
// group goes first, flagged, then the evicted head; the groups between the
// head and s are the old ones shifted by the group's tokens, variance and the
// change of costs at the head; the position after s is formed afresh (its
// tokens and variance ahead are the old ones: the group is ahead of it either
// way); past it only the costs change.  Each wavefront stages the tail
// records of its queues in LDS when they fit (st: kRelStage per wavefront).
__device__ inline void frel_body(const SearchArgs &a, int bid, float2 *tab, float *st_c,
                                 double *lmin, TRec *stall)
{
    const int64_t b = bid / a.nwg_r;
    const int wg = bid % a.nwg_r;
    if (a.done[b]) return;                    // the same in the whole workgroup
    const int G = a.G, I = a.I;
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const TRec *__restrict__ tr = a.trec + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    TRec *st = stall + wave_id() * kRelStage;
    const int ncost = a.swap_cost ? a.C * a.M * a.M : 0;
    const bool cost_lds = ncost <= kSwapCostStage;
    for (int k = threadIdx.x; k < qlm_tail::kCells; k += kThreads) tab[k] = a.tail[k];
    if (cost_lds)
        for (int k = threadIdx.x; k < ncost; k += kThreads) st_c[k] = a.swap_cost[k];
    __syncthreads();
    const float *swc = cost_lds ? st_c : nullptr;
    const int s = wg * kThreads + threadIdx.x;
    bool valid = false, force = false, on1 = false, on2 = false;
    int g = 0, lo1 = 0, hi1 = 0, lo2 = 0, hi2 = 0;
    double q = 0.0, dE1 = 0.0, dE2 = 0.0, vscale = 0.0;
    float dvz1 = 0.0f;
    if (s < G) {
        SRec x = sr[s];
        g = (int)min(x.q, (uint32_t)(I - 1));
        const int bq = qof[g], eq = qof[g + 1];
        if (s > bq) {
            valid = true;
            x.nmf |= kFlagBit;
            const double theta = (double)a.inst_tput[g];
            const double inv_theta = 1.0 / theta;
            vscale = qlm_tail::kVarScale / (theta * theta);
            const int cls = clampi(a.inst_class[g], 0, a.C - 1);
            const double eps = margin_eps(eq - bq);
            const double es = a.Es[b * I + g];
            Run r{0.0, 0.0, 0.0, 0.0, model0_of(a, g)};
            screen_visit(r, x, theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
            screen_visit(r, sr[bq], theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
            q = r.sc;
            const double dK1 = r.K - ss[bq].K;
            if (bq + 1 < s) {
                dE1 = x.a * inv_theta + dK1;
                dvz1 = (float)(x.b * vscale);
                lo1 = bq + 1;
                hi1 = s;
                on1 = true;
                force = force || !((double)(tr[lo1].vz + dvz1) >= vz_floor(eps, es + fabs(dE1)));
            }
            if (s + 1 < eq) {
                const SSt t = ss[s + 1];
                const SRec y = sr[s - 1];
                Run r2{t.A, t.V, s - 1 == bq ? r.K : ss[s - 1].K + dK1, 0.0,
                       (int)(y.nmf & 0xFFu)};
                // its sums ahead come from the cache, not from the exact walk's
                // order: an indicator (nothing ahead with variance) is not trusted
                force = force || !(t.V > 0.0);
                screen_visit(r2, sr[s + 1], theta, inv_theta, cls, vscale, eps, tab, a, force, swc);
                q += r2.sc;
                const double dK2 = r2.K - t.K;
                if (s + 2 < eq) {
                    lo2 = s + 2;
                    hi2 = eq;
                    force = force || !((double)tr[lo2].vz >= vz_floor(eps, es + fabs(dK2)));
                    if (dK2 == 0.0)
                        q += a.Q[b * I + g] - ss[lo2].C;
                    else {
                        dE2 = dK2;
                        on2 = true;
                    }
                }
            }
        }
    }
    // the positions the wavefront walks, staged in LDS when they fit
    const int wlo = __builtin_amdgcn_readfirstlane((int)wave_min(
        on1 ? (double)lo1 : (on2 ? (double)lo2 : 1e9)));
    const int whi = __builtin_amdgcn_readfirstlane((int)wave_max(
        on2 ? (double)hi2 : (on1 ? (double)hi1 : -1.0)));
    const bool staged = wlo < whi && whi - wlo <= kRelStage;
    if (staged)
        for (int u = wlo + (int)(threadIdx.x & (kWave - 1)); u < whi; u += kWave)
            st[u - wlo] = tr[u];
    __syncthreads();
    auto v_at = [&](int u) { return ss[u].V; };    // (not read: exactv is off)
    if (staged) {
        auto st_at = [&](int u) { return st[u - wlo]; };
        q += tail_walk(st_at, v_at, tab, on1, lo1, hi1, dE1, dvz1, 0.0, vscale, false);
        q += tail_walk(st_at, v_at, tab, on2, lo2, hi2, dE2, 0.0f, 0.0, vscale, false);
    } else {
        auto tr_at = [&](int u) { return tr[u]; };
        q += tail_walk(tr_at, v_at, tab, on1, lo1, hi1, dE1, dvz1, 0.0, vscale, false);
        q += tail_walk(tr_at, v_at, tab, on2, lo2, hi2, dE2, 0.0f, 0.0, vscale, false);
    }
    double F = INFINITY, D = 0.0;
    if (valid) {
        const double cur = a.cur[b];
        const double nq = a.Nq[b * I + g];
        F = cur - a.Q[b * I + g] + q;
        D = force ? INFINITY : kEpsP * nq + 1e-12 * (fabs(cur) + nq);
    }
    if (s < G) {
        const int64_t k = (int64_t)G * a.W + (int64_t)G * I + (int64_t)s * I + g;
        a.F[b * a.n_moves + k] = F;
        a.D[b * a.n_moves + k] = D;
    }
    const double m = block_min(F + D, lmin);
    if (threadIdx.x == 0) a.smin[b * a.nws + a.nwg_f + (int64_t)I * a.nwg_b + wg] = m;
}

// The screens of moves into another queue and of relocations, in one launch
// (more wavefronts to hide each one's set-up; the short own-queue relocation
// screens run beside the long ones).  Per launch: nwg_r * B workgroups screen
// the relocations within a queue, then I * nwg_b * B the MOVEs and RELOCATEs
// into another queue.
// (six wavefronts per SIMD: the compiler keeps it within 80 registers, and
// more wavefronts cover the lanes' chain of dependent reads before the walk)
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(6))) void k_fmove(
    SearchArgs a)
{
    __shared__ float2 tab[qlm_tail::kCells];
    __shared__ double lmin[kWaves];
    __shared__ int lint[kWaves];
    // (the move screens stage kStage records and seven blank ones)
    static_assert(kWaves * kRelStage >= kStage + 7, "the screens' staging buffer");
    __shared__ TRec stage[kWaves * kRelStage];
    __shared__ float st_c[kSwapCostStage];    // the swap costs, when they fit
    const int nrel = (int)((int64_t)a.nwg_r * a.B);
    const int bid = (int)blockIdx.x;
    if (bid < nrel)
        frel_body(a, bid, tab, st_c, lmin, stage);
    else
        fmove_body(a, bid - nrel, tab, st_c, lmin, lint, stage);
}

// The bound of the chain's lowest exact score, min(F + D); the candidate list
// starts empty.
__global__ __launch_bounds__(kThreads) void k_sbound(SearchArgs a)
{
    __shared__ double lmin[kWaves];
    const int64_t b = blockIdx.x;
    if (a.done[b]) return;
    double m = INFINITY;
    for (int w = threadIdx.x; w < a.nws; w += kThreads) m = fmin(m, a.smin[b * a.nws + w]);
    m = block_min(m, lmin);
    if (threadIdx.x == 0) {
        a.U[b] = m;
        a.ncand[b] = 0;
    }
}

// Candidates: moves whose exact score may be the lowest and below the plan's.
__global__ __launch_bounds__(kThreads) void k_sselect(SearchArgs a)
{
    const int nblk = (int)((a.n_moves + kThreads - 1) / kThreads);
    const int64_t b = blockIdx.x / nblk;
    if (a.done[b]) return;
    const int64_t k = (int64_t)(blockIdx.x % nblk) * kThreads + threadIdx.x;
    bool c = false;
    if (k < a.n_moves) {
        const double lo = a.F[b * a.n_moves + k] - a.D[b * a.n_moves + k];
        c = lo <= a.U[b] && lo < a.cur[b];
    }
    const uint64_t mask = __ballot(c);
    if (!mask) return;
    const int lane = threadIdx.x & (kWave - 1);
    int base = 0;
    if (lane == 0) base = atomicAdd(&a.ncand[b], __popcll(mask));
    base = __shfl(base, 0, kWave);
    if (c) {
        const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        a.cand[b * a.n_moves + base + below] = (int32_t)k;
    }
}

// Exact scores of the candidates, two wavefronts per candidate: a move into
// another queue walks the target queue (the first wavefront) and the source
// queue from the moved slot on (the second) side by side, and the first adds
// the two into the plan score; a move within one queue is one walk (the second
// idles).  Every walk is the one a single wavefront made in turn, so the
// scores do not change.
__global__ __launch_bounds__(kThreads) void k_sexact(SearchArgs a)
{
    __shared__ double src_part[kWaves];
    const int64_t b = blockIdx.x / kExactBlocks;
    if (a.done[b]) return;
    const int G = a.G, I = a.I, W = a.W;
    const SRec *__restrict__ sr = a.srec + b * G;
    const SSt *__restrict__ ss = a.sst + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const double *T = a.T + b * (I + 1);
    const double *Q = a.Q + b * I;
    const int nc = a.ncand[b];
    const int lane = threadIdx.x & (kWave - 1);
    constexpr int kPairs = kWaves / 2;
    const int pair = wave_id() >> 1;
    const bool second = (wave_id() & 1) != 0;
    // (the loop's trip count is the same in the whole workgroup: barriers)
    for (int c0 = (int)(blockIdx.x % kExactBlocks) * kPairs; c0 < nc;
         c0 += kExactBlocks * kPairs) {
        const int c = c0 + pair;
        double score = INFINITY;              // for a number that names no move
        bool two = false;                     // a move into another queue
        int g2 = 0, h2 = 0;
        double nh2 = 0.0;                     // (first wavefront) the target queue's sum
        double mine = 0.0;                    // (second wavefront) the source queue's sum
        if (c < nc) {
            const int64_t k = __builtin_amdgcn_readfirstlane(a.cand[b * a.n_moves + c]);
            if (k < (int64_t)G * W) {
                const int s = (int)(k / W), d = (int)(k % W) + 1;
                const int g = (int)sr[s].q;
                const int bq = qof[g], eq = qof[g + 1];
                if (!(s + d >= eq || s == bq) && !second) {
                    Run r = start_at(a, sr, ss, s, bq, g);
                    wave_walk(r, eq - s,
                              [&](int v) { return sr[v == 0 ? s + d : (v == d ? s : s + v)]; },
                              (double)a.inst_tput[g], clampi(a.inst_class[g], 0, a.C - 1), a,
                              NoOut{});
                    score = total_with(T, Q, I, g, r.sc);
                }
            } else if (k >= (int64_t)G * W + (int64_t)G * I) {
                // RELOCATE(s, h): the group first in h, flagged, then h's groups
                const int64_t rr = k - (int64_t)G * W - (int64_t)G * I;
                const int s = (int)(rr / I), h = (int)(rr % I);
                SRec x = sr[s];
                x.nmf |= kFlagBit;
                const int g = (int)x.q;
                const int bq = qof[h], eq = qof[h + 1];
                if (!(s == qof[g] || bq == eq)) {
                    const double theta = (double)a.inst_tput[h];
                    const int cls = clampi(a.inst_class[h], 0, a.C - 1);
                    Run r{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
                    if (g == h) {
                        if (!second) {
                            wave_walk(r, eq - bq, [&](int v) {
                                return v == 0 ? x : (bq + v - 1 < s ? sr[bq + v - 1] : sr[bq + v]);
                            }, theta, cls, a, NoOut{});
                            score = total_with(T, Q, I, g, r.sc);
                        }
                    } else {
                        two = true;
                        g2 = g;
                        h2 = h;
                        if (!second) {
                            wave_walk(r, eq - bq + 1, [&](int v) { return v == 0 ? x : sr[bq + v - 1]; },
                                      theta, cls, a, NoOut{});
                            nh2 = r.sc;
                        } else {
                            const int bg = qof[g], eg = qof[g + 1];
                            Run rg = start_at(a, sr, ss, s, bg, g);
                            wave_walk(rg, eg - s - 1, [&](int v) { return sr[s + 1 + v]; },
                                      (double)a.inst_tput[g], clampi(a.inst_class[g], 0, a.C - 1),
                                      a, NoOut{});
                            mine = rg.sc;
                        }
                    }
                }
            } else {
                const int64_t rr = k - (int64_t)G * W;
                const int s = (int)(rr / I), h = (int)(rr % I);
                const SRec x = sr[s];
                const int g = (int)x.q;
                if (!(g == h || s == qof[g])) {
                    two = true;
                    g2 = g;
                    h2 = h;
                    if (!second) {
                        const int bq = qof[h], eq = qof[h + 1];
                        const double theta = (double)a.inst_tput[h];
                        const int cls = clampi(a.inst_class[h], 0, a.C - 1);
                        Run r;
                        if (bq == eq) {
                            r = Run{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
                            wave_walk(r, 1, [&](int) { return x; }, theta, cls, a, NoOut{});
                        } else {
                            const int p = edf_point(sr, bq, eq, x.slo);
                            if (p == eq) {
                                r = start_at(a, sr, ss, eq - 1, bq, h);
                                wave_walk(r, 2, [&](int v) { return v == 0 ? sr[eq - 1] : x; }, theta,
                                          cls, a, NoOut{});
                            } else {
                                r = start_at(a, sr, ss, p, bq, h);
                                wave_walk(r, eq - p + 1,
                                          [&](int v) { return v == 0 ? x : sr[p + v - 1]; }, theta,
                                          cls, a, NoOut{});
                            }
                        }
                        nh2 = r.sc;
                    } else {
                        const int bg = qof[g], eg = qof[g + 1];
                        Run rg = start_at(a, sr, ss, s, bg, g);
                        wave_walk(rg, eg - s - 1, [&](int v) { return sr[s + 1 + v]; },
                                  (double)a.inst_tput[g], clampi(a.inst_class[g], 0, a.C - 1), a,
                                  NoOut{});
                        mine = rg.sc;
                    }
                }
            }
        }
        if (second && lane == 0) src_part[wave_id()] = mine;
        __syncthreads();
        if (!second && c < nc) {
            if (two) score = total_with2(T, Q, I, g2, src_part[wave_id() + 1], h2, nh2);
            if (lane == 0) a.cex[b * a.n_moves + c] = score;
        }
        __syncthreads();
    }
}

#pragma clang fp contract(on)

// Moves the group at slot s of chain b to queue h, at insertion point p_known
// (by default its EDF position after h's head: a reassignment, or with h its
// own queue a re-insertion; a relocation passes h's head slot and `evict`,
// which sets the group's flag): the slots between its old and new place
// rotate by one (with the slot index of each group moved), and the queue
// offsets between the two queues shift.  Run by a whole workgroup.
__device__ void place_apply(const SearchArgs &a, int64_t b, int s, int h, int p_known = -1,
                            int g_known = -1, bool evict = false)
{
    // the slots that move, staged in LDS when they fit (else in the workspace)
    __shared__ int32_t st_perm[kStageSlots];
    __shared__ uint8_t st_flag[kStageSlots];
    const int G = a.G, I = a.I;
    int32_t *perm = a.perm + b * G;
    uint8_t *flag = a.flag + b * G;
    int32_t *qof = a.qof + b * (I + 1);
    int32_t *inv = a.inv + b * G;
    const SRec *sr = a.srec + b * G;
    const int g = g_known >= 0 ? g_known : (int)sr[s].q;
    const int p = p_known >= 0 ? p_known : edf_point(sr, qof[h], qof[h + 1], sr[s].slo);
    // left: the group goes later (to slot p - 1); right: earlier (to slot p)
    const bool left = h > g || (h == g && p > s);
    const int lo = left ? s : p;
    const int hi = left ? p - 1 : s;
    if (hi - lo < kStageSlots) {
        // 16 reads in flight per thread before any is stored: the slots
        // between two far queues are thousands
        constexpr int kBatch = 16;
        for (int u0 = lo + (int)threadIdx.x; u0 <= hi; u0 += kBatch * kThreads) {
            int32_t pv[kBatch];
            uint8_t fv[kBatch];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int u = u0 + j * kThreads;
                if (u <= hi) {
                    pv[j] = perm[u];
                    fv[j] = flag[u];
                }
            }
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int u = u0 + j * kThreads;
                if (u <= hi) {
                    st_perm[u - lo] = pv[j];
                    st_flag[u - lo] = fv[j];
                }
            }
        }
        __syncthreads();
        for (int u = lo + threadIdx.x; u <= hi; u += kThreads) {
            const int v = left ? (u == hi ? s : u + 1) : (u == lo ? s : u - 1);
            const int32_t i = st_perm[v - lo];
            perm[u] = i;
            flag[u] = st_flag[v - lo];
            inv[clampi(i, 0, G - 1)] = u;
        }
    } else {
        int32_t *sp = a.scratch + b * 2 * G;
        int32_t *sf = sp + G;
        for (int u = lo + threadIdx.x; u <= hi; u += kThreads) {
            sp[u] = perm[u];
            sf[u] = flag[u];
        }
        __syncthreads();
        for (int u = lo + threadIdx.x; u <= hi; u += kThreads) {
            const int v = left ? (u == hi ? s : u + 1) : (u == lo ? s : u - 1);
            const int32_t i = sp[v];
            perm[u] = i;
            flag[u] = (uint8_t)sf[v];
            inv[clampi(i, 0, G - 1)] = u;
        }
    }
    if (h > g) {
        for (int q = g + 1 + threadIdx.x; q <= h; q += kThreads) qof[q] -= 1;
    } else if (h < g) {
        for (int q = h + 1 + threadIdx.x; q <= g; q += kThreads) qof[q] += 1;
    }
    if (evict) {
        __syncthreads();                     // every slot of the rotation written
        if (threadIdx.x == 0) flag[left ? p - 1 : p] = 1;
    }
}

// The lowest exact score among the candidates (lowest k on ties); applied when
// it improves on the plan.
__global__ __launch_bounds__(kThreads) void k_spick(SearchArgs a, int step)
{
    __shared__ double ls[kWaves];
    __shared__ int64_t lk[kWaves];
    __shared__ int apply;
    __shared__ int64_t kk;
    const int64_t b = blockIdx.x;
    if (a.done[b]) return;
    const int G = a.G, I = a.I, W = a.W;
    const int nc = a.ncand[b];
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    for (int c = threadIdx.x; c < nc; c += kThreads) {
        const double s = a.cex[b * a.n_moves + c];
        const int64_t k = a.cand[b * a.n_moves + c];
        if (better(s, k, best, bk)) {
            best = s;
            bk = k;
        }
    }
    block_best(best, bk, ls, lk);
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
    if (r < (int64_t)G * I) {
        place_apply(a, b, (int)(r / I), (int)(r % I));
    } else {
        const int s = (int)((r - (int64_t)G * I) / I), h = (int)((r - (int64_t)G * I) % I);
        place_apply(a, b, s, h, a.qof[b * (I + 1) + h], -1, true);
    }
}

// Final plans to the caller's slot-major arrays, with their scores and steps.
__global__ __launch_bounds__(kThreads) void k_sout(SearchArgs a, qlm_plans_out out,
                                                   double *score, int32_t *steps)
{
    const int G = a.G, I = a.I;
    const int64_t B = a.B;
    const int nw = (G + 31) >> 5;
    const int64_t rows = (int64_t)G + (I + 1) + (out.evict_bits ? nw : 0) + 1;
    for (int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x; x < rows * B;
         x += (int64_t)gridDim.x * kThreads) {
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
// Placement of one group (qlm_place_group)

#pragma clang fp contract(off)

// Exact score of each plan with its group `group` at each of its 2I places:
// c < I the EDF position of queue c after its head (as the queue stands
// without the group), c >= I the head of the non-empty queue c - I with the
// group flagged.  One wavefront per (chain, w), w in [0, 2I]: w < I the place
// c = w, w = I the group's own queue without it (which every other queue's
// score shares, in U), w > I the place c = w - 1.  Each place is scored as
// the score of the queue that receives the group (its own queue without it
// and with it, or queue h with it); k_place_pick completes the plan scores.
// The walks read the plan itself (group ids, flags, group records): a
// placement session keeps only the plan, the slot of every group and the
// queue scores up to date between its steps.  A group at its queue's head is
// running and is not placed (k_place_pick keeps the plan).
__global__ __launch_bounds__(kThreads) void k_place_eval(SearchArgs a, int group)
{
    const int G = a.G, I = a.I;
    const int nblk = (2 * I + 1 + kWaves - 1) / kWaves;
    const int64_t b = blockIdx.x / nblk;
    const int w = (blockIdx.x % nblk) * kWaves + wave_id();
    if (w > 2 * I) return;
    const int32_t *__restrict__ perm = a.perm + b * G;
    const uint8_t *__restrict__ flag = a.flag + b * G;
    const int32_t *__restrict__ qof = a.qof + b * (I + 1);
    const int lane = threadIdx.x & (kWave - 1);
    const int s = __builtin_amdgcn_readfirstlane(clampi(a.inv[b * G + group], 0, G - 1));
    // the group's queue: the last g with qof[g] <= s
    int g = 0;
    {
        int lo = 0, hi = I - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (qof[mid] <= s)
                lo = mid;
            else
                hi = mid - 1;
        }
        g = __builtin_amdgcn_readfirstlane(lo);
    }
    const int bg = clampi(qof[g], 0, G);
    const bool lead = lane == 0;
    if (w == I && lead) {
        a.dq[b * 4] = s;
        a.dq[b * 4 + 1] = g;
        a.dq[b * 4 + 2] = s == bg;             // running: it stays
    }
    if (s == bg) return;                       // running: it stays
    auto rec_at = [&](int u) __attribute__((always_inline)) {
        const GRec gr = a.grec[clampi(perm[u], 0, G - 1)];
        SRec x{};
        x.a = gr.a;
        x.b = gr.b;
        x.slo = gr.slo;
        x.nmf = gr.nm | (flag[u] ? kFlagBit : 0u);
        return x;
    };
    SRec x = rec_at(s);
    // the place: w = I its own queue without it; else queue h, the group at the
    // head (flagged) or at its EDF position
    const int c = w < I ? w : w - 1;
    const bool head = w != I && c >= I;
    const int h = w == I ? g : (head ? c - I : c);
    const int bq = clampi(qof[h], 0, G), eq = clampi(qof[h + 1], bq, G);
    const bool own = h == g;
    const int L = eq - bq - (own ? 1 : 0);     // the queue's positions without the group
    auto src = [&](int v) __attribute__((always_inline)) {
        return bq + v + (own && bq + v >= s ? 1 : 0);
    };
    auto raw = [&](int v) __attribute__((always_inline)) { return rec_at(src(v)); };
    const double theta = (double)a.inst_tput[h];
    const int cls = clampi(a.inst_class[h], 0, a.C - 1);
    Run r{0.0, 0.0, 0.0, 0.0, model0_of(a, h)};
    if (w == I) {
        wave_walk(r, L, raw, theta, cls, a, NoOut{});
        if (lead) a.U[b] = r.sc;
        return;
    }
    double score = INFINITY;
    int p = bq;                                // insertion slot, in the plan as it stands
    int ip = 0;                                // the group's position in the walk
    if (head) {
        // at the head, ahead of the running group (an empty queue has none to
        // evict: no place)
        x.nmf |= kFlagBit;
    } else {
        // the EDF position: before the first group after the head whose SLO
        // is strictly later (position ip of the queue without the group)
        ip = L;
        for (int v0 = 0; v0 < L; v0 += kWave) {
            const int v = v0 + lane;
            const uint64_t m =
                __builtin_amdgcn_ballot_w64(v >= 1 && v < L && raw(min(v, L - 1)).slo > x.slo);
            if (m) {
                ip = v0 + (int)__builtin_ctzll(m);
                break;
            }
        }
        ip = __builtin_amdgcn_readfirstlane(ip);
        p = ip < L ? src(ip) : eq;
    }
    if (!head || L > 0) {
        wave_walk(r, L + 1, [&](int v) { return v == ip ? x : raw(v < ip ? v : v - 1); }, theta,
                  cls, a, NoOut{});
        score = r.sc;
    }
    if (lead) {
        a.cex[b * a.n_moves + c] = score;      // completed by k_place_pick
        a.cand[b * a.n_moves + c] = p;         // the insertion point, for the pick
    }
}

#pragma clang fp contract(on)

// The place with the lowest exact score (lowest c on ties), applied; a running
// group stays, and the plan keeps its score.  The plan's queue scores are
// summed here, in queue order (the running sums the totals need).
__global__ __launch_bounds__(kThreads) void k_place_pick(SearchArgs a, int32_t *queue,
                                                         double *score)
{
    __shared__ double ls[kWaves];
    __shared__ int64_t lk[kWaves];
    __shared__ int64_t kk;
    __shared__ int kp, kg, stay;
    // the queue scores and their running sums, staged for the totals
    __shared__ double sT[kMaxSearchInstances + 1], sQ[kMaxSearchInstances];
    __shared__ int scand[kThreads];
    __shared__ double scex[kThreads];
    const int64_t b = blockIdx.x;
    const int G = a.G, I = a.I;
    const int n = 2 * I;
    // every independent load at once: the queue scores, the moved group's
    // slot and queue, and (up to kThreads places) each thread's candidate
    // score and insertion point
    const bool one = n <= kThreads;
    double v1 = 0.0;
    if (one && threadIdx.x < n) {
        v1 = a.cex[b * a.n_moves + threadIdx.x];
        scex[threadIdx.x] = v1;
        scand[threadIdx.x] = a.cand[b * a.n_moves + threadIdx.x];
    }
    for (int q = threadIdx.x; q < I; q += kThreads) sQ[q] = a.Q[b * I + q];
    const int s0 = clampi(a.dq[b * 4], 0, G - 1);
    const int g0 = clampi(a.dq[b * 4 + 1], 0, I - 1);
    if (threadIdx.x == 0) {
        kg = g0;
        stay = a.dq[b * 4 + 2];
    }
    __syncthreads();
    // the running sums of the queue scores, in queue order (the additions of a
    // serial sum, rippled across the first wavefront's lanes)
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        double carry = 0.0;
        if (lane == 0) sT[0] = 0.0;
        for (int q0 = 0; q0 < I; q0 += kWave) {
            const int cnt = min(kWave, I - q0);
            const double x = lane < cnt ? sQ[q0 + lane] : 0.0;
            const double lx = from_left0(x);
            double t = carry;
            const int steps = __builtin_amdgcn_readfirstlane(cnt - 1);
            for (int j = 0; j < steps; j += 8) {
#pragma unroll
                for (int u = 0; u < 8; ++u) t = from_left(t) + lx;
            }
            const double t1 = t + x;
            if (lane < cnt) sT[q0 + lane + 1] = t1;
            carry = lane_value(t1, cnt - 1);
        }
    }
    __syncthreads();
    if (stay) {
        if (threadIdx.x == 0) {
            a.cur[b] = sT[I];
            if (queue) queue[b] = g0;
            if (score) score[b] = sT[I];
        }
        return;
    }
    const double *T = sT;
    const double *Q = sQ;
    const double rg = a.U[b];
    double best = INFINITY;
    int64_t bk = INT64_MAX;
    // a place's plan score: its queue's new score (the candidate's) with the
    // group's own queue without it, the other queues as they stand
    auto total = [&](int c, double v) __attribute__((always_inline)) {
        const int h = c < I ? c : c - I;
        return h != g0 ? total_with2(T, Q, I, g0, rg, h, v) : total_with(T, Q, I, g0, v);
    };
    for (int c = threadIdx.x; c < n; c += kThreads) {
        const double v = total(c, one ? v1 : a.cex[b * a.n_moves + c]);
        if (better(v, c, best, bk)) {
            best = v;
            bk = c;
        }
    }
    block_best(best, bk, ls, lk);
    if (threadIdx.x == 0) {
        const bool none = bk < 0 || bk >= n;
        if (none) bk = 0;                         // every score NaN: the first place
        kk = bk;
        const double vq = one ? scex[bk] : a.cex[b * a.n_moves + bk];   // its queue's new score
        const double cur = none ? total((int)bk, vq) : best;
        a.cur[b] = cur;
        if (queue) queue[b] = (int32_t)bk;
        if (score) score[b] = cur;
        const int h = (int)(bk < I ? bk : bk - I);
        kp = clampi(one ? scand[bk] : a.cand[b * a.n_moves + bk], 0, G);
        // the queue scores of the plan after the move
        if (h != g0) {
            a.Q[b * I + g0] = rg;
            a.Q[b * I + h] = vq;
        } else {
            a.Q[b * I + g0] = vq;
        }
    }
    __syncthreads();
    const int c = (int)kk;
    place_apply(a, b, s0, c < I ? c : c - I, kp, kg, c >= I);
}

// ---------------------------------------------------------------------------
// Seed plans: groups taken in EDF order (SLO, id) or grouped by model (model,
// SLO, id), each appended to the queue whose drain time after taking it,
// (A_q + n mu) / Theta_q + (K_q + model-change cost), is smallest (the lowest
// queue on ties).  No evictions.

constexpr int kMaxSeeds = 64;
constexpr size_t kSeedSwapLds = 48 * 1024;     // largest swap table staged in LDS

struct SeedArgs {
    int32_t G, I, M, C;
    const int32_t *grp_count;
    const float *grp_mu, *grp_slo;
    const int32_t *grp_model;
    const float *inst_tput;
    const int32_t *inst_class, *inst_model0;
    const float *swap_cost;
    int32_t n;                    // seeds
    int32_t swap_in_lds;          // the swap table is staged in LDS
    int8_t policy[kMaxSeeds];     // 0 EDF, 1 grouped
    int32_t *order, *owner, *pos; // [n][G]: groups in order, their queue and position
    int32_t *qcount;              // [n][I]
    qlm_plans_out out;
};

// Order key of group i: model (when grouping), then the SLO as a number (-0
// counts as +0); ties go to the lower id.
__device__ inline uint64_t seed_key(const SeedArgs &a, int pol, int i)
{
    float f = a.grp_slo[i];
    if (f == 0.0f) f = 0.0f;
    const uint64_t hi = pol == 1 ? (uint64_t)(uint32_t)a.grp_model[i] : 0u;
    return (hi << 32) | order_key(f);
}

// Each group's rank in its seed's order (grid: 64 groups x seeds).
__global__ __launch_bounds__(kThreads) void k_seedrank(SeedArgs a)
{
    __shared__ uint64_t keys[kRankTile];
    __shared__ int part[kThreads];
    const int seed = blockIdx.y;
    const int pol = a.policy[seed];
    const int G = a.G;
    const int li = threadIdx.x & (kWave - 1), quarter = threadIdx.x / kWave;
    const int i = blockIdx.x * kWave + li;
    const uint64_t mine = i < G ? seed_key(a, pol, i) : 0u;
    int cnt = 0;
    for (int t0 = 0; t0 < G; t0 += kRankTile) {
        __syncthreads();
        for (int k = threadIdx.x; k < kRankTile; k += kThreads)
            keys[k] = t0 + k < G ? seed_key(a, pol, t0 + k) : ~0ull;
        __syncthreads();
        const int base = quarter * (kRankTile / kWaves);
#pragma unroll 4
        for (int k = 0; k < kRankTile / kWaves; ++k) {
            const uint64_t o = keys[base + k];
            const int id = t0 + base + k;       // ids past G hold the largest key
            cnt += (o < mine || (o == mine && id < i)) ? 1 : 0;
        }
    }
    part[threadIdx.x] = cnt;
    __syncthreads();
    if (quarter == 0 && i < G)
        a.order[(int64_t)seed * G + part[li] + part[li + kWave] + part[li + 2 * kWave] +
                part[li + 3 * kWave]] = i;
}

#pragma clang fp contract(off)

// Placement, one wavefront per seed: groups in order; each lane evaluates the
// drain time of its queues (q = lane, lane + 64, ...), the lowest drain time
// (then the lowest queue) wins, and the winning queue takes the group.
__global__ __launch_bounds__(kWave) void k_seedassign(SeedArgs a)
{
    extern __shared__ __align__(16) unsigned char dyn[];
    const int seed = blockIdx.x;
    const int G = a.G, I = a.I, M = a.M;
    const int lane = threadIdx.x;
    double *qA = reinterpret_cast<double *>(dyn);
    double *qK = qA + I;
    int *qlast = reinterpret_cast<int *>(qK + I);
    int *qcnt = qlast + I;
    float *sw = reinterpret_cast<float *>(qcnt + I);
    for (int q = lane; q < I; q += kWave) {
        qA[q] = 0.0;
        qK[q] = 0.0;
        qlast[q] = a.inst_model0 ? clampi(a.inst_model0[q], -1, M - 1) : -1;
        qcnt[q] = 0;
    }
    if (a.swap_in_lds)
        for (int k = lane; k < a.C * M * M; k += kWave) sw[k] = a.swap_cost[k];
    const float *swt = a.swap_in_lds ? sw : a.swap_cost;
    __syncthreads();
    const int32_t *order = a.order + (int64_t)seed * G;
    int32_t *owner = a.owner + (int64_t)seed * G;
    int32_t *pos = a.pos + (int64_t)seed * G;
    for (int k0 = 0; k0 < G; k0 += kWave) {
        const int cnt = min(kWave, G - k0);
        const int il = lane < cnt ? order[k0 + lane] : 0;
        const double al = (double)a.grp_count[il] * (double)a.grp_mu[il];
        const int ml = clampi(a.grp_model[il], 0, M - 1);
        for (int j = 0; j < cnt; ++j) {
            const double ag = lane_value(al, j);
            const int mg = __builtin_amdgcn_readlane(ml, j);
            double bd = INFINITY;
            int bq = INT_MAX;
            for (int q = lane; q < I; q += kWave) {
                const int l = qlast[q];
                double sc = 0.0;
                if (l >= 0 && l != mg && a.swap_cost)
                    sc = (double)swt[((int64_t)clampi(a.inst_class[q], 0, a.C - 1) * M + l) * M + mg];
                const double d = (qA[q] + ag) / (double)a.inst_tput[q] + (qK[q] + sc);
                if (d < bd) {
                    bd = d;
                    bq = q;
                }
            }
            for (int o = kWave / 2; o > 0; o >>= 1) {
                const double d2 = __shfl_xor(bd, o, kWave);
                const int q2 = __shfl_xor(bq, o, kWave);
                if (d2 < bd || (d2 == bd && q2 < bq)) {
                    bd = d2;
                    bq = q2;
                }
            }
            int best = __builtin_amdgcn_readfirstlane(bq);
            if (best == INT_MAX) best = 0;          // every drain time NaN: the first queue
            if (lane == (best & (kWave - 1))) {
                const int l = qlast[best];
                double sc = 0.0;
                if (l >= 0 && l != mg && a.swap_cost)
                    sc = (double)swt[((int64_t)clampi(a.inst_class[best], 0, a.C - 1) * M + l) * M + mg];
                qA[best] += ag;
                qK[best] += sc;
                qlast[best] = mg;
                owner[k0 + j] = best;
                pos[k0 + j] = qcnt[best];
                qcnt[best] += 1;
            }
            __syncthreads();
        }
    }
    for (int q = lane; q < I; q += kWave) a.qcount[(int64_t)seed * I + q] = qcnt[q];
}

#pragma clang fp contract(on)

// The seed plans into the caller's slot-major arrays (one workgroup per seed).
__global__ __launch_bounds__(kThreads) void k_seedwrite(SeedArgs a)
{
    __shared__ int32_t qo[kMaxSearchInstances + 1];
    const int seed = blockIdx.x;
    const int G = a.G, I = a.I;
    const int64_t st = a.out.plan_stride;
    if (threadIdx.x == 0) {
        int t = 0;
        qo[0] = 0;
        for (int q = 0; q < I; ++q) {
            t += a.qcount[(int64_t)seed * I + q];
            qo[q + 1] = t;
        }
    }
    __syncthreads();
    for (int q = threadIdx.x; q <= I; q += kThreads) a.out.qoff[(int64_t)q * st + seed] = qo[q];
    for (int k = threadIdx.x; k < G; k += kThreads) {
        const int64_t o = (int64_t)seed * G + k;
        const int slot = clampi(qo[clampi(a.owner[o], 0, I - 1)] + a.pos[o], 0, G - 1);
        a.out.perm[(int64_t)slot * st + seed] = a.order[o];
    }
    if (a.out.evict_bits)
        for (int w = threadIdx.x; w < (G + 31) / 32; w += kThreads)
            a.out.evict_bits[(int64_t)w * st + seed] = 0u;
}

// ---------------------------------------------------------------------------
// Host side

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

struct Layout {
    int nwg_a, nwg_b, nwg, nwg_f, nwg_r, nws;
    int64_t n_moves;
    size_t grec, by_slo, rank_part, perm, flag, qof, inv, srec, sst, trec, R, RD, Q, Nq, Es, T, cur, done, steps,
        wmin_s, wmin_i, smin, F, D, cand, cex, ncand, U, scratch, dq, tail, total;
};

Layout layout(int G, int I, int W, int64_t B)
{
    Layout L{};
    L.nwg_a = (int)(((int64_t)G * (W + 1) + kThreads - 1) / kThreads);
    L.nwg_b = (G + kThreads - 1) / kThreads;
    L.nwg = L.nwg_a + 2 * I * L.nwg_b;
    L.nwg_f = (int)(((int64_t)G * (W + 1) + kThreads - 1) / kThreads);
    L.nwg_r = (G + kThreads - 1) / kThreads;
    L.nws = L.nwg_f + I * L.nwg_b + L.nwg_r;
    L.n_moves = (int64_t)G * W + 2 * (int64_t)G * I;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align256(bytes);
        return at;
    };
    const size_t b = (size_t)B;
    const size_t nm = (size_t)L.n_moves;
    L.grec = take(sizeof(GRec) * G);
    L.by_slo = take(4 * (size_t)G);
    L.rank_part = take(4 * (size_t)G * (size_t)((G + kRankTile - 1) / kRankTile));
    L.perm = take(4 * (size_t)G * b);
    L.flag = take((size_t)G * b);
    L.qof = take(4 * (size_t)(I + 1) * b);
    L.inv = take(4 * (size_t)G * b);
    L.srec = take(sizeof(SRec) * G * b);
    L.sst = take(sizeof(SSt) * G * b);
    L.trec = take(sizeof(TRec) * G * b);
    L.R = take(8 * (size_t)G * b);
    L.RD = take(8 * (size_t)G * b);
    L.Q = take(8 * (size_t)I * b);
    L.Nq = take(8 * (size_t)I * b);
    L.Es = take(8 * (size_t)I * b);
    L.T = take(8 * (size_t)(I + 1) * b);
    L.cur = take(8 * b);
    L.done = take(4 * b);
    L.steps = take(4 * b);
    L.wmin_s = take(8 * (size_t)L.nwg * b);
    L.wmin_i = take(8 * (size_t)L.nwg * b);
    L.smin = take(8 * (size_t)L.nws * b);
    L.F = take(8 * nm * b);
    L.D = take(8 * nm * b);
    L.cand = take(4 * nm * b);
    L.cex = take(8 * nm * b);
    L.ncand = take(4 * b);
    L.U = take(8 * b);
    L.scratch = take(8 * (size_t)G * b);
    L.dq = take(16 * b);
    L.tail = take(sizeof(float2) * qlm_tail::kCells);
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
    const Layout L = layout(pr->n_groups, pr->n_instances, W, 1);
    const int64_t Bc = B > 0 ? B : 1;
    const int64_t sel = (L.n_moves + kThreads - 1) / kThreads;
    if ((int64_t)L.nwg * Bc > INT_MAX || sel * Bc > INT_MAX || (int64_t)L.nws * Bc > INT_MAX ||
        (int64_t)kExactBlocks * Bc > INT_MAX ||
        (int64_t)((pr->n_groups + kWaves - 1) / kWaves) * Bc > INT_MAX ||
        (int64_t)((pr->n_instances + kWaves - 1) / kWaves) * Bc > INT_MAX ||
        (int64_t)((pr->n_groups + kThreads - 1) / kThreads) * Bc > INT_MAX)
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
    a.rank_part = (int32_t *)(ws + L.rank_part);
    a.perm = (int32_t *)(ws + L.perm);
    a.flag = ws + L.flag;
    a.qof = (int32_t *)(ws + L.qof);
    a.inv = (int32_t *)(ws + L.inv);
    a.srec = (SRec *)(ws + L.srec);
    a.sst = (SSt *)(ws + L.sst);
    a.trec = (TRec *)(ws + L.trec);
    a.R = (double *)(ws + L.R);
    a.RD = (double *)(ws + L.RD);
    a.Q = (double *)(ws + L.Q);
    a.Nq = (double *)(ws + L.Nq);
    a.Es = (double *)(ws + L.Es);
    a.T = (double *)(ws + L.T);
    a.cur = (double *)(ws + L.cur);
    a.done = (int32_t *)(ws + L.done);
    a.steps = (int32_t *)(ws + L.steps);
    a.wmin_s = (double *)(ws + L.wmin_s);
    a.wmin_i = (int64_t *)(ws + L.wmin_i);
    a.smin = (double *)(ws + L.smin);
    a.F = (double *)(ws + L.F);
    a.D = (double *)(ws + L.D);
    a.cand = (int32_t *)(ws + L.cand);
    a.cex = (double *)(ws + L.cex);
    a.ncand = (int32_t *)(ws + L.ncand);
    a.U = (double *)(ws + L.U);
    a.scratch = (int32_t *)(ws + L.scratch);
    a.dq = (int32_t *)(ws + L.dq);
    a.tail = (float2 *)(ws + L.tail);
    a.nwg_a = L.nwg_a;
    a.nwg_b = L.nwg_b;
    a.nwg = L.nwg;
    a.nwg_f = L.nwg_f;
    a.nwg_r = L.nwg_r;
    a.nws = L.nws;
    a.n_moves = L.n_moves;
    return a;
}

int launched(const char *what)
{
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? QLM_OK : hip_fail(e, what);
}

// Checks, the group records, and (for the screens) the SLO ranks and the tail
// table.
int search_begin(const qlm_problem *pr, const qlm_plans *pl, int32_t W, void *ws, size_t ws_bytes,
                 SearchArgs *out, hipStream_t stream, bool screens = true)
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
    if (!screens) {
        hipLaunchKernelGGL(k_sgrec, dim3((a.G + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, a);
        return launched("k_sgrec launch");
    }
    {
        const int nb = (a.G + kWave - 1) / kWave;
        const int ntiles = (a.G + kRankTile - 1) / kRankTile;
        hipLaunchKernelGGL(k_srank, dim3((unsigned)(nb * ntiles)), dim3(kThreads), 0, stream, a);
        rc = launched("k_srank launch");
        if (rc) return rc;
        hipLaunchKernelGGL(k_srankout, dim3((a.G + kThreads - 1) / kThreads), dim3(kThreads), 0,
                           stream, a, ntiles);
        rc = launched("k_srankout launch");
    }
    if (rc) return rc;
    hipLaunchKernelGGL(k_stail, dim3(1), dim3(kThreads), 0, stream, a);
    return launched("k_stail launch");
}

int launch_state(SearchArgs &a, int force, hipStream_t stream)
{
    const int nblk = (a.I + kWaves - 1) / kWaves;
    hipLaunchKernelGGL(k_sstate, dim3((unsigned)(nblk * a.B)), dim3(kThreads), 0, stream, a, force);
    int rc = launched("k_sstate launch");
    if (rc) return rc;
    hipLaunchKernelGGL(k_stotal, dim3((unsigned)a.B), dim3(kThreads), 0, stream, a, force);
    return launched("k_stotal launch");
}

int load_and_state(SearchArgs &a, const qlm_plans *pl, hipStream_t stream)
{
    const int nblk = (a.G + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(k_sload, dim3((unsigned)(nblk * a.B)), dim3(kThreads), 0, stream, a, *pl);
    int rc = launched("k_sload launch");
    if (rc) return rc;
    return launch_state(a, 1, stream);
}

// Exact scores of every move (one lane per move).
int exact_moves(SearchArgs &a, hipStream_t stream)
{
    hipLaunchKernelGGL(k_sswap, dim3((unsigned)(a.nwg_a * a.B)), dim3(kThreads), 0, stream, a);
    int rc = launched("k_sswap launch");
    if (rc) return rc;
    qlm_internal::TimedLaunch tl;
    if ((rc = qlm_internal::timing_begin(stream, &tl))) return rc;
    hipLaunchKernelGGL(k_smove, dim3((unsigned)((int64_t)a.I * a.nwg_b * a.B)), dim3(kThreads), 0,
                       stream, a);
    if ((rc = launched("k_smove launch"))) return rc;
    qlm_internal::timing_end(stream, &tl);
    hipLaunchKernelGGL(k_sreloc, dim3((unsigned)((int64_t)a.I * a.nwg_b * a.B)), dim3(kThreads), 0,
                       stream, a);
    return launched("k_sreloc launch");
}

// The screens of every move (removals and swaps, then reassignments, then
// relocations into other queues and within a queue).
int screen_moves(SearchArgs &a, hipStream_t stream)
{
    hipLaunchKernelGGL(k_fswap, dim3((unsigned)(a.nwg_f * a.B)), dim3(kThreads), 0, stream, a);
    int rc = launched("k_fswap launch");
    if (rc) return rc;
    const dim3 mgrid((unsigned)(((int64_t)a.I * a.nwg_b + a.nwg_r) * a.B));
    qlm_internal::TimedLaunch tl;
    if ((rc = qlm_internal::timing_begin(stream, &tl))) return rc;
    hipLaunchKernelGGL(k_fmove, mgrid, dim3(kThreads), 0, stream, a);
    if ((rc = launched("k_fmove launch"))) return rc;
    qlm_internal::timing_end(stream, &tl);
    return QLM_OK;
}

// The placement of one group in every chain: the candidate places scored
// exactly, the lowest applied (the plan, the slot of every group and the queue
// scores kept up to date, which is all the next placement reads).
int place_step(SearchArgs &a, int32_t group, int32_t *queue, double *score, hipStream_t stream)
{
    int rc;
    qlm_internal::TimedLaunch tl;
    if ((rc = qlm_internal::timing_begin(stream, &tl))) return rc;
    const int eblk = (2 * a.I + 1 + kWaves - 1) / kWaves;
    hipLaunchKernelGGL(k_place_eval, dim3((unsigned)(eblk * a.B)), dim3(kThreads), 0, stream, a,
                       group);
    if ((rc = launched("k_place_eval launch"))) return rc;
    qlm_internal::timing_end(stream, &tl);
    hipLaunchKernelGGL(k_place_pick, dim3((unsigned)a.B), dim3(kThreads), 0, stream, a, queue,
                       score);
    return launched("k_place_pick launch");
}

// The chains' plans back to the caller's layout, with their scores.
int write_plans(SearchArgs &a, qlm_plans_out o, double *score, hipStream_t stream)
{
    const int64_t rows = (int64_t)a.G + a.I + 1 + (o.evict_bits ? (a.G + 31) / 32 : 0) + 1;
    int64_t grid = (rows * a.B + kThreads - 1) / kThreads;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(k_sout, dim3((unsigned)grid), dim3(kThreads), 0, stream, a, o, score,
                       (int32_t *)nullptr);
    return launched("k_sout launch");
}

// The arguments of a placement session's later calls: the workspace as
// qlm_place_begin left it, for the same problem and plan count.
int session_args(const qlm_problem *pr, int64_t B, void *ws, size_t ws_bytes, SearchArgs *out)
{
    int rc = check_search(pr, B, 0);
    if (rc) return rc;
    const Layout L = layout(pr->n_groups, pr->n_instances, 0, B);
    if (!ws || ((uintptr_t)ws & 255u))
        return fail(QLM_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    if (ws_bytes < L.total) return fail(QLM_ERR_WORKSPACE, "workspace too small");
    *out = search_args(pr, B, 0, (unsigned char *)ws, L);
    return QLM_OK;
}

// One search step after the screens: candidates, their exact scores, the pick.
int pick_step(SearchArgs &a, int step, hipStream_t stream)
{
    hipLaunchKernelGGL(k_sbound, dim3((unsigned)a.B), dim3(kThreads), 0, stream, a);
    int rc = launched("k_sbound launch");
    if (rc) return rc;
    const int64_t sel = (a.n_moves + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(k_sselect, dim3((unsigned)(sel * a.B)), dim3(kThreads), 0, stream, a);
    if ((rc = launched("k_sselect launch"))) return rc;
    hipLaunchKernelGGL(k_sexact, dim3((unsigned)(kExactBlocks * a.B)), dim3(kThreads), 0, stream, a);
    if ((rc = launched("k_sexact launch"))) return rc;
    hipLaunchKernelGGL(k_spick, dim3((unsigned)a.B), dim3(kThreads), 0, stream, a, step);
    return launched("k_spick launch");
}

struct SeedLayout {
    size_t order, owner, pos, qcount, total;
};

SeedLayout seed_layout(int G, int I, int n)
{
    SeedLayout L{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align256(bytes);
        return at;
    };
    L.order = take(4 * (size_t)G * n);
    L.owner = take(4 * (size_t)G * n);
    L.pos = take(4 * (size_t)G * n);
    L.qcount = take(4 * (size_t)I * n);
    L.total = o;
    return L;
}

}  // namespace

// ---------------------------------------------------------------------------
// C interface

extern "C" {

size_t qlm_seed_workspace_bytes(const qlm_problem *problem, int32_t n_seeds)
{
    if (!problem || problem->n_groups < 1 || problem->n_instances < 1 || n_seeds < 0)
        return 0;
    return seed_layout(problem->n_groups, problem->n_instances, n_seeds > 0 ? n_seeds : 1).total;
}

int qlm_seed_plans(const qlm_problem *problem, int32_t n, const int32_t *policy,
                   const qlm_plans_out *out, void *ws, size_t ws_bytes, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    int rc = check_search(problem, 1, 0);
    if (rc) return rc;
    if (n < 0 || n > kMaxSeeds) return fail(QLM_ERR_ARG, "seeds: n must be in [0, 64]");
    if (n == 0) return QLM_OK;
    if (!policy) return fail(QLM_ERR_ARG, "seeds: policy is NULL");
    for (int k = 0; k < n; ++k)
        if (policy[k] != 0 && policy[k] != 1)
            return fail(QLM_ERR_ARG, "seeds: a policy is neither 0 (EDF) nor 1 (grouped)");
    if (!out || !out->perm || !out->qoff) return fail(QLM_ERR_ARG, "seeds: out perm and qoff are required");
    if (out->plan_stride < n) return fail(QLM_ERR_ARG, "seeds: out plan_stride must be >= n");
    const int G = problem->n_groups, I = problem->n_instances;
    const SeedLayout L = seed_layout(G, I, n);
    if (!ws || ((uintptr_t)ws & 255u))
        return fail(QLM_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    if (ws_bytes < L.total) return fail(QLM_ERR_WORKSPACE, "workspace too small");
    SeedArgs a{};
    a.G = G;
    a.I = I;
    a.M = problem->n_models;
    a.C = problem->n_classes;
    a.grp_count = problem->grp_count;
    a.grp_mu = problem->grp_mu;
    a.grp_slo = problem->grp_slo;
    a.grp_model = problem->grp_model;
    a.inst_tput = problem->inst_tput;
    a.inst_class = problem->inst_class;
    a.inst_model0 = problem->inst_model0;
    a.swap_cost = problem->swap_cost;
    a.n = n;
    for (int k = 0; k < n; ++k) a.policy[k] = (int8_t)policy[k];
    unsigned char *w = (unsigned char *)ws;
    a.order = (int32_t *)(w + L.order);
    a.owner = (int32_t *)(w + L.owner);
    a.pos = (int32_t *)(w + L.pos);
    a.qcount = (int32_t *)(w + L.qcount);
    a.out = *out;
    const size_t swap_bytes = problem->swap_cost ? sizeof(float) * (size_t)a.C * a.M * a.M : 0;
    a.swap_in_lds = swap_bytes > 0 && swap_bytes <= kSeedSwapLds;
    const size_t lds = 24 * (size_t)I + (a.swap_in_lds ? swap_bytes : 0);
    hipError_t e = hipFuncSetAttribute((const void *)k_seedassign,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return hip_fail(e, "hipFuncSetAttribute");
    hipLaunchKernelGGL(k_seedrank, dim3((G + kWave - 1) / kWave, n), dim3(kThreads), 0, stream, a);
    if ((rc = launched("k_seedrank launch"))) return rc;
    hipLaunchKernelGGL(k_seedassign, dim3(n), dim3(kWave), lds, stream, a);
    if ((rc = launched("k_seedassign launch"))) return rc;
    hipLaunchKernelGGL(k_seedwrite, dim3(n), dim3(kThreads), 0, stream, a);
    return launched("k_seedwrite launch");
}

int qlm_place_group(const qlm_problem *problem, const qlm_plans *start, const qlm_plans_out *out,
                    int32_t group, void *ws, size_t ws_bytes, double *score, int32_t *queue,
                    qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!out) return fail(QLM_ERR_ARG, "out is NULL");
    if (!problem || group < 0 || group >= problem->n_groups)
        return fail(QLM_ERR_ARG, "group must be in [0, n_groups)");
    if (start && start->n_plans > 0) {
        if (!out->perm || !out->qoff || !out->evict_bits)
            return fail(QLM_ERR_ARG, "out perm, qoff and evict_bits are required (a relocation "
                                     "sets eviction flags)");
        if (out->plan_stride < start->n_plans)
            return fail(QLM_ERR_ARG, "out plan_stride must be >= n_plans");
    }
    SearchArgs a;
    int rc = search_begin(problem, start, 0, ws, ws_bytes, &a, stream, false);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    rc = load_and_state(a, start, stream);
    if (rc) return rc;
    if ((rc = place_step(a, group, queue, nullptr, stream))) return rc;
    return write_plans(a, *out, score, stream);
}

int qlm_place_begin(const qlm_problem *problem, const qlm_plans *plans, void *ws, size_t ws_bytes,
                    qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    SearchArgs a;
    int rc = search_begin(problem, plans, 0, ws, ws_bytes, &a, stream, false);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    return load_and_state(a, plans, stream);
}

int qlm_place_step(const qlm_problem *problem, int64_t n_plans, int32_t group, void *ws,
                   size_t ws_bytes, double *score, int32_t *queue, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!problem || group < 0 || group >= problem->n_groups)
        return fail(QLM_ERR_ARG, "group must be in [0, n_groups)");
    SearchArgs a;
    int rc = session_args(problem, n_plans, ws, ws_bytes, &a);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    return place_step(a, group, queue, score, stream);
}

int qlm_place_end(const qlm_problem *problem, int64_t n_plans, const qlm_plans_out *out, void *ws,
                  size_t ws_bytes, double *score, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!out) return fail(QLM_ERR_ARG, "out is NULL");
    SearchArgs a;
    int rc = session_args(problem, n_plans, ws, ws_bytes, &a);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    if (!out->perm || !out->qoff || !out->evict_bits)
        return fail(QLM_ERR_ARG, "out perm, qoff and evict_bits are required (a relocation sets "
                                 "eviction flags)");
    if (out->plan_stride < n_plans) return fail(QLM_ERR_ARG, "out plan_stride must be >= n_plans");
    return write_plans(a, *out, score, stream);
}

int64_t qlm_search_n_moves(int32_t n_groups, int32_t n_instances, int32_t window)
{
    if (n_groups < 1 || n_instances < 1 || window < 0) return 0;
    return (int64_t)n_groups * window + 2 * (int64_t)n_groups * n_instances;
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
    return exact_moves(a, stream);
}

int qlm_search_screen(const qlm_problem *problem, const qlm_plans *plans, int32_t window,
                      void *ws, size_t ws_bytes, double *score, double *bound, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!score || !bound) return fail(QLM_ERR_ARG, "score and bound are required");
    SearchArgs a;
    int rc = search_begin(problem, plans, window, ws, ws_bytes, &a, stream);
    if (rc) return rc;
    if (a.B == 0) return QLM_OK;
    rc = load_and_state(a, plans, stream);
    if (rc) return rc;
    a.F = score;
    a.D = bound;
    return screen_moves(a, stream);
}

int qlm_local_search(const qlm_problem *problem, const qlm_plans *start, const qlm_plans_out *out,
                     int32_t window, int32_t max_steps, void *ws, size_t ws_bytes, double *score,
                     int32_t *steps, int64_t *trace, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!out) return fail(QLM_ERR_ARG, "out is NULL");
    if (max_steps < 0) return fail(QLM_ERR_ARG, "max_steps must be >= 0");
    if (start && start->n_plans > 0) {
        if (!out->perm || !out->qoff || !out->evict_bits)
            return fail(QLM_ERR_ARG, "out perm, qoff and evict_bits are required (a relocation "
                                     "sets eviction flags)");
        if (out->plan_stride < start->n_plans)
            return fail(QLM_ERR_ARG, "out plan_stride must be >= n_plans");
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
        if (t > 0 && (rc = launch_state(a, 0, stream))) return rc;
        if ((rc = screen_moves(a, stream))) return rc;
        if ((rc = pick_step(a, t, stream))) return rc;
    }
    if (max_steps > 0 && (rc = launch_state(a, 1, stream))) return rc;
    const qlm_plans_out o = *out;
    const int64_t rows = (int64_t)a.G + a.I + 1 + (o.evict_bits ? (a.G + 31) / 32 : 0) + 1;
    int64_t grid = (rows * a.B + kThreads - 1) / kThreads;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(k_sout, dim3((unsigned)grid), dim3(kThreads), 0, stream, a, o, score, steps);
    return launched("k_sout launch");
}

}  // extern "C"
