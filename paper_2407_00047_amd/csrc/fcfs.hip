// fcfs.hip -- the per-request variant of the plan score: first come, first
// served inside each group, every request with its own SLO.  Interface:
// qlm_fcfs_* in include/qlm.h.
//
// Request r (r = 0 the first to arrive) of the group i at position j of queue
// g has ahead of it the groups before j and the r earlier requests of group i
// (Sec. 4 request groups are served first come, first served; Sec. 6, Eq.
// output_token_dist counts every request ahead), and carries its own TTFT SLO
// (Sec. 3, Definition "SLO"):
//
//   E[W_r]  = A / Theta_g + K + r (mu_i / Theta_g)
//   SD[W_r] = sqrt(V + r sigma_i^2) / Theta_g
//   P_r     = Q((slo_r - E[W_r]) / SD[W_r]),  [E[W_r] > slo_r] at SD = 0
//   score_p = sum of P_r over every request of the plan
//
// A, V are the tokens and the token variance of the groups ahead of position
// j, K the swap and eviction seconds up to and including it.  At 8192 groups
// of 128 requests a plan holds 1,048,576 requests, each with its own tail: the
// work is arithmetic, one tail per request, and the kernels are laid out for
// that, not for memory traffic.
//
// Screen.  The running sums are per position (one walk of each plan), the
// tails are per request.  The walk produces, for every group and plan, the
// group's start E[W] = A/Theta + K (double), its variance ahead (single,
// scaled for the tail table) and its queue, gathered group by group; the
// screen then takes one lane per plan and one wavefront per (64 plans, one
// group): all 64 lanes work on the same group at a time, so the request SLOs
// are the same across the wavefront and come through the scalar cache, the
// request's position in its group is a constant of the unrolled loop, and
// each request costs a margin in double, a variance in single and one read of
// the normal-tail table (11 vector instructions).
//
// The walk reads the plans slot-major with every lane (plan) of a wavefront at
// the same slot, so its reads are coalesced.  It is cut into segments of 128
// slots: k_fseg sums each segment's trailing queue piece, k_fstart chains the
// pieces into each segment's starting sums, and k_frec walks each segment
// again from them and forms the records.  The records belong in the rows of
// the groups, a different row in every lane: this transposition from the
// plans' slot order to group order is the price of the screen's shared SLOs.
// It runs in two passes: k_frec sorts every 8 slots' records by block of 128
// groups in LDS and appends each block's run to the block's bucket of the
// tile; k_fbscreen places each bucket's records in LDS by (group, plan) and
// screens them there.
//
// Screening bound, per request: table error below 2.2e-6; single-precision
// rounding of the cell coordinate, of the line's evaluation, of the margin and
// of the variance below 1.7e-6; the sum of at most 32 terms in single
// precision below 1.9e-6 per term; so |screened - exact| <= 8e-6 per request.
// The margin is formed in double from the start E[W], whose rounding stays
// below 2^-50 E[W_r]: negligible while E[W_r] <= 2^30 SD[W_r] (true of any
// plan whose variances are not zero or vanishingly small).  A request with
// SD = 0 at r = 0 (a queue's first group, or one behind groups without
// variance) takes the exact comparison with the oracle's E[W] (formed in the
// oracle's order: where a segment starts with nothing varying ahead, its sums
// are formed again from the queue's first slot); a group without variance is
// walked with exact comparisons throughout.
//
// Exact argmin.  Plans whose screened score is within twice the bound of the
// lowest are re-scored exactly (k_fexact: one workgroup per queue, the running
// sums rippled from lane to lane in position order, each request's term in
// double with erfc, its 16 wavefronts over slices of every group's requests),
// and the lowest exact score, the lowest index on ties, wins.
//
// Kernels
//   k_fprep     per group: clamped count, request offset, statistics; the
//               request total; per instance: Theta, the variance scale, class
//               and first model; k_fslo: the SLOs widened to double; k_ftail:
//               the normal-tail table
//   k_fseg      one lane per plan, one wavefront per (64 plans, segment):
//               each segment's trailing queue piece
//   k_fstart    one lane per plan: the sums at each segment's first slot
//   k_frec      as k_fseg: the records of the segment's groups, into the
//               buckets of their group blocks (k_fbzero clears the counts);
//               a tile's workgroups on one XCD
//   k_fbscreen  one workgroup per (64 plans, 128 groups): the bucket into LDS
//               by (group, plan), then the partial screened scores, one
//               wavefront per group at a time (lane = plan)
//   k_fsum      partial scores -> screened plan scores, and the per-block
//               minimum
//   k_fselect   the plans within the bound of the lowest -> candidates
//   k_fexact    one workgroup per (candidate, queue): exact queue scores
//   k_fpick / k_fplan   exact plan scores; the lowest (score, index)
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "internal.h"
#include "qlm.h"
#include "ripple.h"
#include "tail.h"

namespace {

using qlm_internal::check_plans;
using qlm_internal::check_problem;
using qlm_internal::fail;
using qlm_internal::hip_fail;
using qlm_ripple::from_left;
using qlm_ripple::from_left0;
using qlm_ripple::lane_value;
using qlm_ripple::wave_id;

constexpr int kWave = 64;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kSeg = 128;                   // slots per segment of the queue walks
constexpr int kSegThreads = 1024;           // k_fseg: 16 wavefronts, one workgroup per CU
constexpr int kSegWaves = kSegThreads / kWave;
constexpr size_t kSegLdsLimit = 160 * 1024; // LDS of one workgroup
constexpr int kBlk = 128;                   // groups per bucket of the transposition
constexpr int kBlkCap = kBlk * 64;          // records per bucket (a tile's plans)
constexpr int kSub = 8;                     // slots a walk sorts into buckets at a time
constexpr int kRecWaves = 4;                // wavefronts of a k_frec workgroup
constexpr int kXcds = 8;                    // XCDs of the device (workgroups dealt in turn)
constexpr size_t kFrecTabLimit = 16 * 1024; // k_frec: most bytes of tables copied into LDS
constexpr size_t kCuLds = 160 * 1024;       // LDS of one CU
constexpr int kMaxFcfsGroups = 1 << 16;
constexpr int kMaxFcfsInstances = 4096;
constexpr int kMaxBlocks = kMaxFcfsGroups / kBlk;
constexpr int kSumBlocks = 1024;            // k_fsum blocks (per-block minima)
constexpr int kExactBlocks = 256;
constexpr int kPickThreads = 256;
constexpr uint32_t kCountMask = (1u << 21) - 1u;
constexpr uint32_t kNoVar = 1u << 31;       // record flag: no variance ahead
constexpr double kEpsP = 8e-6;              // screening bound per request
constexpr int64_t kMaxRequests = (int64_t)1 << 31;
constexpr size_t kRecBudget = (size_t)1 << 30;    // bytes of group records per chunk

// Per group, built once per call: for the walks (the count clamped to 21 bits,
// the model clamped to [0, M)) ...
struct FGrp {
    float mu, var;
    uint32_t cnt;
    uint32_t model;
};

// ... and for the requests: how many are scored (clamped to n_requests).
struct FReq {
    float mu, var;
    uint32_t n;
    uint32_t pad;
};

// Per instance, for the walks: Theta, the table scale over Theta^2, the class
// clamped to [0, C), the model loaded at the start (-1: none).
struct FInst {
    double theta, vscale;
    int32_t cls, m0;
    int32_t pad[2];
};

// A slot's group start in one plan: E[W] of its first request, its variance
// ahead V / Theta^2 times the table's scale, and its queue (| kNoVar when
// V = 0).
struct FRec {
    double c0;
    float v0;
    uint32_t q;
};

// The transposition's streaming reads (each bucket record read once):
// non-temporal.  (For k_frec's bucket appends, runs of a few records merged
// into lines in L2, non-temporal stores were slower.)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ inline FRec ld_rec_nt(const FRec *p)
{
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    FRec r;
    r.c0 = __hiloint2double((int)v.y, (int)v.x);
    r.v0 = __uint_as_float(v.z);
    r.q = v.w;
    return r;
}

// Sums over the slots of one segment of a plan that belong to the queue open
// at the segment's end (tokens, variance, fixed costs), whether that queue
// starts inside the segment, and the queue open at the segment's start.
struct Piece {
    double A, V, K;
    int32_t head, q0;
};

// The running sums at a segment's first slot (those of its queue so far).
struct Start {
    double A, V, K;
    int32_t pad[2];
};

struct FArgs {
    int32_t G, I, M, C;
    const int32_t *grp_count;
    const float *grp_mu, *grp_var;
    const int32_t *grp_model;
    const float *inst_tput;
    const int32_t *inst_class, *inst_model0;
    const float *swap_cost;
    float evict_cost;
    int64_t P, ld;
    const int32_t *perm, *qoff;
    const uint32_t *evict_bits;
    const float *req_slo;
    int64_t n_req;
    // workspace
    FGrp *grp;                // [G]
    FReq *req;                // [G]
    FInst *inst;              // [I]
    int32_t *first;           // [G + 1] request offsets in req_slo
    double *slo64;            // [n_req] the SLOs in double
    float2 *tail;             // [kCells]
    double *nreq;             // [1] requests scored
    FRec *bucket;             // [tiles][nblk][kBlkCap] the transposition's buckets
    int32_t *bcnt;            // [tiles][nblk] records in each bucket
    Piece *piece;             // [nseg][chunk]
    Start *start;             // [nseg][chunk]
    double *part;             // [ceil(G / kBlk)][chunk] partial screened scores
    double *F;                // [P] screened scores
    double *bmin;             // [kSumBlocks]
    int32_t *ncand;           // [1]
    int64_t *cand;            // [P]
    double *Q;                // [P][I] exact queue scores
    int64_t chunk;
};

__device__ inline int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

template <class T>
__device__ inline const __attribute__((address_space(4))) T *as_const(const T *p)
{
    return (const __attribute__((address_space(4))) T *)p;
}

__device__ inline double wave_min(double v)
{
    for (int o = kWave / 2; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, kWave));
    return v;
}

__device__ inline int wave_max_int(int v)
{
    for (int o = kWave / 2; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, kWave));
    return v;
}

// (score, index) is better than (s2, i2): lower score, then lower index; a NaN
// score is never better.
__device__ inline bool better(double s, int64_t i, double s2, int64_t i2)
{
    return s < s2 || (s == s2 && i < i2);
}

#pragma clang fp contract(off)

// ---------------------------------------------------------------------------
// Per-call tables

// One workgroup: clamped counts, request offsets (an exclusive scan), group
// statistics, the request total.
__global__ __launch_bounds__(kThreads) void k_fprep(FArgs a)
{
    __shared__ int64_t part[kThreads];
    const int t = threadIdx.x;
    const int per = (a.G + kThreads - 1) / kThreads;
    const int b = t * per, e = min(a.G, b + per);
    int64_t s = 0;
    for (int i = b; i < e; ++i) s += (int64_t)((uint32_t)a.grp_count[i] & kCountMask);
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
    int64_t off = part[t];
    for (int i = b; i < e; ++i) {
        const int64_t want = (int64_t)((uint32_t)a.grp_count[i] & kCountMask);
        const int64_t lo = off < a.n_req ? off : a.n_req;
        const int64_t hi = off + want < a.n_req ? off + want : a.n_req;
        a.first[i] = (int32_t)lo;
        FGrp g;
        g.mu = a.grp_mu[i];
        g.var = a.grp_var[i];
        g.cnt = (uint32_t)want;
        g.model = (uint32_t)clampi(a.grp_model[i], 0, a.M - 1);
        a.grp[i] = g;
        FReq r;
        r.mu = g.mu;
        r.var = g.var;
        r.n = (uint32_t)(hi - lo);
        r.pad = 0u;
        a.req[i] = r;
        off += want;
    }
    for (int q = t; q < a.I; q += kThreads) {
        FInst v;
        v.theta = (double)a.inst_tput[q];
        v.vscale = qlm_tail::kVarScale / (v.theta * v.theta);
        v.cls = clampi(a.inst_class[q], 0, a.C - 1);
        v.m0 = a.inst_model0 ? clampi(a.inst_model0[q], -1, a.M - 1) : -1;
        v.pad[0] = v.pad[1] = 0;
        a.inst[q] = v;
    }
    // the last thread's range ends at G: its offset is then the total
    if (t == kThreads - 1) {
        a.first[a.G] = (int32_t)(off < a.n_req ? off : a.n_req);
        a.nreq[0] = (double)(off < a.n_req ? off : a.n_req);
    }
}

__global__ __launch_bounds__(kThreads) void k_fslo(FArgs a)
{
    for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < a.n_req;
         k += (int64_t)gridDim.x * kThreads)
        a.slo64[k] = (double)a.req_slo[k];
}

__global__ __launch_bounds__(kThreads) void k_ftail(FArgs a)
{
    __shared__ float2 tab[qlm_tail::kCells];
    qlm_tail::build<kThreads>(tab);
    __syncthreads();
    for (int k = threadIdx.x; k < qlm_tail::kCells; k += kThreads) a.tail[k] = tab[k];
}

// ---------------------------------------------------------------------------
// Screen

// The walk of one plan's slots in order, one lane per plan, every lane of a
// wavefront at the same slot (so the reads of the plan rows are coalesced).
// Queues are contiguous slot ranges; at a queue's first slot the running sums
// restart.  The sums and costs are formed with the oracle's operations in the
// oracle's order.
constexpr int kAhead = 3;      // queue boundaries a walk holds beyond the open queue's
static_assert(kAhead == 3, "open_queue settles nh and three boundaries");

struct Walk {
    int q, nh;                 // open queue, first slot of the next queue
    int nx[kAhead];            // qoff[q + 2 + j] (j < kAhead), -1 where not read
    double theta, vscale;
    int cls, prev;
    double A, V, K;
};

__device__ inline void set_queue(const FInst *inst, int q, Walk &w)
{
    const FInst v = inst[q];
    w.q = q;
    w.theta = v.theta;
    w.vscale = v.vscale;
    w.cls = v.cls;
    w.prev = v.m0;
    w.A = w.V = w.K = 0.0;
}

// Open queue q: its end boundary and the next kAhead ones are read together
// and waited for at once, so that no later read of the walk waits behind
// them (memory reads complete in order), and the switches to the next
// queues read nothing.  inst: the per-instance table (in LDS or global
// memory).
__device__ inline void open_queue(const FArgs &a, const FInst *inst, int64_t p, int q, Walk &w)
{
    w.nh = a.qoff[(int64_t)(q + 1) * a.ld + p];
#pragma unroll
    for (int j = 0; j < kAhead; ++j)
        w.nx[j] = q + 2 + j <= a.I ? a.qoff[(int64_t)(q + 2 + j) * a.ld + p] : -1;
    asm volatile("" ::"v"(w.nh), "v"(w.nx[0]), "v"(w.nx[1]), "v"(w.nx[2]));
    set_queue(inst, q, w);
}

// The queue holding slot s: the largest q with qoff[q] <= s.
__device__ inline int queue_at(const FArgs &a, int64_t p, int s)
{
    int lo = 0, hi = a.I - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.qoff[(int64_t)mid * a.ld + p] <= s)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Slots [s0, s1) of the walk, B at a time: a batch's reads (group ids, one
// eviction word, the group records) are issued together, and with kPipe the
// next batch's reads are issued while a batch is walked.  Batches start at
// multiples of B (so one eviction word covers a batch); slots before s0 are
// passed over.  At a queue's first slot (the next queue's first slot reached,
// empty queues skipped) the sums restart; then the slot's model-change and
// eviction costs; visit(s, i, w) sees the sums on entry to the slot (fixed
// costs included); then the group's tokens and variance join the sums.  Ids
// out of range (a malformed plan) are skipped.  The group records and swap
// costs are read from grp and swc: the problem's own arrays, or copies in LDS.
template <int B>
struct Batch {
    int ids[B];
    uint32_t ev;
};

template <int B>
__device__ inline void batch_ids(const FArgs &a, int64_t p, int sb, int s1, Batch<B> &b)
{
    // (rows past s1 clamp to its last one: the walk stops at s1, and no read
    // waits behind a conditional one)
#pragma unroll
    for (int u = 0; u < B; ++u) b.ids[u] = a.perm[(int64_t)min(sb + u, s1 - 1) * a.ld + p];
    b.ev = a.evict_bits ? a.evict_bits[(int64_t)(sb >> 5) * a.ld + p] : 0u;
}

// (every gather is issued, at a clamped id, so that all of a batch's are in
// flight together; the walk does not use the record of an id out of range)
template <int B>
__device__ inline void batch_groups(const FArgs &a, const FGrp *grp, const Batch<B> &b, FGrp *gr)
{
#pragma unroll
    for (int u = 0; u < B; ++u) gr[u] = grp[clampi(b.ids[u], 0, a.G - 1)];
}

struct NoPost {
    __device__ void operator()(int) const {}
};

template <int B, bool kPipe, class Visit, class Post = NoPost>
__device__ inline void walk(const FArgs &a, const FGrp *grp, const float *swc, const FInst *inst,
                            int64_t p, int s0, int s1, Walk &w, bool *fresh, const Visit &visit,
                            const Post &post = Post{})
{
    static_assert(B <= 32 && (B & (B - 1)) == 0, "a batch lies in one eviction word");
    if (s0 >= s1) return;
    int sb = s0 & ~(B - 1);
    Batch<B> cur;
    FGrp gr[B];
    batch_ids<B>(a, p, sb, s1, cur);
    batch_groups<B>(a, grp, cur, gr);
    for (; sb < s1; sb += B) {
        Batch<B> nxt;
        const bool more = sb + B < s1;
        if (kPipe && more) batch_ids<B>(a, p, sb + B, s1, nxt);
#pragma unroll
        for (int u = 0; u < B; ++u) {
            const int s = sb + u;
            if (s < s0) continue;
            if (s >= s1) break;
            if (s >= w.nh) {
                if (w.q + 1 < a.I && w.nx[0] >= 0 && (w.q + 2 >= a.I || w.nx[0] > s)) {
                    // the next queue (qoff[q+1] <= s < qoff[q+2]), from the
                    // boundaries held (a negative one is taken as not held)
                    w.nh = w.nx[0];
#pragma unroll
                    for (int j = 0; j + 1 < kAhead; ++j) w.nx[j] = w.nx[j + 1];
                    w.nx[kAhead - 1] = -1;
                    set_queue(inst, w.q + 1, w);
                } else {
                    int q = w.q;
                    while (q + 1 < a.I && a.qoff[(int64_t)(q + 1) * a.ld + p] <= s) ++q;
                    open_queue(a, inst, p, q, w);
                }
                *fresh = true;
            }
            const int i = cur.ids[u];
            if (i < 0 || i >= a.G) continue;
            const int m = (int)gr[u].model;
            if (w.prev >= 0 && w.prev != m && a.swap_cost)
                w.K += (double)swc[((int64_t)w.cls * a.M + w.prev) * a.M + m];
            if ((cur.ev >> (s & 31)) & 1u) w.K += (double)a.evict_cost;
            visit(s, i, w);
            const double n = (double)gr[u].cnt;
            w.A += n * (double)gr[u].mu;
            w.V += n * (double)gr[u].var;
            w.prev = m;
        }
        // the next batch's gathers go out before post: waiting for them then
        // waits for none of post's stores
        if (more) {
            if (kPipe)
                cur = nxt;
            else
                batch_ids<B>(a, p, sb + B, s1, cur);
            batch_groups<B>(a, grp, cur, gr);
        }
        post(sb);                       // every lane, after each batch
    }
}

// Bytes of the swap-cost table, rounded up to 16.
__device__ __host__ inline size_t swap_bytes(const FArgs &a)
{
    return a.swap_cost ? ((sizeof(float) * (size_t)a.C * a.M * a.M + 15) & ~(size_t)15) : 0;
}

// Copies of the swap costs and the instance table in LDS at t (swap_bytes(a)
// then I FInst); every thread of the workgroup takes part.
__device__ inline void stage_tables(const FArgs &a, unsigned char *t, int nthreads,
                                    const float **swc, const FInst **inst)
{
    float *sc = reinterpret_cast<float *>(t);
    FInst *si = reinterpret_cast<FInst *>(t + swap_bytes(a));
    if (a.swap_cost)
        for (int k = threadIdx.x; k < a.C * a.M * a.M; k += nthreads) sc[k] = a.swap_cost[k];
    for (int q = threadIdx.x; q < a.I; q += nthreads) si[q] = a.inst[q];
    *swc = a.swap_cost ? sc : nullptr;
    *inst = si;
}

struct NoVisit {
    __device__ void operator()(int, int, const Walk &) const {}
};

// Grid: ceil(chunk/64) tiles x ceil(nseg/16); wavefront = (tile, segment).
// Pass 1: each segment's trailing piece (the sums of its last queue over the
// segment's slots).  With kLds the group records, the swap costs and the
// instance table are first copied into LDS (dynamic: 16 G bytes, the costs,
// 32 I bytes), so that every slot's gather is an LDS read, not a random L2
// access.
template <bool kLds>
__global__ __launch_bounds__(kSegThreads) void k_fseg(FArgs a, int64_t p0, int64_t pc)
{
    extern __shared__ __align__(16) unsigned char fseg_lds[];
    const FGrp *grp = a.grp;
    const float *swc = a.swap_cost;
    const FInst *inst = a.inst;
    if (kLds) {
        FGrp *sg = reinterpret_cast<FGrp *>(fseg_lds);
        for (int i = threadIdx.x; i < a.G; i += kSegThreads) sg[i] = a.grp[i];
        stage_tables(a, fseg_lds + sizeof(FGrp) * (size_t)a.G, kSegThreads, &swc, &inst);
        __syncthreads();
        grp = sg;
    }
    const int nseg = (a.G + kSeg - 1) / kSeg;
    const int sq = (nseg + kSegWaves - 1) / kSegWaves;
    const int64_t tile = blockIdx.x / sq;
    const int k = (int)(blockIdx.x % sq) * kSegWaves + wave_id();
    if (k >= nseg) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t col = tile * kWave + lane;
    const bool on = col < pc;
    const int64_t p = p0 + (on ? col : pc - 1);
    const int s0 = k * kSeg, s1 = min(a.G, s0 + kSeg);
    Walk w;
    const int q0 = queue_at(a, p, s0);
    open_queue(a, inst, p, q0, w);
    bool fresh = s0 == 0 || a.qoff[(int64_t)q0 * a.ld + p] >= s0;
    if (!fresh) {
        const int i = a.perm[(int64_t)(s0 - 1) * a.ld + p];
        if (i >= 0 && i < a.G) w.prev = (int)grp[i].model;
    }
    walk<8, true>(a, grp, swc, inst, p, s0, s1, w, &fresh, NoVisit{});
    if (on) {
        Piece t;
        t.A = w.A;
        t.V = w.V;
        t.K = w.K;
        t.head = fresh ? 1 : 0;
        t.q0 = q0;
        a.piece[(int64_t)k * a.chunk + col] = t;
    }
}

// Pass 2: one lane per plan, the segments in order: the sums at each
// segment's first slot.
__global__ __launch_bounds__(kThreads) void k_fstart(FArgs a, int64_t pc)
{
    const int64_t col = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (col >= pc) return;
    const int nseg = (a.G + kSeg - 1) / kSeg;
    double A = 0.0, V = 0.0, K = 0.0;
    for (int k = 0; k < nseg; ++k) {
        Start st;
        st.A = A;
        st.V = V;
        st.K = K;
        st.pad[0] = st.pad[1] = 0;
        a.start[(int64_t)k * a.chunk + col] = st;
        const Piece t = a.piece[(int64_t)k * a.chunk + col];
        if (t.head) {
            A = t.A;
            V = t.V;
            K = t.K;
        } else {
            A = A + t.A;
            V = V + t.V;
            K = K + t.K;
        }
    }
}

// Pass 3: each slot's record (its group's start E[W] = A/Theta + K, its
// variance ahead, its queue), on its way to the group's row.  A queue open at
// the segment's start continues from the sums of pass 2; where nothing varies
// ahead (V = 0) those sums are formed again slot by slot from the queue's
// first slot, so that E[W] is the oracle's bit for bit wherever an exact
// comparison uses it.
//
// The records go to group rows, a different row in every lane, so they are
// not stored directly (every store would be a partial line).  Every kSub
// slots the wavefront sorts its records by group block (kBlk groups) in LDS
// and appends each block's run to that block's bucket of the tile, in
// consecutive addresses; k_fbscreen then places each bucket by group.  A
// record carries its group within the block and its lane in the word of its
// queue (the queue < 4096 in bits 0-11, the group in bits 12-18, the lane in
// bits 19-24, kNoVar in bit 31).
template <int kNB>
struct WaveBuf {
    // the records as four arrays of 32-bit words (c0's low and high words, v0,
    // q): a gather of records in sorted order then spreads its lanes over the
    // banks by entry, where 16-byte records would give it 16 bank groups
    uint32_t rw[4][kSub * kWave];
    uint32_t sidx[kSub * kWave];    // sorted position -> entry | group block << 16
    uint16_t sgb[kSub * kWave];     // entry -> group block
    uint8_t val[kSub * kWave];      // entry holds a record
    int cnt[kNB];                   // per group block (nblk <= kNB)
    uint16_t boff[kNB], gbase[kNB];
};

__device__ inline void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The wavefront's buffered records into the buckets of tile `tile`.
template <int kNB>
__device__ inline void flush(const FArgs &a, WaveBuf<kNB> &wb, int64_t tile, int nblk)
{
    const int lane = threadIdx.x & (kWave - 1);
    for (int k = lane; k < nblk; k += kWave) wb.cnt[k] = 0;
    wave_sync();
    int rank[kSub];
#pragma unroll
    for (int j = 0; j < kSub; ++j) {
        const int e = j * kWave + lane;
        rank[j] = wb.val[e] ? atomicAdd(&wb.cnt[wb.sgb[e]], 1) : 0;
    }
    wave_sync();
    // offsets of the blocks' runs (a scan over the blocks), and their room in
    // the buckets
    int run = 0;
    for (int k0 = 0; k0 < nblk; k0 += kWave) {
        const int k = k0 + lane;
        const int c = k < nblk ? wb.cnt[k] : 0;
        int x = c;
        for (int o = 1; o < kWave; o <<= 1) {
            const int y = __shfl_up(x, o, kWave);
            if (lane >= o) x += y;
        }
        if (k < nblk) {
            wb.boff[k] = (uint16_t)(run + x - c);
            const int at = c > 0 ? atomicAdd(&a.bcnt[tile * nblk + k], c) : 0;
            wb.gbase[k] = (uint16_t)min(at, kBlkCap);
        }
        run += __shfl(x, kWave - 1, kWave);
    }
    wave_sync();
#pragma unroll
    for (int j = 0; j < kSub; ++j) {
        const int e = j * kWave + lane;
        if (wb.val[e]) {
            const uint32_t k = wb.sgb[e];
            wb.sidx[wb.boff[k] + rank[j]] = (uint32_t)e | (k << 16);
        }
    }
    wave_sync();
    for (int pos = lane; pos < run; pos += kWave) {
        const uint32_t se = wb.sidx[pos];
        const int e = (int)(se & 0xFFFFu);
        const int k = (int)(se >> 16);
        const int dst = wb.gbase[k] + (pos - wb.boff[k]);
        if (dst < kBlkCap) {
            FRec r;
            r.c0 = __hiloint2double((int)wb.rw[1][e], (int)wb.rw[0][e]);
            r.v0 = __uint_as_float(wb.rw[2][e]);
            r.q = wb.rw[3][e];
            a.bucket[(tile * nblk + k) * (int64_t)kBlkCap + dst] = r;
        }
    }
    wave_sync();
#pragma unroll
    for (int j = 0; j < kSub; ++j) wb.val[j * kWave + lane] = 0;
    wave_sync();
}

// kNB: group blocks the wavefront buffers hold (64 or kMaxBlocks); kTab: the
// swap costs and the instance table copied into (dynamic) LDS.
template <int kNB, bool kTab>
__global__ __launch_bounds__(kRecWaves * kWave) void k_frec(FArgs a, int64_t p0, int64_t pc)
{
    __shared__ WaveBuf<kNB> bufs[kRecWaves];
    extern __shared__ __align__(16) unsigned char frec_lds[];
    const float *swc = a.swap_cost;
    const FInst *inst = a.inst;
    if (kTab) {
        stage_tables(a, frec_lds, kRecWaves * kWave, &swc, &inst);
        __syncthreads();
    }
    const int nseg = (a.G + kSeg - 1) / kSeg;
    const int nblk = (a.G + kBlk - 1) / kBlk;
    const int sq = (nseg + kRecWaves - 1) / kRecWaves;
    // Workgroups are dealt to the XCDs in turn; all workgroups of a tile get
    // the same XCD (xcd = blockIdx mod kXcds), so that the bucket lines their
    // appends share fill up in that XCD's L2 before they are written back
    // (from several L2s they went out in pieces).  The grid holds the tiles
    // rounded up to a multiple of kXcds.
    const int64_t local = blockIdx.x / kXcds;
    const int64_t tile = (local / sq) * kXcds + blockIdx.x % kXcds;
    const int k = (int)(local % sq) * kRecWaves + wave_id();
    if (tile * kWave >= pc || k >= nseg) return;
    WaveBuf<kNB> &wb = bufs[wave_id()];
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t col = tile * kWave + lane;
    const bool on = col < pc;
    const int64_t c = on ? col : pc - 1;
    const int64_t p = p0 + c;
    const int s0 = k * kSeg, s1 = min(a.G, s0 + kSeg);
#pragma unroll
    for (int j = 0; j < kSub; ++j) wb.val[j * kWave + lane] = 0;
    Walk w;
    const int q0 = a.piece[(int64_t)k * a.chunk + c].q0;
    open_queue(a, inst, p, q0, w);
    const int b = a.qoff[(int64_t)q0 * a.ld + p];
    if (s0 > 0 && b < s0) {
        const Start st = a.start[(int64_t)k * a.chunk + c];
        if (st.V == 0.0) {
            // nothing varies ahead: form the sums again in the oracle's order
            bool f = false;
            walk<8, true>(a, a.grp, swc, inst, p, max(b, 0), s0, w, &f, NoVisit{});
        } else {
            w.A = st.A;
            w.V = st.V;
            w.K = st.K;
            const int i = a.perm[(int64_t)(s0 - 1) * a.ld + p];
            if (i >= 0 && i < a.G) w.prev = (int)a.grp[i].model;
        }
    }
    wave_sync();
    bool f = false;
    // batches of kSub slots (s0 is a multiple of kSub); the next batch's reads
    // are in flight while a batch's records are sorted into the buckets
    walk<kSub, true>(a, a.grp, swc, inst, p, s0, s1, w, &f, [&](int s, int i, const Walk &x) {
        if (on) {
            const int e = (s & (kSub - 1)) * kWave + lane;
            FRec r;
            r.c0 = x.A / x.theta + x.K;
            r.v0 = (float)(x.V * x.vscale);
            r.q = (uint32_t)x.q | ((uint32_t)(i & (kBlk - 1)) << 12) |
                  ((uint32_t)lane << 19) | (x.V == 0.0 ? kNoVar : 0u);
            wb.rw[0][e] = (uint32_t)__double2loint(r.c0);
            wb.rw[1][e] = (uint32_t)__double2hiint(r.c0);
            wb.rw[2][e] = __float_as_uint(r.v0);
            wb.rw[3][e] = r.q;
            wb.sgb[e] = (uint16_t)(i / kBlk);
            wb.val[e] = 1;
        }
    }, [&](int) {
        wave_sync();
        flush(a, wb, tile, nblk);
    });
}

__global__ __launch_bounds__(kThreads) void k_fbzero(FArgs a, int64_t n)
{
    for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < n;
         k += (int64_t)gridDim.x * kThreads)
        a.bcnt[k] = 0;
}

// Q of the margin m (seconds) at scaled variance vz, from the table in LDS.
__device__ inline float tail_q(const float2 *tab, float m, float vz)
{
    return qlm_tail::q_of(tab, m, vz);
}

// The screened sum of P over the requests of group i in one plan (lane = plan;
// every lane of a wavefront at the same request of the same group, whose SLO
// is read through the scalar cache), from the group's start record rc.
__device__ inline double group_screen(const FArgs &a, const float2 *tab, int i, const FRec &rc)
{
    const auto req = as_const(a.req);
    const auto first = as_const(a.first);
    const int n = (int)req[i].n;
    if (n == 0) return 0.0;
    const float mu = req[i].mu, var = req[i].var;
    const auto slo = as_const(a.slo64 + first[i]);
    const int g = min((int)(rc.q & ~kNoVar), a.I - 1);
    const bool novar = (rc.q & kNoVar) != 0u;
    const double theta = (double)a.inst_tput[g];
    const double c1 = (double)mu / theta;
    const float v1 = (float)((double)var * (qlm_tail::kVarScale / (theta * theta)));
    const double c0 = rc.c0;
    const float v0 = rc.v0;
    const double s0 = slo[0];
    double Sg = novar ? (c0 > s0 ? 1.0 : 0.0) : (double)tail_q(tab, (float)(s0 - c0), v0);
    if (var == 0.0f) {
        for (int r = 1; r < n; ++r) {
            const double Er = c0 + (double)r * c1;
            const double sr = slo[r];
            Sg += novar ? (Er > sr ? 1.0 : 0.0) : (double)tail_q(tab, (float)(sr - Er), v0);
        }
    } else {
        int r = 1;
        for (; r + 32 <= n; r += 32) {
            const double eb = c0 + (double)r * c1;
            const float vb = fmaf((float)r, v1, v0);
            float S = 0.0f;
#pragma unroll
            for (int k = 0; k < 32; ++k) {
                const float m = (float)fma(-(double)k, c1, slo[r + k] - eb);
                const float v = fmaf((float)k, v1, vb);
                S += tail_q(tab, m, v);
            }
            Sg += (double)S;
        }
        float S = 0.0f;
        for (; r < n; ++r) {
            const double e = c0 + (double)r * c1;
            const float m = (float)(slo[r] - e);
            const float v = fmaf((float)r, v1, v0);
            S += tail_q(tab, m, v);
        }
        Sg += (double)S;
    }
    return Sg;
}

// The second pass of the transposition and the screen in one: one workgroup
// per bucket (tile, block of kBlk groups), group block major (the workgroups
// running at one time share their groups' SLOs in the caches).  The bucket's
// records go into LDS at their (group, plan) place; the 16 wavefronts then
// take the block's groups one at a time from a counter in LDS and screen each
// from LDS, leaving the group's sum for every plan in the place of its record;
// these are added in a fixed order (blocks of consecutive groups, then the
// blocks), the block's partial score of each plan.  The records sit in LDS as four arrays of 32-bit words (the low and
// high words of c0, v0, q), so that a scattered store's lanes land in banks by
// their plan's lane alone: a 16-byte record per place would give the 64 lanes
// of a store only 16 bank groups.  (Writing the records out as group rows for
// a separate screen moved 2 GiB more per chunk at large.)
constexpr int kTransThreads = 1024;

__global__ __launch_bounds__(kTransThreads) void k_fbscreen(FArgs a, int64_t pc)
{
    extern __shared__ __align__(16) unsigned char dyn[];
    uint32_t *w0 = reinterpret_cast<uint32_t *>(dyn);      // [kBlkCap] each
    uint32_t *w1 = w0 + kBlkCap;
    uint32_t *w2 = w1 + kBlkCap;
    uint32_t *w3 = w2 + kBlkCap;
    __shared__ float2 tab[qlm_tail::kCells];
    __shared__ int next;
    for (int k = threadIdx.x; k < qlm_tail::kCells; k += kTransThreads) tab[k] = a.tail[k];
    if (threadIdx.x == 0) next = 0;
    const int nblk = (a.G + kBlk - 1) / kBlk;
    const int64_t tiles = (pc + kWave - 1) / kWave;
    const int gb = (int)(blockIdx.x / tiles);
    const int64_t tile = blockIdx.x % tiles;
    const int i0 = gb * kBlk;
    const int ng = min(kBlk, a.G - i0);
    const int n = min(a.bcnt[tile * nblk + gb], kBlkCap);
    const FRec *src = a.bucket + (tile * nblk + gb) * (int64_t)kBlkCap;
    constexpr int kU = kBlkCap / kTransThreads;       // 8 records a thread, read together
    FRec x[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int r = u * kTransThreads + (int)threadIdx.x;
        if (r < n) x[u] = ld_rec_nt(src + r);
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int r = u * kTransThreads + (int)threadIdx.x;
        if (r < n) {
            const int gi = (int)((x[u].q >> 12) & (kBlk - 1));
            const int ln = (int)((x[u].q >> 19) & (kWave - 1));
            const int at = gi * kWave + ln;
            w0[at] = (uint32_t)__double2loint(x[u].c0);
            w1[at] = (uint32_t)__double2hiint(x[u].c0);
            w2[at] = __float_as_uint(x[u].v0);
            w3[at] = x[u].q & (0xFFFu | kNoVar);
        }
    }
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t col0 = tile * kWave + lane;
    const bool on = col0 < pc;
    // a lane past the chunk takes the record of the tile's last plan
    const int ln = on ? lane : (int)(pc - 1 - tile * kWave);
    for (;;) {
        int gi = 0;
        if (lane == 0) gi = atomicAdd(&next, 1);
        gi = __builtin_amdgcn_readfirstlane(__shfl(gi, 0, kWave));
        if (gi >= ng) break;
        const int at = gi * kWave + ln;
        FRec rc;
        rc.c0 = __hiloint2double((int)w1[at], (int)w0[at]);
        rc.v0 = __uint_as_float(w2[at]);
        rc.q = w3[at];
        const double Sg = group_screen(a, tab, i0 + gi, rc);
        // (every lane has read its record: the wavefront moves in step)
        const int me = gi * kWave + lane;
        w0[me] = (uint32_t)__double2loint(Sg);
        w1[me] = (uint32_t)__double2hiint(Sg);
    }
    __syncthreads();
    // the sums in a fixed order: each wavefront adds kBlk / 16 consecutive
    // groups, then one wavefront adds the 16 partials (in the record words
    // v0, q, free now)
    constexpr int kPer = kBlk / (kTransThreads / kWave);
    const int wv = wave_id();
    double part = 0.0;
    for (int gi = wv * kPer; gi < min(ng, wv * kPer + kPer); ++gi)
        part += __hiloint2double((int)w1[gi * kWave + lane], (int)w0[gi * kWave + lane]);
    w2[wv * kWave + lane] = (uint32_t)__double2loint(part);
    w3[wv * kWave + lane] = (uint32_t)__double2hiint(part);
    __syncthreads();
    if (threadIdx.x < kWave) {
        double tot = 0.0;
        for (int k = 0; k < kTransThreads / kWave; ++k)
            tot += __hiloint2double((int)w3[k * kWave + lane], (int)w2[k * kWave + lane]);
        if (on) a.part[(int64_t)gb * a.chunk + col0] = tot;
    }
}

// Screened plan scores of the chunk (partials in group-block order) and the
// running minimum per block (grid-stride over plans, fixed grid).
__global__ __launch_bounds__(kThreads) void k_fsum(FArgs a, int64_t p0, int64_t pc, int first_chunk)
{
    __shared__ double lmin[kWaves];
    const int nb = (a.G + kBlk - 1) / kBlk;
    double mn = first_chunk ? INFINITY : a.bmin[blockIdx.x];
    for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < pc;
         c += (int64_t)gridDim.x * kThreads) {
        double s = 0.0;
        for (int b = 0; b < nb; ++b) s += a.part[(int64_t)b * a.chunk + c];
        a.F[p0 + c] = s;
        mn = fmin(mn, s);
    }
    mn = wave_min(mn);
    if ((threadIdx.x & (kWave - 1)) == 0) lmin[threadIdx.x / kWave] = mn;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kWaves; ++w) mn = fmin(mn, lmin[w]);
        a.bmin[blockIdx.x] = mn;
    }
}

// Candidates: plans whose screened score lies within twice the bound of the
// lowest (their exact score can be the lowest), and plans with a NaN score.
// Block 0 clears the counter first in a kernel of its own (k_fzero).
__global__ void k_fzero(FArgs a) { if (threadIdx.x == 0) a.ncand[0] = 0; }

__global__ __launch_bounds__(kThreads) void k_fselect(FArgs a, int nbmin)
{
    __shared__ double smin;
    if (threadIdx.x < kWave) {
        double m = INFINITY;
        for (int b = threadIdx.x; b < nbmin; b += kWave) m = fmin(m, a.bmin[b]);
        m = wave_min(m);
        if (threadIdx.x == 0) smin = m;
    }
    __syncthreads();
    const double lim = smin + 2.0 * kEpsP * a.nreq[0] + 1e-9 * fabs(smin);
    for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < a.P;
         p += (int64_t)gridDim.x * kThreads) {
        const double f = a.F[p];
        if (f <= lim || f != f) {
            const int k = atomicAdd(a.ncand, 1);
            a.cand[k] = p;
        }
    }
}

// ---------------------------------------------------------------------------
// Exact scores

// The oracle's terms for one group in double, for its requests in slice j of
// nsl (consecutive arrivals): the slice's sum starts at 0 and adds its P_r in
// arrival order.
__device__ inline double slot_exact(const FArgs &a, int i, double A, double V, double K,
                                    double theta, int j, int nsl)
{
    const int n = (int)a.req[i].n;
    const double mu = (double)a.grp[i].mu;
    const double var = (double)a.grp[i].var;
    const float *slo = a.req_slo + a.first[i];
    const double EW = A / theta + K;
    double slot = 0.0;
    const int r0 = (int)((int64_t)n * j / nsl), r1 = (int)((int64_t)n * (j + 1) / nsl);
    for (int r = r0; r < r1; ++r) {
        const double sl = (double)slo[r];
        const double Er = EW + (double)r * (mu / theta);
        const double SDr = sqrt(V + (double)r * var) / theta;
        double P;
        if (SDr > 0.0)
            P = 0.5 * erfc((sl - Er) / (SDr * 1.4142135623730951));
        else
            P = (Er > sl) ? 1.0 : 0.0;
        slot += P;
    }
    return slot;
}

// One workgroup per (candidate k, queue g), over a fixed grid; each of its 16
// wavefronts takes one slice of every group's requests (consecutive
// arrivals).  A wavefront walks the queue's positions 64 at a time, one per
// lane; the running sums ripple from lane to lane in position order, then each
// lane forms its slice of its group's requests' terms, and those sums ripple
// into the slice's queue sum the same way.  The queue score is the slices'
// sums added in slice order (the oracle's sum reassociated: equal to within
// the rounding of a sum of that many terms).  Sixteen wavefronts per queue
// instead of one keep the requests' erfc chains short and the chip busy when
// only a few plans are re-scored.
constexpr int kExactThreads = 1024;
constexpr int kExactSlices = kExactThreads / kWave;

__global__ __launch_bounds__(kExactThreads) void k_fexact(FArgs a, const int64_t *plan_index,
                                                           const int32_t *count_dev, int64_t count)
{
    __shared__ double part[kExactSlices];
    const int lane = threadIdx.x & (kWave - 1);
    const int js = wave_id();
    const int64_t n = count_dev ? (int64_t)__builtin_amdgcn_readfirstlane(count_dev[0]) : count;
    const int64_t tasks = n * a.I;
    const double ecost = (double)a.evict_cost;
    for (int64_t t = blockIdx.x; t < tasks; t += gridDim.x) {
        const int64_t k = t / a.I;
        const int g = (int)(t % a.I);
        int64_t p = plan_index[k];
        p = p < 0 ? 0 : (p >= a.P ? a.P - 1 : p);
        const int G = a.G;
        const int bq = clampi(a.qoff[(int64_t)g * a.ld + p], 0, G);
        const int eq = clampi(a.qoff[(int64_t)(g + 1) * a.ld + p], bq, G);
        const double theta = (double)a.inst_tput[g];
        const int cls = clampi(a.inst_class[g], 0, a.C - 1);
        int prev = a.inst_model0 ? clampi(a.inst_model0[g], -1, a.M - 1) : -1;
        double rA = 0.0, rV = 0.0, rK = 0.0, rC = 0.0;
        for (int v0 = bq; v0 < eq; v0 += kWave) {
            const int cnt = min(kWave, eq - v0);
            const bool on = lane < cnt;
            int i = -1;
            if (on) {
                i = a.perm[(int64_t)(v0 + lane) * a.ld + p];
                if (i < 0 || i >= G) i = -1;
            }
            const int m = i >= 0 ? (int)a.grp[i].model : -1;
            // an invalid id (malformed plan) keeps the model before it
            int pm = __shfl_up(m, 1, kWave);
            if (lane == 0) pm = prev;
            const int mm = m >= 0 ? m : pm;
            double xa = 0.0, xb = 0.0, c1 = 0.0, c2 = 0.0;
            if (i >= 0) {
                const double nn = (double)a.grp[i].cnt;
                xa = nn * (double)a.grp[i].mu;
                xb = nn * (double)a.grp[i].var;
                if (pm >= 0 && pm != m && a.swap_cost)
                    c1 = (double)a.swap_cost[((int64_t)cls * a.M + pm) * a.M + m];
                const int s = v0 + lane;
                if (a.evict_bits && ((a.evict_bits[(int64_t)(s >> 5) * a.ld + p] >> (s & 31)) & 1u))
                    c2 = ecost;
            }
            const double la = from_left0(xa), lb = from_left0(xb);
            const double l1 = from_left0(c1), l2 = from_left0(c2);
            double A = rA, V = rV, K0 = rK;
            // cnt - 1 steps, rounded up to blocks of 8 (a step past the last
            // position leaves every position's sums unchanged), the count in
            // a scalar register so that only a block ends in a branch
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
            const double term = i >= 0 ? slot_exact(a, i, A, V, K, theta, js, kExactSlices) : 0.0;
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
            // the model the next round starts from: the last valid one
            int carry = __builtin_amdgcn_readlane(mm, last);
            prev = carry;
        }
        if (lane == 0) part[js] = rC;
        __syncthreads();
        if (threadIdx.x == 0) {
            double q = 0.0;
            for (int j = 0; j < kExactSlices; ++j) q += part[j];
            a.Q[k * a.I + g] = q;
        }
        __syncthreads();
    }
}

// Exact plan scores of the listed plans (queue scores summed in order).
__global__ __launch_bounds__(kThreads) void k_fplan(FArgs a, int64_t n, double *score)
{
    for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < n;
         k += (int64_t)gridDim.x * kThreads) {
        double s = 0.0;
        for (int g = 0; g < a.I; ++g) s += a.Q[k * a.I + g];
        score[k] = s;
    }
}

// The lowest (exact score, plan index) over the candidates.
__global__ __launch_bounds__(kPickThreads) void k_fpick(FArgs a, int64_t *best_index,
                                                        double *best_score)
{
    __shared__ double ls[kPickThreads / kWave];
    __shared__ int64_t li[kPickThreads / kWave];
    const int n = a.ncand[0];
    double bs = INFINITY;
    int64_t bi = -1;
    for (int k = threadIdx.x; k < n; k += kPickThreads) {
        double s = 0.0;
        for (int g = 0; g < a.I; ++g) s += a.Q[(int64_t)k * a.I + g];
        const int64_t p = a.cand[k];
        if (s == s && (bi < 0 || better(s, p, bs, bi))) {   // a NaN score never wins
            bs = s;
            bi = p;
        }
    }
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const double s2 = __shfl_xor(bs, o, kWave);
        const int64_t i2 = __shfl_xor(bi, o, kWave);
        if (i2 >= 0 && (bi < 0 || better(s2, i2, bs, bi))) {
            bs = s2;
            bi = i2;
        }
    }
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        ls[w] = bs;
        li[w] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < kPickThreads / kWave; ++k)
            if (li[k] >= 0 && (bi < 0 || better(ls[k], li[k], bs, bi))) {
                bs = ls[k];
                bi = li[k];
            }
        best_index[0] = bi;
        best_score[0] = bi < 0 ? INFINITY : bs;
    }
}

#pragma clang fp contract(on)

// ---------------------------------------------------------------------------
// Host side

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Plans per chunk: as many as `want` asks for (0 = up to kRecBudget bytes of
// group records), a multiple of 64, no more than the plans rounded up.
int64_t chunk_of(int32_t G, int64_t P, int64_t want)
{
    int64_t c = (int64_t)(kRecBudget / (sizeof(FRec) * (size_t)(G > 0 ? G : 1)));
    if (want > 0) c = want;
    c = (c + kWave - 1) / kWave * kWave;
    const int64_t all = (P + kWave - 1) / kWave * kWave;
    if (all < c) c = all;
    return c < kWave ? kWave : c;
}

struct FLayout {
    size_t grp, req, inst, first, slo64, tail, nreq, bucket, bcnt, piece, start, part, F, bmin, ncand,
        cand, Q, total;
    int64_t chunk;
};

FLayout flayout(const qlm_problem *pr, int64_t P, int64_t n_req, int64_t chunk)
{
    FLayout L{};
    const int32_t G = pr->n_groups, I = pr->n_instances;
    L.chunk = chunk_of(G, P, chunk);
    const int64_t Pn = P > 0 ? P : 1;
    const int nb = (G + kBlk - 1) / kBlk;
    size_t o = 0;
    auto put = [&](size_t &field, size_t bytes) {
        field = o;
        o += align256(bytes);
    };
    put(L.grp, sizeof(FGrp) * (size_t)G);
    put(L.req, sizeof(FReq) * (size_t)G);
    put(L.inst, sizeof(FInst) * (size_t)I);
    put(L.first, 4 * ((size_t)G + 1));
    put(L.slo64, 8 * ((size_t)n_req + 1));
    put(L.tail, 8 * (size_t)qlm_tail::kCells);
    put(L.nreq, 8);
    const size_t tiles = (size_t)(L.chunk / kWave);
    const size_t nblk = (size_t)((G + kBlk - 1) / kBlk);
    put(L.bucket, sizeof(FRec) * tiles * nblk * (size_t)kBlkCap);
    put(L.bcnt, 4 * tiles * nblk);
    const size_t nseg = (size_t)((G + kSeg - 1) / kSeg);
    put(L.piece, sizeof(Piece) * nseg * (size_t)L.chunk);
    put(L.start, sizeof(Start) * nseg * (size_t)L.chunk);
    put(L.part, 8 * (size_t)nb * (size_t)L.chunk);
    put(L.F, 8 * (size_t)Pn);
    put(L.bmin, 8 * (size_t)kSumBlocks);
    put(L.ncand, 256);
    put(L.cand, 8 * (size_t)Pn);
    put(L.Q, 8 * (size_t)Pn * (size_t)I);
    L.total = o;
    return L;
}

int check_requests(const qlm_problem *pr, const float *req_slo, int64_t n_req)
{
    (void)pr;
    if (n_req < 0 || n_req >= kMaxRequests)
        return fail(QLM_ERR_ARG, "n_requests must be in [0, 2^31)");
    if (n_req > 0 && !req_slo) return fail(QLM_ERR_ARG, "req_slo is NULL");
    return QLM_OK;
}

FArgs fargs(const qlm_problem *pr, const qlm_plans *pl, const float *req_slo, int64_t n_req,
            void *ws, const FLayout &L)
{
    FArgs a{};
    a.G = pr->n_groups;
    a.I = pr->n_instances;
    a.M = pr->n_models;
    a.C = pr->n_classes;
    a.grp_count = pr->grp_count;
    a.grp_mu = pr->grp_mu;
    a.grp_var = pr->grp_var;
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
    a.evict_bits = pl->evict_bits;
    a.req_slo = req_slo;
    a.n_req = n_req;
    unsigned char *w = (unsigned char *)ws;
    a.grp = (FGrp *)(w + L.grp);
    a.req = (FReq *)(w + L.req);
    a.inst = (FInst *)(w + L.inst);
    a.first = (int32_t *)(w + L.first);
    a.slo64 = (double *)(w + L.slo64);
    a.tail = (float2 *)(w + L.tail);
    a.nreq = (double *)(w + L.nreq);
    a.bucket = (FRec *)(w + L.bucket);
    a.bcnt = (int32_t *)(w + L.bcnt);
    a.piece = (Piece *)(w + L.piece);
    a.start = (Start *)(w + L.start);
    a.part = (double *)(w + L.part);
    a.F = (double *)(w + L.F);
    a.bmin = (double *)(w + L.bmin);
    a.ncand = (int32_t *)(w + L.ncand);
    a.cand = (int64_t *)(w + L.cand);
    a.Q = (double *)(w + L.Q);
    a.chunk = L.chunk;
    return a;
}

int launched(const char *what)
{
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? QLM_OK : hip_fail(e, what);
}

// Common start of every call: argument checks, the workspace, the per-call
// tables.
int fbegin(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
           int64_t n_req, void *ws, size_t ws_bytes, FArgs *out, FLayout *lay, bool need_tail,
           bool prep, hipStream_t stream)
{
    int rc = check_problem(problem);
    if (rc) return rc;
    rc = check_plans(problem, plans);
    if (rc) return rc;
    rc = check_requests(problem, req_slo, n_req);
    if (rc) return rc;
    if (problem->n_groups > kMaxFcfsGroups || problem->n_instances > kMaxFcfsInstances)
        return fail(QLM_ERR_CAPACITY, "the per-request calls take at most 65536 groups and 4096 "
                                      "instances");
    if (!ws || ((uintptr_t)ws & 255u))
        return fail(QLM_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    // the largest chunk the workspace holds, from the default down to 64 plans
    FLayout L = flayout(problem, plans->n_plans, n_req, 0);
    if (ws_bytes < L.total) {
        const FLayout L64 = flayout(problem, plans->n_plans, n_req, kWave);
        if (ws_bytes < L64.total) return fail(QLM_ERR_WORKSPACE, "workspace too small");
        const size_t per = (L.total - L64.total) / (size_t)(L.chunk - kWave);
        int64_t c = kWave + (int64_t)((ws_bytes - L64.total) / (per > 0 ? per : 1));
        c = c / kWave * kWave;
        L = flayout(problem, plans->n_plans, n_req, c);
        while (L.total > ws_bytes && c > kWave) L = flayout(problem, plans->n_plans, n_req, c -= kWave);
    }
    *out = fargs(problem, plans, req_slo, n_req, ws, L);
    *lay = L;
    if (plans->n_plans == 0 || !prep) return QLM_OK;
    hipLaunchKernelGGL(k_fprep, dim3(1), dim3(kThreads), 0, stream, *out);
    if ((rc = launched("k_fprep launch"))) return rc;
    if (n_req > 0 && need_tail) {
        int64_t blocks = (n_req + kThreads - 1) / kThreads;
        if (blocks > 4096) blocks = 4096;
        hipLaunchKernelGGL(k_fslo, dim3((unsigned)blocks), dim3(kThreads), 0, stream, *out);
        if ((rc = launched("k_fslo launch"))) return rc;
    }
    if (need_tail) {
        hipLaunchKernelGGL(k_ftail, dim3(1), dim3(kThreads), 0, stream, *out);
        if ((rc = launched("k_ftail launch"))) return rc;
    }
    return QLM_OK;
}

// k_frec in the form the problem allows: wavefront buffers for 64 group
// blocks where they suffice, and the tables in LDS where they leave as many
// workgroups on a CU as there are without them.
template <int kNB>
int launch_frec_nb(const FArgs &a, size_t tab_bytes, dim3 grid, hipStream_t stream, int64_t p0,
                   int64_t pc)
{
    const size_t fixed = sizeof(WaveBuf<kNB>) * kRecWaves;
    if (tab_bytes <= kFrecTabLimit &&
        kCuLds / (fixed + tab_bytes) == kCuLds / fixed) {
        hipLaunchKernelGGL((k_frec<kNB, true>), grid, dim3(kRecWaves * kWave), tab_bytes, stream, a,
                           p0, pc);
    } else {
        hipLaunchKernelGGL((k_frec<kNB, false>), grid, dim3(kRecWaves * kWave), 0, stream, a, p0,
                           pc);
    }
    return launched("k_frec launch");
}

int launch_frec(const FArgs &a, size_t tab_bytes, dim3 grid, hipStream_t stream, int64_t p0,
                int64_t pc)
{
    const int nblk = (a.G + kBlk - 1) / kBlk;
    if (nblk <= 64) return launch_frec_nb<64>(a, tab_bytes, grid, stream, p0, pc);
    return launch_frec_nb<kMaxBlocks>(a, tab_bytes, grid, stream, p0, pc);
}

// The screen over every plan, chunk by chunk: F and the per-block minima.
int screen_all(const FArgs &a, hipStream_t stream)
{
    int rc;
    for (int64_t p0 = 0; p0 < a.P; p0 += a.chunk) {
        const int64_t pc = a.P - p0 < a.chunk ? a.P - p0 : a.chunk;
        const int64_t tiles = (pc + kWave - 1) / kWave;
        const int64_t sq = ((a.G + kSeg - 1) / kSeg + kSegWaves - 1) / kSegWaves;
        const size_t tab_bytes = swap_bytes(a) + sizeof(FInst) * (size_t)a.I;
        const size_t seg_lds = sizeof(FGrp) * (size_t)a.G + tab_bytes;
        if (seg_lds <= kSegLdsLimit) {
            const hipError_t e = hipFuncSetAttribute((const void *)k_fseg<true>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     (int)seg_lds);
            if (e != hipSuccess) return hip_fail(e, "hipFuncSetAttribute");
            hipLaunchKernelGGL(k_fseg<true>, dim3((unsigned)(tiles * sq)), dim3(kSegThreads),
                               seg_lds, stream, a, p0, pc);
        } else {
            hipLaunchKernelGGL(k_fseg<false>, dim3((unsigned)(tiles * sq)), dim3(kSegThreads), 0,
                               stream, a, p0, pc);
        }
        if ((rc = launched("k_fseg launch"))) return rc;
        hipLaunchKernelGGL(k_fstart, dim3((unsigned)((pc + kThreads - 1) / kThreads)),
                           dim3(kThreads), 0, stream, a, pc);
        if ((rc = launched("k_fstart launch"))) return rc;
        const int64_t nblk = (a.G + kBlk - 1) / kBlk;
        int64_t zb = (tiles * nblk + kThreads - 1) / kThreads;
        if (zb > 1024) zb = 1024;
        hipLaunchKernelGGL(k_fbzero, dim3((unsigned)zb), dim3(kThreads), 0, stream, a, tiles * nblk);
        if ((rc = launched("k_fbzero launch"))) return rc;
        const int64_t sq2 = ((a.G + kSeg - 1) / kSeg + kRecWaves - 1) / kRecWaves;
        const int64_t tiles8 = (tiles + kXcds - 1) / kXcds * kXcds;
        if ((rc = launch_frec(a, tab_bytes, dim3((unsigned)(tiles8 * sq2)), stream, p0, pc)))
            return rc;
        const hipError_t ea = hipFuncSetAttribute((const void *)k_fbscreen,
                                                  hipFuncAttributeMaxDynamicSharedMemorySize,
                                                  (int)(sizeof(FRec) * kBlkCap));
        if (ea != hipSuccess) return hip_fail(ea, "hipFuncSetAttribute");
        qlm_internal::TimedLaunch tl;
        if ((rc = qlm_internal::timing_begin(stream, &tl))) return rc;
        hipLaunchKernelGGL(k_fbscreen, dim3((unsigned)(tiles * nblk)), dim3(kTransThreads),
                           sizeof(FRec) * kBlkCap, stream, a, pc);
        if ((rc = launched("k_fbscreen launch"))) return rc;
        qlm_internal::timing_end(stream, &tl);
        hipLaunchKernelGGL(k_fsum, dim3(kSumBlocks), dim3(kThreads), 0, stream, a, p0, pc,
                           p0 == 0 ? 1 : 0);
        if ((rc = launched("k_fsum launch"))) return rc;
    }
    return QLM_OK;
}

int exact_grid(int64_t tasks)
{
    int64_t b = tasks;                         // a workgroup per task
    if (b > kExactBlocks) b = kExactBlocks;
    return (int)(b < 1 ? 1 : b);
}

}  // namespace

// ---------------------------------------------------------------------------
// C interface

extern "C" {

size_t qlm_fcfs_workspace_bytes(const qlm_problem *problem, int64_t n_plans, int64_t n_requests,
                                int64_t chunk_plans)
{
    if (!problem || problem->n_groups < 1 || problem->n_instances < 1) return 0;
    if (n_plans < 0) n_plans = 0;
    if (n_requests < 0) n_requests = 0;
    return flayout(problem, n_plans, n_requests, chunk_plans > 0 ? chunk_plans : 0).total;
}

int qlm_fcfs_score(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
                   int64_t n_requests, void *ws, size_t ws_bytes, double *score,
                   qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    FArgs a;
    FLayout L;
    if (plans && plans->n_plans > 0 && !score) return fail(QLM_ERR_ARG, "score is NULL");
    int rc = fbegin(problem, plans, req_slo, n_requests, ws, ws_bytes, &a, &L, true, true, stream);
    if (rc) return rc;
    if (plans->n_plans == 0) return QLM_OK;
    a.F = score;
    return screen_all(a, stream);
}

int qlm_fcfs_score_exact(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
                         int64_t n_requests, const int64_t *plan_index, int64_t n, void *ws,
                         size_t ws_bytes, double *score, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (n < 0) return fail(QLM_ERR_ARG, "n must be >= 0");
    FArgs a;
    FLayout L;
    if (n > 0 && (!plan_index || !score))
        return fail(QLM_ERR_ARG, "plan_index and score are required");
    if (plans && n > plans->n_plans) return fail(QLM_ERR_ARG, "n must be <= n_plans");
    int rc = fbegin(problem, plans, req_slo, n_requests, ws, ws_bytes, &a, &L, false, n > 0,
                    stream);
    if (rc) return rc;
    if (n == 0) return QLM_OK;
    hipLaunchKernelGGL(k_fexact, dim3((unsigned)exact_grid(n * a.I)), dim3(kExactThreads), 0, stream, a,
                       plan_index, (const int32_t *)nullptr, n);
    if ((rc = launched("k_fexact launch"))) return rc;
    int64_t blocks = (n + kThreads - 1) / kThreads;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(k_fplan, dim3((unsigned)blocks), dim3(kThreads), 0, stream, a, n, score);
    return launched("k_fplan launch");
}

int qlm_fcfs_best_plan(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
                       int64_t n_requests, void *ws, size_t ws_bytes, int64_t *best_index,
                       double *best_score, qlm_stream stream_)
{
    hipStream_t stream = (hipStream_t)stream_;
    if (!best_index || !best_score)
        return fail(QLM_ERR_ARG, "best_index and best_score are required");
    FArgs a;
    FLayout L;
    int rc = fbegin(problem, plans, req_slo, n_requests, ws, ws_bytes, &a, &L, true, true, stream);
    if (rc) return rc;
    hipLaunchKernelGGL(k_fzero, dim3(1), dim3(kWave), 0, stream, a);
    if ((rc = launched("k_fzero launch"))) return rc;
    if (plans->n_plans > 0) {
        if ((rc = screen_all(a, stream))) return rc;
        hipLaunchKernelGGL(k_fselect, dim3(kSumBlocks), dim3(kThreads), 0, stream, a, kSumBlocks);
        if ((rc = launched("k_fselect launch"))) return rc;
        hipLaunchKernelGGL(k_fexact, dim3(kExactBlocks), dim3(kExactThreads), 0, stream, a,
                           (const int64_t *)a.cand, (const int32_t *)a.ncand, (int64_t)0);
        if ((rc = launched("k_fexact launch"))) return rc;
    }
    hipLaunchKernelGGL(k_fpick, dim3(1), dim3(kPickThreads), 0, stream, a, best_index, best_score);
    return launched("k_fpick launch");
}

}  // extern "C"
