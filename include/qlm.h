/*
 * qlm.h -- C interface of libqlm: batched request waiting time (RWT) estimation
 * and SLO-violation scoring of candidate virtual-queue plans on an MI355X
 * (gfx950), after "Queue Management for SLO-Oriented Large Language Model
 * Serving" (QLM, arXiv 2407.00047).
 *
 * Model (paper Secs. 6 and 7).  Request groups (Sec. 4, Definition "Request
 * Group") carry n_i requests of one model whose output tokens have mean mu_i
 * and variance sigma_i^2, and one TTFT SLO.  A plan places every group in
 * exactly one position of exactly one virtual queue (Sec. 7, Eq.
 * slot_assignment); queue g is served by an instance of token throughput
 * Theta_g.  For the group at position j of queue g:
 *
 *   E[W] = (sum_{k<j} n_k mu_k) / Theta_g + K_j          (Eq. base_equation;
 *   SD[W] = sqrt(sum_{k<j} n_k sigma_k^2) / Theta_g       Eq. output_token_dist)
 *   K_j  = sum_{k<=j} ( t_k * S[class_g][m_{k-1}][m_k] + evicted_k * E )
 *          with t_k = (m_{k-1} != m_k)                    (Eq. transition_time,
 *          and m_{-1} = inst_model0[g] (none if -1)        swap term of Eq.
 *                                                          completion_time)
 *   P    = P(W > slo), W ~ N(E[W], SD^2); for SD = 0, P = [E[W] > slo]
 *   score_p = sum over queues, then positions, of n * P   (expected number of
 *                                                          requests missing their SLO)
 *   penalty_p = sum of (E[W] - slo)                        (Eq. penalty, objective)
 *
 * The group's own incoming model swap and its own eviction count in its wait;
 * an eviction adds a fixed cost and no variance.
 *
 * Conventions for every entry point:
 *  - All array pointers are DEVICE pointers owned by the caller, unless stated.
 *    The library allocates no device memory.  Scalars and the structs themselves
 *    live in host memory and are read during the call only.
 *  - Work is enqueued on `stream` (0 = the null stream) and is asynchronous:
 *    outputs are valid once the stream reaches that point.  Calls keep no state
 *    between them, may run concurrently on different streams, and are
 *    thread-safe (the error text is per host thread).
 *  - The return value is a status (QLM_OK = 0).  Nothing is enqueued when a call
 *    returns an argument, capacity or workspace error.  No exception crosses
 *    the interface.
 *  - Plan contents are not checked by the scoring calls (use
 *    qlm_validate_plans): a malformed plan yields an unspecified score for that
 *    plan, never an out-of-bounds access.  Group ids are clamped to [0, G],
 *    models and classes to their ranges, counts to 21 bits.
 */
#ifndef QLM_H
#define QLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A HIP stream (hipStream_t); 0 is the null stream. */
typedef void *qlm_stream;

enum {
    QLM_OK = 0,
    QLM_ERR_ARG = 1,        /* null required pointer, bad size or stride      */
    QLM_ERR_CAPACITY = 2,   /* tables exceed the on-chip (LDS) budget         */
    QLM_ERR_WORKSPACE = 3,  /* workspace missing, too small or misaligned     */
    QLM_ERR_HIP = 4         /* a HIP call or kernel launch failed             */
};

/* Request groups, instances and swap costs (Sec. 7, table of LP symbols:
 * models_i, slos_i, S; Sec. 6: mu_o, sigma_o, Theta).                       */
typedef struct qlm_problem {
    int32_t n_groups;            /* G >= 1                                       */
    int32_t n_instances;         /* I >= 1 (one virtual queue per instance)      */
    int32_t n_models;            /* M, 1 <= M <= 255                             */
    int32_t n_classes;           /* C >= 1 hardware classes                      */
    const int32_t *grp_count;    /* [G] requests per group, 0 <= n < 2^21        */
    const float   *grp_mu;       /* [G] mean output tokens per request           */
    const float   *grp_var;      /* [G] variance of output tokens, >= 0          */
    const int32_t *grp_model;    /* [G] model of the group, in [0, M)            */
    const float   *grp_slo;      /* [G] TTFT SLO, seconds                        */
    const float   *inst_tput;    /* [I] token throughput Theta, tokens/s, > 0    */
    const int32_t *inst_class;   /* [I] class of the instance, in [0, C)         */
    const int32_t *inst_model0;  /* [I] model loaded before the head, -1 = none;
                                    NULL = none for every instance               */
    const float   *swap_cost;    /* [C][M][M] seconds to swap from model a (row)
                                    to model b (column) on class c; the diagonal
                                    is ignored; NULL = no swap cost              */
    float          evict_cost;   /* seconds added at an evicted slot             */
} qlm_problem;

/* A batch of candidate plans, slot-major ("structure of arrays" over plans):
 * entry (s, p) of perm is perm[s * plan_stride + p].  Consecutive plans are
 * contiguous, so a wavefront reading one slot of 64 plans reads 256 bytes.    */
typedef struct qlm_plans {
    int64_t n_plans;             /* P >= 0                                      */
    int64_t plan_stride;         /* elements between slot rows, P <= . <= 2^22   */
    const int32_t  *perm;        /* [G][stride]: group at slot s of plan p; each
                                    plan's column is a permutation of 0..G-1   */
    const int32_t  *qoff;        /* [I+1][stride]: queue g holds slots
                                    [qoff[g], qoff[g+1]); 0 = qoff[0] <= ... <=
                                    qoff[I] = G; empty queues allowed           */
    const uint32_t *evict_bits;  /* [ceil(G/32)][stride]: slot s is evicted when
                                    bit s%32 of word s/32 is set; NULL = none   */
} qlm_plans;

/* Per-slot outputs for plans [plan_begin, plan_begin + plan_count), each array
 * [G][plan_count] slot-major (entry (s, q) at s * plan_count + q, where plan
 * p = plan_begin + q); any of the three pointers may be NULL.                */
typedef struct qlm_detail {
    int64_t plan_begin, plan_count;
    float *wait_mean;            /* E[W], seconds                                */
    float *wait_sd;              /* SD[W], seconds                               */
    float *prob;                 /* P(W > slo)                                   */
} qlm_detail;

/*
 * Scores every plan (Secs. 6-7, the model above).
 *   score   [P] out: score_p = expected requests missing their SLO
 *   penalty [P] out or NULL: sum of (E[W] - slo) (Eq. penalty)
 *   detail  NULL or per-slot outputs for a plan range (must lie in [0, P))
 * Accuracy: per slot |dP| <= 1e-5 and E[W], SD[W] within 1e-5 relative of the
 * double-precision definition; |d score_p| <= 8e-6 * (total requests).  At a
 * position with SD = 0, P is the indicator [E[W] > slo] decided exactly as the
 * definition decides it.  The result is bit-for-bit reproducible for the same
 * inputs.  Method: waits in double precision, variances in single precision
 * per block of 32 positions on top of a double sum, and P from a 1024-cell
 * linear table of the normal tail over |z| <= 6 (error below 2.2e-6; beyond,
 * P is exactly 0 or 1).  Two forms (qlm_score_form): the fast path, for
 * problems whose groups all have requests and variance (SD = 0 then occurs
 * only at queue heads, where the wait is the head's cost seconds and Theta
 * times it is exact); and a general walk that forms A / Theta + K as the
 * definition does, taken for every other problem.
 */
int qlm_rwt_score(const qlm_problem *problem, const qlm_plans *plans, double *score,
                  double *penalty, const qlm_detail *detail, qlm_stream stream);

/*
 * Exact (double precision) scores of selected plans: plan_index[k] (device
 * array of n, each in [0, P)) -> score[k] (device); an index outside [0, P)
 * gives NaN.  Every step is the definition above in double precision, with
 * IEEE division and square root and the device erfc; each queue's terms are
 * added in position order, then the queue sums in queue order.
 */
int qlm_rwt_score_exact(const qlm_problem *problem, const qlm_plans *plans,
                        const int64_t *plan_index, int64_t n, double *score,
                        qlm_stream stream);

/*
 * Bytes of device workspace qlm_best_plan needs for n_plans plans: about 16
 * bytes per plan, plus 8 bytes per instance for each candidate whose queue
 * scores it holds (min(n_plans, max(256, 4Mi / n_instances)) candidates, 32
 * MiB at most).  0 when problem is NULL or has no instances.
 */
size_t qlm_best_plan_workspace_bytes(const qlm_problem *problem, int64_t n_plans);

/*
 * The plan the scheduler should pick (Sec. 7, objective; the scoring above in
 * place of the LP): argmin over p of the exact score, the lowest index on ties.
 * Screens every plan with the qlm_rwt_score arithmetic, then re-scores exactly
 * every plan that can still be the minimum given the screening error bound
 * (the candidates): one wavefront per (candidate, queue) while the workspace
 * holds the candidates' queue scores, else one workgroup per candidate.
 *   ws          device workspace of at least qlm_best_plan_workspace_bytes,
 *               256-byte aligned; its contents are scratch.  A larger one
 *               holds the queue scores of more candidates.
 *   best_index  [1] device out: index of the best plan (-1 when P = 0)
 *   best_score  [1] device out: its exact score (+inf when P = 0)
 */
int qlm_best_plan(const qlm_problem *problem, const qlm_plans *plans, void *ws,
                  size_t ws_bytes, int64_t *best_index, double *best_score,
                  qlm_stream stream);

/*
 * qlm_best_plan for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same computation and result, with the workspace in a static device
 * array of the library (64 MiB, on each GPU the library runs on, held until
 * the process ends) instead of a caller's buffer.  Allocates nothing and
 * creates no events.  The caller still passes the problem, the plans and the
 * two outputs (device pointers, as for qlm_best_plan).
 *   QLM_ERR_CAPACITY  when qlm_best_plan_workspace_bytes(problem, n_plans)
 *                     exceeds 64 MiB (nothing is enqueued)
 * Every call on a GPU shares that GPU's array, and calls that overlap on one
 * GPU (different streams or threads without ordering) race on it.
 */
int qlm_best_plan_static(const qlm_problem *problem, const qlm_plans *plans,
                         int64_t *best_index, double *best_score, qlm_stream stream);

/*
 * Checks plan structure (Eq. slot_assignment): qoff starts at 0, ends at G and
 * never decreases; perm is a permutation of 0..G-1; no eviction bit is set
 * beyond slot G-1.
 *   n_invalid   [1] device out: number of malformed plans
 *   plan_status [P] device out or NULL: 0 ok, 1 bad qoff, 2 bad perm, 4 bad
 *               eviction bits (bitwise or)
 */
int qlm_validate_plans(const qlm_problem *problem, const qlm_plans *plans,
                       int64_t *n_invalid, int32_t *plan_status, qlm_stream stream);

/*
 * Checks the tables: 0 <= n < 2^21, var >= 0, models in [0, M), classes in
 * [0, C), throughputs finite and > 0, inst_model0 in [-1, M).
 *   n_invalid   [1] device out: number of bad entries
 */
int qlm_validate_problem(const qlm_problem *problem, int64_t *n_invalid,
                         qlm_stream stream);

/* Writable plans (the output of qlm_local_search), laid out as qlm_plans.   */
typedef struct qlm_plans_out {
    int64_t plan_stride;         /* elements between slot rows, >= n_plans      */
    int32_t  *perm;              /* [G][stride]                                  */
    int32_t  *qoff;              /* [I+1][stride]                                */
    uint32_t *evict_bits;        /* [ceil(G/32)][stride]; required by the search
                                    and the placements (a relocation sets flags,
                                    also in plans that had none)                */
} qlm_plans_out;

/*
 * Plan search.  The paper's scheduler places groups by solving an LP over the
 * assignment of groups to queue positions (Sec. 7) and is compared with EDF
 * and same-model grouping (Secs. 2, 8).  This library instead improves plans
 * by local search whose moves are the scheduler's actions on virtual queues
 * (Sec. 5: reordering within a queue, reassigning a group to another
 * instance, evicting the running group), each scored exactly by the plan
 * score above.  The first slot of a non-empty queue holds the group its
 * instance is running: a group that has started stays on its instance
 * (Sec. 5), and only an eviction puts a group ahead of it.
 *
 *   SWAP(s, d)      k = s*W + d - 1          (s in [0,G), d in [1,W]): the
 *                   groups at slots s and s + d trade places, if both slots
 *                   lie in one queue and s is not its head;
 *   MOVE(s, h)      k = G*W + s*I + h        (h in [0,I)): the group at slot s
 *                   (not a head) leaves its queue g for queue h != g, placed
 *                   before the first group after h's head whose SLO is
 *                   strictly later than its own (else at the end; into an
 *                   empty h, as its head);
 *   RELOCATE(s, h)  k = G*W + G*I + s*I + h  (h in [0,I)): the group at slot s
 *                   (not a head) becomes the head of the non-empty queue h
 *                   (its own or another) ahead of the running group, and its
 *                   eviction flag is set (it pays evict_cost at its start).
 *
 * Any other moved group keeps its eviction flag.  A number k whose slot s is
 * a queue's head, whose partner slot lies in another queue or beyond G, whose
 * h is the group's own queue (MOVE) or an empty queue (RELOCATE), names no
 * move.  A move's score is the exact plan score (the arithmetic and summation
 * order of qlm_rwt_score_exact) of the plan the move makes; the library
 * computes it incrementally, from the first position the move changes.
 *
 * Limits: G <= 65536, I <= 4096, 0 <= W <= 1024.  SLOs must not be NaN.
 * Malformed start plans give unspecified results, never out-of-bounds access.
 */
int64_t qlm_search_n_moves(int32_t n_groups, int32_t n_instances, int32_t window);

/* Bytes of device workspace for n_plans plans with window W (0 on bad sizes). */
size_t qlm_search_workspace_bytes(const qlm_problem *problem, int64_t n_plans,
                                  int32_t window);

/*
 * Scores every move of every plan: move_score [P][qlm_search_n_moves] device
 * out, plan-major (entry (p, k) at p * n_moves + k); +inf where k names no
 * move.  ws: device workspace of at least qlm_search_workspace_bytes, 256-byte
 * aligned, scratch.
 */
int qlm_search_moves(const qlm_problem *problem, const qlm_plans *plans, int32_t window,
                     void *ws, size_t ws_bytes, double *move_score, qlm_stream stream);

/*
 * Screened scores of every move, the first stage of every qlm_local_search
 * step: score [P][n_moves] and bound [P][n_moves] device out, plan-major like
 * qlm_search_moves.  For every move |score - exact score| <= bound, where the
 * exact score is the one qlm_search_moves returns.  The screen walks a move's
 * target queue from cached waits and variances with the normal tail read from
 * the table of qlm_rwt_score; its bound is 8e-6 times the requests of that
 * queue plus 1e-12 of the scores.  bound = +inf marks a move the screen cannot
 * bound (a spread too small for the rounding of its margin; the search scores
 * it exactly); score = +inf with bound 0 where k names no move.
 */
int qlm_search_screen(const qlm_problem *problem, const qlm_plans *plans, int32_t window,
                      void *ws, size_t ws_bytes, double *score, double *bound,
                      qlm_stream stream);

/*
 * Steepest-descent local search from every start plan, independently: each
 * step scores every move, takes the lowest score (the lowest k on ties) and
 * applies it when it is strictly below the current plan's score; otherwise
 * that plan has converged and stops.  At most max_steps steps.  Each step
 * screens every move (qlm_search_screen), scores exactly only the moves that
 * can still be the lowest and improve, and decides on the exact scores, so
 * the steps are those of a search that scores every move exactly.
 *   start   the start plans (read before any output is written, so `out` may
 *           name the same arrays)
 *   out     the final plans, with their eviction words (required; QLM_ERR_ARG
 *           when evict_bits is NULL)
 *   score   [P] device out or NULL: exact score of each final plan
 *   steps   [P] device out or NULL: moves applied
 *   trace   [P][max_steps] device out or NULL: the move applied at each step,
 *           -1 from the step that found no improving move
 */
int qlm_local_search(const qlm_problem *problem, const qlm_plans *start,
                     const qlm_plans_out *out, int32_t window, int32_t max_steps,
                     void *ws, size_t ws_bytes, double *score, int32_t *steps,
                     int64_t *trace, qlm_stream stream);

/*
 * Placement of one group in every plan: the scheduler call of Sec. 5 when a
 * group arrives (the caller parks it behind the head of any non-empty queue
 * first) or when its wait violates its SLO (request eviction is how it can go
 * ahead of a running group).  In plan p the group leaves its slot and goes to
 * one of 2I places c:
 *   c = h       (h in [0,I)) queue h before the first group after h's head (as
 *               h stands without the group) whose SLO is strictly later, at
 *               the end when there is none, at the head of an empty h; its
 *               eviction flag kept (MOVE; with h its own queue, a reinsertion)
 *   c = I + h   the head of the non-empty queue h, ahead of its running group,
 *               with the group's eviction flag set (RELOCATE)
 * The place with the lowest exact plan score wins, the lowest c on ties.  A
 * group at its queue's head is running and stays: the plan is unchanged and c
 * is its queue.  Only the two queues that change are walked, from the first
 * position that changes.
 *   start/out  as for qlm_local_search (out may name the start arrays; its
 *              eviction words are required)
 *   group      the group's id; every plan holds it
 *   ws         device workspace of at least qlm_search_workspace_bytes(problem,
 *              P, 0), 256-byte aligned, scratch
 *   score [P]  device out or NULL: exact score of each placed plan
 *   queue [P]  device out or NULL: the place c chosen
 */
int qlm_place_group(const qlm_problem *problem, const qlm_plans *start,
                    const qlm_plans_out *out, int32_t group, void *ws, size_t ws_bytes,
                    double *score, int32_t *queue, qlm_stream stream);

/*
 * A placement session: the plans stay in the workspace between placements, so
 * that a stream of arrivals and violations is placed one group after another
 * without reloading the plans; each placement changes the plan in place and
 * keeps the queue scores and every group's slot up to date.
 *   qlm_place_begin  loads the plans (as qlm_place_group reads them) and
 *                    forms their cache in ws (qlm_search_workspace_bytes(
 *                    problem, P, 0) bytes, 256-byte aligned)
 *   qlm_place_step   places `group` in every plan, as qlm_place_group does;
 *                    score [P] and queue [P] (device out or NULL): each
 *                    plan's exact score after the placement, the place chosen
 *   qlm_place_end    writes the plans (as qlm_place_group writes them, with
 *                    their eviction words, required) and their exact scores
 *                    (score [P] or NULL); the session may continue after it
 * Every call names the same problem and plan count.  The workspace is the
 * session's state: between qlm_place_begin and the last call that uses it, no
 * other call may use it, and the calls of a session must be ordered (one
 * stream, or synchronized).
 */
int qlm_place_begin(const qlm_problem *problem, const qlm_plans *plans, void *ws, size_t ws_bytes,
                    qlm_stream stream);
int qlm_place_step(const qlm_problem *problem, int64_t n_plans, int32_t group, void *ws,
                   size_t ws_bytes, double *score, int32_t *queue, qlm_stream stream);
int qlm_place_end(const qlm_problem *problem, int64_t n_plans, const qlm_plans_out *out, void *ws,
                  size_t ws_bytes, double *score, qlm_stream stream);

/*
 * Seed plans for the search: the paper's reference orders, EDF (Sec. 8
 * baselines) and same-model grouping (Sec. 2, Insight #3).  Groups are taken
 * in EDF order (SLO, then group id) for policy 0, or by model, then SLO, then
 * id for policy 1; each is appended to the queue whose drain time after taking
 * it is smallest, (A_q + n mu) / Theta_q + (K_q + S[class_q][last model][model])
 * with A_q the queue's tokens and K_q its model-change costs so far (load
 * balancing by drain time, Sec. 8), the lowest queue on ties.  Seeds evict
 * nothing.  Limits as for the search; SLOs must not be NaN.
 *   policy  host array [n], 0 <= n <= 64: the policy of plan k of out
 *   out     plans 0..n-1 are written (eviction bits, when given, cleared)
 *   ws      device workspace of at least qlm_seed_workspace_bytes, 256-byte
 *           aligned, scratch
 */
size_t qlm_seed_workspace_bytes(const qlm_problem *problem, int32_t n_seeds);
int qlm_seed_plans(const qlm_problem *problem, int32_t n, const int32_t *policy,
                   const qlm_plans_out *out, void *ws, size_t ws_bytes, qlm_stream stream);

/*
 * Per-request variant: first come, first served inside each group, every
 * request with its own TTFT SLO (Sec. 3, Definition "SLO"; Sec. 4, requests
 * of a group are served first come, first served; Sec. 5, request pulling).
 * Request r (r = 0 the first to arrive) of the group at position j of queue g
 * has ahead of it the groups before j and the r earlier requests of its own
 * group, so by Eq. output_token_dist, with E[W] and K as above:
 *
 *   E[W_r]  = E[W] + r * (mu_i / Theta_g)
 *   SD[W_r] = sqrt(sum_{k<j} n_k sigma_k^2 + r sigma_i^2) / Theta_g
 *   P_r     = P(W_r > slo_{i,r}), W_r ~ N(E[W_r], SD[W_r]^2); [E[W_r] > slo] at SD = 0
 *   score_p = sum over queues, then positions, then requests in arrival order,
 *             of P_r (expected number of requests missing their own SLO)
 *
 * req_slo [n_requests] (device) holds the SLOs (seconds) of group 0's requests
 * in arrival order, then group 1's, and so on: group i's start at
 * n_0 + ... + n_{i-1}.  n_requests must equal sum n_i; the calls clamp every
 * group's requests to the array, so a mismatch gives unspecified scores, never
 * an out-of-bounds read.
 * With one request per group and req_slo = grp_slo this is the group score.
 *
 * Every call takes a device workspace, 256-byte aligned, used as scratch.
 * The plans are screened in chunks: a chunk of c plans needs 16 bytes per
 * group and plan for the groups' starts, and every call 8 bytes per request
 * and 8 (I + 2) bytes per plan.  qlm_fcfs_workspace_bytes(problem, n_plans,
 * n_requests, chunk_plans) is the size for chunks of chunk_plans plans
 * (rounded up to a multiple of 64; 0 = as many as 1 GiB of starts holds, the
 * size to use), 0 for an invalid problem.  A call uses the largest chunk the
 * workspace it is given holds, so any workspace of at least the size for
 * chunk_plans = 64 works; smaller chunks only take more launches.  Calls that
 * share a workspace must not overlap.
 */
size_t qlm_fcfs_workspace_bytes(const qlm_problem *problem, int64_t n_plans, int64_t n_requests,
                                int64_t chunk_plans);

/*
 * Screened per-request scores of every plan: score [P] device out.
 * Accuracy: |score_p - exact| <= 8e-6 * n_requests, when every request with
 * SD[W_r] > 0 has E[W_r] <= 2^30 SD[W_r] (any plan whose token variances are
 * zero or not vanishingly small); requests with SD = 0 are decided exactly at
 * r = 0 and throughout groups without variance.  Method: per group and plan,
 * the start E[W] in double (one walk of each queue); per request, the margin
 * in double, the variance in single precision and the normal tail from the
 * 1024-cell table; single-precision sums of at most 32 terms.
 */
int qlm_fcfs_score(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
                   int64_t n_requests, void *ws, size_t ws_bytes, double *score,
                   qlm_stream stream);

/*
 * Exact (double precision) per-request scores of selected plans: plan_index
 * [n] (device, each in [0, P), n <= P) -> score [n] (device).  The
 * definition above in double precision, in the order stated, with IEEE
 * division and square root and the device erfc.
 */
int qlm_fcfs_score_exact(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
                         int64_t n_requests, const int64_t *plan_index, int64_t n, void *ws,
                         size_t ws_bytes, double *score, qlm_stream stream);

/*
 * argmin over plans of the exact per-request score, the lowest index on ties
 * (a NaN score never wins; -1 and +inf when there is no plan): every plan is
 * screened, the plans whose screened score lies within twice the bound of the
 * lowest are scored exactly, and the lowest exact score wins.
 *   best_index [1], best_score [1]: device out
 */
int qlm_fcfs_best_plan(const qlm_problem *problem, const qlm_plans *plans, const float *req_slo,
                       int64_t n_requests, void *ws, size_t ws_bytes, int64_t *best_index,
                       double *best_score, qlm_stream stream);

/*
 * A hardware profile (Sec. 6, "Offline profiling": workload and hardware
 * profiling of the estimator's constants), per model m and per (instance
 * class c, model m), row-major [C][M].  Device arrays; any may be NULL, which
 * leaves out the terms that need it.
 */
typedef struct qlm_profile {
    const float *prefill;        /* [M]    P, prefill time of a request, seconds
                                    (constant per model, Sec. 6)                */
    const float *decode_time;    /* [C][M] d, seconds per output token          */
    const float *ineff;          /* [C][M] eps, inefficiency of continuous batching */
    const float *max_tokens;     /* [M]    O_max, the model's largest output     */
    const float *kv_tokens;      /* [C][M] GPU, tokens the GPU memory holds      */
    const float *mean_tokens;    /* [M]    E[I + O], tokens per request          */
} qlm_profile;

/*
 * Problem tables with the estimator's prefill, drain and throughput terms
 * folded in (Sec. 6, Eqs. total_completion_time, total_decode_time,
 * group_completion_time; Sec. 7, Eq. completion_time; Appendix, waiting time
 * predictability), for the scoring calls to read in place of the problem's own:
 *   slo_out  [G]      grp_slo[i] - P[m_i]: the SLO bounds the time to the
 *                     first token, the wait plus the request's own prefill
 *   swap_out [C][M][M] S[c][a][b] + (P[a] + O_max[a] eps[c][a] d[c][a]) for
 *                     a != b (the running requests of model a finish before
 *                     the swap: the completion time Eq. completion_time
 *                     charges at each transition); S = 0 where swap_cost is
 *                     NULL; the diagonal is copied
 *   tput_out [I]      Theta = (GPU[c][m] / E[I+O][m]) / (d[c][m] eps[c][m])
 *                     for instance g of class c serving inst_model[g] = m (the
 *                     batch the memory holds over one decode step); the
 *                     problem's inst_tput where inst_model is NULL or -1
 *   req_slo_out [n]   per-request SLOs (qlm_fcfs_* layout) less the prefill of
 *                     their group's model; req_slo and req_slo_out both NULL
 *                     or both given
 * The drain needs prefill, decode_time, ineff and max_tokens; the throughput
 * needs kv_tokens, decode_time, ineff, mean_tokens and inst_model.  Each value
 * is formed in double precision in the order written and stored in single
 * precision.  The outputs are device arrays of the caller and may not alias
 * the inputs.
 */
int qlm_apply_profile(const qlm_problem *problem, const qlm_profile *profile,
                      const int32_t *inst_model, float *swap_out, float *slo_out, float *tput_out,
                      const float *req_slo, int64_t n_requests, float *req_slo_out,
                      qlm_stream stream);

/* Largest G the scoring kernels accept for these M, C, I (on-chip budget). */
int32_t qlm_max_groups(int32_t n_models, int32_t n_classes, int32_t n_instances,
                       int32_t with_eviction);

/* Text of a status code; the last error's detail for this host thread. */
/*
 * Which form of the scoring kernel a problem gets (qlm_rwt_score and
 * qlm_best_plan decide it on the device, from the tables, at every launch):
 *   form [1] device out: 1 the fast path -- every group with 0 < n <= 2048
 *        requests and a variance that keeps n var / (1024/12)^2 a normal
 *        single-precision number, at most 64 models, a cost table (swap
 *        seconds, plus the eviction cost) whose entries have at most 29
 *        significant bits, and with eviction a cost table whose half fits 8
 *        KiB; 0 the general exact walk (the same results within the same
 *        bounds, slower).
 *   with_eviction  nonzero when the plans carry eviction bits
 */
int qlm_score_form(const qlm_problem *problem, int32_t with_eviction, int32_t *form,
                   qlm_stream stream);

const char *qlm_status_string(int status);
const char *qlm_last_error(void);

/*
 * Optional launch timing for benchmarks: when enabled, the dominant kernel of
 * each call is bracketed by HIP events on the call's stream: the plan-scoring
 * kernel of every qlm_rwt_score / qlm_best_plan call, the kernel that scores
 * the reassignment moves in every qlm_search_moves / qlm_search_screen call
 * and every step of qlm_local_search, the candidate kernel of every
 * qlm_place_group call, and the per-request screening kernel of every plan
 * chunk of qlm_fcfs_score / qlm_fcfs_best_plan.  qlm_timing_read waits for the recorded events and
 * returns the number of timed launches and their summed duration in
 * milliseconds since the last reset, then resets.
 */
int qlm_timing_enable(int on);
int qlm_timing_read(int64_t *launches, double *total_ms);

#ifdef __cplusplus
}
#endif

#endif /* QLM_H */
