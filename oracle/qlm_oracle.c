/*
 * qlm_oracle.c -- plain, slow, fp64 CPU oracle for QLM's request waiting time
 * (RWT) estimation and SLO-violation scoring of candidate virtual-queue plans
 * (Queue Management for SLO-Oriented LLM Serving, arXiv 2407.00047).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this file's library.  It shares no
 * code, header, table or constant with the HIP path: everything below is
 * written from the paper's definitions, in the paper's order, in double
 * precision, with no blocking, fusion or reordering.
 *
 * What is computed, per plan p, per virtual queue g (ascending), per queue
 * position j (ascending); slot s = qoff[g] + j holds request group i:
 *
 *   tokens ahead      A = sum_{k<j} n_k mu_k            (Sec. 6, Eq. base_equation
 *   variance ahead    V = sum_{k<j} n_k sigma_k^2        and Eq. output_token_dist:
 *                                                        the tokens ahead of a request
 *                                                        are Normal, mean and variance
 *                                                        add over the requests ahead)
 *   model transition  t = (m_prev >= 0 && m_prev != m_i) (Sec. 7, Eq. transition_time;
 *                     m_prev = model of the previous      the queue head compares with
 *                     position, or the instance's loaded  the model already loaded,
 *                     model at the head (-1 = none)       Sec. 5 "Model Swapping")
 *   fixed costs       K += t * S[class_g][m_prev][m_i]   (Sec. 7, Eq. completion_time,
 *                          + evicted(s) * E              swap term; the eviction LSO of
 *                                                        Sec. 5 adds a fixed cost)
 *   waiting time      E[W] = A / Theta_g + K             (Eq. base_equation + swaps)
 *                     SD[W] = sqrt(V) / Theta_g          (Theta constant, Sec. 6)
 *   violation prob.   P = P(W > slo_i), W ~ N(E[W], SD^2)
 *                       = 0.5 erfc((slo_i - E[W]) / (SD sqrt 2)),  SD > 0
 *                       = [E[W] > slo_i],                          SD = 0
 *   plan score        score_p = sum_g sum_j n_i P        (expected number of requests
 *                                                        that miss their SLO; the
 *                                                        objective of Sec. 7 summed
 *                                                        over queues then positions)
 *   plan penalty      pen_p   = sum_g sum_j (E[W] - slo_i)  (Sec. 7, Eq. penalty and
 *                                                        the optimisation goal)
 *   best plan         argmin_p score_p, lowest p on ties.
 *
 * The plan search at the end of the file (local search with the scheduler's
 * reorder, reassign and evict actions as moves) scores each move by building the
 * moved plan and scoring it with the definition above, from scratch.
 *
 * The readings behind the choices that the paper leaves open (probability of
 * violation as the score, the group's own swap counted in its waiting time,
 * eviction as a fixed cost, the exclusive token prefix) are listed in the
 * design notes of the repository.
 *
 * Parity status: every function here is pinned by tests (closed forms,
 * textbook normal-table values, invariants, Monte Carlo of the stated Normal
 * model, brute force over orderings on tiny inputs; for the search, moves
 * worked by hand, an independent re-implementation of the moves, and brute
 * force over every move of tiny plans).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Problem tables, as the caller holds them (fp32 / int32; widened to double
 * on use).  Layout and meaning follow the public C interface of the library,
 * but the struct is declared here on its own.                              */
typedef struct {
    int32_t n_groups, n_instances, n_models, n_classes;
    const int32_t *grp_count;   /* [G] requests in group i               */
    const float   *grp_mu;      /* [G] mean output tokens per request    */
    const float   *grp_var;     /* [G] variance of output tokens         */
    const int32_t *grp_model;   /* [G] model of the group                */
    const float   *grp_slo;     /* [G] TTFT SLO in seconds               */
    const float   *inst_tput;   /* [I] token throughput Theta, tokens/s  */
    const int32_t *inst_class;  /* [I] hardware class                    */
    const int32_t *inst_model0; /* [I] loaded model or -1; NULL = none   */
    const float   *swap_cost;   /* [C][M][M] from-model row, to-model column; NULL = 0 */
    float          evict_cost;  /* seconds added at an evicted slot      */
} oracle_problem;

/* A batch of plans, slot-major: entry (s, p) of perm is at perm[s*ld + p].  */
typedef struct {
    int64_t n_plans;
    int64_t ld;                 /* plan stride of every array, >= n_plans */
    const int32_t  *perm;       /* [G][ld]  group at slot s               */
    const int32_t  *qoff;       /* [I+1][ld] queue g holds slots [qoff[g], qoff[g+1]) */
    const uint32_t *evict_bits; /* [ceil(G/32)][ld] bit s%32 of word s/32; NULL = none */
} oracle_plans;

static int evicted(const oracle_plans *pl, int64_t p, int32_t s)
{
    if (!pl->evict_bits) return 0;
    uint32_t w = pl->evict_bits[(int64_t)(s / 32) * pl->ld + p];
    return (int)((w >> (s % 32)) & 1u);
}

/* One plan, written out exactly as the definitions above read.  Any output
 * pointer may be NULL.  Per-slot outputs are indexed by slot s (0..G-1).
 * Returns 0, or -1 when the plan is malformed (the caller's problem; the
 * oracle refuses to guess).                                                */
int oracle_plan(const oracle_problem *pr, const oracle_plans *pl, int64_t p,
                double *wait_mean, double *wait_sd, double *prob,
                double *score_out, double *penalty_out)
{
    const int G = pr->n_groups, I = pr->n_instances, M = pr->n_models;
    double score = 0.0, penalty = 0.0;

    if (pl->qoff[p] != 0 || pl->qoff[(int64_t)I * pl->ld + p] != G) return -1;

    for (int g = 0; g < I; ++g) {                       /* queues ascending */
        const int32_t begin = pl->qoff[(int64_t)g * pl->ld + p];
        const int32_t end   = pl->qoff[(int64_t)(g + 1) * pl->ld + p];
        if (begin > end) return -1;
        const double theta = (double)pr->inst_tput[g];
        const int    cls   = pr->inst_class[g];
        int m_prev = pr->inst_model0 ? pr->inst_model0[g] : -1;

        double A = 0.0;   /* tokens of the groups ahead on this queue    */
        double V = 0.0;   /* variance of those tokens                    */
        double K = 0.0;   /* swap and eviction seconds, up to and incl. j */
        double score_g = 0.0, penalty_g = 0.0;

        for (int32_t s = begin; s < end; ++s) {         /* positions ascending */
            const int32_t i = pl->perm[(int64_t)s * pl->ld + p];
            if (i < 0 || i >= G) return -1;
            const int    m   = pr->grp_model[i];
            const double n   = (double)pr->grp_count[i];
            const double mu  = (double)pr->grp_mu[i];
            const double var = (double)pr->grp_var[i];
            const double slo = (double)pr->grp_slo[i];

            if (m_prev >= 0 && m_prev != m && pr->swap_cost)
                K += (double)pr->swap_cost[((int64_t)cls * M + m_prev) * M + m];
            if (evicted(pl, p, s))
                K += (double)pr->evict_cost;

            const double EW = A / theta + K;
            const double SD = sqrt(V) / theta;
            double P;
            if (SD > 0.0)
                P = 0.5 * erfc((slo - EW) / (SD * sqrt(2.0)));
            else
                P = (EW > slo) ? 1.0 : 0.0;

            if (wait_mean) wait_mean[s] = EW;
            if (wait_sd)   wait_sd[s]   = SD;
            if (prob)      prob[s]      = P;

            score_g   += n * P;
            penalty_g += EW - slo;

            A += n * mu;
            V += n * var;
            m_prev = m;
        }
        score   += score_g;
        penalty += penalty_g;
    }
    if (score_out)   *score_out   = score;
    if (penalty_out) *penalty_out = penalty;
    return 0;
}

/* Scores of plans [p0, p0+count).  score/penalty are indexed from 0.  Plans
 * are independent, so they are spread over threads; nothing inside a plan is
 * reordered.  Returns the number of malformed plans (their score is NaN).   */
int64_t oracle_score_plans(const oracle_problem *pr, const oracle_plans *pl,
                           int64_t p0, int64_t count,
                           double *score, double *penalty, int n_threads)
{
    int64_t bad = 0;
#ifdef _OPENMP
    if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel for schedule(static) num_threads(n_threads) reduction(+ : bad)
#endif
    for (int64_t k = 0; k < count; ++k) {
        double sc = 0.0, pe = 0.0;
        if (oracle_plan(pr, pl, p0 + k, NULL, NULL, NULL, &sc, &pe) != 0) {
            sc = NAN;
            pe = NAN;
            bad += 1;
        }
        if (score)   score[k]   = sc;
        if (penalty) penalty[k] = pe;
    }
    (void)n_threads;
    return bad;
}

/* argmin over plans of the score, lowest index on ties (the first minimum
 * in index order).  NaN scores (malformed plans) never win.              */
int64_t oracle_argmin(const double *score, int64_t count, double *best_score)
{
    int64_t best = -1;
    double bs = INFINITY;
    for (int64_t p = 0; p < count; ++p) {
        if (score[p] < bs) {
            bs = score[p];
            best = p;
        }
    }
    if (best_score) *best_score = bs;
    return best;
}

/* The number of threads OpenMP would use, for reporting. */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------
 * Per-request variant: first-come-first-served order inside each group.
 *
 * The requests of a group are served in their arrival order (Sec. 4, request
 * group creation; Sec. 5, request pulling takes the head group's requests
 * first come, first served), and every request carries its own TTFT SLO
 * (Sec. 3, Definition "SLO").  Request r of the group at position j of queue g
 * (r = 0 is the first to arrive) has ahead of it the requests of the groups
 * before position j and the r earlier requests of its own group.  By Eq.
 * output_token_dist its tokens ahead are Normal with mean A + r mu_i and
 * variance V + r sigma_i^2, so with E[W] = A / Theta_g + K as above:
 *
 *   E[W_r]  = E[W] + r * (mu_i / Theta_g)
 *   SD[W_r] = sqrt(V + r * sigma_i^2) / Theta_g
 *   P_r     = 0.5 erfc((slo_{i,r} - E[W_r]) / (SD[W_r] sqrt 2)),   SD > 0
 *           = [E[W_r] > slo_{i,r}],                                SD = 0
 *   score_p = sum over queues, then positions, then requests, of P_r
 *             (the expected number of requests that miss their own SLO;
 *             the group's slot sum starts at 0 and adds P_0, P_1, ... in
 *             order, the queue sum adds the slot sums in position order,
 *             the plan sum adds the queue sums in queue order)
 *
 * req_slo[n_requests] holds the SLOs of group 0's requests in arrival order,
 * then group 1's, and so on: group i's start at n_0 + ... + n_{i-1}.  With one
 * request per group (and its SLO equal to the group's) this is the group
 * model above.
 */
int oracle_plan_fcfs(const oracle_problem *pr, const oracle_plans *pl, int64_t p,
                     const float *req_slo, int64_t n_requests, double *prob,
                     double *score_out)
{
    const int G = pr->n_groups, I = pr->n_instances, M = pr->n_models;
    int64_t *first = (int64_t *)malloc(sizeof(int64_t) * (size_t)(G + 1));
    if (!first) return -1;
    first[0] = 0;
    for (int i = 0; i < G; ++i) first[i + 1] = first[i] + pr->grp_count[i];
    int rc = 0;
    double score = 0.0;
    if (first[G] != n_requests) rc = -1;
    if (pl->qoff[p] != 0 || pl->qoff[(int64_t)I * pl->ld + p] != G) rc = -1;

    for (int g = 0; g < I && rc == 0; ++g) {                 /* queues ascending */
        const int32_t begin = pl->qoff[(int64_t)g * pl->ld + p];
        const int32_t end   = pl->qoff[(int64_t)(g + 1) * pl->ld + p];
        if (begin > end) { rc = -1; break; }
        const double theta = (double)pr->inst_tput[g];
        const int    cls   = pr->inst_class[g];
        int m_prev = pr->inst_model0 ? pr->inst_model0[g] : -1;
        double A = 0.0, V = 0.0, K = 0.0;
        double score_g = 0.0;

        for (int32_t s = begin; s < end; ++s) {             /* positions ascending */
            const int32_t i = pl->perm[(int64_t)s * pl->ld + p];
            if (i < 0 || i >= G) { rc = -1; break; }
            const int    m   = pr->grp_model[i];
            const int32_t n  = pr->grp_count[i];
            const double mu  = (double)pr->grp_mu[i];
            const double var = (double)pr->grp_var[i];

            if (m_prev >= 0 && m_prev != m && pr->swap_cost)
                K += (double)pr->swap_cost[((int64_t)cls * M + m_prev) * M + m];
            if (evicted(pl, p, s))
                K += (double)pr->evict_cost;

            const double EW = A / theta + K;                 /* the group's start */
            double slot = 0.0;
            for (int32_t r = 0; r < n; ++r) {                /* arrival order */
                const double slo = (double)req_slo[first[i] + r];
                const double Er  = EW + (double)r * (mu / theta);
                const double SDr = sqrt(V + (double)r * var) / theta;
                double P;
                if (SDr > 0.0)
                    P = 0.5 * erfc((slo - Er) / (SDr * sqrt(2.0)));
                else
                    P = (Er > slo) ? 1.0 : 0.0;
                if (prob) prob[first[i] + r] = P;
                slot += P;
            }
            score_g += slot;

            A += (double)n * mu;
            V += (double)n * var;
            m_prev = m;
        }
        score += score_g;
    }
    free(first);
    if (score_out) *score_out = (rc == 0) ? score : NAN;
    return rc;
}

/* FCFS scores of plans [p0, p0+count), spread over threads by plan.  Returns
 * the number of malformed plans (their score is NaN).                       */
int64_t oracle_score_plans_fcfs(const oracle_problem *pr, const oracle_plans *pl,
                                const float *req_slo, int64_t n_requests,
                                int64_t p0, int64_t count, double *score, int n_threads)
{
    int64_t bad = 0;
#ifdef _OPENMP
    if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads) reduction(+ : bad)
#endif
    for (int64_t k = 0; k < count; ++k) {
        double sc = 0.0;
        if (oracle_plan_fcfs(pr, pl, p0 + k, req_slo, n_requests, NULL, &sc) != 0) bad += 1;
        if (score) score[k] = sc;
    }
    (void)n_threads;
    return bad;
}

/* ------------------------------------------------------------------------
 * Problem tables from a hardware profile: prefill, drain and throughput.
 *
 * The completion time of a request is its wait, its prefill and its decode,
 * C_q = W_q + P + D_q (Sec. 6, Eq. total_completion_time), with P constant per
 * model, D_q = O_q * eps * d (Eq. total_decode_time; O_q taken as the
 * model's largest output, the estimator's conservative choice) and a group's
 * completion the latest of its requests' (Eq. group_completion_time).
 *
 *   prefill   The SLO bounds the time to the first token (Sec. 3, Definition
 *             "SLO"), which is the wait plus the request's own prefill, so a
 *             request misses it when W > slo - P[m].  The SLO table becomes
 *             slo - P[m_i].
 *   drain     Before an instance of class c changes from model a to model b,
 *             the requests already running must complete: the latest of them,
 *             admitted last, needs its prefill and up to O_max decode steps,
 *             P[a] + O_max[a] * eps[c][a] * d[c][a].  This is the completion
 *             time that Eq. completion_time charges at every model transition
 *             (its third term), so the swap table becomes
 *             S[c][a][b] + P[a] + O_max[a] * eps[c][a] * d[c][a] for a != b.
 *   Theta     The token throughput of an instance is its batch over the time
 *             of one decode step, Theta = B / (d * eps), and the batch is what
 *             the GPU's token memory holds, B = GPU / E[I + O] (Appendix,
 *             waiting time predictability).  Instance g of class c serving
 *             model m gets Theta[c][m].
 *
 * Each value is formed in double precision and stored in single precision,
 * the precision of the problem tables.  A NULL profile array leaves its term
 * out (no prefill; no drain; the throughputs as given).
 */
typedef struct {
    const float *prefill;      /* [M]    P, seconds                           */
    const float *decode_time;  /* [C][M] d, seconds per output token          */
    const float *ineff;        /* [C][M] eps, inefficiency factor             */
    const float *max_tokens;   /* [M]    O_max, largest output of the model   */
    const float *kv_tokens;    /* [C][M] GPU, tokens the memory holds         */
    const float *mean_tokens;  /* [M]    E[I + O], tokens per request         */
} oracle_profile;

void oracle_apply_profile(const oracle_problem *pr, const oracle_profile *pf,
                          const int32_t *inst_model, float *swap_out, float *slo_out,
                          float *tput_out, const float *req_slo, int64_t n_requests,
                          float *req_slo_out)
{
    const int G = pr->n_groups, I = pr->n_instances, M = pr->n_models, C = pr->n_classes;
    const int drain = pf->prefill && pf->decode_time && pf->ineff && pf->max_tokens;
    for (int c = 0; c < C; ++c)
        for (int a = 0; a < M; ++a)
            for (int b = 0; b < M; ++b) {
                const int64_t k = ((int64_t)c * M + a) * M + b;
                double S = pr->swap_cost ? (double)pr->swap_cost[k] : 0.0;
                if (drain && a != b) {
                    const int64_t ca = (int64_t)c * M + a;
                    const double D = (double)pf->max_tokens[a] * (double)pf->ineff[ca] *
                                     (double)pf->decode_time[ca];
                    S = S + ((double)pf->prefill[a] + D);
                }
                swap_out[k] = (float)S;
            }
    for (int i = 0; i < G; ++i) {
        double slo = (double)pr->grp_slo[i];
        if (pf->prefill) slo = slo - (double)pf->prefill[pr->grp_model[i]];
        slo_out[i] = (float)slo;
    }
    if (req_slo && req_slo_out) {
        int64_t r = 0;
        for (int i = 0; i < G && r < n_requests; ++i)
            for (int32_t k = 0; k < pr->grp_count[i] && r < n_requests; ++k, ++r) {
                double slo = (double)req_slo[r];
                if (pf->prefill) slo = slo - (double)pf->prefill[pr->grp_model[i]];
                req_slo_out[r] = (float)slo;
            }
    }
    for (int g = 0; g < I; ++g) {
        double theta = (double)pr->inst_tput[g];
        const int m = inst_model ? inst_model[g] : -1;
        if (pf->kv_tokens && pf->decode_time && pf->ineff && pf->mean_tokens && m >= 0) {
            const int64_t cm = (int64_t)pr->inst_class[g] * M + m;
            const double B = (double)pf->kv_tokens[cm] / (double)pf->mean_tokens[m];
            theta = B / ((double)pf->decode_time[cm] * (double)pf->ineff[cm]);
        }
        tput_out[g] = (float)theta;
    }
}

/* ------------------------------------------------------------------------
 * Plan search: a local search over plans.
 *
 * The paper's global scheduler places groups by solving the assignment
 * x_{g,i,j} of Sec. 7 as an LP and compares with EDF and with same-model
 * grouping (Secs. 2 and 8).  This library searches plans directly with the
 * scheduler's own actions on virtual queues as moves.  The first slot of a
 * non-empty queue holds the group its instance is running; a group that has
 * started does not go to another instance (Sec. 5, load balancing), and only
 * an eviction puts a group ahead of it (Sec. 5, request eviction):
 *
 *   SWAP(s, d)      reordering within a queue: the groups at slots s and
 *                   s + d (1 <= d <= W) trade places when both slots lie in
 *                   one queue and s is not its head;
 *   MOVE(s, h)      reassignment (load balancing, Sec. 5): the group at slot s
 *                   (not a head) leaves its queue g and joins queue h != g,
 *                   placed before the first group of h after h's head whose
 *                   SLO is strictly later than its own (at the end of h when
 *                   there is none; the head of h when h is empty);
 *   RELOCATE(s, h)  eviction: the group at slot s (not a head) leaves its
 *                   queue and becomes the head of the non-empty queue h (its
 *                   own queue or another), ahead of the running group, with
 *                   its eviction flag set.
 *
 * Any other moved group keeps its eviction flag (the flag belongs to the
 * group's placement, not to the slot number).  Moves are numbered
 *   SWAP(s, d):      k = s*W + (d - 1)             s in [0, G), d in [1, W]
 *   MOVE(s, h):      k = G*W + s*I + h             s in [0, G), h in [0, I)
 *   RELOCATE(s, h):  k = G*W + G*I + s*I + h       s in [0, G), h in [0, I)
 * and a number whose slot s is a queue's head, whose partner slot lies in
 * another queue (or beyond G), whose h is the group's own queue (MOVE) or an
 * empty queue (RELOCATE), names no move.
 *
 * One step scores every move (the exact score above of the plan the move
 * makes), takes the lowest score, the lowest k on ties, and applies that move
 * when its score is strictly below the current plan's; otherwise the search
 * has converged and stops.
 */
int64_t oracle_n_moves(int32_t G, int32_t I, int32_t W)
{
    return (int64_t)G * W + 2 * (int64_t)G * I;
}

/* queue holding slot s: the g with qoff[g] <= s < qoff[g+1] */
static int queue_of(const int32_t *qoff, int I, int32_t s)
{
    for (int g = 0; g < I; ++g)
        if (qoff[g] <= s && s < qoff[g + 1]) return g;
    return -1;
}

/* The plan with the group at slot s (not a head) taken out of its queue and
 * put into queue h: at the head with its flag set when `head`, else before
 * the first group after h's head (as h stands without the group) whose SLO is
 * strictly later, else at the end.  Written to (perm2, qoff2, flag2) queue by
 * queue. */
static void insert_into(const oracle_problem *pr, const int32_t *perm, const int32_t *qoff,
                        const uint8_t *flag, int32_t s, int h, int head, int32_t *perm2,
                        int32_t *qoff2, uint8_t *flag2)
{
    const int I = pr->n_instances;
    const int32_t gi = perm[s];
    const float slo_i = pr->grp_slo[gi];
    int32_t out = 0;
    for (int q = 0; q < I; ++q) {
        qoff2[q] = out;
        if (q == h && head) {
            perm2[out] = gi;  flag2[out] = 1;  ++out;
        }
        int placed = (q != h) || head;
        int seen = 0;                           /* groups of q already written */
        for (int32_t u = qoff[q]; u < qoff[q + 1]; ++u) {
            if (u == s) continue;                       /* the group leaves */
            if (!placed && seen > 0 && pr->grp_slo[perm[u]] > slo_i) {
                perm2[out] = gi;  flag2[out] = flag[s];  ++out;  placed = 1;
            }
            perm2[out] = perm[u];  flag2[out] = flag[u];  ++out;
            ++seen;
        }
        if (!placed) { perm2[out] = gi;  flag2[out] = flag[s];  ++out; }
    }
    qoff2[I] = out;
}

/* Applies move k to the plan (perm, qoff, flag) of one plan; writes the new
 * plan to (perm2, qoff2, flag2).  Returns 1 when k names a move, else 0
 * (outputs untouched). */
int oracle_move_apply(const oracle_problem *pr, int32_t W, int64_t k,
                      const int32_t *perm, const int32_t *qoff, const uint8_t *flag,
                      int32_t *perm2, int32_t *qoff2, uint8_t *flag2)
{
    const int G = pr->n_groups, I = pr->n_instances;
    if (k < 0 || k >= oracle_n_moves(G, I, W)) return 0;
    if (k < (int64_t)G * W) {                                  /* SWAP */
        const int32_t s = (int32_t)(k / W), t = s + (int32_t)(k % W) + 1;
        if (t >= G) return 0;
        const int g = queue_of(qoff, I, s);
        if (s == qoff[g] || t >= qoff[g + 1]) return 0;
        memcpy(perm2, perm, sizeof(int32_t) * G);
        memcpy(qoff2, qoff, sizeof(int32_t) * (I + 1));
        memcpy(flag2, flag, G);
        perm2[s] = perm[t];  perm2[t] = perm[s];
        flag2[s] = flag[t];  flag2[t] = flag[s];
        return 1;
    }
    int64_t r = k - (int64_t)G * W;
    const int relocate = r >= (int64_t)G * I;
    if (relocate) r -= (int64_t)G * I;
    const int32_t s = (int32_t)(r / I);
    const int h = (int)(r % I);
    const int g = queue_of(qoff, I, s);
    if (s == qoff[g]) return 0;                          /* the running group */
    if (relocate ? qoff[h] == qoff[h + 1] : h == g) return 0;
    insert_into(pr, perm, qoff, flag, s, h, relocate, perm2, qoff2, flag2);
    return 1;
}

/* Exact score of one plan given as arrays (flags one byte per slot; a search
 * can set flags, so they are always passed). */
static double score_one(const oracle_problem *pr, const int32_t *perm, const int32_t *qoff,
                        const uint8_t *flag, uint32_t *words)
{
    const int G = pr->n_groups;
    oracle_plans one;
    one.n_plans = 1;
    one.ld = 1;
    one.perm = perm;
    one.qoff = qoff;
    memset(words, 0, sizeof(uint32_t) * (size_t)((G + 31) / 32));
    for (int s = 0; s < G; ++s)
        if (flag[s]) words[s / 32] |= 1u << (s % 32);
    one.evict_bits = words;
    double sc = NAN;
    if (oracle_plan(pr, &one, 0, NULL, NULL, NULL, &sc, NULL) != 0) return NAN;
    return sc;
}

/* The plan p of a batch as arrays. */
static void take_plan(const oracle_problem *pr, const oracle_plans *pl, int64_t p,
                      int32_t *perm, int32_t *qoff, uint8_t *flag)
{
    for (int s = 0; s < pr->n_groups; ++s) {
        perm[s] = pl->perm[(int64_t)s * pl->ld + p];
        flag[s] = (uint8_t)evicted(pl, p, s);
    }
    for (int g = 0; g <= pr->n_instances; ++g) qoff[g] = pl->qoff[(int64_t)g * pl->ld + p];
}

/* Scores of moves of one plan given as arrays: ks[0..n) (NULL = every move,
 * n = oracle_n_moves).  A number that names no move scores +inf. */
static void move_scores_of(const oracle_problem *pr, int32_t W, const int32_t *perm,
                           const int32_t *qoff, const uint8_t *flag, const int64_t *ks,
                           int64_t n, double *out, int n_threads)
{
    const int G = pr->n_groups, I = pr->n_instances;
#ifdef _OPENMP
    if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel num_threads(n_threads)
#endif
    {
        int32_t *perm2 = malloc(sizeof(int32_t) * G);
        int32_t *qoff2 = malloc(sizeof(int32_t) * (I + 1));
        uint8_t *flag2 = malloc(G);
        uint32_t *words = malloc(sizeof(uint32_t) * ((G + 31) / 32));
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 64)
#endif
        for (int64_t j = 0; j < n; ++j) {
            const int64_t k = ks ? ks[j] : j;
            if (oracle_move_apply(pr, W, k, perm, qoff, flag, perm2, qoff2, flag2))
                out[j] = score_one(pr, perm2, qoff2, flag2, words);
            else
                out[j] = INFINITY;
        }
        free(perm2); free(qoff2); free(flag2); free(words);
    }
    (void)n_threads;
}

/* Scores of moves ks[0..n) (NULL = all) of plan p of the batch. */
int oracle_move_scores(const oracle_problem *pr, const oracle_plans *pl, int64_t p, int32_t W,
                       const int64_t *ks, int64_t n, double *out, int n_threads)
{
    const int G = pr->n_groups, I = pr->n_instances;
    int32_t *perm = malloc(sizeof(int32_t) * G);
    int32_t *qoff = malloc(sizeof(int32_t) * (I + 1));
    uint8_t *flag = malloc(G);
    take_plan(pr, pl, p, perm, qoff, flag);
    if (!ks) n = oracle_n_moves(G, I, W);
    move_scores_of(pr, W, perm, qoff, flag, ks, n, out, n_threads);
    free(perm); free(qoff); free(flag);
    return 0;
}

/* Local search from plan p of the batch, at most max_steps steps.  Writes the
 * final plan (perm_out[G], qoff_out[I+1], evict_out[ceil(G/32)] or NULL), its
 * exact score, the number of moves applied, and trace[max_steps] (the move
 * applied at each step, -1 from the step that found no improving move on). */
int oracle_local_search(const oracle_problem *pr, const oracle_plans *pl, int64_t p, int32_t W,
                        int32_t max_steps, int32_t *perm_out, int32_t *qoff_out,
                        uint32_t *evict_out, double *score, int32_t *steps, int64_t *trace,
                        int n_threads)
{
    const int G = pr->n_groups, I = pr->n_instances;
    const int64_t nm = oracle_n_moves(G, I, W);
    int32_t *perm = malloc(sizeof(int32_t) * G), *perm2 = malloc(sizeof(int32_t) * G);
    int32_t *qoff = malloc(sizeof(int32_t) * (I + 1)), *qoff2 = malloc(sizeof(int32_t) * (I + 1));
    uint8_t *flag = malloc(G), *flag2 = malloc(G);
    uint32_t *words = malloc(sizeof(uint32_t) * ((G + 31) / 32));
    double *sc = malloc(sizeof(double) * (size_t)(nm > 0 ? nm : 1));
    take_plan(pr, pl, p, perm, qoff, flag);
    double cur = score_one(pr, perm, qoff, flag, words);
    int32_t done = 0;
    for (int32_t t = 0; t < max_steps; ++t) trace[t] = -1;
    for (int32_t t = 0; t < max_steps; ++t) {
        move_scores_of(pr, W, perm, qoff, flag, NULL, nm, sc, n_threads);
        int64_t best = -1;
        double bs = INFINITY;
        for (int64_t k = 0; k < nm; ++k)
            if (sc[k] < bs) { bs = sc[k]; best = k; }
        if (best < 0 || !(bs < cur)) break;             /* converged */
        oracle_move_apply(pr, W, best, perm, qoff, flag, perm2, qoff2, flag2);
        memcpy(perm, perm2, sizeof(int32_t) * G);
        memcpy(qoff, qoff2, sizeof(int32_t) * (I + 1));
        memcpy(flag, flag2, G);
        cur = score_one(pr, perm, qoff, flag, words);
        trace[t] = best;
        ++done;
    }
    memcpy(perm_out, perm, sizeof(int32_t) * G);
    memcpy(qoff_out, qoff, sizeof(int32_t) * (I + 1));
    if (evict_out) {
        memset(evict_out, 0, sizeof(uint32_t) * (size_t)((G + 31) / 32));
        for (int s = 0; s < G; ++s)
            if (flag[s]) evict_out[s / 32] |= 1u << (s % 32);
    }
    *score = cur;
    *steps = done;
    free(perm); free(perm2); free(qoff); free(qoff2); free(flag); free(flag2); free(words); free(sc);
    return 0;
}

/* ------------------------------------------------------------------------
 * Seed plans for the search: the paper's reference orders.
 *
 *   policy 0, EDF: groups taken by SLO (earliest deadline first, the EDF
 *             baseline of Sec. 8), ties by group id;
 *   policy 1, grouped: groups taken by model, then SLO, then id (same-model
 *             requests kept together to avoid repeated model swaps, Sec. 2,
 *             Insight #3).
 *
 * Groups are placed one at a time, in that order, at the end of the queue
 * whose drain time after taking the group is smallest (load balancing by
 * queue drain time, Sec. 8's load-balancing study): for queue q holding
 * tokens A_q and fixed costs K_q, whose last model is l_q (the loaded model
 * inst_model0[q] while empty, -1 = none),
 *   drain_q(i) = (A_q + n_i mu_i) / Theta_q + (K_q + s),
 *   s = S[class_q][l_q][m_i] if l_q >= 0 and l_q != m_i, else 0,
 * the lowest q on ties.  Seeds evict nothing.
 */
static const oracle_problem *g_seed_pr;
static int g_seed_policy;

static int seed_cmp(const void *pa, const void *pb)
{
    const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    const oracle_problem *pr = g_seed_pr;
    if (g_seed_policy == 1 && pr->grp_model[a] != pr->grp_model[b])
        return pr->grp_model[a] < pr->grp_model[b] ? -1 : 1;
    if (pr->grp_slo[a] < pr->grp_slo[b]) return -1;
    if (pr->grp_slo[a] > pr->grp_slo[b]) return 1;
    return a < b ? -1 : (a > b ? 1 : 0);
}

/* One seed plan: perm_out[G], qoff_out[I+1].  Returns 0, or -1 on a bad policy. */
int oracle_seed_plan(const oracle_problem *pr, int32_t policy, int32_t *perm_out,
                     int32_t *qoff_out)
{
    const int G = pr->n_groups, I = pr->n_instances, M = pr->n_models;
    if (policy != 0 && policy != 1) return -1;
    int32_t *order = malloc(sizeof(int32_t) * G);
    int32_t *owner = malloc(sizeof(int32_t) * G);
    double *A = calloc((size_t)I, sizeof(double)), *K = calloc((size_t)I, sizeof(double));
    int32_t *last = malloc(sizeof(int32_t) * I), *count = calloc((size_t)I, sizeof(int32_t));
    for (int i = 0; i < G; ++i) order[i] = i;
    g_seed_pr = pr;
    g_seed_policy = policy;
    qsort(order, (size_t)G, sizeof(int32_t), seed_cmp);
    for (int q = 0; q < I; ++q) last[q] = pr->inst_model0 ? pr->inst_model0[q] : -1;
    for (int k = 0; k < G; ++k) {
        const int i = order[k];
        const int m = pr->grp_model[i];
        const double a = (double)pr->grp_count[i] * (double)pr->grp_mu[i];
        int best = -1;
        double bd = INFINITY;
        for (int q = 0; q < I; ++q) {
            double s = 0.0;
            if (last[q] >= 0 && last[q] != m && pr->swap_cost)
                s = (double)pr->swap_cost[((int64_t)pr->inst_class[q] * M + last[q]) * M + m];
            const double d = (A[q] + a) / (double)pr->inst_tput[q] + (K[q] + s);
            if (d < bd) { bd = d; best = q; }
        }
        if (best < 0) best = 0;                        /* all NaN: the first queue */
        {
            double s = 0.0;
            if (last[best] >= 0 && last[best] != m && pr->swap_cost)
                s = (double)pr->swap_cost[((int64_t)pr->inst_class[best] * M + last[best]) * M + m];
            A[best] += a;
            K[best] += s;
        }
        last[best] = m;
        owner[k] = best;
        count[best] += 1;
    }
    qoff_out[0] = 0;
    for (int q = 0; q < I; ++q) qoff_out[q + 1] = qoff_out[q] + count[q];
    for (int q = 0; q < I; ++q) count[q] = 0;
    for (int k = 0; k < G; ++k) {
        const int q = owner[k];
        perm_out[qoff_out[q] + count[q]] = order[k];
        count[q] += 1;
    }
    free(order); free(owner); free(A); free(K); free(last); free(count);
    return 0;
}

/* ------------------------------------------------------------------------
 * Placement of one group (a new arrival parked behind the head of a queue, or
 * a group whose wait violates its SLO): the scheduler call of Sec. 5 for one
 * group.  The group leaves its slot and goes to one of 2I places c:
 *   c = h       queue h before the first group after h's head (as h stands
 *               without the group) whose SLO is strictly later, at the end
 *               when there is none, at the head of an empty h; its flag kept
 *               (the MOVE of the search; with h its own queue, a reinsertion);
 *   c = I + h   the head of the non-empty queue h, ahead of the running
 *               group, with its eviction flag set (the RELOCATE of the search).
 * The c giving the lowest exact plan score wins, the lowest c on ties (c = 0
 * when every score is NaN).  A group at its queue's head is running and stays
 * where it is: the plan comes back unchanged and c is its queue.
 */

/* Places group `group` of plan p; writes the new plan, its exact score and the
 * chosen place c.  Returns 0, or -1 when the group is not in the plan. */
int oracle_place_group(const oracle_problem *pr, const oracle_plans *pl, int64_t p, int32_t group,
                       int32_t *perm_out, int32_t *qoff_out, uint32_t *evict_out, double *score,
                       int32_t *queue)
{
    const int G = pr->n_groups, I = pr->n_instances;
    int32_t *perm = malloc(sizeof(int32_t) * G), *perm2 = malloc(sizeof(int32_t) * G);
    int32_t *qoff = malloc(sizeof(int32_t) * (I + 1)), *qoff2 = malloc(sizeof(int32_t) * (I + 1));
    uint8_t *flag = malloc(G), *flag2 = malloc(G);
    uint32_t *words = malloc(sizeof(uint32_t) * ((G + 31) / 32));
    take_plan(pr, pl, p, perm, qoff, flag);
    int32_t s = -1;
    for (int u = 0; u < G; ++u)
        if (perm[u] == group) s = u;
    if (s >= 0) {
        const int g = queue_of(qoff, I, s);
        int best = -1;
        if (s == qoff[g]) {                              /* running: it stays */
            memcpy(perm2, perm, sizeof(int32_t) * G);
            memcpy(qoff2, qoff, sizeof(int32_t) * (I + 1));
            memcpy(flag2, flag, G);
            best = g;
        } else {
            double bs = INFINITY;
            for (int c = 0; c < 2 * I; ++c) {
                const int head = c >= I, h = head ? c - I : c;
                if (head && qoff[h] == qoff[h + 1]) continue;   /* nothing to evict */
                insert_into(pr, perm, qoff, flag, s, h, head, perm2, qoff2, flag2);
                const double sc = score_one(pr, perm2, qoff2, flag2, words);
                if (sc < bs) { bs = sc; best = c; }
            }
            if (best < 0) best = 0;
            insert_into(pr, perm, qoff, flag, s, best >= I ? best - I : best, best >= I, perm2,
                        qoff2, flag2);
        }
        memcpy(perm_out, perm2, sizeof(int32_t) * G);
        memcpy(qoff_out, qoff2, sizeof(int32_t) * (I + 1));
        if (evict_out) {
            memset(evict_out, 0, sizeof(uint32_t) * (size_t)((G + 31) / 32));
            for (int u = 0; u < G; ++u)
                if (flag2[u]) evict_out[u / 32] |= 1u << (u % 32);
        }
        *score = score_one(pr, perm2, qoff2, flag2, words);
        *queue = best;
    }
    free(perm); free(perm2); free(qoff); free(qoff2); free(flag); free(flag2); free(words);
    return s >= 0 ? 0 : -1;
}
