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
 * The readings behind the choices that the paper leaves open (probability of
 * violation as the score, the group's own swap counted in its waiting time,
 * eviction as a fixed cost, the exclusive token prefix) are listed in the
 * design notes of the repository.
 *
 * Parity status: every function here is pinned by tests (closed forms,
 * textbook normal-table values, invariants, Monte Carlo of the stated Normal
 * model, brute force over orderings on tiny inputs).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

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
