"""The pins must catch plausible mistakes in the oracle.

Each case below plants one mistake in a copy of oracle/qlm_oracle.c (on the CPU,
in a temporary directory), builds it with gcc, and runs every pin against it; at
least one pin must fail.  A mutant that survives means a blind spot in the pins.
The pins run in a child process: a mistake in an index can make the mutant
read out of bounds, and a crash there (reported as such) must not take the
test run down with it.
"""
import json
import os
import signal
import subprocess
import sys

import pytest

import oracle
import pins

_SRC = os.path.join(os.path.dirname(oracle.__file__), "qlm_oracle.c")

# (name, text in the committed source, replacement)
MUTANTS = [
    ("inclusive_token_prefix",
     "const double EW = A / theta + K;",
     "A += n * mu; const double EW = A / theta + K; A -= n * mu;"),
    ("tokens_not_scaled_by_count", "A += n * mu;", "A += mu;"),
    ("variance_not_scaled_by_count", "V += n * var;", "V += var;"),
    ("variance_scaled_by_count_squared", "V += n * var;", "V += n * n * var;"),
    ("sd_without_sqrt", "const double SD = sqrt(V) / theta;", "const double SD = V / theta;"),
    ("sd_divided_by_theta_squared", "const double SD = sqrt(V) / theta;",
     "const double SD = sqrt(V) / (theta * theta);"),
    ("tokens_times_theta", "const double EW = A / theta + K;", "const double EW = A * theta + K;"),
    ("z_sign_flipped", "erfc((slo - EW) / (SD * sqrt(2.0)))", "erfc((EW - slo) / (SD * sqrt(2.0)))"),
    ("missing_sqrt2", "erfc((slo - EW) / (SD * sqrt(2.0)))", "erfc((slo - EW) / SD)"),
    ("missing_half", "P = 0.5 * erfc(", "P = erfc("),
    ("erf_instead_of_erfc", "P = 0.5 * erfc(", "P = 0.5 * erf("),
    ("sd_zero_non_strict", "P = (EW > slo) ? 1.0 : 0.0;", "P = (EW >= slo) ? 1.0 : 0.0;"),
    ("swap_dropped",
     "K += (double)pr->swap_cost[((int64_t)cls * M + m_prev) * M + m];", "(void)cls;"),
    ("swap_transposed",
     "pr->swap_cost[((int64_t)cls * M + m_prev) * M + m]",
     "pr->swap_cost[((int64_t)cls * M + m) * M + m_prev]"),
    ("swap_class_ignored",
     "pr->swap_cost[((int64_t)cls * M + m_prev) * M + m]",
     "pr->swap_cost[((int64_t)0 * M + m_prev) * M + m]"),
    ("swap_paid_after_the_group",     # the literal sum over k < j of the LP
     "            if (m_prev >= 0 && m_prev != m && pr->swap_cost)\n"
     "                K += (double)pr->swap_cost[((int64_t)cls * M + m_prev) * M + m];\n",
     "            const double K_before = K;\n"
     "            if (m_prev >= 0 && m_prev != m && pr->swap_cost)\n"
     "                K += (double)pr->swap_cost[((int64_t)cls * M + m_prev) * M + m];\n"
     "            const double K_swap = K - K_before; K = K_before;\n"),
    ("head_model_ignored", "int m_prev = pr->inst_model0 ? pr->inst_model0[g] : -1;",
     "int m_prev = -1;"),
    ("eviction_dropped", "K += (double)pr->evict_cost;", "(void)0;"),
    ("eviction_bit_off_by_one", "return (int)((w >> (s % 32)) & 1u);",
     "return (int)((w >> ((s + 1) % 32)) & 1u);"),
    ("costs_not_carried", "double K = 0.0;   /* swap", "double K = 0.0; double K0 = 0.0; /* swap"),
    ("score_not_weighted_by_count", "score_g   += n * P;", "score_g   += P;"),
    ("penalty_sign", "penalty_g += EW - slo;", "penalty_g += slo - EW;"),
    ("prefix_not_reset_per_queue", "        double A = 0.0;   /* tokens",
     "        static double A_carry = 0.0; double A = A_carry; (void)A_carry;   /* tokens"),
    ("argmin_last_on_ties", "if (score[p] < bs) {", "if (score[p] <= bs) {"),
    ("theta_of_first_queue", "const double theta = (double)pr->inst_tput[g];",
     "const double theta = (double)pr->inst_tput[0];"),
    # plan search
    ("insert_before_equal_slo", "seen > 0 && pr->grp_slo[perm[u]] > slo_i) {",
     "seen > 0 && pr->grp_slo[perm[u]] >= slo_i) {"),
    ("insert_before_earlier_slo", "seen > 0 && pr->grp_slo[perm[u]] > slo_i) {",
     "seen > 0 && pr->grp_slo[perm[u]] < slo_i) {"),
    ("insert_passes_running_head", "if (!placed && seen > 0 && ", "if (!placed && "),
    ("swap_flags_stay", "flag2[s] = flag[t];  flag2[t] = flag[s];", "(void)0;"),
    ("move_flag_dropped", "perm2[out] = gi;  flag2[out] = flag[s];  ++out;  placed = 1;",
     "perm2[out] = gi;  flag2[out] = 0;  ++out;  placed = 1;"),
    ("swap_across_queues", "if (s == qoff[g] || t >= qoff[g + 1]) return 0;",
     "if (s == qoff[g]) return 0;"),
    ("swap_takes_running_head", "if (s == qoff[g] || t >= qoff[g + 1]) return 0;",
     "if (t >= qoff[g + 1]) return 0;"),
    ("swap_distance_short", "t = s + (int32_t)(k % W) + 1;", "t = s + (int32_t)(k % W);"),
    ("move_index_transposed",
     "const int32_t s = (int32_t)(r / I);\n    const int h = (int)(r % I);",
     "const int32_t s = (int32_t)(r % G);\n    const int h = (int)(r / G);"),
    ("move_takes_running_head",
     "if (s == qoff[g]) return 0;                          /* the running group */", "(void)0;"),
    ("relocate_flag_not_set", "perm2[out] = gi;  flag2[out] = 1;  ++out;",
     "perm2[out] = gi;  flag2[out] = flag[s];  ++out;"),
    ("relocate_into_empty_queue", "if (relocate ? qoff[h] == qoff[h + 1] : h == g) return 0;",
     "if (relocate ? 0 : h == g) return 0;"),
    ("relocate_not_to_own_queue", "if (relocate ? qoff[h] == qoff[h + 1] : h == g) return 0;",
     "if (relocate ? (qoff[h] == qoff[h + 1] || h == g) : h == g) return 0;"),
    ("relocate_index_off_by_one", "if (relocate) r -= (int64_t)G * I;",
     "if (relocate) r -= (int64_t)G * I - 1;"),
    ("relocate_to_edf_place", "insert_into(pr, perm, qoff, flag, s, h, relocate, perm2, qoff2, flag2);",
     "insert_into(pr, perm, qoff, flag, s, h, 0, perm2, qoff2, flag2);"),
    ("relocate_moves_not_counted", "return (int64_t)G * W + 2 * (int64_t)G * I;",
     "return (int64_t)G * W + (int64_t)G * I;"),
    ("last_move_on_ties", "if (sc[k] < bs) { bs = sc[k]; best = k; }",
     "if (sc[k] <= bs) { bs = sc[k]; best = k; }"),
    ("move_on_equal_score", "if (best < 0 || !(bs < cur)) break;",
     "if (best < 0 || !(bs <= cur)) break;"),
    # seed plans
    ("seed_last_queue_on_ties", "if (d < bd) { bd = d; best = q; }",
     "if (d <= bd) { bd = d; best = q; }"),
    ("seed_grouping_ignores_model", "if (g_seed_policy == 1 && pr->grp_model[a] != pr->grp_model[b])",
     "if (g_seed_policy == 2 && pr->grp_model[a] != pr->grp_model[b])"),
    ("seed_latest_deadline_first",
     "if (pr->grp_slo[a] < pr->grp_slo[b]) return -1;\n    if (pr->grp_slo[a] > pr->grp_slo[b]) return 1;",
     "if (pr->grp_slo[a] > pr->grp_slo[b]) return -1;\n    if (pr->grp_slo[a] < pr->grp_slo[b]) return 1;"),
    ("seed_drain_without_own_tokens",
     "const double d = (A[q] + a) / (double)pr->inst_tput[q] + (K[q] + s);",
     "const double d = A[q] / (double)pr->inst_tput[q] + (K[q] + s);"),
    ("seed_swap_not_kept", "            K[best] += s;", "            (void)s;"),
    # placement of one group
    ("place_last_place_on_ties", "if (sc < bs) { bs = sc; best = c; }",
     "if (sc <= bs) { bs = sc; best = c; }"),
    ("place_own_queue_skipped",
     "                insert_into(pr, perm, qoff, flag, s, h, head, perm2, qoff2, flag2);\n",
     "                if (!head && h == g) continue;\n"
     "                insert_into(pr, perm, qoff, flag, s, h, head, perm2, qoff2, flag2);\n"),
    ("place_without_head_places", "for (int c = 0; c < 2 * I; ++c) {",
     "for (int c = 0; c < I; ++c) {"),
    ("place_running_group_moved", "if (s == qoff[g]) {                              /* running: it stays */",
     "if (0) {"),
    # per-request (FCFS) variant
    ("fcfs_own_requests_dropped", "const double Er  = EW + (double)r * (mu / theta);",
     "const double Er  = EW;"),
    ("fcfs_own_variance_dropped", "sqrt(V + (double)r * var)", "sqrt(V)"),
    ("fcfs_own_request_counted", "(double)r * (mu / theta)", "(double)(r + 1) * (mu / theta)"),
    ("fcfs_variance_times_r_squared", "sqrt(V + (double)r * var)", "sqrt(V + (double)r * r * var)"),
    ("fcfs_mean_over_theta_squared", "(double)r * (mu / theta)", "(double)r * (mu / (theta * theta))"),
    ("fcfs_group_slo_for_all", "(double)req_slo[first[i] + r];", "(double)req_slo[first[i]];"),
    ("fcfs_reversed_arrival", "(double)req_slo[first[i] + r];", "(double)req_slo[first[i] + (n - 1 - r)];"),
    ("fcfs_sd_zero_non_strict", "P = (Er > slo) ? 1.0 : 0.0;", "P = (Er >= slo) ? 1.0 : 0.0;"),
    ("fcfs_weighted_by_count", "slot += P;", "slot += (double)n * P;"),
    ("fcfs_eviction_dropped",
     "                K += (double)pr->evict_cost;\n\n            const double EW = A / theta + K;  "
     "               /* the group's start */",
     "                (void)0;\n\n            const double EW = A / theta + K;"),
    ("fcfs_head_model_ignored",
     "int m_prev = pr->inst_model0 ? pr->inst_model0[g] : -1;\n        double A = 0.0, V = 0.0, K = 0.0;",
     "int m_prev = -1;\n        double A = 0.0, V = 0.0, K = 0.0;"),
    # problem tables from a hardware profile
    ("profile_drain_of_new_model", "const int64_t ca = (int64_t)c * M + a;",
     "const int64_t ca = (int64_t)c * M + b;"),
    ("profile_drain_without_prefill", "S = S + ((double)pf->prefill[a] + D);", "S = S + D;"),
    ("profile_drain_on_diagonal", "if (drain && a != b) {", "if (drain) {"),
    ("profile_drain_without_ineff",
     "const double D = (double)pf->max_tokens[a] * (double)pf->ineff[ca] *",
     "const double D = (double)pf->max_tokens[a] * 1.0 *"),
    ("profile_prefill_added", "if (pf->prefill) slo = slo - (double)pf->prefill[pr->grp_model[i]];",
     "if (pf->prefill) slo = slo + (double)pf->prefill[pr->grp_model[i]];"),
    ("profile_theta_ineff_inverted",
     "theta = B / ((double)pf->decode_time[cm] * (double)pf->ineff[cm]);",
     "theta = B * (double)pf->ineff[cm] / (double)pf->decode_time[cm];"),
    ("profile_batch_inverted",
     "const double B = (double)pf->kv_tokens[cm] / (double)pf->mean_tokens[m];",
     "const double B = (double)pf->mean_tokens[m] / (double)pf->kv_tokens[cm];"),
    ("profile_class_of_first_instance",
     "const int64_t cm = (int64_t)pr->inst_class[g] * M + m;",
     "const int64_t cm = (int64_t)pr->inst_class[0] * M + m;"),
]


def _fix_costs_not_carried(src):
    # make the eviction/swap total restart at every position (K not carried)
    return src.replace("            if (m_prev >= 0 && m_prev != m && pr->swap_cost)",
                       "            K = K0;\n            if (m_prev >= 0 && m_prev != m && pr->swap_cost)",
                       1)


def _fix_swap_after(src):
    # the swap reaches the waits of later groups only
    return src.replace("            A += n * mu;\n", "            A += n * mu; K += K_swap;\n")


def _fix_prefix_carry(src):
    return src.replace("            A += n * mu;\n", "            A += n * mu; A_carry = A;\n")


def _mutant_source(name, old, new):
    src = open(_SRC).read()
    assert src.count(old) >= 1, name
    src = src.replace(old, new, 1)
    if name == "costs_not_carried":
        src = _fix_costs_not_carried(src)
    if name == "swap_paid_after_the_group":
        src = _fix_swap_after(src)
    if name == "prefix_not_reset_per_queue":
        src = _fix_prefix_carry(src)
    return src


def _run_mutant(tmp, name, old, new):
    """Builds the mutant and runs the pins on it in a child process; returns
    (return code, failed pins or the child's error output)."""
    src = _mutant_source(name, old, new)
    c = os.path.join(tmp, name + ".c")
    so = os.path.join(tmp, "lib" + name + ".so")
    with open(c, "w") as f:
        f.write(src)
    subprocess.run(["gcc", "-O1", "-fopenmp", "-ffp-contract=off", "-std=c11", "-shared", "-fPIC",
                    "-w", "-o", so, c, "-lm"], check=True)
    here = os.path.dirname(os.path.abspath(__file__))
    env = dict(os.environ, OMP_NUM_THREADS="1",
               PYTHONPATH=os.pathsep.join([here, os.path.dirname(here),
                                           os.environ.get("PYTHONPATH", "")]))
    child = subprocess.run([sys.executable, "-c", _CHILD, so], capture_output=True, text=True,
                           cwd=here, timeout=900, env=env)
    if child.returncode != 0:
        return child.returncode, child.stderr[-2000:]
    return 0, json.loads(child.stdout.strip().splitlines()[-1])


@pytest.fixture(scope="module")
def mutant_results(tmp_path_factory):
    """Every mutant's result, the children run side by side."""
    from concurrent.futures import ThreadPoolExecutor
    tmp = str(tmp_path_factory.mktemp("mutants"))
    workers = max(1, min(8, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        futs = {m[0]: ex.submit(_run_mutant, tmp, *m) for m in MUTANTS}
        return {k: f.result() for k, f in futs.items()}


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_mutant_is_caught(mutant_results, name):
    rc, out = mutant_results[name]
    if rc < 0:
        # killed by a signal inside the mutant (an access out of bounds): the
        # mistake did not pass unnoticed
        print("mutant %s crashed the oracle (%s)" % (name, signal.Signals(-rc).name))
        return
    assert rc == 0, out
    print("mutant %s caught by %s" % (name, ", ".join(out)))
    assert out, "mutant %s survived every pin" % name


# Runs every pin against the oracle library named on the command line and
# prints the names of the pins that failed, as one JSON line.
_CHILD = """
import json, sys
import oracle, pins
orc = oracle.Oracle(sys.argv[1])
failed = []
for pin in pins.ALL_PINS:
    try:
        pin(orc)
    except (AssertionError, ValueError, FloatingPointError):
        failed.append(pin.__name__)
print(json.dumps(failed))
"""
