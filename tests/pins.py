"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each ``pin_*`` takes a loaded oracle (``oracle.Oracle``) and raises
AssertionError when the oracle disagrees.  They are run against the committed
oracle by ``test_oracle_pins.py`` and against deliberately broken builds of it
by ``test_oracle_mutants.py`` (every planted mistake must fail at least one).

Expected values are hand-derived for hand-built inputs, textbook normal-table
values (tests/golden/normal_upper_tail.txt), invariants, a Monte Carlo of the
stated Normal model, or brute force over all orderings of tiny inputs.
"""
from __future__ import annotations

import os

import numpy as np

from cases import all_orders, plans, problem

_GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def normal_table():
    rows = []
    with open(os.path.join(_GOLDEN, "normal_upper_tail.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                z, q = line.split()
                rows.append((float(z), float(q)))
    return rows


# ---------------------------------------------------------------------------
# Closed forms on hand-built queues


def pin_deterministic_queue(orc):
    """One queue, sigma^2 = 0 (Sec. 6, Eq. base_equation with known tokens).
    Each group carries n*mu = 400 tokens and Theta = 400 tok/s, so the group at
    position j waits exactly j seconds (the tokens of the j groups ahead)."""
    n = [4, 2, 8, 1, 5]
    mu = [100, 200, 50, 400, 80]
    slo = [0.5, 0.5, 2.5, 3.0, 10.0]
    pr = problem([(n[k], mu[k], 0.0, 0, slo[k]) for k in range(5)], [(400.0, 0)])
    pl = plans([[[0, 1, 2, 3, 4]]], 5)
    d = orc.plan_detail(pr, pl, 0)
    assert np.array_equal(d["wait_mean"], [0.0, 1.0, 2.0, 3.0, 4.0]), d["wait_mean"]
    assert np.array_equal(d["wait_sd"], [0.0] * 5), d["wait_sd"]
    # SD = 0: violated iff the wait strictly exceeds the SLO; 3.0 > 3.0 is met
    assert np.array_equal(d["prob"], [0.0, 1.0, 0.0, 0.0, 0.0]), d["prob"]
    assert d["score"] == 2.0, d["score"]          # n of the violated group
    assert d["penalty"] == -6.5, d["penalty"]     # sum of (wait - slo), Eq. penalty
    # a different order moves the waits with the groups
    pl2 = plans([[[4, 3, 2, 1, 0]]], 5)
    d2 = orc.plan_detail(pr, pl2, 0)
    assert np.array_equal(d2["wait_mean"], [0.0, 1.0, 2.0, 3.0, 4.0])
    # slots hold groups 4,3,2,1,0 (slo 10, 3, 2.5, .5, .5) waiting 0..4 s: groups 1 and 0
    # (n = 2 and 4) miss their SLO
    assert np.array_equal(d2["prob"], [0.0, 0.0, 0.0, 1.0, 1.0]), d2["prob"]
    assert d2["score"] == 2.0 + 4.0


def pin_variance_queue(orc):
    """Same queue with n*sigma^2 = 40000 per group (Eq. output_token_dist): the
    variance of the tokens ahead adds up, so SD[W_j] = sqrt(40000 j)/400 = sqrt(j)/2.
    SLOs are placed at exact z-scores, so P(W > slo) = Q(z) from the normal table."""
    n = [4, 2, 8, 1, 5]
    mu = [100, 200, 50, 400, 80]
    var = [10000, 20000, 5000, 40000, 8000]
    table = dict(normal_table())
    # wait = 0,1,2,3,4 ; sd = 0, .5, .707, .866, 1
    slo = [10.0, 2.0, 2.0, 1.0e9, 5.0]            # z: -, 2, 0, huge, 1
    pr = problem([(n[k], mu[k], var[k], 0, slo[k]) for k in range(5)], [(400.0, 0)])
    pl = plans([[[0, 1, 2, 3, 4]]], 5)
    d = orc.plan_detail(pr, pl, 0)
    sd = np.array([0.0, 0.5, np.sqrt(2.0) / 2, np.sqrt(3.0) / 2, 1.0])
    assert np.allclose(d["wait_sd"], sd, rtol=1e-15, atol=0), d["wait_sd"]
    want = [0.0, table[2.0], 0.5, 0.0, table[1.0]]
    assert np.allclose(d["prob"], want, rtol=1e-12, atol=1e-15), (d["prob"], want)
    assert abs(d["score"] - (2 * table[2.0] + 8 * 0.5 + 5 * table[1.0])) < 1e-12
    # mirrored SLOs: z = -2 at slot 1 and z = -1 at slot 4 give 1 - Q(z)
    slo_m = [10.0, 0.0, 2.0, 1.0e9, 3.0]
    pr_m = problem([(n[k], mu[k], var[k], 0, slo_m[k]) for k in range(5)], [(400.0, 0)])
    dm = orc.plan_detail(pr_m, pl, 0)
    assert abs(dm["prob"][1] - (1 - table[2.0])) < 1e-13, dm["prob"]
    assert abs(dm["prob"][4] - (1 - table[1.0])) < 1e-13, dm["prob"]


def pin_normal_table(orc):
    """P(W > slo) against the textbook Q(z) at every tabulated z, both signs.
    A head group of 400 tokens with variance 160000 on Theta = 400 gives the
    second group W ~ N(1, 1) (seconds), so slo = 1 + z puts it at z."""
    rows = normal_table()
    for z, q in rows:
        for sign in (+1, -1):
            slo = 1.0 + sign * z
            pr = problem([(1, 400.0, 160000.0, 0, 100.0), (3, 7.0, 9.0, 0, slo)], [(400.0, 0)])
            d = orc.plan_detail(pr, plans([[[0, 1]]], 2), 0)
            assert d["wait_mean"][1] == 1.0 and d["wait_sd"][1] == 1.0
            want = q if sign > 0 else 1.0 - q
            got = d["prob"][1]
            assert abs(got - want) <= 1e-12 * max(want, 1e-300) + 1e-15, (z, sign, got, want)
            assert abs(d["score"] - 3 * want) <= 1e-12 * 3 * max(want, 1e-300) + 1e-15


def _swap_table():
    """[C=2][M=3][M=3] swap costs, from-model row, to-model column; every
    off-diagonal entry distinct (100c + 10a + b + 1) so that a transposed or
    misplaced lookup shows; the diagonal is never a swap and holds 5000."""
    S = np.zeros((2, 3, 3), np.float32)
    for c in range(2):
        for a in range(3):
            for b in range(3):
                S[c, a, b] = 5000.0 if a == b else 100 * c + 10 * a + b + 1
    return S


def pin_swap_costs(orc):
    """Model transitions (Sec. 7, Eq. transition_time) add the swap time to the
    waiting time of the group whose model is loaded and of every group behind it.
    No tokens (mu = 0), so the wait is the swap sum alone."""
    models = [0, 1, 1, 2, 0, 2, 2, 0]
    groups = [(1, 0.0, 0.0, m, 1e6) for m in models]
    pr = problem(groups, [(400.0, 1), (250.0, 0)], n_models=3, n_classes=2,
                 swap=_swap_table(), model0=[-1, 1])
    pl = plans([[[0, 1, 2, 3, 4], [5, 6, 7]]], 8)
    d = orc.plan_detail(pr, pl, 0)
    # queue 0 (class 1, nothing loaded): 0->1 costs 102, 1->2 costs 113, 2->0 costs 121
    # queue 1 (class 0, model 1 loaded): head 1->2 costs 13, then 2->2 free, 2->0 costs 21
    want = [0.0, 102.0, 102.0, 215.0, 336.0, 13.0, 13.0, 34.0]
    assert np.array_equal(d["wait_mean"], want), d["wait_mean"]


def pin_eviction_costs(orc):
    """An evicted slot adds the eviction cost to its own wait and to every later
    wait on the same queue, never to another queue."""
    groups = [(1, 0.0, 0.0, 0, 1e6)] * 8
    pr = problem(groups, [(400.0, 0), (400.0, 0)], evict_cost=2.5)
    pl = plans([[[0, 1, 2, 3, 4], [5, 6, 7]]], 8, evict=[[1, 3, 7]])
    d = orc.plan_detail(pr, pl, 0)
    want = [0.0, 2.5, 2.5, 5.0, 5.0, 0.0, 0.0, 2.5]
    assert np.array_equal(d["wait_mean"], want), d["wait_mean"]


def pin_throughput_per_queue(orc):
    """Each queue divides its own tokens by its own throughput (Eq. base_equation
    with Theta per instance), and variances by Theta^2."""
    groups = [(2, 300.0, 800.0, 0, 1e6)] * 4     # 600 tokens, variance 1600 each
    pr = problem(groups, [(600.0, 0), (150.0, 0)])
    pl = plans([[[0, 1], [2, 3]]], 4)
    d = orc.plan_detail(pr, pl, 0)
    assert np.array_equal(d["wait_mean"], [0.0, 1.0, 0.0, 4.0]), d["wait_mean"]
    assert np.allclose(d["wait_sd"], [0.0, 40.0 / 600.0, 0.0, 40.0 / 150.0], rtol=1e-15)


# ---------------------------------------------------------------------------
# Invariants on random inputs


def _random_case(rng, G=12, I=3, M=3, C=2, P=40, evict=True, model0=True):
    groups = []
    for _ in range(G):
        n = int(rng.integers(1, 20))
        mu = float(np.float32(rng.uniform(50, 500)))
        var = float(np.float32(rng.uniform(0, 4e4)))
        groups.append((n, mu, var, int(rng.integers(0, M)), float(np.float32(rng.uniform(1, 60)))))
    inst = [(float(np.float32(rng.choice([800.0, 1500.0, 3000.0]))), int(rng.integers(0, C)))
            for _ in range(I)]
    S = rng.uniform(0.5, 10.0, (C, M, M)).astype(np.float32)
    m0 = [int(x) for x in rng.integers(-1, M, I)] if model0 else None
    pr = problem(groups, inst, n_models=M, n_classes=C, swap=S, evict_cost=1.5, model0=m0)
    qls, evs = [], []
    for _ in range(P):
        order = rng.permutation(G)
        owner = rng.integers(0, I, G)
        qls.append([[int(i) for i in order if owner[i] == g] for g in range(I)])
        evs.append(list(rng.choice(G, size=2, replace=False)) if evict else [])
    pl = plans(qls, G, evict=evs if evict else None)
    return pr, pl


def pin_invariants(orc):
    rng = np.random.default_rng(1234)
    pr, pl = _random_case(rng)
    for p in range(pl["n_plans"]):
        d = orc.plan_detail(pr, pl, p)
        q = pl["qoff"][:, p]
        for g in range(pr["n_instances"]):
            w = d["wait_mean"][q[g]:q[g + 1]]
            s = d["wait_sd"][q[g]:q[g + 1]]
            assert np.all(np.diff(w) >= 0) and np.all(np.diff(s) >= 0)
            if q[g + 1] > q[g]:
                assert s[0] == 0.0                     # nothing ahead of the head
        assert np.all((d["prob"] >= 0) & (d["prob"] <= 1))
    # P is non-increasing in the SLO, and 1/2 exactly at slo = E[W] (SD > 0)
    d = orc.plan_detail(pr, pl, 0)
    s = int(np.argmax(d["wait_sd"]))
    i = int(pl["perm"][s, 0])
    last = 2.0
    for slo in np.linspace(d["wait_mean"][s] - 4 * d["wait_sd"][s],
                           d["wait_mean"][s] + 4 * d["wait_sd"][s], 17):
        pr2 = dict(pr)
        pr2["grp_slo"] = pr["grp_slo"].copy()
        pr2["grp_slo"][i] = np.float32(slo)
        pv = orc.plan_detail(pr2, pl, 0)["prob"][s]
        assert pv <= last + 1e-300
        last = pv
    # an SLO no wait can reach: nothing is violated
    pr3 = dict(pr)
    pr3["grp_slo"] = np.full(pr["n_groups"], 3.0e38, np.float32)
    sc, _ = orc.score_plans(pr3, pl)
    assert np.all(sc == 0.0)
    # an SLO far below every wait: everything is violated
    pr4 = dict(pr)
    pr4["grp_slo"] = np.full(pr["n_groups"], -3.0e38, np.float32)
    sc4, _ = orc.score_plans(pr4, pl)
    assert np.all(sc4 == float(pr["grp_count"].sum()))


def pin_half_at_mean(orc):
    """P = 1/2 when the SLO equals the mean wait and SD > 0 (Normal symmetry)."""
    pr = problem([(2, 300.0, 500.0, 0, 99.0), (1, 10.0, 10.0, 0, 1.5)], [(400.0, 0)])
    d = orc.plan_detail(pr, plans([[[0, 1]]], 2), 0)
    assert d["wait_mean"][1] == 1.5 and d["prob"][1] == 0.5


def pin_identical_instances_symmetry(orc):
    """Swapping the whole queues of two identical instances leaves every wait,
    probability and the score unchanged (the score is a sum over queues)."""
    rng = np.random.default_rng(7)
    pr, pl = _random_case(rng, I=2, C=1, model0=False, evict=False)
    pr["inst_tput"][:] = np.float32(1500.0)
    for p in range(10):
        q = pl["qoff"][:, p]
        a = [int(x) for x in pl["perm"][q[0]:q[1], p]]
        b = [int(x) for x in pl["perm"][q[1]:q[2], p]]
        pl2 = plans([[a, b], [b, a]], pr["n_groups"])
        s, _ = orc.score_plans(pr, pl2)
        assert abs(s[0] - s[1]) <= 1e-12 * max(1.0, abs(s[0]))


# ---------------------------------------------------------------------------
# Monte Carlo of the stated model


def _simulate(pr, queues, evicted, rng, n_samples):
    """Draw every request's output tokens from N(mu, sigma^2) (the per-request
    model of Sec. 6), serve each queue in order on its own throughput, and add
    swap and eviction seconds as the queue is walked.  Returns W[sample, slot]
    with slots in plan order."""
    G = pr["n_groups"]
    W = np.zeros((n_samples, G))
    s = 0
    S = pr["swap_cost"]
    M = pr["n_models"]
    for g, q in enumerate(queues):
        theta = float(pr["inst_tput"][g])
        c = int(pr["inst_class"][g])
        prev = -1 if pr["inst_model0"] is None else int(pr["inst_model0"][g])
        tokens = np.zeros(n_samples)
        fixed = 0.0
        for i in q:
            m = int(pr["grp_model"][i])
            if prev >= 0 and prev != m:
                fixed += float(S[(c * M + prev) * M + m])
            if s in evicted:
                fixed += pr["evict_cost"]
            W[:, s] = tokens / theta + fixed
            n = int(pr["grp_count"][i])
            draws = rng.normal(float(pr["grp_mu"][i]), np.sqrt(float(pr["grp_var"][i])),
                               (n_samples, n))
            tokens = tokens + draws.sum(axis=1)
            prev = m
            s += 1
    return W


def pin_monte_carlo(orc):
    rng = np.random.default_rng(99)
    groups = [(3, 200.0, 9000.0, 0, 0.0), (5, 120.0, 2500.0, 1, 0.0), (2, 400.0, 20000.0, 1, 0.0),
              (4, 150.0, 4000.0, 0, 0.0), (6, 90.0, 1000.0, 1, 0.0), (3, 250.0, 12000.0, 0, 0.0)]
    S = np.array([[[0, 2.0], [3.0, 0]], [[0, 0.5], [0.75, 0]]], np.float32)
    pr = problem(groups, [(1000.0, 0), (600.0, 1)], n_models=2, n_classes=2, swap=S,
                 evict_cost=0.4, model0=[1, -1])
    queues = [[4, 0, 2], [1, 5, 3]]
    evicted = {1, 4}
    # SLOs at quantiles of an independent draw (so they sit inside each W's spread)
    W0 = _simulate(pr, queues, evicted, rng, 20000)
    levels = [0.15, 0.35, 0.5, 0.65, 0.85, 0.25]
    slo_slot = [np.float32(np.quantile(W0[:, s], levels[s])) for s in range(6)]
    perm = [i for q in queues for i in q]
    for s, i in enumerate(perm):
        pr["grp_slo"][i] = slo_slot[s]
    pl = plans([queues], 6, evict=[sorted(evicted)])
    d = orc.plan_detail(pr, pl, 0)
    N = 400000
    W = _simulate(pr, queues, evicted, rng, N)
    slo = np.array([pr["grp_slo"][i] for i in perm], np.float64)
    hat = (W > slo[None, :]).mean(axis=0)
    se = np.sqrt(np.maximum(d["prob"] * (1 - d["prob"]), 1e-12) / N)
    assert np.all(np.abs(hat - d["prob"]) <= 5 * se), (hat, d["prob"], se)
    mean = W.mean(axis=0)
    sd = W.std(axis=0)
    assert np.allclose(mean, d["wait_mean"], rtol=0, atol=5 * sd.max() / np.sqrt(N) + 1e-9)
    assert np.allclose(sd, d["wait_sd"], rtol=0.01, atol=1e-9), (sd, d["wait_sd"])
    n = np.array([pr["grp_count"][i] for i in perm], np.float64)
    score_hat = ((W > slo[None, :]) * n[None, :]).sum(axis=1)
    assert abs(score_hat.mean() - d["score"]) <= 5 * score_hat.std() / np.sqrt(N)


# ---------------------------------------------------------------------------
# Brute force over orderings


def pin_edf_special_case(orc):
    """Sec. 2 Insight #3: with negligible swap cost EDF is the order to use.
    With deterministic, equal-size groups the waiting time is the start time, and
    Jackson's rule says EDF order minimises the maximum lateness max_j(W_j - slo_j);
    so EDF also meets every SLO whenever any order does (score 0)."""
    rng = np.random.default_rng(3)
    for trial in range(6):
        G = 6
        slo = np.sort(rng.uniform(0.0, 6.0, G)).astype(np.float32)
        rng.shuffle(slo)
        groups = [(2, 200.0, 0.0, 0, float(slo[k])) for k in range(G)]   # 1 s each
        pr = problem(groups, [(400.0, 0)])
        pl = plans(all_orders(G), G)
        score, _ = orc.score_plans(pr, pl)
        lateness = []
        for p in range(pl["n_plans"]):
            d = orc.plan_detail(pr, pl, p)
            sl = pr["grp_slo"][pl["perm"][:, p]].astype(np.float64)
            lateness.append(np.max(d["wait_mean"] - sl))
        edf = [[int(i) for i in np.argsort(slo, kind="stable")]]
        ed = orc.plan_detail(pr, plans([edf], G), 0)
        sl = pr["grp_slo"][edf[0]].astype(np.float64)
        assert abs(np.max(ed["wait_mean"] - sl) - min(lateness)) < 1e-12
        if score.min() == 0.0:
            assert ed["score"] == 0.0
        # brute-force argmin agrees with the oracle's argmin (first minimum)
        best, bs = orc.argmin(score)
        assert bs == score.min() and best == int(np.flatnonzero(score == score.min())[0])


def pin_grouping_special_case(orc):
    """Sec. 2 Insight #3: grouping same-model requests minimises the queue drain
    time.  With no tokens, the last group's wait is the total swap time, which is
    least (models - 1 swaps) exactly for the orders that keep each model together."""
    models = [0, 0, 1, 1, 2, 2]
    groups = [(1, 0.0, 0.0, m, 1e6) for m in models]
    pr = problem(groups, [(400.0, 0)], n_models=3, swap=7.0)
    pl = plans(all_orders(6), 6)
    last = []
    contiguous = []
    for p in range(pl["n_plans"]):
        d = orc.plan_detail(pr, pl, p)
        last.append(d["wait_mean"][-1])
        ms = [models[i] for i in pl["perm"][:, p]]
        runs = 1 + sum(1 for k in range(1, 6) if ms[k] != ms[k - 1])
        contiguous.append(runs == 3)
    last = np.array(last)
    assert last.min() == 14.0
    assert np.array_equal(last == 14.0, np.array(contiguous))
    assert int(np.sum(contiguous)) == 48          # 3! model orders x 2!^3 within


def pin_argmin_ties(orc):
    """Equal scores (duplicate plans) go to the lowest plan index."""
    pr = problem([(3, 100.0, 500.0, 0, 0.2), (2, 50.0, 300.0, 0, 0.3), (4, 80.0, 100.0, 0, 0.5)],
                 [(400.0, 0)])
    orders = [[[2, 1, 0]], [[1, 0, 2]], [[0, 1, 2]], [[1, 0, 2]], [[0, 2, 1]], [[1, 0, 2]]]
    pl = plans(orders, 3)
    score, _ = orc.score_plans(pr, pl)
    assert score[1] == score[3] == score[5]
    best, bs = orc.argmin(score)
    assert bs == score.min()
    assert best == int(np.flatnonzero(score == bs)[0])
    # put the best order first, then later duplicates of it: index 0 must win
    b = orders[best]
    pl2 = plans([b, orders[0], b, b], 3)
    s2, _ = orc.score_plans(pr, pl2)
    assert orc.argmin(s2)[0] == (0 if s2[0] <= s2[1] else 1)


# ---------------------------------------------------------------------------
# Plan search (local search with reorder, reassign and evict moves)
#
# The first slot of a non-empty queue holds its running group, which no move
# takes and only a relocation passes.  SWAP(s, d), k = s*W + d - 1: the groups
# at slots s and s+d trade places when both are in one queue.  MOVE(s, h),
# k = G*W + s*I + h: the group at slot s leaves its queue for queue h != g,
# placed before the first group after h's head with a strictly later SLO
# (else at the end; the head of an empty h).  RELOCATE(s, h),
# k = G*W + G*I + s*I + h: the group at slot s becomes the head of the
# non-empty queue h with its eviction flag set.  Other flags go with their
# group.


def _queues_of(perm, qoff):
    return [list(perm[qoff[g]:qoff[g + 1]]) for g in range(len(qoff) - 1)]


def _n_moves(G, I, W):
    return G * W + 2 * G * I


def _edf_index(q, slo, item_slo):
    """Where a group goes in the list q (its head excluded from the search):
    before the first later SLO after the head, else the end."""
    later = [j for j in range(1, len(q)) if slo[q[j][0]] > item_slo]
    return later[0] if later else len(q)


def _apply_move_py(pr, perm, qoff, flag, W, k):
    """The moves restated on Python lists (independent of the oracle's code):
    returns (perm, qoff, flag) or None."""
    G, I = int(pr["n_groups"]), int(pr["n_instances"])
    slo = pr["grp_slo"]
    owner = {}
    for g in range(I):
        for s in range(qoff[g], qoff[g + 1]):
            owner[s] = g
    heads = {int(qoff[g]) for g in range(I) if qoff[g] < qoff[g + 1]}
    # carry (group, flag) pairs per queue
    qs = [[(int(perm[s]), int(flag[s])) for s in range(qoff[g], qoff[g + 1])] for g in range(I)]
    if k < G * W:
        s, d = divmod(k, W)
        t = s + d + 1
        if t >= G or owner[s] != owner[t] or s in heads:
            return None
        g = owner[s]
        a, b = s - qoff[g], t - qoff[g]
        qs[g][a], qs[g][b] = qs[g][b], qs[g][a]
    elif k < G * W + G * I:
        s, h = divmod(k - G * W, I)
        g = owner[s]
        if h == g or s in heads:
            return None
        item = qs[g].pop(s - qoff[g])
        qs[h].insert(_edf_index(qs[h], slo, slo[item[0]]), item)
    else:
        s, h = divmod(k - G * W - G * I, I)
        g = owner[s]
        if s in heads or not qs[h]:
            return None
        item = qs[g].pop(s - qoff[g])
        qs[h].insert(0, (item[0], 1))
    flat = [x for q in qs for x in q]
    lens = [len(q) for q in qs]
    return (np.array([x[0] for x in flat], np.int32),
            np.concatenate([[0], np.cumsum(lens)]).astype(np.int32),
            np.array([x[1] for x in flat], np.uint8))


def _flags_of(pl, p, G):
    if pl.get("evict_bits") is None:
        return np.zeros(G, np.uint8)
    w = pl["evict_bits"][:, p]
    return np.array([(int(w[s // 32]) >> (s % 32)) & 1 for s in range(G)], np.uint8)


def _one_plan(perm, qoff, flag, with_flags):
    G = len(perm)
    ev = None
    if with_flags:
        ev = np.zeros(((G + 31) // 32, 1), np.uint32)
        for s in range(G):
            if flag[s]:
                ev[s // 32, 0] |= np.uint32(1) << np.uint32(s % 32)
    return {"n_plans": 1, "perm": np.asarray(perm, np.int32).reshape(G, 1),
            "qoff": np.asarray(qoff, np.int32).reshape(-1, 1), "evict_bits": ev}


def pin_moves_by_hand(orc):
    """Moves worked by hand on one plan: queues [[0, 1, 2], [3], [4, 5, 6]] with
    SLOs 0:5 1:1 2:9 3:3 4:5 5:1 6:9, group 2 flagged (slot 2), W = 2.  Slots
    0, 3 and 4 hold the running groups."""
    slo = [5, 1, 9, 3, 5, 1, 9]
    pr = problem([(1, 10.0, 0.0, 0, float(x)) for x in slo], [(100.0, 0)] * 3)
    perm = np.array([0, 1, 2, 3, 4, 5, 6], np.int32)
    qoff = np.array([0, 3, 4, 7], np.int32)
    flag = np.array([0, 0, 1, 0, 0, 0, 0], np.uint8)
    G, I, W = 7, 3, 2
    MV, RL = G * W, G * W + G * I

    def mv(k):
        return orc.move_apply(pr, perm, qoff, flag, W, k)

    def check(k, p, q, f):
        r = mv(k)
        assert r is not None, k
        assert list(r[0]) == p and list(r[1]) == q and list(r[2]) == f, (k, r)
    # SWAP(1, 1) = k 2: groups 1 and 2 trade places, and the flag goes with group 2
    check(1 * W + 0, [0, 2, 1, 3, 4, 5, 6], [0, 3, 4, 7], [0, 1, 0, 0, 0, 0, 0])
    check(5 * W + 0, [0, 1, 2, 3, 4, 6, 5], [0, 3, 4, 7], [0, 0, 1, 0, 0, 0, 0])
    # SWAP(0, 1), SWAP(0, 2), SWAP(4, 1): a running group; SWAP(2, 1): slot 3 is
    # in the next queue; SWAP(6, 1): beyond G
    for k in (0, 1, 4 * W, 2 * W, 6 * W):
        assert mv(k) is None, k
    # MOVE(slot 1 = group 1, SLO 1, to queue 2 = [4(5), 5(1), 6(9)]): the head 4
    # stays first; 5's SLO 1 is not later; before 6 (9)
    check(MV + 1 * I + 2, [0, 2, 3, 4, 5, 1, 6], [0, 2, 3, 7], [0, 1, 0, 0, 0, 0, 0])
    # MOVE(slot 5 = group 5, SLO 1, to queue 0 = [0(5), 1(1), 2(9)]): behind the
    # running group 0 although its SLO is later; before 2 (9)
    check(MV + 5 * I + 0, [0, 1, 5, 2, 3, 4, 6], [0, 4, 5, 7], [0, 0, 0, 1, 0, 0, 0])
    # MOVE(slot 2 = flagged group 2, SLO 9, to queue 1 = [3(3)]): at the end, flag kept
    check(MV + 2 * I + 1, [0, 1, 3, 2, 4, 5, 6], [0, 2, 4, 7], [0, 0, 0, 1, 0, 0, 0])
    # MOVE of a running group (slots 0, 3, 4), MOVE to the group's own queue: no move
    for k in (MV + 0 * I + 1, MV + 3 * I + 2, MV + 4 * I + 0, MV + 5 * I + 2):
        assert mv(k) is None, k
    # RELOCATE(slot 2 = group 2, its own queue 0): ahead of the running group 0,
    # flagged (it already was)
    check(RL + 2 * I + 0, [2, 0, 1, 3, 4, 5, 6], [0, 3, 4, 7], [1, 0, 0, 0, 0, 0, 0])
    # RELOCATE(slot 5 = group 5, queue 1 = [3]): [5*, 3]; the flag is set
    check(RL + 5 * I + 1, [0, 1, 2, 5, 3, 4, 6], [0, 3, 5, 7], [0, 0, 1, 1, 0, 0, 0])
    # RELOCATE(slot 1 = group 1, queue 2): [1*, 4, 5, 6]; group 2 keeps its flag
    check(RL + 1 * I + 2, [0, 2, 3, 1, 4, 5, 6], [0, 2, 3, 7], [0, 1, 0, 1, 0, 0, 0])
    # RELOCATE(slot 6 = group 6, its own queue 2): [6*, 4, 5]
    check(RL + 6 * I + 2, [0, 1, 2, 3, 6, 4, 5], [0, 3, 4, 7], [0, 0, 1, 0, 1, 0, 0])
    # RELOCATE of a running group: no move
    for k in (RL + 0 * I + 0, RL + 3 * I + 0, RL + 4 * I + 1):
        assert mv(k) is None, k
    assert orc.n_moves(G, I, W) == G * W + 2 * G * I
    # an empty queue: MOVE makes the group its head, RELOCATE names no move
    pr2 = problem([(1, 10.0, 0.0, 0, 1.0), (1, 10.0, 0.0, 0, 2.0)], [(100.0, 0)] * 2)
    p0, q0, f0 = np.array([0, 1], np.int32), np.array([0, 2, 2], np.int32), np.zeros(2, np.uint8)
    r = orc.move_apply(pr2, p0, q0, f0, 1, 2 * 1 + 1 * 2 + 1)
    assert list(r[0]) == [0, 1] and list(r[1]) == [0, 1, 2] and list(r[2]) == [0, 0]
    assert orc.move_apply(pr2, p0, q0, f0, 1, 2 + 4 + 1 * 2 + 1) is None
    r = orc.move_apply(pr2, p0, q0, f0, 1, 2 + 4 + 1 * 2 + 0)
    assert list(r[0]) == [1, 0] and list(r[1]) == [0, 2, 2] and list(r[2]) == [1, 0]


def _search_case(rng, G, I, M=2, C=2, evict=True):
    pr, pl = _random_case(rng, G=G, I=I, M=M, C=C, P=3, evict=evict)
    return pr, pl


def pin_moves_independent(orc):
    """Every move of random tiny plans, against the moves restated in Python,
    and every move's score against the plan score of the moved plan."""
    rng = np.random.default_rng(77)
    for G, I, W, evict in [(7, 3, 3, True), (9, 2, 9, False), (5, 4, 1, True)]:
        pr, pl = _search_case(rng, G, I, evict=evict)
        nm = _n_moves(G, I, W)
        for p in range(pl["n_plans"]):
            perm = pl["perm"][:, p].copy()
            qoff = pl["qoff"][:, p].copy()
            flag = _flags_of(pl, p, G)
            sc = orc.move_scores(pr, pl, p, W)
            assert sc.size == nm
            for k in range(nm):
                a = orc.move_apply(pr, perm, qoff, flag, W, k)
                b = _apply_move_py(pr, perm, qoff, flag, W, k)
                if b is None:
                    assert a is None and sc[k] == np.inf, (G, I, W, p, k)
                    continue
                assert a is not None, (G, I, W, p, k)
                for x, y in zip(a, b):
                    assert np.array_equal(x, y), (G, I, W, p, k, a, b)
                ref = orc.plan_detail(pr, _one_plan(*b, True), 0)["score"]
                assert sc[k] == ref, (k, sc[k], ref)
            # a sample of moves by number gives the same scores
            ks = np.array([0, G * W + 1, G * W + G * I - 1, nm - 1, G * W + G * I + 2, 2],
                          np.int64)
            assert np.array_equal(orc.move_scores(pr, pl, p, W, ks=ks), sc[ks])


def pin_search_by_hand(orc):
    """Two identical instances (400 tok/s); queue 0 holds group 0 (2 x 200
    tokens, 1 s; running) then group 1 (3 x 100 tokens), both with a 0.5 s SLO;
    queue 1 is empty.  Group 1 waits 1 s and misses: score 3.  With G = 2,
    W = 1, I = 2 (MOVEs from k = 2, RELOCATEs from k = 6): k0 SWAP(0, 1), k2,
    k3, k6, k7: the running group; k1: beyond G; k4 MOVE(1, 0): own queue;
    k9 RELOCATE(1, 1): queue 1 is empty; k5 MOVE(1, 1): alone in queue 1,
    nobody waits, score 0; k8 RELOCATE(1, 0): group 1 first (waits E = 0),
    group 0 waits 0.75 s and misses, score 2.  The search takes k5, after which
    nothing improves on 0."""
    pr = problem([(2, 200.0, 0.0, 0, 0.5), (3, 100.0, 0.0, 0, 0.5)], [(400.0, 0), (400.0, 0)])
    pl = plans([[[0, 1], []]], 2)
    sc = orc.move_scores(pr, pl, 0, 1)
    inf = np.inf
    assert list(sc) == [inf, inf, inf, inf, inf, 0.0, inf, inf, 2.0, inf], sc
    r = orc.local_search(pr, pl, 0, 1, 4)
    assert r["steps"] == 1 and list(r["trace"]) == [5, -1, -1, -1]
    assert list(r["perm"]) == [0, 1] and list(r["qoff"]) == [0, 1, 2] and r["score"] == 0.0
    # a plan that meets every SLO does not move
    r = orc.local_search(pr, plans([[[0], [1]]], 2), 0, 1, 4)
    assert r["steps"] == 0 and list(r["perm"]) == [0, 1] and r["score"] == 0.0
    # one instance: only RELOCATE(1, 0) = k 3 is a move.  With E = 0.25 s group 1
    # waits 0.25 s (met) and group 0 1 s (misses): 2 < 3, taken.  With E = 0.6 s
    # both miss: 5, not taken.
    for E, steps, score in ((0.25, 1, 2.0), (0.6, 0, 3.0)):
        pr1 = problem([(2, 200.0, 0.0, 0, 0.5), (3, 100.0, 0.0, 0, 0.5)], [(400.0, 0)],
                      evict_cost=E)
        assert list(orc.move_scores(pr1, plans([[[0, 1]]], 2), 0, 0)) == [inf, inf, inf,
                                                                          5.0 - 3.0 * (E < 0.5)]
        r = orc.local_search(pr1, plans([[[0, 1]]], 2), 0, 0, 3)
        assert r["steps"] == steps and r["score"] == score, (E, r)
        if steps:
            assert list(r["trace"]) == [3, -1, -1] and list(r["perm"]) == [1, 0]
            assert list(_flags_of({"evict_bits": r["evict_bits"].reshape(-1, 1)}, 0, 2)) == [1, 0]
        else:
            assert list(r["trace"]) == [-1, -1, -1] and list(r["perm"]) == [0, 1]


def pin_relocate_by_hand(orc):
    """Head-of-line blocking (Sec. 5, request eviction): one 100 tok/s instance
    runs a batch group (1 request of 1000 tokens, 10 s, SLO 60 s); behind it an
    interactive group (2 requests of 10 tokens, SLO 1 s) waits 10 s and both
    its requests miss: score 2.  Relocating it to the head with E = 0.5 s: it
    waits 0.5 s, the batch group 0.5 + 0.2 s, every SLO met: score 0.  With
    E = 2 s the interactive group still misses (2 s > 1 s) and the batch group
    meets its SLO: score 2, not below 2, so the plan stays.  With E = 1 s the
    wait equals the SLO, which is met (a strict miss): score 0."""
    for E, score, moved in ((0.5, 0.0, True), (2.0, 2.0, False), (1.0, 0.0, True)):
        pr = problem([(1, 1000.0, 0.0, 0, 60.0), (2, 10.0, 0.0, 0, 1.0)], [(100.0, 0)],
                     evict_cost=E)
        pl = plans([[[0, 1]]], 2)
        sc = orc.move_scores(pr, pl, 0, 1)
        # k0 SWAP(0, 1): running; k1 beyond G; k2, k3 MOVE: running / own queue;
        # k4 RELOCATE(0, 0): running; k5 RELOCATE(1, 0)
        assert list(sc) == [np.inf] * 5 + [0.0 if moved else 2.0], (E, sc)
        d = orc.plan_detail(pr, _one_plan([1, 0], [0, 2], [1, 0], True), 0)
        assert d["wait_mean"][0] == E and d["wait_mean"][1] == E + 0.2, d["wait_mean"]
        r = orc.local_search(pr, pl, 0, 1, 2)
        assert r["score"] == score and r["steps"] == (1 if moved else 0), (E, r)
        if moved:
            assert list(r["perm"]) == [1, 0] and list(r["trace"]) == [5, -1]


def pin_search_steepest(orc):
    """Brute force: at every step of the search on tiny random plans, the move
    taken is the first minimum over every move (each scored by building the
    moved plan in Python and scoring it), it strictly improves, and the search
    stops exactly when no move improves."""
    rng = np.random.default_rng(5)
    for G, I, W, evict in [(7, 3, 2, True), (6, 2, 6, False)]:
        pr, pl = _search_case(rng, G, I, evict=evict)
        for p in range(pl["n_plans"]):
            r = orc.local_search(pr, pl, p, W, 12)
            perm = pl["perm"][:, p].copy()
            qoff = pl["qoff"][:, p].copy()
            flag = _flags_of(pl, p, G)
            cur = orc.plan_detail(pr, _one_plan(perm, qoff, flag, True), 0)["score"]
            for t in range(13):
                best, bs = -1, np.inf
                for k in range(_n_moves(G, I, W)):
                    b = _apply_move_py(pr, perm, qoff, flag, W, k)
                    if b is None:
                        continue
                    v = orc.plan_detail(pr, _one_plan(*b, True), 0)["score"]
                    if v < bs:
                        best, bs = k, v
                if t == 12 or not bs < cur:
                    break
                assert r["trace"][t] == best, (p, t, r["trace"], best)
                perm, qoff, flag = _apply_move_py(pr, perm, qoff, flag, W, best)
                cur = bs
            assert r["steps"] == t, (r["steps"], t)
            assert np.array_equal(r["perm"], perm) and np.array_equal(r["qoff"], qoff)
            assert r["score"] == cur
            assert np.array_equal(_flags_of({"evict_bits": r["evict_bits"].reshape(-1, 1)}, 0, G),
                                  flag)


# ---------------------------------------------------------------------------
# Seed plans (EDF order / same-model grouping, each group at the end of the
# queue with the smallest drain time after taking it, the lowest queue on ties)


def _seed_py(pr, policy):
    """The seed construction restated in Python (float64, same operations)."""
    G, I, M = int(pr["n_groups"]), int(pr["n_instances"]), int(pr["n_models"])
    slo = pr["grp_slo"]
    model = pr["grp_model"]
    ids = list(range(G))
    if policy == 0:
        ids.sort(key=lambda i: (float(slo[i]), i))
    else:
        ids.sort(key=lambda i: (int(model[i]), float(slo[i]), i))
    m0 = pr.get("inst_model0")
    last = [int(m0[q]) if m0 is not None else -1 for q in range(I)]
    A = [0.0] * I
    K = [0.0] * I
    queues = [[] for _ in range(I)]
    S = pr.get("swap_cost")
    for i in ids:
        m = int(model[i])
        a = float(pr["grp_count"][i]) * float(pr["grp_mu"][i])
        best, bd = -1, np.inf
        for q in range(I):
            sw = 0.0
            if last[q] >= 0 and last[q] != m and S is not None:
                sw = float(S[(int(pr["inst_class"][q]) * M + last[q]) * M + m])
            d = (A[q] + a) / float(pr["inst_tput"][q]) + (K[q] + sw)
            if d < bd:
                best, bd = q, d
        sw = 0.0
        if last[best] >= 0 and last[best] != m and S is not None:
            sw = float(S[(int(pr["inst_class"][best]) * M + last[best]) * M + m])
        A[best] += a
        K[best] += sw
        last[best] = m
        queues[best].append(i)
    perm = np.array([i for q in queues for i in q], np.int32)
    qoff = np.concatenate([[0], np.cumsum([len(q) for q in queues])]).astype(np.int32)
    return perm, qoff


def pin_seed_by_hand(orc):
    """Four 1-s groups on two 100 tok/s instances, 10 s per model change.
    EDF order 1 (m1), 3 (m1), 2 (m0), 0 (m0): 1 -> q0 (tie, 1 s each); 3 -> q1
    (2 s on q0, 1 s on q1); 2 -> q0 (2 + 10 = 12 s either way, tie); 0 -> q1
    (13 s on q0, 12 s on q1).  Grouped order 2, 0 (m0), 1, 3 (m1): 2 -> q0,
    0 -> q1, 1 -> q0 (12 s both), 3 -> q1 (13 s against 12 s)."""
    pr = problem([(1, 100.0, 0.0, 0, 5.0), (1, 100.0, 0.0, 1, 1.0), (1, 100.0, 0.0, 0, 3.0),
                  (1, 100.0, 0.0, 1, 2.0)], [(100.0, 0), (100.0, 0)], n_models=2, swap=10.0)
    p, q = orc.seed_plan(pr, 0)
    assert list(p) == [1, 2, 3, 0] and list(q) == [0, 2, 4], (p, q)
    p, q = orc.seed_plan(pr, 1)
    assert list(p) == [2, 1, 0, 3] and list(q) == [0, 2, 4], (p, q)


def pin_seed_special_cases(orc):
    """One queue: the EDF seed is the SLO order (ties by id), the grouped seed
    the (model, SLO) order.  Equal groups on identical instances go round-robin.
    On instances of 100 and 300 tok/s, equal 1-s groups split 1 : 3 (the faster
    instance drains three groups in the time of one)."""
    rng = np.random.default_rng(8)
    G = 9
    slo = np.float32(rng.choice([3.0, 1.0, 7.0], G))
    model = rng.integers(0, 3, G)
    pr = problem([(2, 50.0, 10.0, int(model[k]), float(slo[k])) for k in range(G)], [(400.0, 0)],
                 n_models=3, swap=5.0)
    p, q = orc.seed_plan(pr, 0)
    assert list(p) == list(np.lexsort((np.arange(G), slo))) and list(q) == [0, G]
    p, q = orc.seed_plan(pr, 1)
    assert list(p) == list(np.lexsort((np.arange(G), slo, model)))
    # SLOs falling as the ids rise: EDF reverses the ids
    pr = problem([(1, 10.0, 1.0, 0, float(20 - k)) for k in range(12)], [(400.0, 0)])
    p, q = orc.seed_plan(pr, 0)
    assert list(p) == list(range(11, -1, -1)), p
    pr = problem([(1, 100.0, 0.0, 0, float(k)) for k in range(8)], [(100.0, 0)] * 3)
    p, q = orc.seed_plan(pr, 0)
    assert list(p) == [0, 3, 6, 1, 4, 7, 2, 5] and list(q) == [0, 3, 6, 8], (p, q)
    pr = problem([(1, 100.0, 0.0, 0, float(k)) for k in range(8)], [(100.0, 0), (300.0, 0)])
    p, q = orc.seed_plan(pr, 0)
    assert list(q) == [0, 2, 8] and list(p) == [2, 6, 0, 1, 3, 4, 5, 7], (p, q)


def pin_seed_restated(orc):
    """Random problems (heterogeneous instances, swap costs, loaded models):
    both seeds equal the construction restated in Python, and are plans."""
    rng = np.random.default_rng(21)
    for G, I in [(12, 3), (30, 5), (7, 7), (20, 1)]:
        pr, _ = _random_case(rng, G=G, I=I, M=3, C=2, P=1)
        for policy in (0, 1):
            p, q = orc.seed_plan(pr, policy)
            rp, rq = _seed_py(pr, policy)
            assert np.array_equal(p, rp) and np.array_equal(q, rq), (G, I, policy)
            assert sorted(p) == list(range(G)) and q[0] == 0 and q[-1] == G
            assert np.all(np.diff(q) >= 0)


# ---------------------------------------------------------------------------
# Placement of one group (arrival / violation trigger)


def _place_py(pr, perm, qoff, flag, s, c):
    """Group at slot s out of its queue, into place c (restated on Python
    lists): c < I the EDF position of queue c after its head (as it stands
    after the removal), c >= I the head of queue c - I, flagged.  None when
    that queue is empty (nothing to evict)."""
    I = int(pr["n_instances"])
    slo = pr["grp_slo"]
    qs = [[(int(perm[u]), int(flag[u])) for u in range(qoff[g], qoff[g + 1])] for g in range(I)]
    g = next(q for q in range(I) if qoff[q] <= s < qoff[q + 1])
    item = qs[g].pop(s - qoff[g])
    if c < I:
        qs[c].insert(_edf_index(qs[c], slo, slo[item[0]]), item)
    else:
        if not qs[c - I]:
            return None
        qs[c - I].insert(0, (item[0], 1))
    flat = [x for q in qs for x in q]
    return (np.array([x[0] for x in flat], np.int32),
            np.concatenate([[0], np.cumsum([len(q) for q in qs])]).astype(np.int32),
            np.array([x[1] for x in flat], np.uint8))


def pin_place_by_hand(orc):
    """Queue 0 holds groups 0, 1, 2 (1.33, 1 and 1.33 s; SLOs 0.5, 0.6, 0.7 s),
    queue 1 is empty: groups 1 and 2 miss (score 7).  Placing group 2: back at
    the end of queue 0 (no later SLO; 7), alone in queue 1 (3), or at the head
    of queue 0 (groups 0 and 1 miss: 5): queue 1.  With one instance, a group
    with a 0.5 s SLO behind two 1 s groups with 10 s SLOs goes behind the
    running group (it misses: 5) or, evicting it, ahead (everything met when
    E = 0: c = I + 0 = 1; with E = 0.6 s it misses there too, a tie at 5 that
    the lower c wins)."""
    pr = problem([(2, 200.0, 0.0, 0, 0.5), (3, 100.0, 0.0, 0, 0.6), (4, 100.0, 0.0, 0, 0.7)],
                 [(300.0, 0), (300.0, 0)])
    pl = plans([[[0, 1, 2], []]], 3)
    r = orc.place_group(pr, pl, 0, 2)
    assert r["queue"] == 1 and list(r["perm"]) == [0, 1, 2] and list(r["qoff"]) == [0, 2, 3]
    assert r["score"] == 3.0, r["score"]
    for E, c, perm, flags, score in ((0.0, 1, [2, 0, 1], [1, 0, 0], 0.0),
                                     (0.6, 0, [0, 2, 1], [0, 0, 0], 5.0)):
        pr = problem([(1, 100.0, 0.0, 0, 10.0), (1, 100.0, 0.0, 0, 10.0), (5, 20.0, 0.0, 0, 0.5)],
                     [(100.0, 0)], evict_cost=E)
        r = orc.place_group(pr, plans([[[0, 1, 2]]], 3), 0, 2)
        assert r["queue"] == c and list(r["perm"]) == perm and r["score"] == score, (E, r)
        assert list(_flags_of({"evict_bits": r["evict_bits"].reshape(-1, 1)}, 0, 3)) == flags
    # equal SLOs are not later: group 0 goes behind the groups that share its
    # SLO (waits 0, 1, 2 s against 1 s: one miss either way, so c = 0 wins
    # the tie with the head place)
    pr = problem([(1, 100.0, 0.0, 0, 1.0)] * 3, [(100.0, 0)])
    r = orc.place_group(pr, plans([[[2, 0, 1]]], 3), 0, 0)
    assert list(r["perm"]) == [2, 1, 0] and r["queue"] == 0 and r["score"] == 1.0, r
    # the running group stays where it is
    r = orc.place_group(pr, plans([[[2, 0, 1]]], 3), 0, 2)
    assert list(r["perm"]) == [2, 0, 1] and r["queue"] == 0 and r["score"] == 1.0, r


def pin_place_restated(orc):
    """Random plans: the placed plan is the first minimum over every place of
    the placement restated in Python and scored as a plan; the places in other
    queues are the moves MOVE(s, h), the head places RELOCATE(s, h); a running
    group stays."""
    rng = np.random.default_rng(31)
    for G, I, evict in [(9, 3, True), (12, 4, False), (6, 1, True)]:
        pr, pl = _random_case(rng, G=G, I=I, M=2, C=2, P=3, evict=evict)
        for p in range(pl["n_plans"]):
            perm = pl["perm"][:, p].copy()
            qoff = pl["qoff"][:, p].copy()
            flag = _flags_of(pl, p, G)
            ms = orc.move_scores(pr, pl, p, 0)
            assert ms.size == _n_moves(G, I, 0)
            for group in range(G):
                s = int(np.flatnonzero(perm == group)[0])
                g = next(q for q in range(I) if qoff[q] <= s < qoff[q + 1])
                r = orc.place_group(pr, pl, p, group)
                got = _flags_of({"evict_bits": r["evict_bits"].reshape(-1, 1)}, 0, G)
                if s == qoff[g]:
                    assert r["queue"] == g and np.array_equal(r["perm"], perm)
                    assert np.array_equal(r["qoff"], qoff) and np.array_equal(got, flag)
                    continue
                best, bs, bplan = -1, np.inf, None
                for c in range(2 * I):
                    cand = _place_py(pr, perm, qoff, flag, s, c)
                    if cand is None:
                        continue
                    v = orc.plan_detail(pr, _one_plan(*cand, True), 0)["score"]
                    if c < I and c != g:
                        assert v == ms[s * I + c], (c, v, ms[s * I + c])
                    if c >= I:
                        assert v == ms[G * I + s * I + c - I], (c, v)
                    if v < bs:
                        best, bs, bplan = c, v, cand
                assert r["queue"] == best and r["score"] == bs, (r["queue"], best, r["score"], bs)
                assert np.array_equal(r["perm"], bplan[0]) and np.array_equal(r["qoff"], bplan[1])
                assert np.array_equal(got, bplan[2])


# ---------------------------------------------------------------------------
# Per-request variant: first come, first served inside each group


def _req_first(pr):
    return np.concatenate([[0], np.cumsum(np.asarray(pr["grp_count"], np.int64))])


def pin_fcfs_by_hand(orc):
    """One queue at Theta = 100 tok/s.  Group 0 holds 3 requests of 100 tokens
    (1 s each), group 1 two of 50 (0.5 s each).  Deterministic (sigma = 0):
    request r of group 0 waits r s; group 1 starts after the 300 tokens of
    group 0, so its requests wait 3 and 3.5 s.  With SD = 0 a request misses
    its SLO when its wait is strictly later."""
    pr = problem([(3, 100.0, 0.0, 0, 9.0), (2, 50.0, 0.0, 0, 9.0)], [(100.0, 0)])
    pl = plans([[[0, 1]]], 2)
    req = np.array([0.5, 0.5, 2.5, 3.0, 3.4], np.float32)
    d = orc.plan_fcfs(pr, pl, req, 0)
    assert np.array_equal(d["prob"], [0.0, 1.0, 0.0, 0.0, 1.0]), d["prob"]
    assert d["score"] == 2.0
    # the other order: group 1 first (waits 0, 0.5 s), then group 0 (1, 2, 3 s)
    d2 = orc.plan_fcfs(pr, plans([[[1, 0]]], 2), req, 0)
    assert np.array_equal(d2["prob"], [1.0, 1.0, 1.0, 0.0, 0.0]), d2["prob"]
    # sigma = 100 tokens = 1 s per request: request r of group 0 has SD sqrt(r) s;
    # SLOs at z = 2 for r = 1 (1 + 2) and z = 1 for r = 2 (2 + sqrt 2); r = 0 has
    # SD 0 and a wait of 0 > -1
    table = dict(normal_table())
    pr3 = problem([(3, 100.0, 10000.0, 0, 9.0)], [(100.0, 0)])
    req3 = np.array([-1.0, 3.0, 2.0 + np.sqrt(2.0)], np.float32)
    d3 = orc.plan_fcfs(pr3, plans([[[0]]], 1), req3, 0)
    z2 = (float(req3[2]) - 2.0) / np.sqrt(2.0)      # 1 up to the float rounding of the SLO
    want = [1.0, table[2.0], table[1.0] - (z2 - 1.0) * np.exp(-0.5) / np.sqrt(2 * np.pi)]
    assert np.allclose(d3["prob"], want, rtol=0, atol=1e-8), (d3["prob"], want)


def _explode(pr, queues, req, evicted):
    """Every request as a group of its own (n = 1, its own SLO), in arrival order
    at its group's place; a group's eviction goes to its first request."""
    first = _req_first(pr)
    groups, qs, ev, slot = [], [], [], 0
    for q in queues:
        out = []
        for i in q:
            s_here = slot
            slot += 1
            for r in range(int(pr["grp_count"][i])):
                if r == 0 and s_here in evicted:
                    ev.append(len(groups))
                out.append(len(groups))
                groups.append((1, float(pr["grp_mu"][i]), float(pr["grp_var"][i]),
                               int(pr["grp_model"][i]), float(req[first[i] + r])))
        qs.append(out)
    G = len(groups)
    # group ids = exploded positions, so the plan's slot s holds exploded group s
    pe = problem(groups, np.stack([pr["inst_tput"], pr["inst_class"]], 1).tolist(),
                 n_models=pr["n_models"], n_classes=pr["n_classes"],
                 swap=None if pr["swap_cost"] is None else
                 pr["swap_cost"].reshape(pr["n_classes"], pr["n_models"], pr["n_models"]),
                 evict_cost=pr["evict_cost"], model0=pr["inst_model0"])
    return pe, plans([qs], G, evict=[ev])


def pin_fcfs_exploded(orc):
    """Request r of a group has ahead of it the groups before the group and the
    group's r earlier requests (Eq. output_token_dist counts every request
    ahead): the per-request score of a plan equals the group score of the plan
    in which every request is a group of one, with its own SLO, at its place in
    arrival order.  One request per group, with the group's SLO, gives the group
    score itself, exactly."""
    rng = np.random.default_rng(41)
    for trial in range(5):
        G, I, M, C = 7, 3, 3, 2
        groups = [(int(rng.integers(0, 6)), float(rng.uniform(20, 400)),
                   float(rng.uniform(0, 3e4)), int(rng.integers(0, M)), 0.0) for _ in range(G)]
        S = rng.uniform(0.5, 8.0, (C, M, M)).astype(np.float32)
        pr = problem(groups, [(float(rng.choice([300.0, 800.0])), int(rng.integers(0, C)))
                              for _ in range(I)], n_models=M, n_classes=C, swap=S,
                     evict_cost=0.7, model0=[int(x) for x in rng.integers(-1, M, I)])
        order = rng.permutation(G)
        owner = rng.integers(0, I, G)
        queues = [[int(i) for i in order if owner[i] == g] for g in range(I)]
        evicted = set(int(x) for x in rng.choice(G, 2, replace=False))
        pl = plans([queues], G, evict=[sorted(evicted)])
        N = int(sum(g[0] for g in groups))
        # SLOs near each request's wait, so that P spreads over (0, 1)
        waits = rng.uniform(0.0, 60.0, N)
        req = waits.astype(np.float32)
        f = orc.score_plans_fcfs(pr, pl, req)[0]
        pe, ple = _explode(pr, queues, req, evicted)
        g, _ = orc.score_plans(pe, ple)
        assert abs(f - g[0]) <= 1e-12 * max(1.0, abs(g[0])), (trial, f, g[0])
        assert 0.0 < f < N
        # one request per group: the group model, bit for bit
        pr1 = dict(pr)
        pr1["grp_count"] = np.ones(G, np.int32)
        req1 = pr1["grp_slo"] = rng.uniform(0, 30, G).astype(np.float32)
        assert orc.score_plans_fcfs(pr1, pl, req1)[0] == orc.score_plans(pr1, pl)[0][0]


def _simulate_requests(pr, queues, evicted, rng, n_samples):
    """Every request's tokens drawn from N(mu, sigma^2); each queue served in
    order, each group's requests in arrival order.  Returns W[sample, request]
    with requests indexed as the SLO array."""
    first = _req_first(pr)
    W = np.zeros((n_samples, int(first[-1])))
    S, M, s = pr["swap_cost"], pr["n_models"], 0
    for g, q in enumerate(queues):
        theta = float(pr["inst_tput"][g])
        c = int(pr["inst_class"][g])
        prev = -1 if pr["inst_model0"] is None else int(pr["inst_model0"][g])
        tokens = np.zeros(n_samples)
        fixed = 0.0
        for i in q:
            m = int(pr["grp_model"][i])
            if prev >= 0 and prev != m:
                fixed += float(S[(c * M + prev) * M + m])
            if s in evicted:
                fixed += pr["evict_cost"]
            for r in range(int(pr["grp_count"][i])):
                W[:, first[i] + r] = tokens / theta + fixed
                tokens = tokens + rng.normal(float(pr["grp_mu"][i]),
                                             np.sqrt(float(pr["grp_var"][i])), n_samples)
            prev = m
            s += 1
    return W


def pin_fcfs_monte_carlo(orc):
    """Per-request violation probabilities against a simulation of the stated
    model: each request's tokens drawn, requests served one after another."""
    rng = np.random.default_rng(7)
    groups = [(3, 200.0, 9000.0, 0, 0.0), (4, 120.0, 2500.0, 1, 0.0), (2, 400.0, 20000.0, 1, 0.0),
              (3, 150.0, 4000.0, 0, 0.0)]
    S = np.array([[[0, 2.0], [3.0, 0]]], np.float32)
    pr = problem(groups, [(1000.0, 0), (600.0, 0)], n_models=2, n_classes=1, swap=S,
                 evict_cost=0.4, model0=[1, -1])
    queues = [[3, 0], [1, 2]]
    evicted = {2}
    W0 = _simulate_requests(pr, queues, evicted, rng, 20000)
    levels = np.linspace(0.1, 0.9, W0.shape[1])
    req = np.array([np.quantile(W0[:, k], levels[k]) for k in range(W0.shape[1])], np.float32)
    req[0] = -1.0                       # group 0's first request waits behind group 3
    pl = plans([queues], 4, evict=[sorted(evicted)])
    d = orc.plan_fcfs(pr, pl, req, 0)
    N = 200000
    W = _simulate_requests(pr, queues, evicted, rng, N)
    hat = (W > req[None, :].astype(np.float64)).mean(axis=0)
    se = np.sqrt(np.maximum(d["prob"] * (1 - d["prob"]), 1e-12) / N)
    assert np.all(np.abs(hat - d["prob"]) <= 5 * se), (hat, d["prob"], se)
    tot = (W > req[None, :].astype(np.float64)).sum(axis=1)
    assert abs(tot.mean() - d["score"]) <= 5 * tot.std() / np.sqrt(N)


# ---------------------------------------------------------------------------
# Problem tables from a hardware profile


def _profile_by_hand():
    # two classes, two models; decode times and factors chosen so that the
    # derived throughputs and drains are exact in binary
    return {"prefill": [0.25, 0.5],
            "decode_time": [1 / 32, 1 / 64, 1 / 16, 1 / 128],   # [c][m]
            "ineff": [2.0, 1.5, 1.0, 2.0],
            "max_tokens": [512.0, 256.0],
            "kv_tokens": [4096.0, 8192.0, 2048.0, 65536.0],
            "mean_tokens": [512.0, 256.0]}


def pin_profile_by_hand(orc):
    """Sec. 6 (completion = wait + prefill + decode, decode = O eps d, a group
    completes with its last request) and the Appendix (Theta = B / (d eps),
    B = GPU / E[I + O]), worked by hand:
      Theta[0][0] = (4096/512) / (2/32) = 128 tok/s, Theta[1][1] = (65536/256) / (2/128) = 16384;
      drain[0][0] = 0.25 + 512*2/32 = 32.25 s, drain[0][1] = 0.5 + 256*1.5/64 = 6.5 s,
      drain[1][0] = 0.25 + 512/16 = 32.25 s, drain[1][1] = 0.5 + 256*2/128 = 4.5 s;
    the swap table gains the drain of the model left behind; SLOs lose the
    prefill of the group's model."""
    S = np.array([[[99, 10], [20, 99]], [[99, 1], [2, 99]]], np.float32)
    groups = [(1, 128.0, 0.0, 0, 100.0), (2, 64.0, 0.0, 1, 43.5), (1, 128.0, 0.0, 1, 45.0),
              (1, 128.0, 0.0, 0, 50.0)]
    pr = problem(groups, [(999.0, 0), (999.0, 1)], n_models=2, n_classes=2, swap=S)
    out, _ = orc.apply_profile(pr, _profile_by_hand(), inst_model=[0, 1])
    assert list(out["inst_tput"]) == [128.0, 16384.0], out["inst_tput"]
    want = np.array([[[99, 42.25], [26.5, 99]], [[99, 33.25], [6.5, 99]]], np.float32)
    assert np.array_equal(out["swap_cost"], want.reshape(-1)), out["swap_cost"]
    assert list(out["grp_slo"]) == [99.75, 43.0, 44.5, 49.75], out["grp_slo"]
    # queue 0 (Theta 128): groups 0 (model 0, 1 s of tokens), 1 and 2 (model 1,
    # 1 s each): waits 0, 1 + 42.25, 44.25.  Group 1's TTFT (43.25 + 0.5) is
    # past its SLO of 43.5, group 2's (44.25 + 0.5) is not
    d = orc.plan_detail(out, plans([[[0, 1, 2], [3]]], 4), 0)
    assert list(d["wait_mean"]) == [0.0, 43.25, 44.25, 0.0], d["wait_mean"]
    assert list(d["prob"]) == [0.0, 1.0, 0.0, 0.0], d["prob"]
    assert d["score"] == 2.0
    # no profile: the tables as given
    same, _ = orc.apply_profile(pr, {})
    assert np.array_equal(same["swap_cost"], pr["swap_cost"])
    assert np.array_equal(same["grp_slo"], pr["grp_slo"])
    assert np.array_equal(same["inst_tput"], pr["inst_tput"])
    # per-request SLOs lose the prefill of their group's model
    req = np.arange(5, dtype=np.float32) + 10.0
    _, rs = orc.apply_profile(pr, {"prefill": [0.25, 0.5]}, req_slo=req)
    assert list(rs) == [9.75, 10.5, 11.5, 12.5, 13.75], rs


def pin_profile_scaling(orc):
    """Theta grows with the token memory and falls with the decode time, the
    inefficiency and the tokens per request, each in proportion (Appendix):
    random profiles, each factor doubled in turn."""
    rng = np.random.default_rng(17)
    C, M = 2, 3
    pr = problem([(1, 100.0, 10.0, m % M, 50.0) for m in range(4)],
                 [(1000.0, c % C) for c in range(4)], n_models=M, n_classes=C)
    base = {"prefill": rng.uniform(0.05, 0.5, M), "decode_time": rng.uniform(0.01, 0.05, C * M),
            "ineff": rng.uniform(1.0, 1.6, C * M), "max_tokens": rng.uniform(256, 4096, M),
            "kv_tokens": rng.uniform(1e5, 1e6, C * M), "mean_tokens": rng.uniform(200, 900, M)}
    base = {k: np.float32(v) for k, v in base.items()}
    im = [0, 1, 2, 1]
    t0 = orc.apply_profile(pr, base, inst_model=im)[0]["inst_tput"].astype(np.float64)
    for f, power in (("kv_tokens", 1), ("decode_time", -1), ("ineff", -1), ("mean_tokens", -1)):
        p2 = dict(base)
        p2[f] = base[f] * np.float32(2)
        t = orc.apply_profile(pr, p2, inst_model=im)[0]["inst_tput"].astype(np.float64)
        assert np.allclose(t / t0, 2.0 ** power, rtol=2e-7), (f, t / t0)
    # an instance without a model keeps its throughput
    t = orc.apply_profile(pr, base, inst_model=[-1, 1, 2, 1])[0]["inst_tput"]
    assert t[0] == 1000.0


ALL_PINS = [pin_deterministic_queue, pin_variance_queue, pin_normal_table, pin_swap_costs,
            pin_eviction_costs, pin_throughput_per_queue, pin_invariants, pin_half_at_mean,
            pin_identical_instances_symmetry, pin_monte_carlo, pin_edf_special_case,
            pin_grouping_special_case, pin_argmin_ties, pin_moves_by_hand, pin_moves_independent,
            pin_search_by_hand, pin_relocate_by_hand, pin_search_steepest, pin_seed_by_hand, pin_seed_special_cases,
            pin_seed_restated, pin_place_by_hand, pin_place_restated, pin_fcfs_by_hand,
            pin_fcfs_exploded, pin_fcfs_monte_carlo, pin_profile_by_hand, pin_profile_scaling]
