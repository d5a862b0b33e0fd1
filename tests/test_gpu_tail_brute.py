"""Parity at the places where the screened score is most fragile, through the
C interface:

- the normal tail on a dense grid of standardised margins: every cell edge
  of the 1024-cell table over |z| <= 6, points inside the cells, both clamp
  ends and beyond, in the fast path and in the general exact walk;
- positions with SD = 0 whose wait sits exactly on the SLO or one float away
  (zero-variance groups: the general walk; queue heads with swap and
  eviction seconds: the fast path);
- brute force: every order of 8 groups on one queue, and every assignment
  and order of 5 groups on 2 instances, with swap costs and evictions,
  with random and with deterministic (tie-rich) lengths, and the paper's two
  special cases (earliest deadline first on one queue; same-model grouping
  under costly swaps).  qlm_best_plan must return the oracle's argmin.
"""
import numpy as np
import pytest

import cases
from gpu_util import P_ABS, SCORE_REL, assert_argmin, device_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qlm():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_00047_amd import qlm as q
    q.library()
    return q


def _run(qlm, pr, pl, detail=True):
    import torch
    dpr, dpl = device_inputs(pr, pl)
    P = pl["n_plans"]
    res = qlm.rwt_score(dpr, dpl, detail=(0, P) if detail else None)
    bi, bs = qlm.best_plan(dpr, dpl)
    torch.cuda.synchronize()
    form = qlm.score_form(dpr, pl["evict_bits"] is not None)
    out = {k: v.cpu().numpy() for k, v in res.items() if v is not None}
    return out, int(bi.item()), float(bs.item()), form, dpr.total_requests


def _check_scores(orc, pr, pl, out, bi, bs, N, label):
    osc, _ = orc.score_plans(pr, pl)
    err = np.abs(out["score"] - osc)
    assert np.all(err <= SCORE_REL * max(N, 1)), (label, float(err.max()))
    oi, obs = assert_argmin(bi, osc, label)
    assert abs(bs - obs) <= 1e-12 * max(abs(obs), 1e-300), (label, bs, obs)
    return osc


# ---------------------------------------------------------------------------
# Dense sweep of the normal tail

THETA = 1000.0


def _sweep_points():
    """Margins z = slo - E[W] (with SD = 1 s) that put the kernel's table
    coordinate t = 1536 - z * 1024 / 12 on every cell edge (integer t), at
    quarter, half and nearly whole steps inside each cell, at the clamp ends
    t = 1024, 2048 and beyond them (|z| up to about 7.5)."""
    t = []
    for k in range(1024 - 90, 2048 + 91):
        t += [k, k + 0.25, k + 0.5, k + 0.999]
    t = np.array(t, np.float64)
    return (1536.0 - t) * 12.0 / 1024.0


def _sweep_problem(z, zero_variance_extra):
    """One plan; queue q holds [a_q, b_q]: a_q (1 request of 1000 tokens,
    variance 1e6 tokens^2) ahead of b_q, so b_q waits E = 1 s with SD = 1 s on
    a 1000 tok/s instance; b_q's SLO is 1 + z_q.  With zero_variance_extra a
    last queue holds a group without variance (the problem then takes the
    general exact walk)."""
    groups, queues = [], []
    for zq in z:
        a = len(groups)
        groups.append((1, 1000.0, 1.0e6, 0, 1.0e9))
        groups.append((1, 1.0, 1.0, 0, float(np.float32(1.0 + zq))))
        queues.append([a, a + 1])
    if zero_variance_extra:
        g = len(groups)
        groups.append((3, 100.0, 0.0, 0, 5.0))
        queues.append([g])
    inst = [(THETA, 0)] * len(queues)
    pr = cases.problem(groups, inst)
    pl = cases.plans([queues], len(groups))
    return pr, pl


@pytest.mark.parametrize("general", [False, True], ids=["fast", "general"])
def test_tail_dense_sweep(qlm, orc, general):
    z = _sweep_points()
    worst = 0.0
    for part in np.array_split(z, 3):
        pr, pl = _sweep_problem(part, general)
        print("case tail sweep", "general" if general else "fast", len(part), "points", flush=True)
        out, bi, bs, form, N = _run(qlm, pr, pl)
        assert form == (0 if general else 1)
        d = orc.plan_detail(pr, pl, 0)
        e = np.abs(out["prob"][:, 0].astype(np.float64) - d["prob"])
        worst = max(worst, float(e.max()))
        assert np.all(e <= P_ABS), (float(e.max()), int(np.argmax(e)))
        _check_scores(orc, pr, pl, out, bi, bs, N, "tail sweep")
    print("tail sweep (%s): max |dP| = %.3e over %d margins"
          % ("general" if general else "fast", worst, len(z)))


# ---------------------------------------------------------------------------
# SD = 0: waits exactly on the SLO, or one float away

def _f32_below(x):
    return float(np.nextafter(np.float32(x), np.float32(-np.inf)))


def _f32_above(x):
    return float(np.nextafter(np.float32(x), np.float32(np.inf)))


def test_zero_sd_ties_general(qlm, orc):
    """Zero-variance groups ahead: SD = 0 and P = [E[W] > slo] exactly as the
    definition reads (A / theta + K in double precision)."""
    groups, queues, inst, ev = [], [], [], []
    # (tokens ahead n mu, theta, evicted b?) -> E[W] of the second group
    setups = [(3000.0, 1500.0, False),        # E = 2 exactly
              (3000.0, 1500.0, True),         # E = 2 + 1.25 exactly
              (1000.0, 3.0, False),           # E = 333.33.. (not a float)
              (1000.0, 7.0, True),            # E = 142.857.. + 1.25
              (123456.0, 800.0, False)]
    slot = 0
    for tok, th, evicted in setups:
        E = tok / th + (1.25 if evicted else 0.0)
        for slo in (E, _f32_below(E), _f32_above(E)):
            a = len(groups)
            groups.append((1, tok, 0.0, 0, 1.0e9))
            groups.append((1, 5.0, 0.0, 0, float(np.float32(slo))))
            queues.append([a, a + 1])
            inst.append((th, 0))
            if evicted:
                ev.append(slot + 1)
            slot += 2
    pr = cases.problem(groups, inst, evict_cost=1.25)
    pl = cases.plans([queues], len(groups), evict=[ev])
    out, bi, bs, form, N = _run(qlm, pr, pl)
    assert form == 0
    d = orc.plan_detail(pr, pl, 0)
    assert np.array_equal(out["prob"][:, 0].astype(np.float64), d["prob"]), \
        (out["prob"][:, 0], d["prob"])
    assert set(np.unique(d["prob"][1::2])) == {0.0, 1.0}
    _check_scores(orc, pr, pl, out, bi, bs, N, "zero sd")


def test_head_ties_fast(qlm, orc):
    """Queue heads (SD = 0 in every problem) in the fast path: the head's wait
    is its swap from the loaded model plus its eviction, and the SLO sits on it
    or one float either side."""
    S = np.zeros((1, 3, 3), np.float32)
    S[0, 0, 1], S[0, 1, 0], S[0, 2, 1], S[0, 0, 2] = 7.5, 12.25, 0.8125, 30.0
    groups, queues, inst, m0, ev = [], [], [], [], []
    slot = 0
    for loaded, model, evicted in [(0, 1, False), (1, 0, False), (2, 1, True), (0, 2, True),
                                   (-1, 1, True), (1, 1, False)]:
        K = (float(S[0, loaded, model]) if loaded >= 0 and loaded != model else 0.0) + \
            (2.0 if evicted else 0.0)
        for slo in (K, _f32_below(K), _f32_above(K)):
            h = len(groups)
            groups.append((4, 200.0, 900.0, model, float(np.float32(slo))))
            groups.append((2, 50.0, 100.0, 0, 60.0))
            queues.append([h, h + 1])
            inst.append((1500.0, 0))
            m0.append(loaded)
            if evicted:
                ev.append(slot)
            slot += 2
    pr = cases.problem(groups, inst, n_models=3, swap=S, evict_cost=2.0, model0=m0)
    pl = cases.plans([queues], len(groups), evict=[ev])
    out, bi, bs, form, N = _run(qlm, pr, pl)
    assert form == 1
    d = orc.plan_detail(pr, pl, 0)
    heads = np.arange(0, len(groups), 2)
    assert np.array_equal(out["prob"][heads, 0].astype(np.float64), d["prob"][heads])
    assert set(np.unique(d["prob"][heads])) == {0.0, 1.0}
    _check_scores(orc, pr, pl, out, bi, bs, N, "head ties")


# ---------------------------------------------------------------------------
# Brute force over every plan of tiny problems

def _random_groups(rng, G, M, deterministic):
    groups = []
    for _ in range(G):
        n = 3 if deterministic else int(rng.integers(1, 20))
        mu = 400.0 if deterministic else float(rng.uniform(10, 600))
        var = 0.0 if deterministic else float(rng.uniform(10, 4e4))
        groups.append((n, mu, var, int(rng.integers(0, M)), float(rng.uniform(0.5, 12.0))))
    return groups


@pytest.mark.parametrize("deterministic", [False, True], ids=["random", "deterministic"])
def test_brute_force_orders_one_queue(qlm, orc, deterministic):
    """All 8! orders of 8 groups on one queue, with swap costs and a loaded
    model."""
    rng = np.random.default_rng(11 + deterministic)
    M = 3
    S = rng.uniform(0.5, 6.0, (1, M, M)).astype(np.float32)
    pr = cases.problem(_random_groups(rng, 8, M, deterministic), [(1000.0, 0)], n_models=M,
                       swap=S, model0=[1])
    pl = cases.plans(cases.all_orders(8), 8)
    print("case all orders of 8, deterministic", deterministic, pl["n_plans"], "plans", flush=True)
    out, bi, bs, form, N = _run(qlm, pr, pl, detail=False)
    assert form == (0 if deterministic else 1)
    osc = _check_scores(orc, pr, pl, out, bi, bs, N, ("orders", deterministic))
    print("exact ties at the minimum: %d plans" % int(np.sum(osc == osc.min())))


@pytest.mark.parametrize("deterministic", [False, True], ids=["random", "deterministic"])
def test_brute_force_assignments(qlm, orc, deterministic):
    """Every assignment and order of 5 groups on 2 instances (different
    throughputs and classes), with swap costs, loaded models and an evicted
    slot."""
    rng = np.random.default_rng(21 + deterministic)
    M = 2
    S = rng.uniform(0.5, 6.0, (2, M, M)).astype(np.float32)
    pr = cases.problem(_random_groups(rng, 5, M, deterministic), [(800.0, 0), (1500.0, 1)],
                       n_models=M, n_classes=2, swap=S, evict_cost=1.5, model0=[0, 1])
    qls = cases.all_assignments(5, 2)
    pl = cases.plans(qls, 5, evict=[[2]] * len(qls))
    print("case all assignments of 5 on 2, deterministic", deterministic, len(qls), "plans",
          flush=True)
    out, bi, bs, form, N = _run(qlm, pr, pl)
    assert form == (0 if deterministic else 1)
    for p in range(0, len(qls), 97):
        d = orc.plan_detail(pr, pl, p)
        assert np.all(np.abs(out["prob"][:, p] - d["prob"]) <= P_ABS)
    osc = _check_scores(orc, pr, pl, out, bi, bs, N, ("assignments", deterministic))
    print("exact ties at the minimum: %d plans" % int(np.sum(osc == osc.min())))


def test_edf_special_case(qlm, orc):
    """One queue, deterministic equal groups, no swaps: only the earliest-
    deadline-first order meets every SLO (Jackson's rule, the paper's EDF
    baseline), so it is the best plan."""
    # each group takes 1 s; group i's SLO is its EDF finish-start plus slack
    slos = [3.5, 0.5, 5.5, 2.5, 1.5, 6.5, 4.5]
    groups = [(1, 1000.0, 0.0, 0, s) for s in slos]
    pr = cases.problem(groups, [(1000.0, 0)])
    pl = cases.plans(cases.all_orders(7), 7)
    out, bi, bs, form, N = _run(qlm, pr, pl, detail=False)
    osc = _check_scores(orc, pr, pl, out, bi, bs, N, "edf")
    edf = [int(i) for i in np.argsort(slos, kind="stable")]
    assert list(pl["perm"][:, bi]) == edf
    assert bs == 0.0 and np.sum(osc == 0.0) == 1


def test_grouping_special_case(qlm, orc):
    """Costly swaps: the model-0 groups (tight SLOs) must all run before the
    first swap, so the best plans keep each model's groups together (the
    paper's same-model grouping)."""
    groups = [(1, 500.0, 0.0, 0, 10.0)] * 3 + [(1, 500.0, 0.0, 1, 200.0)] * 3
    pr = cases.problem(groups, [(1000.0, 0)], n_models=2, swap=100.0, model0=[0])
    pl = cases.plans(cases.all_orders(6), 6)
    out, bi, bs, form, N = _run(qlm, pr, pl, detail=False)
    osc = _check_scores(orc, pr, pl, out, bi, bs, N, "grouping")
    models = [int(pr["grp_model"][i]) for i in pl["perm"][:, bi]]
    assert models == [0, 0, 0, 1, 1, 1] and bs == 0.0
