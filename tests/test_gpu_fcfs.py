"""Parity of the per-request (first come, first served) score with the oracle.

  - exact scores (qlm_fcfs_score_exact) of every plan of hand-built and
    generated cases against the oracle: both double precision in the same
    order, so they agree to the last bits of erfc;
  - screened scores (qlm_fcfs_score) within the stated bound, 8e-6 per
    request, of the oracle's;
  - the best plan (qlm_fcfs_best_plan): the oracle's argmin, lowest index on
    ties, with its exact score;
  - chunking (a workspace too small for one pass) changes nothing;
  - at the benchmarked size (8192 groups of 128 requests, 16,384 plans) a
    sample of plans against the oracle, and the best plan against the
    screened scores of every plan.
"""
import time

import numpy as np
import pytest

from cases import hand_case, plans as make_plans_by_hand, problem as make_problem_by_hand
from gpu_util import assert_argmin, device_inputs

pytestmark = pytest.mark.gpu

EXACT_REL = 1e-12
EPS_P = 8e-6


@pytest.fixture(scope="module")
def qlm():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_00047_amd import qlm as q
    q.library()
    return q


def _req_slos(rng, pr, lo=0.0, hi=120.0):
    """Per-request SLOs drawn uniformly; a group's requests in arrival order."""
    N = int(np.asarray(pr["grp_count"], np.int64).sum())
    return rng.uniform(lo, hi, N).astype(np.float32)


CASES = [
    dict(G=1, I=1, P=3),
    dict(G=7, I=2, P=70),
    dict(G=40, I=3, P=130, empty_queues=True),
    dict(G=70, I=4, P=65, model0=False),
    dict(G=97, I=1, P=5, evict=False),
    dict(G=64, I=64, P=9),
    dict(G=300, I=12, P=66, skewed=True),
    # more groups than the segment sums' LDS copy of the group table holds
    # (16 B a group, 160 KiB): they read the problem's own arrays instead
    dict(G=10500, I=40, P=70),
]


def _case(kw, seed):
    rng = np.random.default_rng(seed)
    kw = dict(kw)
    pr, pl = hand_case(rng, **kw)
    # a few groups without variance, and a few without requests
    G = pr["n_groups"]
    pr["grp_var"][rng.choice(G, size=max(1, G // 6), replace=False)] = 0.0
    if G > 4:
        pr["grp_count"][rng.choice(G, size=G // 8, replace=False)] = 0
    return pr, pl, _req_slos(rng, pr)


def _run(qlm, pr, pl, req, chunk_plans=0):
    import torch
    dpr, dpl = device_inputs(pr, pl)
    dreq = qlm.device_requests(req)
    ws = qlm.fcfs_workspace(dpr, pl["n_plans"], req.size, chunk_plans=chunk_plans)
    F = qlm.fcfs_score(dpr, dpl, dreq, ws=ws).cpu().numpy()
    X = qlm.fcfs_score_exact(dpr, dpl, dreq, np.arange(pl["n_plans"]), ws=ws).cpu().numpy()
    bi, bs = qlm.fcfs_best_plan(dpr, dpl, dreq, ws=ws)
    torch.cuda.synchronize()
    return F, X, int(bi.item()), float(bs.item())


def _check(orc, pr, pl, req, F, X, bi, bs, label):
    S = orc.score_plans_fcfs(pr, pl, req)
    N = req.size
    assert np.all(np.abs(X - S) <= EXACT_REL * (np.abs(S) + 1.0)), (label, np.abs(X - S).max())
    err = np.abs(F - S)
    assert np.all(err <= EPS_P * N + 1e-9), (label, err.max(), EPS_P * N)
    oi, os_ = orc.argmin(S)
    assert bi == oi, (label, bi, oi, bs, os_)
    assert abs(bs - os_) <= EXACT_REL * (abs(os_) + 1.0), (label, bs, os_)
    return err.max() / max(N, 1)


@pytest.mark.parametrize("k", range(len(CASES)))
def test_fcfs_hand_cases(qlm, orc, k):
    pr, pl, req = _case(CASES[k], 100 + k)
    F, X, bi, bs = _run(qlm, pr, pl, req)
    r = _check(orc, pr, pl, req, F, X, bi, bs, CASES[k])
    print("case", k, "screen error per request", r)


def test_fcfs_chunks_change_nothing(qlm, orc):
    """A workspace for chunks of 64 plans: 3 chunks and a ragged tail."""
    pr, pl, req = _case(dict(G=50, I=5, P=200), 7)
    full = _run(qlm, pr, pl, req)
    small = _run(qlm, pr, pl, req, chunk_plans=64)
    assert np.array_equal(full[0], small[0])
    assert np.array_equal(full[1], small[1])
    assert full[2:] == small[2:]
    _check(orc, pr, pl, req, *small, "chunks")


def test_fcfs_by_hand(qlm):
    """The worked case of the oracle's pins, on the GPU: no variance, waits of
    whole seconds, one SLO met exactly (3 s against 3.0)."""
    pr = make_problem_by_hand([(3, 100.0, 0.0, 0, 9.0), (2, 50.0, 0.0, 0, 9.0)], [(100.0, 0)])
    pl = make_plans_by_hand([[[0, 1]], [[1, 0]]], 2)
    req = np.array([0.5, 0.5, 2.5, 3.0, 3.4], np.float32)
    F, X, bi, bs = _run(qlm, pr, pl, req)
    assert list(F) == [2.0, 3.0] and list(X) == [2.0, 3.0]
    assert (bi, bs) == (0, 2.0)


def test_fcfs_one_request_per_group_is_the_group_score(qlm, orc):
    """n = 1 and req_slo = grp_slo: the group model's exact score, bit for bit
    on the GPU as in the oracle."""
    rng = np.random.default_rng(5)
    pr, pl = hand_case(rng, G=60, I=4, P=40)
    pr["grp_count"][:] = 1
    req = pr["grp_slo"].copy()
    dpr, dpl = device_inputs(pr, pl)
    X = qlm.fcfs_score_exact(dpr, dpl, qlm.device_requests(req), np.arange(40)).cpu().numpy()
    Y = qlm.rwt_score_exact(dpr, dpl, np.arange(40)).cpu().numpy()
    assert np.array_equal(X, Y)
    S, _ = orc.score_plans(pr, pl)
    assert np.all(np.abs(X - S) <= EXACT_REL * (np.abs(S) + 1.0))


def test_fcfs_edges(qlm, orc):
    import torch
    # no requests at all: every score is 0, the lowest index wins
    rng = np.random.default_rng(9)
    pr, pl = hand_case(rng, G=12, I=3, P=5)
    pr["grp_count"][:] = 0
    req = np.zeros(0, np.float32)
    F, X, bi, bs = _run(qlm, pr, pl, req)
    assert np.all(F == 0) and np.all(X == 0) and (bi, bs) == (0, 0.0)
    # no plans: nothing to score, no best plan
    pr, pl = hand_case(rng, G=12, I=3, P=1)
    req = _req_slos(rng, pr)
    dpr, dpl = device_inputs(pr, pl)
    empty = qlm.DevicePlans(dpl.perm, dpl.qoff, None, 0)
    dreq = qlm.device_requests(req)
    bi, bs = qlm.fcfs_best_plan(dpr, empty, dreq)
    torch.cuda.synchronize()
    assert int(bi.item()) == -1 and np.isinf(bs.item())
    # one group holding every request, on one queue of several
    pr = make_problem_by_hand([(300, 250.0, 9000.0, 0, 50.0)], [(500.0, 0), (800.0, 0)])
    pl = make_plans_by_hand([[[0], []], [[], [0]]], 1)
    req = np.linspace(0.0, 200.0, 300).astype(np.float32)
    F, X, bi, bs = _run(qlm, pr, pl, req)
    _check(orc, pr, pl, req, F, X, bi, bs, "one group")


@pytest.mark.parametrize("name,P", [("tiny", 256), ("mixed", 256), ("hetero", 96),
                                     ("heavy", 64)])
def test_fcfs_workloads(qlm, orc, name, P):
    from paper_2407_00047_amd import workload
    pr = workload.make_problem(name)
    pl = workload.make_plans(pr, 0, P)
    req = workload.make_request_slos(pr)
    F, X, bi, bs = _run(qlm, pr, pl, req)
    r = _check(orc, pr, pl, req, F, X, bi, bs, name)
    print(name, "screen error per request", r)


def test_fcfs_large(qlm, orc):
    """The benchmarked configuration: 8192 groups of 128 requests on 64
    instances, 16,384 plans (two chunks).  The oracle scores every plan (all
    host threads): each screened score within the bound of it, the best plan
    the oracle's argmin, its exact score the oracle's; exact scores of a
    sample of plans against the oracle's."""
    import torch
    from paper_2407_00047_amd import workload
    pr = workload.make_problem("large")
    P = 16384
    pl = workload.make_plans(pr, 0, P)
    req = workload.make_request_slos(pr)
    dpr, dpl = device_inputs(pr, pl)
    dreq = qlm.device_requests(req)
    ws = qlm.fcfs_workspace(dpr, P, req.size)
    F = qlm.fcfs_score(dpr, dpl, dreq, ws=ws).cpu().numpy()
    bi, bs = qlm.fcfs_best_plan(dpr, dpl, dreq, ws=ws)
    torch.cuda.synchronize()
    bi, bs = int(bi.item()), float(bs.item())
    N = req.size
    sample = [0, 1, 8191, 8192, P - 1, bi]
    X = qlm.fcfs_score_exact(dpr, dpl, dreq, np.array(sample), ws=ws).cpu().numpy()
    for k, p in enumerate(sample):
        sub = {"n_plans": 1, "perm": np.ascontiguousarray(pl["perm"][:, p:p + 1]),
               "qoff": np.ascontiguousarray(pl["qoff"][:, p:p + 1]),
               "evict_bits": np.ascontiguousarray(pl["evict_bits"][:, p:p + 1])}
        S = orc.score_plans_fcfs(pr, sub, req)[0]
        assert abs(X[k] - S) <= EXACT_REL * (abs(S) + 1.0), (p, X[k], S)
        assert abs(F[p] - S) <= EPS_P * N, (p, F[p], S)
    assert bs == X[-1]
    t0 = time.perf_counter()
    S_all = orc.score_plans_fcfs(pr, pl, req)
    print("oracle: %d plans in %.1f s" % (P, time.perf_counter() - t0), flush=True)
    err = np.abs(F - S_all)
    print("large: screen error per request, max %.3e (bound %.1e)" % (err.max() / N, EPS_P))
    assert np.all(err <= EPS_P * N), (int(np.argmax(err)), float(err.max()))
    oi, obs = assert_argmin(bi, S_all, "fcfs large")
    assert abs(bs - obs) <= EXACT_REL * (abs(obs) + 1.0), (bs, obs)
    print("large: best", bi, bs, "oracle", oi, obs)
