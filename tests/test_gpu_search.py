"""Parity of the GPU plan search with the oracle.

  - every move score of every plan (qlm_search_moves) against the oracle,
    which builds each moved plan and scores it from scratch: both are double
    precision in the same order, so they agree to the last bits of erfc;
  - the search itself (qlm_local_search): the moves taken step by step, the
    steps, the final plans (bit-exact) and their scores.  Where both sides are
    at a near-tie (two moves whose scores differ only in erfc's last bits) the
    GPU may take the other move; that step is then checked for being a valid
    choice, and the comparison ends there;
  - at full workload sizes, a sample of move scores and a few search steps,
    each checked by the oracle on the plan the search holds at that step.
"""
import time
import zlib

import numpy as np
import pytest

from cases import hand_case
from gpu_util import device_inputs

pytestmark = pytest.mark.gpu

# Both sides are double precision with the same operations in the same order;
# only the device and host erfc differ, in their last bits.
MOVE_REL = 1e-12


@pytest.fixture(scope="module")
def qlm():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_00047_amd import qlm as q
    q.library()
    return q


def _close(a, b):
    a = np.atleast_1d(np.asarray(a, np.float64))
    b = np.atleast_1d(np.asarray(b, np.float64))
    same_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    fin = np.isfinite(a) & np.isfinite(b)
    ok = same_inf.copy()
    ok[fin] = np.abs(a[fin] - b[fin]) <= MOVE_REL * (np.abs(b[fin]) + 1.0)
    return ok


def _flags(pl, p, G):
    if pl.get("evict_bits") is None:
        return np.zeros(G, np.uint8)
    w = pl["evict_bits"][:, p]
    return ((w[np.arange(G) // 32] >> (np.arange(G) % 32)) & 1).astype(np.uint8)


def _one(perm, qoff, flag, with_flags):
    G = len(perm)
    ev = None
    if with_flags:
        ev = np.zeros(((G + 31) // 32, 1), np.uint32)
        for s in np.flatnonzero(flag):
            ev[s // 32, 0] |= np.uint32(1) << np.uint32(s % 32)
    return {"n_plans": 1, "perm": np.asarray(perm, np.int32).reshape(G, 1),
            "qoff": np.asarray(qoff, np.int32).reshape(-1, 1), "evict_bits": ev}


SEARCH_CASES = [
    dict(G=1, I=1, P=2, W=1),                       # no move at all
    dict(G=5, I=3, P=9, W=2),
    dict(G=33, I=2, P=8, W=4, evict=False),
    dict(G=70, I=4, P=6, W=8, empty_queues=True),
    dict(G=97, I=1, P=3, W=5, model0=False),        # one queue: no reassignment
    dict(G=40, I=5, P=5, W=0),                      # no swaps
    dict(G=64, I=64, P=4, W=3),                     # about one group per queue
    dict(G=300, I=12, P=4, W=16, skewed=True),      # two rank blocks per queue
    dict(G=160, I=3, P=3, W=200),                   # window beyond every queue
]


def _case(kw):
    kw = dict(kw)
    W = kw.pop("W")
    rng = np.random.default_rng(zlib.crc32(("search" + str(sorted(kw.items()))).encode()))
    pr, pl = hand_case(rng, **kw)
    return pr, pl, W


@pytest.mark.parametrize("kw", SEARCH_CASES, ids=[str(c) for c in SEARCH_CASES])
def test_move_scores(qlm, orc, kw):
    import torch
    pr, pl, W = _case(kw)
    print("case", kw, flush=True)
    dpr, dpl = device_inputs(pr, pl)
    ms = qlm.search_moves(dpr, dpl, W)
    torch.cuda.synchronize()
    ms = ms.cpu().numpy()
    G, I = pr["n_groups"], pr["n_instances"]
    assert ms.shape == (pl["n_plans"], G * W + 2 * G * I)
    exact = 0
    kinds = np.zeros(3, np.int64)
    for p in range(pl["n_plans"]):
        ref = orc.move_scores(pr, pl, p, W)
        ok = _close(ms[p], ref)
        bad = np.flatnonzero(~ok)
        assert ok.all(), (p, bad[:5], ms[p][bad[:5]], ref[bad[:5]])
        exact += int(np.sum(ms[p] == ref))
        fin = np.isfinite(ref)
        kinds += [fin[:G * W].sum(), fin[G * W:G * W + G * I].sum(), fin[G * W + G * I:].sum()]
    print("bit-identical move scores: %d of %d; moves SWAP %d MOVE %d RELOCATE %d"
          % (exact, ms.size, *kinds))


def _check_screen(F, D, ref, label):
    """Screened scores within their bounds of the exact ones; +inf where no move."""
    F = np.asarray(F)
    D = np.asarray(D)
    nomove = np.isinf(ref)
    assert np.all(np.isinf(F[nomove])) and np.all(D[nomove] == 0), label
    mv = ~nomove
    assert np.all(np.isfinite(F[mv])) and np.all(D[mv] >= 0), label
    fin = mv & np.isfinite(D)
    err = np.abs(F[fin] - ref[fin])
    assert np.all(err <= D[fin]), (label, int(np.argmax(err - D[fin])), float(np.max(err - D[fin])))
    return int(np.sum(mv & np.isinf(D))), float(np.max(err / np.maximum(D[fin], 1e-300))) if err.size else 0.0


@pytest.mark.parametrize("kw", SEARCH_CASES, ids=[str(c) for c in SEARCH_CASES])
def test_screen_bounds(qlm, orc, kw):
    """Every screened move score lies within its bound of the oracle's score."""
    import torch
    pr, pl, W = _case(kw)
    print("case", kw, flush=True)
    dpr, dpl = device_inputs(pr, pl)
    F, D = qlm.search_screen(dpr, dpl, W)
    torch.cuda.synchronize()
    F = F.cpu().numpy()
    D = D.cpu().numpy()
    forced, worst = 0, 0.0
    for p in range(pl["n_plans"]):
        ref = orc.move_scores(pr, pl, p, W)
        f, w = _check_screen(F[p], D[p], ref, (kw, p))
        forced += f
        worst = max(worst, w)
    print("unbounded (scored exactly): %d of %d; largest error / bound %.3g" % (forced, F.size, worst))


def test_screen_bounds_long_queue(qlm, orc):
    """A queue of 4300 groups, longer than the reassignment screen stages in
    LDS for its insertion points (4096): the screened scores of every move
    within their bounds of the oracle's."""
    import torch
    rng = np.random.default_rng(52)
    pr, pl = hand_case(rng, G=4500, I=2, P=1)
    pl["qoff"][:, 0] = [0, 4300, 4500]
    dpr, dpl = device_inputs(pr, pl)
    F, D = qlm.search_screen(dpr, dpl, 4)
    torch.cuda.synchronize()
    ref = orc.move_scores(pr, pl, 0, 4)
    f, w = _check_screen(F.cpu().numpy()[0], D.cpu().numpy()[0], ref, "long queue")
    print("unbounded: %d; largest error / bound %.3g" % (f, w))


@pytest.mark.parametrize("kw", [dict(G=600, I=3, P=2, W=500),
                                dict(G=300, I=5, P=2, M=20, C=3, W=8)],
                         ids=["window 500", "1200 swap costs"])
def test_screen_bounds_unstaged(qlm, orc, kw):
    """The removal and swap screen stages its lanes' slot records (up to 384
    slots) and the swap-cost table (up to 1024 entries) in LDS: a window of 500
    takes the records from global memory, 20 models in 3 classes the costs;
    every move's screened score within its bound of the oracle's."""
    import torch
    pr, pl, W = _case(kw)
    dpr, dpl = device_inputs(pr, pl)
    F, D = qlm.search_screen(dpr, dpl, W)
    torch.cuda.synchronize()
    F, D = F.cpu().numpy(), D.cpu().numpy()
    for p in range(pl["n_plans"]):
        _check_screen(F[p], D[p], orc.move_scores(pr, pl, p, W), (kw, p))


def test_screen_bounds_many_groups(qlm, orc):
    """17,000 groups: the SLO ranks are counted over 17 tiles of 1024 groups,
    the last one ragged; every move's screened score within its bound of the
    oracle's."""
    import torch
    rng = np.random.default_rng(53)
    pr, pl = hand_case(rng, G=17000, I=4, P=1)
    dpr, dpl = device_inputs(pr, pl)
    F, D = qlm.search_screen(dpr, dpl, 1)
    torch.cuda.synchronize()
    ref = orc.move_scores(pr, pl, 0, 1)
    f, w = _check_screen(F.cpu().numpy()[0], D.cpu().numpy()[0], ref, "many groups")
    print("unbounded: %d; largest error / bound %.3g" % (f, w))


def _check_search(orc, pr, pl, p, W, T, g_trace, g_steps, g_perm, g_qoff, g_ev, g_score):
    """Compares one chain's search with the oracle's; returns the step where a
    near-tie let the two sides part (None when they agree throughout)."""
    G = pr["n_groups"]
    o = orc.local_search(pr, pl, p, W, T)
    ot = o["trace"]
    diff = np.flatnonzero(g_trace != ot)
    if diff.size == 0:
        assert g_steps == o["steps"]
        assert np.array_equal(g_perm, o["perm"]) and np.array_equal(g_qoff, o["qoff"])
        assert np.array_equal(g_ev, o["evict_bits"])
        assert _close(g_score, o["score"]), (g_score, o["score"])
        return None
    t = int(diff[0])
    # replay the common steps, then judge the GPU's choice at step t
    perm, qoff, flag = pl["perm"][:, p].copy(), pl["qoff"][:, p].copy(), _flags(pl, p, G)
    for k in ot[:t]:
        perm, qoff, flag = orc.move_apply(pr, perm, qoff, flag, W, int(k))
    one = _one(perm, qoff, flag, True)
    cur = orc.plan_detail(pr, one, 0)["score"]
    allm = orc.move_scores(pr, one, 0, W)
    best = float(allm.min())
    gk = int(g_trace[t])
    if gk >= 0:
        # the GPU's move must be a minimum up to erfc's last bits, and an improvement
        assert _close(allm[gk], best), (t, gk, allm[gk], best)
        assert allm[gk] < cur or _close(allm[gk], cur)
    else:
        # the GPU stopped: no move may improve beyond erfc's last bits
        assert _close(best, cur) or best >= cur, (t, best, cur)
    return t


@pytest.mark.parametrize("kw", SEARCH_CASES, ids=[str(c) for c in SEARCH_CASES])
def test_local_search(qlm, orc, kw):
    import torch
    pr, pl, W = _case(kw)
    T = 25
    print("case", kw, "steps", T, flush=True)
    dpr, dpl = device_inputs(pr, pl)
    r = qlm.local_search(dpr, dpl, W, T, trace=True)
    torch.cuda.synchronize()
    out = r["plans"]
    g_perm = out.perm.cpu().numpy()
    g_qoff = out.qoff.cpu().numpy()
    g_ev = out.evict_bits.cpu().numpy().view(np.uint32)
    g_trace = r["trace"].cpu().numpy()
    g_steps = r["steps"].cpu().numpy()
    g_score = r["score"].cpu().numpy()
    moved = 0
    for p in range(pl["n_plans"]):
        t = _check_search(orc, pr, pl, p, W, T, g_trace[p], int(g_steps[p]), g_perm[:, p],
                          g_qoff[:, p], g_ev[:, p], float(g_score[p]))
        if t is not None:
            print("plan %d: near-tie at step %d" % (p, t))
        moved += int(g_steps[p])
    G, I = pr["n_groups"], pr["n_instances"]
    print("moves applied over all plans: %d (relocations %d)"
          % (moved, int(np.sum(g_trace >= G * W + G * I))))
    # scores never rise, and the final scores are those of the final plans
    ex = qlm.rwt_score_exact(dpr, out, np.arange(pl["n_plans"]))
    assert np.array_equal(ex.cpu().numpy(), g_score)


def test_relocate_by_hand(qlm, orc):
    """Head-of-line blocking on one 100 tok/s instance: a running batch group
    (1000 tokens, SLO 60 s), behind it an interactive group (2 x 10 tokens,
    SLO 1 s) that misses (score 2).  Its relocation to the head, paying E, is
    the one move (k 5; the others touch the running group or lie beyond G):
    score 0 for E = 0.5 s and E = 1 s (a wait equal to the SLO meets it), 2
    for E = 2 s, where the search keeps the plan.  Placement of the
    interactive group: the head place c = 1 wins unless E = 2 s."""
    import torch
    from cases import plans as hplans, problem as hproblem
    for E, sc in ((0.5, 0.0), (2.0, 2.0), (1.0, 0.0)):
        pr = hproblem([(1, 1000.0, 0.0, 0, 60.0), (2, 10.0, 0.0, 0, 1.0)], [(100.0, 0)],
                      evict_cost=E)
        pl = hplans([[[0, 1]]], 2)
        dpr, dpl = device_inputs(pr, pl)
        ms = qlm.search_moves(dpr, dpl, 1).cpu().numpy()[0]
        assert list(ms) == [np.inf] * 5 + [sc], (E, ms)
        F, D = qlm.search_screen(dpr, dpl, 1)
        _check_screen(F.cpu().numpy()[0], D.cpu().numpy()[0], ms, ("hand", E))
        r = qlm.local_search(dpr, dpl, 1, 2, trace=True)
        pg = qlm.place_group(dpr, dpl, 1)
        torch.cuda.synchronize()
        moved = sc < 2.0
        assert float(r["score"][0]) == sc and int(r["steps"][0]) == int(moved), (E, r)
        assert list(r["trace"].cpu().numpy()[0]) == ([5, -1] if moved else [-1, -1])
        assert list(r["plans"].perm.cpu().numpy()[:, 0]) == ([1, 0] if moved else [0, 1])
        assert int(r["plans"].evict_bits.cpu().numpy()[0, 0]) == (1 if moved else 0)
        o = orc.place_group(pr, pl, 0, 1)
        assert int(pg["queue"][0]) == o["queue"] == (1 if moved else 0), (E, o["queue"])
        assert float(pg["score"][0]) == o["score"]
        assert list(pg["plans"].perm.cpu().numpy()[:, 0]) == list(o["perm"])


def test_search_edge_calls(qlm, orc):
    """No steps: the start plans and their scores come back unchanged; a search
    in place (output arrays = start arrays); plans that already meet every SLO
    do not move."""
    import torch
    rng = np.random.default_rng(11)
    pr, pl = hand_case(rng, G=50, I=4, P=5)
    dpr, dpl = device_inputs(pr, pl)
    r = qlm.local_search(dpr, dpl, 4, 0, trace=True)
    torch.cuda.synchronize()
    assert np.array_equal(r["plans"].perm.cpu().numpy(), pl["perm"])
    assert np.array_equal(r["plans"].qoff.cpu().numpy(), pl["qoff"])
    assert np.array_equal(r["plans"].evict_bits.cpu().numpy().view(np.uint32), pl["evict_bits"])
    assert np.all(r["steps"].cpu().numpy() == 0)
    osc, _ = orc.score_plans(pr, pl)
    assert np.all(_close(r["score"].cpu().numpy(), osc))
    # in place
    dpl2 = device_inputs(pr, pl)[1]
    r2 = qlm.local_search(dpr, dpl2, 4, 6, out=dpl2)
    ref = qlm.local_search(dpr, dpl, 4, 6)
    torch.cuda.synchronize()
    assert torch.equal(dpl2.perm, ref["plans"].perm) and torch.equal(dpl2.qoff, ref["plans"].qoff)
    assert torch.equal(r2["score"], ref["score"])
    # SLOs no wait reaches: score 0, nothing moves
    pr3 = dict(pr)
    pr3["grp_slo"] = np.full(pr["n_groups"], 3.0e38, np.float32)
    dpr3 = device_inputs(pr3, pl)[0]
    r3 = qlm.local_search(dpr3, dpl, 4, 5)
    torch.cuda.synchronize()
    assert np.all(r3["steps"].cpu().numpy() == 0) and np.all(r3["score"].cpu().numpy() == 0.0)


def test_search_workloads(qlm, orc):
    """Two plans of each generated workload small enough for the oracle's
    full neighbourhoods: all move scores, then five search steps."""
    import torch
    from paper_2407_00047_amd import workload
    for name, W in (("tiny", 4), ("mixed", 8), ("hetero", 8)):
        pr = workload.make_problem(name)
        pl = workload.make_plans(pr, 0, 2)
        print("workload", name, flush=True)
        dpr, dpl = device_inputs(pr, pl)
        ms = qlm.search_moves(dpr, dpl, W).cpu().numpy()
        F, D = qlm.search_screen(dpr, dpl, W)
        F = F.cpu().numpy()
        D = D.cpu().numpy()
        for p in range(2):
            ref = orc.move_scores(pr, pl, p, W)
            assert _close(ms[p], ref).all(), (name, p)
            print(name, "screen: unbounded, worst error/bound", _check_screen(F[p], D[p], ref, (name, p)))
        r = qlm.local_search(dpr, dpl, W, 5, trace=True)
        torch.cuda.synchronize()
        out = r["plans"]
        for p in range(2):
            _check_search(orc, pr, pl, p, W, 5, r["trace"].cpu().numpy()[p],
                          int(r["steps"][p]), out.perm.cpu().numpy()[:, p],
                          out.qoff.cpu().numpy()[:, p],
                          out.evict_bits.cpu().numpy().view(np.uint32)[:, p],
                          float(r["score"][p]))


FULL = [("hetero", 16), ("heavy", 16), ("large", 16)]


@pytest.mark.slow
@pytest.mark.parametrize("name,W", FULL, ids=[f[0] for f in FULL])
def test_search_full_size(qlm, orc, name, W):
    """One plan of the full workload: a sample of move scores (and the best
    one) against the oracle, and three search steps, each move re-scored by
    the oracle on the plan the search held at that step."""
    import torch
    from paper_2407_00047_amd import workload
    pr = workload.make_problem(name)
    pl = workload.make_plans(pr, 0, 1)
    G, I = pr["n_groups"], pr["n_instances"]
    print("full size", name, "G", G, "I", I, "W", W, flush=True)
    dpr, dpl = device_inputs(pr, pl)
    ms = qlm.search_moves(dpr, dpl, W).cpu().numpy()[0]
    # the oracle scores every move (each moved plan from scratch)
    t0 = time.perf_counter()
    ref_all = orc.move_scores(pr, pl, 0, W)
    print("oracle: %d moves in %.1f s" % (ref_all.size, time.perf_counter() - t0), flush=True)
    assert np.array_equal(np.isfinite(ms), np.isfinite(ref_all))
    assert _close(ms, ref_all).all()
    first_min, _ = orc.argmin(ref_all)
    rng = np.random.default_rng(1)
    valid = np.flatnonzero(np.isfinite(ms))
    ks = np.concatenate([rng.choice(valid, 200, replace=False), [first_min],
                         np.flatnonzero(~np.isfinite(ms))[:20]])
    ref = ref_all[ks]
    F, D = qlm.search_screen(dpr, dpl, W)
    F = F.cpu().numpy()[0]
    D = D.cpu().numpy()[0]
    print("screen on the sample: unbounded, worst error/bound", _check_screen(F[ks], D[ks], ref, name))
    # every move: the screen against the exact scores of the GPU's exact kernels
    # (both checked against the oracle above on the sample)
    print("screen on all moves (against the exact kernels):", _check_screen(F, D, ms, name))
    T = 3
    r = qlm.local_search(dpr, dpl, W, T, trace=True)
    torch.cuda.synchronize()
    tr = r["trace"].cpu().numpy()[0]
    # the first step takes the oracle's best move (lowest number on ties)
    assert tr[0] == first_min, (tr[0], first_min)
    perm, qoff, flag = pl["perm"][:, 0].copy(), pl["qoff"][:, 0].copy(), _flags(pl, 0, G)
    cur = orc.plan_detail(pr, _one(perm, qoff, flag, True), 0)["score"]
    for t in range(T):
        k = int(tr[t])
        if k < 0:
            break
        v = orc.move_scores(pr, _one(perm, qoff, flag, True), 0, W, ks=[k])[0]
        assert v < cur
        perm, qoff, flag = orc.move_apply(pr, perm, qoff, flag, W, k)
        cur = v
    out = r["plans"]
    assert np.array_equal(out.perm.cpu().numpy()[:, 0], perm)
    assert np.array_equal(out.qoff.cpu().numpy()[:, 0], qoff)
    assert _close(float(r["score"][0]), cur)


SEED_CASES = [dict(G=1, I=1), dict(G=5, I=3), dict(G=40, I=5, model0=False), dict(G=97, I=1),
              dict(G=300, I=12), dict(G=64, I=64), dict(G=200, I=70)]


@pytest.mark.parametrize("kw", SEED_CASES, ids=[str(c) for c in SEED_CASES])
def test_seed_plans(qlm, orc, kw):
    """Seed plans bit-exact against the oracle's, both policies."""
    import torch
    rng = np.random.default_rng(zlib.crc32(("seed" + str(sorted(kw.items()))).encode()))
    pr, pl = hand_case(rng, P=1, **kw)
    print("case", kw, flush=True)
    dpr = device_inputs(pr, pl)[0]
    sp = qlm.seed_plans(dpr, (0, 1, 0), evict=True)
    torch.cuda.synchronize()
    perm = sp.perm.cpu().numpy()
    qoff = sp.qoff.cpu().numpy()
    assert np.all(sp.evict_bits.cpu().numpy() == 0)
    for k, policy in enumerate((0, 1, 0)):
        p, q = orc.seed_plan(pr, policy)
        assert np.array_equal(perm[:, k], p), (kw, policy)
        assert np.array_equal(qoff[:, k], q), (kw, policy)


def test_seed_plans_workloads(qlm, orc):
    """Seed plans of every generated workload, bit-exact, and a search from them."""
    import torch
    from paper_2407_00047_amd import workload
    for name in ("tiny", "mixed", "hetero", "heavy", "large"):
        pr = workload.make_problem(name)
        dpr = qlm.DeviceProblem(pr)
        sp = qlm.seed_plans(dpr, (0, 1))
        torch.cuda.synchronize()
        for k in (0, 1):
            p, q = orc.seed_plan(pr, k)
            assert np.array_equal(sp.perm.cpu().numpy()[:, k], p), (name, k)
            assert np.array_equal(sp.qoff.cpu().numpy()[:, k], q), (name, k)
        sc = qlm.rwt_score_exact(dpr, sp, [0, 1]).cpu().numpy()
        print(name, "seed scores EDF %.6g grouped %.6g" % tuple(sc), flush=True)


PLACE_CASES = [dict(G=1, I=1, P=2), dict(G=5, I=3, P=9), dict(G=33, I=2, P=8, evict=False),
               dict(G=70, I=4, P=6, empty_queues=True), dict(G=97, I=1, P=3),
               dict(G=64, I=64, P=4), dict(G=300, I=12, P=4, skewed=True)]


@pytest.mark.parametrize("kw", PLACE_CASES, ids=[str(c) for c in PLACE_CASES])
def test_place_group(qlm, orc, kw):
    """Placed plans bit-exact, chosen queues and exact scores against the oracle
    (a near-tie between two queues may pick either; the choice is then checked
    for being a minimum)."""
    import torch
    rng = np.random.default_rng(zlib.crc32(("place" + str(sorted(kw.items()))).encode()))
    pr, pl = hand_case(rng, **kw)
    G = pr["n_groups"]
    dpr, dpl = device_inputs(pr, pl)
    for group in sorted({0, G - 1, G // 2}):
        print("case", kw, "group", group, flush=True)
        r = qlm.place_group(dpr, dpl, group)
        torch.cuda.synchronize()
        out = r["plans"]
        perm = out.perm.cpu().numpy()
        qoff = out.qoff.cpu().numpy()
        sc = r["score"].cpu().numpy()
        qu = r["queue"].cpu().numpy()
        for p in range(pl["n_plans"]):
            o = orc.place_group(pr, pl, p, group)
            if qu[p] != o["queue"]:
                # a near-tie: the GPU's choice must score the same to erfc's last bits
                assert _close(sc[p], o["score"]), (kw, group, p, qu[p], o["queue"])
                continue
            assert np.array_equal(perm[:, p], o["perm"]) and np.array_equal(qoff[:, p], o["qoff"])
            assert np.array_equal(out.evict_bits.cpu().numpy().view(np.uint32)[:, p],
                                  o["evict_bits"])
            assert _close(sc[p], o["score"]), (sc[p], o["score"])
        ex = qlm.rwt_score_exact(dpr, out, np.arange(pl["n_plans"])).cpu().numpy()
        assert np.array_equal(ex, sc)


def test_place_group_arrival(qlm, orc):
    """An arrival: the hetero workload with one more group parked at the end of
    queue 0 of every plan, then placed."""
    import torch
    from paper_2407_00047_amd import workload
    pr = workload.make_problem("hetero")
    pl = workload.make_plans(pr, 0, 4)
    G = pr["n_groups"]
    pr2 = dict(pr)
    pr2["n_groups"] = G + 1
    for k, v in (("grp_count", 7), ("grp_mu", 250.0), ("grp_var", 4e4), ("grp_model", 1),
                 ("grp_slo", 20.0)):
        pr2[k] = np.concatenate([pr[k], np.array([v], pr[k].dtype)])
    e1 = pl["qoff"][1]
    perm = np.concatenate([pl["perm"], np.full((1, 4), -1, np.int32)])
    for p in range(4):
        col = list(pl["perm"][:, p])
        col.insert(int(e1[p]), G)
        perm[:, p] = col
    qoff = pl["qoff"].copy()
    qoff[1:] += 1
    W = (G + 1 + 31) // 32
    ev = np.zeros((W, 4), np.uint32)
    pl2 = {"n_plans": 4, "perm": perm, "qoff": qoff, "evict_bits": ev}
    dpr, dpl = device_inputs(pr2, pl2)
    r = qlm.place_group(dpr, dpl, G)
    torch.cuda.synchronize()
    for p in range(4):
        o = orc.place_group(pr2, pl2, p, G)
        assert int(r["queue"][p]) == o["queue"]
        assert np.array_equal(r["plans"].perm.cpu().numpy()[:, p], o["perm"])
        assert _close(float(r["score"][p]), o["score"])


@pytest.mark.parametrize("fast", [0, 2])
def test_place_group_long_move(qlm, orc, fast):
    """A placement that moves more slots than a workgroup stages in LDS (8192):
    9000 groups on 3 queues, one instance 100 times faster than the others.
    fast = 2: the group is second in queue 0, which holds 8301 groups (the
    slots shift left); fast = 0: the group ends queue 2 and queue 0 holds 100
    groups (they shift right)."""
    import torch
    from cases import plans as make_plans_by_hand, problem as make_problem_by_hand
    rng = np.random.default_rng(31 + fast)
    G = 9000
    groups = [(int(rng.integers(1, 20)), float(rng.uniform(50, 600)), float(rng.uniform(0, 5e4)),
               0, float(rng.uniform(1, 50))) for _ in range(G)]
    inst = [(400.0, 0)] * 3
    inst[fast] = (40000.0, 0)
    pr = make_problem_by_hand(groups, inst)
    order = [int(x) for x in rng.permutation(G)]
    if fast == 2:
        group = order[1]
        queues = [order[:8301], order[8301:8311], order[8311:]]
    else:
        group = order[-1]
        queues = [order[:100], order[100:4600], order[4600:]]
    pl = make_plans_by_hand([queues], G)
    dpr, dpl = device_inputs(pr, pl)
    r = qlm.place_group(dpr, dpl, group)
    torch.cuda.synchronize()
    o = orc.place_group(pr, pl, 0, group)
    span = abs(list(o["perm"]).index(group) - list(pl["perm"][:, 0]).index(group)) + 1
    assert span > 8192 and int(r["queue"][0]) == o["queue"], (span, o["queue"])
    assert np.array_equal(r["plans"].perm.cpu().numpy()[:, 0], o["perm"])
    assert np.array_equal(r["plans"].qoff.cpu().numpy()[:, 0], o["qoff"])
    assert _close(float(r["score"][0]), o["score"])


@pytest.mark.parametrize("kw", [dict(G=9, I=3, P=5), dict(G=70, I=4, P=6, empty_queues=True),
                                dict(G=300, I=12, P=4, skewed=True), dict(G=40, I=1, P=3)])
def test_place_session(qlm, orc, kw):
    """A session places groups one after another with the plans kept in the
    workspace, re-forming only the changed queues' cache: each step's plans and
    scores equal placing the same groups with qlm_place_group, call after call,
    and the oracle's placements of the sequence."""
    import torch
    rng = np.random.default_rng(zlib.crc32(("session" + str(sorted(kw.items()))).encode()))
    pr, pl = hand_case(rng, **kw)
    G, P = pr["n_groups"], pl["n_plans"]
    groups = [int(x) for x in rng.integers(0, G, 8)]
    dpr, dpl = device_inputs(pr, pl)
    ses = qlm.PlaceSession(dpr, dpl)
    cur = dpl
    host = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in pl.items()}
    for k, group in enumerate(groups):
        print("case", kw, "step", k, "group", group, flush=True)
        sc, qu = ses.step(group)
        r = qlm.place_group(dpr, cur, group)
        torch.cuda.synchronize()
        assert np.array_equal(sc.cpu().numpy(), r["score"].cpu().numpy()), (k, group)
        assert np.array_equal(qu.cpu().numpy(), r["queue"].cpu().numpy()), (k, group)
        cur = r["plans"]
        # the oracle, plan by plan, on the host copy of the plans so far
        for p in range(P):
            o = orc.place_group(pr, host, p, group)
            if int(qu[p]) == o["queue"]:
                assert _close(float(sc[p]), o["score"]), (k, p)
        host = {"n_plans": P, "perm": cur.perm.cpu().numpy(), "qoff": cur.qoff.cpu().numpy(),
                "evict_bits": cur.evict_bits.cpu().numpy().view(np.uint32)}
    out, score = ses.end()
    torch.cuda.synchronize()
    assert np.array_equal(out.perm.cpu().numpy(), cur.perm.cpu().numpy())
    assert np.array_equal(out.qoff.cpu().numpy(), cur.qoff.cpu().numpy())
    assert np.array_equal(out.evict_bits.cpu().numpy(), cur.evict_bits.cpu().numpy())
    ex = qlm.rwt_score_exact(dpr, out, np.arange(P)).cpu().numpy()
    assert np.array_equal(score.cpu().numpy(), ex)
