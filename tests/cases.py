"""Hand-built tiny problems and plans for tests.

Builders only: no waiting-time or probability arithmetic lives here.  A plan is
given as queues (one list of group ids per virtual queue); it is laid out
slot-major, the layout both the oracle and the library read.
"""
from __future__ import annotations

import itertools

import numpy as np


def problem(groups, instances, n_models=1, n_classes=1, swap=None, evict_cost=0.0,
            model0=None):
    """groups: list of (n, mu, var, model, slo); instances: list of (tput, cls).
    swap: None, a scalar (same cost for every model change), or a [C][M][M] array."""
    g = np.array(groups, dtype=np.float64).reshape(-1, 5)
    inst = np.array(instances, dtype=np.float64).reshape(-1, 2)
    if swap is not None and np.ndim(swap) == 0:
        s = np.full((n_classes, n_models, n_models), float(swap), np.float32)
        swap = s
    return {
        "n_groups": len(g), "n_instances": len(inst), "n_models": int(n_models),
        "n_classes": int(n_classes),
        "grp_count": g[:, 0].astype(np.int32), "grp_mu": g[:, 1].astype(np.float32),
        "grp_var": g[:, 2].astype(np.float32), "grp_model": g[:, 3].astype(np.int32),
        "grp_slo": g[:, 4].astype(np.float32),
        "inst_tput": inst[:, 0].astype(np.float32), "inst_class": inst[:, 1].astype(np.int32),
        "inst_model0": None if model0 is None else np.asarray(model0, np.int32),
        "swap_cost": None if swap is None else np.asarray(swap, np.float32).reshape(-1),
        "evict_cost": float(evict_cost),
    }


def plans(queue_lists, n_groups, evict=None, ld=None):
    """queue_lists: one entry per plan, each a list (per queue) of group-id lists.
    evict: None or, per plan, an iterable of evicted slot indices."""
    P = len(queue_lists)
    I = len(queue_lists[0])
    ld = P if ld is None else ld
    perm = np.zeros((n_groups, ld), np.int32)
    qoff = np.zeros((I + 1, ld), np.int32)
    W = (n_groups + 31) // 32
    ev = np.zeros((W, ld), np.uint32) if evict is not None else None
    for p, queues in enumerate(queue_lists):
        assert len(queues) == I
        flat = [i for q in queues for i in q]
        assert sorted(flat) == list(range(n_groups)), "each group in exactly one slot"
        perm[:, p] = flat
        qoff[:, p] = np.concatenate([[0], np.cumsum([len(q) for q in queues])])
        if evict is not None:
            for s in evict[p]:
                ev[s // 32, p] |= np.uint32(1) << np.uint32(s % 32)
    # padding columns (p >= P) hold a valid plan too, so strided reads stay sane
    for p in range(P, ld):
        perm[:, p] = perm[:, 0]
        qoff[:, p] = qoff[:, 0]
    return {"n_plans": P, "perm": perm, "qoff": qoff, "evict_bits": ev}


def all_orders(n_groups):
    """Every ordering of groups 0..n-1 on one queue."""
    return [[list(o)] for o in itertools.permutations(range(n_groups))]


def all_assignments(n_groups, n_queues):
    """Every (assignment to queues x order within each queue)."""
    out = []
    for order in itertools.permutations(range(n_groups)):
        for cuts in itertools.combinations_with_replacement(range(n_groups + 1), n_queues - 1):
            bounds = (0,) + cuts + (n_groups,)
            out.append([list(order[bounds[k]:bounds[k + 1]]) for k in range(n_queues)])
    # remove duplicates that differ only in how empty queues were cut
    seen, uniq = set(), []
    for q in out:
        key = tuple(tuple(x) for x in q)
        if key not in seen:
            seen.add(key)
            uniq.append(q)
    return uniq


def subset_plans(pl, idx):
    """Plans pl restricted to the given plan indices (a new, contiguous batch)."""
    idx = np.asarray(idx)
    return {"n_plans": len(idx), "perm": np.ascontiguousarray(pl["perm"][:, idx]),
            "qoff": np.ascontiguousarray(pl["qoff"][:, idx]),
            "evict_bits": None if pl.get("evict_bits") is None
            else np.ascontiguousarray(pl["evict_bits"][:, idx])}


def hand_case(rng, G, I, M=3, C=2, P=70, model0=True, evict=True, empty_queues=False,
              skewed=False, min_count=0):
    """Random groups, instances and plans drawn from rng (uniform sizes, SLOs
    and costs; optional empty queues, skewed queue lengths, eviction flags).
    min_count=1 keeps every group non-empty (with a positive variance)."""
    groups = []
    for _ in range(G):
        groups.append((int(rng.integers(min_count, 30)), float(rng.uniform(1, 600)),
                       float(rng.uniform(min_count, 5e4)), int(rng.integers(0, M)),
                       float(rng.uniform(0.1, 300))))
    inst = [(float(rng.choice([400.0, 1000.0, 5000.0])), int(rng.integers(0, C))) for _ in range(I)]
    S = rng.uniform(0.5, 30.0, (C, M, M)).astype(np.float32)
    m0 = [int(x) for x in rng.integers(-1, M, I)] if model0 else None
    pr = problem(groups, inst, n_models=M, n_classes=C, swap=S, evict_cost=1.25, model0=m0)
    qls, evs = [], []
    for p in range(P):
        order = rng.permutation(G)
        k = I if not empty_queues else max(1, I // 3)
        if skewed:
            # a few long queues and many short ones: 32-slot blocks with one queue
            # head per plan and blocks with several, in the same plan
            w = np.where(np.arange(I) < 3, 30.0, 1.0)
            owner = rng.choice(I, size=G, p=w / w.sum())
        else:
            owner = rng.integers(0, k, G)
        qls.append([[int(i) for i in order if owner[i] == g] for g in range(I)])
        evs.append(list(rng.choice(G, size=min(G, 3), replace=False)))
    pl = plans(qls, G, evict=evs if evict else None)
    return pr, pl
