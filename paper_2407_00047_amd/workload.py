"""Seeded synthetic workloads for QLM plan scoring (input generation only).

The paper (arXiv 2407.00047, Sec. 8) drives its system with ShareGPT requests,
Poisson arrivals and three SLO classes (interactive 20 s, batch 1 min / 1 h).
That dataset is not available here; these workloads stand in for it with
synthetic request groups of the same kind (lognormal or Pareto output tokens,
interactive/batch SLO mixes, heterogeneous instance throughputs, model swaps
and evictions) at five scales, from a one-queue toy to 8192 groups on 64
instances.

Nothing here computes waiting times, probabilities or scores.  The problem
tables are drawn with numpy; the (large) plan batches come from the C
generator ``csrc/qlm_gen.c`` (per-plan streams, so any plan range can be
regenerated alone).  Both the HIP path and the CPU oracle read these arrays.

Layout (slot-major, plan stride ``ld``): perm[G, ld], qoff[I+1, ld],
evict_bits[ceil(G/32), ld].
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_GEN_SRC = os.path.join(_HERE, "csrc", "qlm_gen.c")
_GEN_LIB = os.path.join(_HERE, "libqlm_gen.so")
_lock = threading.Lock()
_gen = None

SEED_BASE = 0x514C4D00

# name -> description.  Sizes: G groups, I instances (classes x throughput),
# M models, requests per group, P plans.
CONFIGS = {
    "tiny": dict(index=0, G=8, I=1, M=1, C=1, tput=[2000.0], group_size=("fixed", 8),
                 tokens=("lognormal", 5.3, 0.9), slo=("uniform", 10.0, 60.0), swap=None,
                 evict_frac=0.0, P=256),
    "mixed": dict(index=1, G=128, I=4, M=2, C=1, tput=[2000.0], group_size=("fixed", 32),
                  tokens=("lognormal", 5.3, 0.9),
                  slo=("mix", [(0.2, 20.0, 20.0), (0.8, 1800.0, 3600.0)]),
                  swap=("flat", 15.0), evict_frac=0.0, P=16384),
    "hetero": dict(index=2, G=1024, I=16, M=4, C=4, tput=[800.0, 1500.0, 3000.0, 6000.0],
                   group_size=("fixed", 64), tokens=("lognormal", 5.3, 0.9),
                   slo=("mix", [(0.2, 20.0, 20.0), (0.8, 1800.0, 3600.0)]),
                   swap=("class_model", 5.0, 40.0), evict_frac=0.05, P=65536),
    "heavy": dict(index=3, G=1024, I=16, M=4, C=4, tput=[800.0, 1500.0, 3000.0, 6000.0],
                  group_size=("loguniform", 16, 256), tokens=("pareto", 1.8, 32.0, 8192.0),
                  slo=("mix", [(0.4, 10.0, 30.0), (0.6, 1800.0, 14400.0)]),
                  swap=("class_model", 5.0, 40.0), evict_frac=0.05, P=262144),
    "large": dict(index=4, G=8192, I=64, M=8, C=4, tput=[800.0, 1500.0, 3000.0, 6000.0],
                  group_size=("fixed", 128), tokens=("lognormal", 5.5, 1.1),
                  slo=("mix", [(0.2, 20.0, 20.0), (0.8, 1800.0, 3600.0)]),
                  swap=("class_model", 5.0, 40.0), evict_frac=0.05, P=131072),
}
EVICT_COST = 2.0
SAMPLES_PER_REQUEST = 8


def build_generator(force: bool = True) -> str:
    if force or not os.path.exists(_GEN_LIB):
        tmp = _GEN_LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-std=c11", "-Wall", "-shared", "-fPIC",
                        "-o", tmp, _GEN_SRC], check=True)
        os.replace(tmp, _GEN_LIB)
    return _GEN_LIB


def _lib():
    global _gen
    with _lock:
        if _gen is None:
            # QLM_GEN_LIB: another build of the same source (the sanitizer test)
            path = os.environ.get("QLM_GEN_LIB")
            if path is None:
                if not os.path.exists(_GEN_LIB):
                    build_generator(force=False)
                path = _GEN_LIB
            lib = ctypes.CDLL(path)
            lib.qlm_gen_plans.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_int]
            lib.qlm_gen_plans.restype = ctypes.c_int
            _gen = lib
    return _gen


def _tokens(rng, spec, size):
    """Output-token draws, rounded to whole tokens (at least one)."""
    if spec[0] == "lognormal":
        x = rng.lognormal(spec[1], spec[2], size)
    elif spec[0] == "pareto":
        alpha, xmin, cap = spec[1], spec[2], spec[3]
        x = np.minimum(xmin * (1.0 - rng.random(size)) ** (-1.0 / alpha), cap)
    else:
        raise ValueError(spec)
    return np.maximum(np.rint(x), 1.0)


def make_problem(name: str, seed: int | None = None):
    """Group, instance and swap tables of a named workload."""
    cfg = CONFIGS[name]
    seed = SEED_BASE + cfg["index"] if seed is None else seed
    rng = np.random.default_rng(seed)
    G, I, M, C = cfg["G"], cfg["I"], cfg["M"], cfg["C"]

    kind = cfg["group_size"]
    if kind[0] == "fixed":
        n = np.full(G, kind[1], np.int64)
    else:
        lo, hi = kind[1], kind[2]
        n = np.floor(np.exp(rng.uniform(np.log(lo), np.log(hi + 1), G))).astype(np.int64)
        n = np.clip(n, lo, hi)

    # group statistics from SAMPLES_PER_REQUEST draws per request: sample mean
    # and unbiased sample variance of the output tokens
    mu = np.empty(G)
    var = np.empty(G)
    for i in range(G):
        x = _tokens(rng, cfg["tokens"], int(n[i]) * SAMPLES_PER_REQUEST)
        mu[i] = x.mean()
        var[i] = x.var(ddof=1)

    model = rng.integers(0, M, G)

    sk = cfg["slo"]
    if sk[0] == "uniform":
        slo = rng.uniform(sk[1], sk[2], G)
    else:
        slo = np.empty(G)
        classes = sk[1]
        counts = [int(round(f * G)) for f, _, _ in classes[:-1]]
        counts.append(G - sum(counts))
        who = rng.permutation(G)
        start = 0
        for (f, lo, hi), cnt in zip(classes, counts):
            idx = who[start:start + cnt]
            slo[idx] = lo if lo == hi else rng.uniform(lo, hi, cnt)
            start += cnt

    cls = (np.arange(I) * C) // I                    # I/C instances per class
    tput = np.asarray(cfg["tput"], np.float64)[cls]

    sw = cfg["swap"]
    if sw is None:
        swap = None
    elif sw[0] == "flat":
        swap = np.full((C, M, M), sw[1])
    else:                                             # per (class, incoming model)
        s = rng.uniform(sw[1], sw[2], (C, M))
        swap = np.repeat(s[:, None, :], M, axis=1)
    if swap is not None:
        for c in range(C):
            np.fill_diagonal(swap[c], 0.0)
        swap = swap.astype(np.float32).reshape(-1)

    return {
        "name": name, "seed": seed,
        "n_groups": G, "n_instances": I, "n_models": M, "n_classes": C,
        "grp_count": n.astype(np.int32), "grp_mu": mu.astype(np.float32),
        "grp_var": var.astype(np.float32), "grp_model": model.astype(np.int32),
        "grp_slo": slo.astype(np.float32), "inst_tput": tput.astype(np.float32),
        "inst_class": cls.astype(np.int32), "inst_model0": None, "swap_cost": swap,
        "evict_cost": EVICT_COST if cfg["evict_frac"] > 0 else 0.0,
        "n_evict": int(round(cfg["evict_frac"] * G)) if cfg["evict_frac"] > 0 else 0,
    }


def plan_seed(problem) -> int:
    return (int(problem["seed"]) * 0x9E3779B1 + 0x5151) & 0xFFFFFFFFFFFFFFFF


def make_plans(problem, p0: int = 0, count: int | None = None, ld: int | None = None,
               threads: int = 0, out=None):
    """Plans [p0, p0+count) of the workload, slot-major with plan stride ld.
    ``out`` may supply preallocated (perm, qoff, evict_bits) arrays."""
    name = problem.get("name")
    if count is None:
        count = CONFIGS[name]["P"] - p0
    ld = count if ld is None else ld
    G, I = problem["n_groups"], problem["n_instances"]
    W = (G + 31) // 32
    has_ev = problem.get("n_evict", 0) > 0
    if out is None:
        perm = np.empty((G, ld), np.int32)
        qoff = np.empty((I + 1, ld), np.int32)
        ev = np.empty((W, ld), np.uint32) if has_ev else None
    else:
        perm, qoff, ev = out
    rc = _lib().qlm_gen_plans(plan_seed(problem), p0, count, G, I,
                              int(problem.get("n_evict", 0)), ld, perm.ctypes.data,
                              qoff.ctypes.data, None if ev is None else ev.ctypes.data,
                              int(threads))
    if rc != 0:
        raise RuntimeError("plan generation failed")
    if ld > count:                                  # keep padding columns valid
        perm[:, count:] = perm[:, :1]
        qoff[:, count:] = qoff[:, :1]
        if ev is not None:
            ev[:, count:] = ev[:, :1]
    return {"n_plans": count, "perm": perm, "qoff": qoff, "evict_bits": ev}


def make(name: str, n_plans: int | None = None, seed: int | None = None, threads: int = 0):
    """Problem and plans of a named workload (all P plans unless n_plans is given)."""
    pr = make_problem(name, seed)
    pl = make_plans(pr, 0, CONFIGS[name]["P"] if n_plans is None else n_plans, threads=threads)
    return pr, pl


def total_requests(problem) -> int:
    return int(np.asarray(problem["grp_count"], np.int64).sum())


ARRIVAL_WINDOW = 0.25


def make_request_slos(problem, seed: int | None = None):
    """Per-request TTFT SLOs for the first-come-first-served variant: every
    request carries its group's SLO target, less the time it has already waited
    since it arrived.  A group's requests arrived as a Poisson stream over about
    ARRIVAL_WINDOW of its SLO, the last one just now; they are listed group by
    group, each group's in arrival order (oldest first).  float32 [sum n_i]."""
    seed = (int(problem["seed"]) ^ 0xFCF5) if seed is None else seed
    rng = np.random.default_rng(seed)
    n = np.asarray(problem["grp_count"], np.int64)
    slo = np.asarray(problem["grp_slo"], np.float64)
    N = int(n.sum())
    grp = np.repeat(np.arange(n.size), n)
    gap = rng.exponential(1.0, N) * (ARRIVAL_WINDOW * slo / np.maximum(n, 1))[grp]
    end = np.cumsum(n)[grp]                          # one past each request's group
    c = np.cumsum(gap)
    age = c[end - 1] - c                             # gaps of the later requests
    return (slo[grp] - age).astype(np.float32)


def make_profile(problem, seed: int | None = None):
    """A synthetic hardware profile for the problem's classes and models (the
    constants the estimator profiles offline): prefill 0.05-0.5 s per model,
    decode time per output token 8-40 ms and inefficiency 1.05-1.5 per (class,
    model), the largest output 1024-4096 tokens per model, a token memory of
    5e4-4e5 tokens per (class, model), 300-1200 tokens per request per model.
    Arrays float32, [M] or [C*M] (class-major)."""
    seed = (int(problem["seed"]) ^ 0x9F0F) if seed is None else seed
    rng = np.random.default_rng(seed)
    C, M = int(problem["n_classes"]), int(problem["n_models"])
    f = np.float32
    return {"prefill": rng.uniform(0.05, 0.5, M).astype(f),
            "decode_time": rng.uniform(0.008, 0.040, C * M).astype(f),
            "ineff": rng.uniform(1.05, 1.5, C * M).astype(f),
            "max_tokens": np.floor(rng.uniform(1024, 4097, M)).astype(f),
            "kv_tokens": np.floor(rng.uniform(5e4, 4e5, C * M)).astype(f),
            "mean_tokens": np.floor(rng.uniform(300, 1201, M)).astype(f)}
