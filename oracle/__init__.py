"""fp64 CPU oracle for QLM plan scoring (arXiv 2407.00047, Secs. 6-7).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no code
with the HIP path and never imports it.

The arithmetic lives in ``qlm_oracle.c`` (plain C, double precision); this
module compiles it with gcc and marshals numpy arrays through ctypes.

Inputs are plain mappings of numpy arrays (the same arrays the GPU reads):

problem: n_groups, n_instances, n_models, n_classes, grp_count[G] int32,
         grp_mu[G] f32, grp_var[G] f32, grp_model[G] int32, grp_slo[G] f32,
         inst_tput[I] f32, inst_class[I] int32, inst_model0[I] int32 or None,
         swap_cost[C*M*M] f32 or None, evict_cost float
plans:   n_plans, perm[G, ld] int32, qoff[I+1, ld] int32,
         evict_bits[ceil(G/32), ld] uint32 or None      (slot-major)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qlm_oracle.c")
_LIB = os.path.join(_HERE, "libqlm_oracle.so")
_lock = threading.Lock()
_default = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (IEEE double, no contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Problem(ctypes.Structure):
    _fields_ = [("n_groups", ctypes.c_int32), ("n_instances", ctypes.c_int32),
                ("n_models", ctypes.c_int32), ("n_classes", ctypes.c_int32),
                ("grp_count", ctypes.c_void_p), ("grp_mu", ctypes.c_void_p),
                ("grp_var", ctypes.c_void_p), ("grp_model", ctypes.c_void_p),
                ("grp_slo", ctypes.c_void_p), ("inst_tput", ctypes.c_void_p),
                ("inst_class", ctypes.c_void_p), ("inst_model0", ctypes.c_void_p),
                ("swap_cost", ctypes.c_void_p), ("evict_cost", ctypes.c_float)]


class _Plans(ctypes.Structure):
    _fields_ = [("n_plans", ctypes.c_int64), ("ld", ctypes.c_int64),
                ("perm", ctypes.c_void_p), ("qoff", ctypes.c_void_p),
                ("evict_bits", ctypes.c_void_p)]


class _Profile(ctypes.Structure):
    _fields_ = [("prefill", ctypes.c_void_p), ("decode_time", ctypes.c_void_p),
                ("ineff", ctypes.c_void_p), ("max_tokens", ctypes.c_void_p),
                ("kv_tokens", ctypes.c_void_p), ("mean_tokens", ctypes.c_void_p)]


PROFILE_FIELDS = ("prefill", "decode_time", "ineff", "max_tokens", "kv_tokens", "mean_tokens")


class Oracle:
    """A loaded oracle library.  ``Oracle()`` is the committed source built by
    ``build()``; tests may load another build of it (for mutation checks)."""

    def __init__(self, path: str | None = None):
        if path is None:
            # QLM_ORACLE_LIB: another build of the same source (the sanitizer test)
            path = os.environ.get("QLM_ORACLE_LIB")
        if path is None:
            if not os.path.exists(_LIB):
                build(force=False)
            path = _LIB
        lib = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        lib.oracle_plan.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans),
                                    ctypes.c_int64, dp, dp, dp, dp, dp]
        lib.oracle_plan.restype = ctypes.c_int
        lib.oracle_score_plans.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans),
                                           ctypes.c_int64, ctypes.c_int64, dp, dp, ctypes.c_int]
        lib.oracle_score_plans.restype = ctypes.c_int64
        lib.oracle_argmin.argtypes = [dp, ctypes.c_int64, dp]
        lib.oracle_argmin.restype = ctypes.c_int64
        lib.oracle_max_threads.restype = ctypes.c_int
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.oracle_n_moves.argtypes = [i32, i32, i32]
        lib.oracle_n_moves.restype = i64
        lib.oracle_move_apply.argtypes = [ctypes.POINTER(_Problem), i32, i64, vp, vp, vp, vp, vp, vp]
        lib.oracle_move_apply.restype = ctypes.c_int
        lib.oracle_move_scores.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans), i64,
                                           i32, vp, i64, dp, ctypes.c_int]
        lib.oracle_move_scores.restype = ctypes.c_int
        lib.oracle_local_search.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans), i64,
                                            i32, i32, vp, vp, vp, dp, vp, vp, ctypes.c_int]
        lib.oracle_local_search.restype = ctypes.c_int
        lib.oracle_seed_plan.argtypes = [ctypes.POINTER(_Problem), i32, vp, vp]
        lib.oracle_seed_plan.restype = ctypes.c_int
        lib.oracle_place_group.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans), i64,
                                           i32, vp, vp, vp, dp, vp]
        lib.oracle_place_group.restype = ctypes.c_int
        lib.oracle_plan_fcfs.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans), i64,
                                         vp, i64, dp, dp]
        lib.oracle_plan_fcfs.restype = ctypes.c_int
        lib.oracle_score_plans_fcfs.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Plans),
                                                vp, i64, i64, i64, dp, ctypes.c_int]
        lib.oracle_score_plans_fcfs.restype = ctypes.c_int64
        lib.oracle_apply_profile.argtypes = [ctypes.POINTER(_Problem), ctypes.POINTER(_Profile),
                                             vp, vp, vp, vp, vp, i64, vp]
        lib.oracle_apply_profile.restype = None
        self.lib = lib
        self.path = path

    def max_threads(self) -> int:
        return int(self.lib.oracle_max_threads())

    def score_plans(self, problem, plans, p0: int = 0, count: int | None = None,
                    threads: int = 0):
        """fp64 score and penalty of plans [p0, p0+count).  Returns (score, penalty)."""
        b = _Bound(problem, plans)
        if count is None:
            count = b.n_plans - p0
        if p0 < 0 or count < 0 or p0 + count > b.n_plans:
            raise ValueError("plan range out of bounds")
        score = np.empty(count, np.float64)
        pen = np.empty(count, np.float64)
        bad = self.lib.oracle_score_plans(ctypes.byref(b.problem), ctypes.byref(b.plans), p0,
                                          count, _dp(score), _dp(pen), int(threads))
        if bad:
            raise ValueError("%d malformed plans" % bad)
        return score, pen

    def plan_detail(self, problem, plans, p: int):
        """Per-slot E[W], SD[W], P and the plan's score and penalty, for plan p."""
        b = _Bound(problem, plans)
        if not 0 <= p < b.n_plans:
            raise ValueError("plan index out of range")
        wm = np.full(b.G, np.nan)
        ws = np.full(b.G, np.nan)
        pr = np.full(b.G, np.nan)
        sc = np.zeros(1)
        pe = np.zeros(1)
        rc = self.lib.oracle_plan(ctypes.byref(b.problem), ctypes.byref(b.plans), p,
                                  _dp(wm), _dp(ws), _dp(pr), _dp(sc), _dp(pe))
        if rc != 0:
            raise ValueError("malformed plan %d" % p)
        return {"wait_mean": wm, "wait_sd": ws, "prob": pr, "score": float(sc[0]),
                "penalty": float(pe[0])}

    def argmin(self, score) -> tuple[int, float]:
        """Lowest score, lowest index on ties."""
        s = np.ascontiguousarray(score, dtype=np.float64)
        bs = np.zeros(1)
        idx = self.lib.oracle_argmin(_dp(s), s.size, _dp(bs))
        return int(idx), float(bs[0])

    def best_plan(self, problem, plans, threads: int = 0) -> tuple[int, float]:
        """argmin_p score_p over all plans, lowest index on ties."""
        score, _ = self.score_plans(problem, plans, threads=threads)
        return self.argmin(score)

    # -- per-request (FCFS within each group) variant ------------------------

    def score_plans_fcfs(self, problem, plans, req_slo, p0: int = 0, count: int | None = None,
                         threads: int = 0):
        """fp64 per-request scores of plans [p0, p0+count); req_slo holds every
        group's request SLOs in arrival order, group by group."""
        b = _Bound(problem, plans)
        slo = np.ascontiguousarray(req_slo, dtype=np.float32)
        if count is None:
            count = b.n_plans - p0
        if p0 < 0 or count < 0 or p0 + count > b.n_plans:
            raise ValueError("plan range out of bounds")
        if slo.size != int(np.asarray(problem["grp_count"], np.int64).sum()):
            raise ValueError("req_slo must hold sum(grp_count) entries")
        score = np.empty(count, np.float64)
        bad = self.lib.oracle_score_plans_fcfs(ctypes.byref(b.problem), ctypes.byref(b.plans),
                                               _ptr(slo), slo.size, p0, count, _dp(score),
                                               int(threads))
        if bad:
            raise ValueError("%d malformed plans" % bad)
        return score

    def plan_fcfs(self, problem, plans, req_slo, p: int):
        """Per-request P (indexed as req_slo) and the score of plan p."""
        b = _Bound(problem, plans)
        slo = np.ascontiguousarray(req_slo, dtype=np.float32)
        if not 0 <= p < b.n_plans:
            raise ValueError("plan index out of range")
        prob = np.full(slo.size, np.nan)
        sc = np.zeros(1)
        if self.lib.oracle_plan_fcfs(ctypes.byref(b.problem), ctypes.byref(b.plans), p,
                                     _ptr(slo), slo.size, _dp(prob), _dp(sc)):
            raise ValueError("malformed plan %d or req_slo size" % p)
        return {"prob": prob, "score": float(sc[0])}

    def best_plan_fcfs(self, problem, plans, req_slo, threads: int = 0) -> tuple[int, float]:
        """argmin_p of the per-request score, lowest index on ties."""
        return self.argmin(self.score_plans_fcfs(problem, plans, req_slo, threads=threads))

    # -- problem tables from a hardware profile -----------------------------

    def apply_profile(self, problem, profile, inst_model=None, req_slo=None):
        """The problem with its swap table (plus the drain before a model
        change), SLOs (less the prefill) and throughputs (from the GPU's token
        memory, the decode step and the inefficiency) derived from a hardware
        profile: a dict of [M] or [C*M] float32 arrays, any of them None.
        Returns (problem, req_slo or None)."""
        G, I = int(problem["n_groups"]), int(problem["n_instances"])
        M, C = int(problem["n_models"]), int(problem["n_classes"])
        plans = {"n_plans": 0, "perm": np.zeros((G, 1), np.int32),
                 "qoff": np.zeros((I + 1, 1), np.int32), "evict_bits": None}
        b = _Bound(problem, plans)
        keep = []
        pf = _Profile()
        sizes = {"prefill": M, "decode_time": C * M, "ineff": C * M, "max_tokens": M,
                 "kv_tokens": C * M, "mean_tokens": M}
        for f in PROFILE_FIELDS:
            x = profile.get(f)
            if x is not None:
                x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
                if x.size != sizes[f]:
                    raise ValueError(f + " has the wrong size")
                keep.append(x)
            setattr(pf, f, _ptr(x))
        im = None if inst_model is None else np.ascontiguousarray(inst_model, np.int32)
        if im is not None and (im.size != I or im.max() >= M or im.min() < -1):
            raise ValueError("inst_model must be [I] in [-1, M)")
        swap = np.empty(C * M * M, np.float32)
        slo = np.empty(G, np.float32)
        tput = np.empty(I, np.float32)
        rs = None if req_slo is None else np.ascontiguousarray(req_slo, np.float32)
        rso = None if rs is None else np.empty_like(rs)
        self.lib.oracle_apply_profile(ctypes.byref(b.problem), ctypes.byref(pf), _ptr(im),
                                      _ptr(swap), _ptr(slo), _ptr(tput), _ptr(rs),
                                      0 if rs is None else rs.size, _ptr(rso))
        out = dict(problem)
        out["swap_cost"] = swap
        out["grp_slo"] = slo
        out["inst_tput"] = tput
        return out, rso

    # -- plan search -------------------------------------------------------

    def n_moves(self, G: int, I: int, window: int) -> int:
        return int(self.lib.oracle_n_moves(G, I, window))

    def move_apply(self, problem, perm, qoff, flag, window: int, k: int):
        """Move k applied to one plan given as arrays (perm[G], qoff[I+1],
        flag[G] 0/1).  Returns (perm, qoff, flag) of the new plan, or None when
        k names no move."""
        b = _Bound(problem, {"perm": np.asarray(perm, np.int32).reshape(-1, 1),
                             "qoff": np.asarray(qoff, np.int32).reshape(-1, 1)})
        G, I = b.G, int(problem["n_instances"])
        perm = np.ascontiguousarray(perm, np.int32)
        qoff = np.ascontiguousarray(qoff, np.int32)
        flag = np.ascontiguousarray(flag, np.uint8)
        p2 = np.empty(G, np.int32)
        q2 = np.empty(I + 1, np.int32)
        f2 = np.empty(G, np.uint8)
        ok = self.lib.oracle_move_apply(ctypes.byref(b.problem), int(window), int(k), _ptr(perm),
                                        _ptr(qoff), _ptr(flag), _ptr(p2), _ptr(q2), _ptr(f2))
        return (p2, q2, f2) if ok else None

    def move_scores(self, problem, plans, p: int, window: int, ks=None, threads: int = 0):
        """Exact scores of the moves ks (default: every move, in index order) of
        plan p; +inf where a number names no move."""
        b = _Bound(problem, plans)
        if not 0 <= p < b.n_plans:
            raise ValueError("plan index out of range")
        if window < 0:
            raise ValueError("window must be >= 0")
        if ks is None:
            n = self.n_moves(b.G, int(problem["n_instances"]), window)
            kp = None
        else:
            ks = np.ascontiguousarray(ks, np.int64)
            n = ks.size
            kp = ks
        out = np.empty(n, np.float64)
        self.lib.oracle_move_scores(ctypes.byref(b.problem), ctypes.byref(b.plans), p, window,
                                    _ptr(kp), n, _dp(out), int(threads))
        return out

    def seed_plan(self, problem, policy: int):
        """Seed plan of a policy (0 EDF, 1 same-model grouped): (perm[G], qoff[I+1])."""
        G, I = int(problem["n_groups"]), int(problem["n_instances"])
        b = _Bound(problem, {"perm": np.zeros((G, 1), np.int32),
                             "qoff": np.zeros((I + 1, 1), np.int32)})
        perm = np.empty(G, np.int32)
        qoff = np.empty(I + 1, np.int32)
        if self.lib.oracle_seed_plan(ctypes.byref(b.problem), int(policy), _ptr(perm), _ptr(qoff)):
            raise ValueError("policy must be 0 (EDF) or 1 (grouped)")
        return perm, qoff

    def place_group(self, problem, plans, p: int, group: int):
        """Plan p with `group` moved to the place giving the lowest exact score:
        the EDF position after the head of queue c, or (c >= I) the head of
        queue c - I with its eviction flag set; the lowest c on ties.  A group
        at its queue's head stays.  Returns a dict perm, qoff, evict_bits,
        score, queue (= c)."""
        b = _Bound(problem, plans)
        if not 0 <= p < b.n_plans:
            raise ValueError("plan index out of range")
        G, I = b.G, int(problem["n_instances"])
        perm = np.empty(G, np.int32)
        qoff = np.empty(I + 1, np.int32)
        ev = np.empty((G + 31) // 32, np.uint32)
        sc = np.zeros(1)
        q = np.zeros(1, np.int32)
        if self.lib.oracle_place_group(ctypes.byref(b.problem), ctypes.byref(b.plans), p,
                                       int(group), _ptr(perm), _ptr(qoff), _ptr(ev), _dp(sc),
                                       _ptr(q)):
            raise ValueError("group not in the plan")
        return {"perm": perm, "qoff": qoff, "evict_bits": ev, "score": float(sc[0]),
                "queue": int(q[0])}

    def local_search(self, problem, plans, p: int, window: int, max_steps: int,
                     threads: int = 0):
        """Steepest-descent search from plan p.  Returns a dict with the final
        perm[G], qoff[I+1], evict_bits[ceil(G/32)] (relocations set flags, so
        they are returned even for start plans without), its score, the number
        of steps applied and trace[max_steps]."""
        b = _Bound(problem, plans)
        if not 0 <= p < b.n_plans:
            raise ValueError("plan index out of range")
        if window < 0 or max_steps < 0:
            raise ValueError("window and max_steps must be >= 0")
        G, I = b.G, int(problem["n_instances"])
        perm = np.empty(G, np.int32)
        qoff = np.empty(I + 1, np.int32)
        ev = np.empty((G + 31) // 32, np.uint32)
        sc = np.zeros(1)
        steps = np.zeros(1, np.int32)
        trace = np.full(max(max_steps, 1), -1, np.int64)
        self.lib.oracle_local_search(ctypes.byref(b.problem), ctypes.byref(b.plans), p, window,
                                     max_steps, _ptr(perm), _ptr(qoff), _ptr(ev), _dp(sc),
                                     _ptr(steps), _ptr(trace), int(threads))
        return {"perm": perm, "qoff": qoff, "evict_bits": ev, "score": float(sc[0]),
                "steps": int(steps[0]), "trace": trace[:max_steps]}


def default() -> Oracle:
    global _default
    with _lock:
        if _default is None:
            _default = Oracle()
    return _default


def _arr(a, dtype):
    if a is None:
        return None
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data


def _dp(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


class _Bound:
    """Keeps the numpy buffers alive while ctypes structs point at them."""

    def __init__(self, problem, plans):
        G = int(problem["n_groups"])
        I = int(problem["n_instances"])
        self.keep = []

        def k(x, dt):
            x = _arr(x, dt)
            self.keep.append(x)
            return x

        pr = _Problem()
        pr.n_groups = G
        pr.n_instances = I
        pr.n_models = int(problem["n_models"])
        pr.n_classes = int(problem["n_classes"])
        pr.grp_count = _ptr(k(problem["grp_count"], np.int32))
        pr.grp_mu = _ptr(k(problem["grp_mu"], np.float32))
        pr.grp_var = _ptr(k(problem["grp_var"], np.float32))
        pr.grp_model = _ptr(k(problem["grp_model"], np.int32))
        pr.grp_slo = _ptr(k(problem["grp_slo"], np.float32))
        pr.inst_tput = _ptr(k(problem["inst_tput"], np.float32))
        pr.inst_class = _ptr(k(problem["inst_class"], np.int32))
        pr.inst_model0 = _ptr(k(problem.get("inst_model0"), np.int32))
        pr.swap_cost = _ptr(k(problem.get("swap_cost"), np.float32))
        pr.evict_cost = float(problem.get("evict_cost", 0.0))
        self.problem = pr
        # the C code trusts sizes and ranges; check them here
        M, C = pr.n_models, pr.n_classes
        for name in ("grp_count", "grp_mu", "grp_var", "grp_model", "grp_slo"):
            if np.asarray(problem[name]).size != G:
                raise ValueError(name + " must have n_groups entries")
        for name in ("inst_tput", "inst_class"):
            if np.asarray(problem[name]).size != I:
                raise ValueError(name + " must have n_instances entries")
        model = np.asarray(problem["grp_model"])
        cls = np.asarray(problem["inst_class"])
        if G < 1 or I < 1 or M < 1 or C < 1:
            raise ValueError("sizes must be positive")
        if model.min() < 0 or model.max() >= M or cls.min() < 0 or cls.max() >= C:
            raise ValueError("model or class index out of range")
        if problem.get("inst_model0") is not None:
            m0 = np.asarray(problem["inst_model0"])
            if m0.size != I or m0.min() < -1 or m0.max() >= M:
                raise ValueError("inst_model0 must be [I] in [-1, M)")
        if problem.get("swap_cost") is not None and np.asarray(problem["swap_cost"]).size != C * M * M:
            raise ValueError("swap_cost must have C*M*M entries")

        perm = k(plans["perm"], np.int32)
        qoff = k(plans["qoff"], np.int32)
        ev = k(plans.get("evict_bits"), np.uint32)
        if perm.ndim != 2 or perm.shape[0] != G:
            raise ValueError("perm must be [G, ld]")
        ld = perm.shape[1]
        if qoff.shape != (I + 1, ld):
            raise ValueError("qoff must be [I+1, ld]")
        if ev is not None and ev.shape != ((G + 31) // 32, ld):
            raise ValueError("evict_bits must be [ceil(G/32), ld]")
        n_plans = int(plans.get("n_plans", ld))
        if not 0 <= n_plans <= ld:
            raise ValueError("n_plans must be in [0, ld]")
        pl = _Plans()
        pl.n_plans = n_plans
        pl.ld = ld
        pl.perm = _ptr(perm)
        pl.qoff = _ptr(qoff)
        pl.evict_bits = _ptr(ev)
        self.plans = pl
        self.n_plans = n_plans
        self.G = G


def max_threads() -> int:
    return default().max_threads()


def score_plans(problem, plans, p0: int = 0, count: int | None = None, threads: int = 0):
    return default().score_plans(problem, plans, p0, count, threads)


def plan_detail(problem, plans, p: int):
    return default().plan_detail(problem, plans, p)


def argmin(score) -> tuple[int, float]:
    return default().argmin(score)


def best_plan(problem, plans, threads: int = 0) -> tuple[int, float]:
    return default().best_plan(problem, plans, threads)


def move_scores(problem, plans, p: int, window: int, ks=None, threads: int = 0):
    return default().move_scores(problem, plans, p, window, ks, threads)


def local_search(problem, plans, p: int, window: int, max_steps: int, threads: int = 0):
    return default().local_search(problem, plans, p, window, max_steps, threads)


def seed_plan(problem, policy: int):
    return default().seed_plan(problem, policy)


def place_group(problem, plans, p: int, group: int):
    return default().place_group(problem, plans, p, group)


def score_plans_fcfs(problem, plans, req_slo, p0: int = 0, count: int | None = None,
                     threads: int = 0):
    return default().score_plans_fcfs(problem, plans, req_slo, p0, count, threads)


def plan_fcfs(problem, plans, req_slo, p: int):
    return default().plan_fcfs(problem, plans, req_slo, p)


def best_plan_fcfs(problem, plans, req_slo, threads: int = 0) -> tuple[int, float]:
    return default().best_plan_fcfs(problem, plans, req_slo, threads)


def apply_profile(problem, profile, inst_model=None, req_slo=None):
    return default().apply_profile(problem, profile, inst_model, req_slo)
