"""Python binding of libqlm (include/qlm.h): argument marshalling only.

Every step of the scoring path runs in the HIP kernels of ``csrc/qlm.hip``;
PyTorch supplies device memory and the current stream.  The binding refuses to
run when the library is not built (there is no fallback of any kind).

Function names follow the C interface: ``rwt_score``, ``rwt_score_exact``,
``best_plan`` (with ``best_plan_workspace_bytes``), ``validate_plans``,
``validate_problem``, ``search_n_moves``, ``search_workspace_bytes``,
``search_moves``, ``search_screen``, ``local_search``, ``seed_plans``,
``place_group``.
"""
from __future__ import annotations

import ctypes
import os
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqlm.so")
_lock = threading.Lock()
_lib = None

QLM_OK, QLM_ERR_ARG, QLM_ERR_CAPACITY, QLM_ERR_WORKSPACE, QLM_ERR_HIP = range(5)


class QlmError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("qlm status %d: %s" % (status, message))
        self.status = status


class Problem(ctypes.Structure):
    _fields_ = [("n_groups", ctypes.c_int32), ("n_instances", ctypes.c_int32),
                ("n_models", ctypes.c_int32), ("n_classes", ctypes.c_int32),
                ("grp_count", ctypes.c_void_p), ("grp_mu", ctypes.c_void_p),
                ("grp_var", ctypes.c_void_p), ("grp_model", ctypes.c_void_p),
                ("grp_slo", ctypes.c_void_p), ("inst_tput", ctypes.c_void_p),
                ("inst_class", ctypes.c_void_p), ("inst_model0", ctypes.c_void_p),
                ("swap_cost", ctypes.c_void_p), ("evict_cost", ctypes.c_float)]


class Plans(ctypes.Structure):
    _fields_ = [("n_plans", ctypes.c_int64), ("plan_stride", ctypes.c_int64),
                ("perm", ctypes.c_void_p), ("qoff", ctypes.c_void_p),
                ("evict_bits", ctypes.c_void_p)]


class PlansOut(ctypes.Structure):
    _fields_ = [("plan_stride", ctypes.c_int64), ("perm", ctypes.c_void_p),
                ("qoff", ctypes.c_void_p), ("evict_bits", ctypes.c_void_p)]


class Detail(ctypes.Structure):
    _fields_ = [("plan_begin", ctypes.c_int64), ("plan_count", ctypes.c_int64),
                ("wait_mean", ctypes.c_void_p), ("wait_sd", ctypes.c_void_p),
                ("prob", ctypes.c_void_p)]


class Profile(ctypes.Structure):
    _fields_ = [("prefill", ctypes.c_void_p), ("decode_time", ctypes.c_void_p),
                ("ineff", ctypes.c_void_p), ("max_tokens", ctypes.c_void_p),
                ("kv_tokens", ctypes.c_void_p), ("mean_tokens", ctypes.c_void_p)]


PROFILE_FIELDS = ("prefill", "decode_time", "ineff", "max_tokens", "kv_tokens", "mean_tokens")


def library():
    """The loaded libqlm; raises when it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError("libqlm.so is not built (run __graft_entry__.build() or "
                                   "python -m paper_2407_00047_amd.build)")
            lib = ctypes.CDLL(LIB_PATH)
            P, PL, D = ctypes.POINTER(Problem), ctypes.POINTER(Plans), ctypes.POINTER(Detail)
            vp, i64 = ctypes.c_void_p, ctypes.c_int64
            lib.qlm_rwt_score.argtypes = [P, PL, vp, vp, D, vp]
            lib.qlm_rwt_score_exact.argtypes = [P, PL, vp, i64, vp, vp]
            lib.qlm_best_plan_workspace_bytes.argtypes = [P, i64]
            lib.qlm_best_plan_workspace_bytes.restype = ctypes.c_size_t
            lib.qlm_best_plan.argtypes = [P, PL, vp, ctypes.c_size_t, vp, vp, vp]
            lib.qlm_best_plan_static.argtypes = [P, PL, vp, vp, vp]
            lib.qlm_score_form.argtypes = [P, ctypes.c_int32, vp, vp]
            lib.qlm_validate_plans.argtypes = [P, PL, vp, vp, vp]
            lib.qlm_validate_problem.argtypes = [P, vp, vp]
            lib.qlm_max_groups.argtypes = [ctypes.c_int32] * 4
            lib.qlm_max_groups.restype = ctypes.c_int32
            lib.qlm_status_string.argtypes = [ctypes.c_int]
            lib.qlm_status_string.restype = ctypes.c_char_p
            lib.qlm_last_error.restype = ctypes.c_char_p
            lib.qlm_timing_enable.argtypes = [ctypes.c_int]
            lib.qlm_timing_read.argtypes = [ctypes.POINTER(ctypes.c_int64),
                                            ctypes.POINTER(ctypes.c_double)]
            i32 = ctypes.c_int32
            lib.qlm_search_n_moves.argtypes = [i32, i32, i32]
            lib.qlm_search_n_moves.restype = i64
            lib.qlm_search_workspace_bytes.argtypes = [P, i64, i32]
            lib.qlm_search_workspace_bytes.restype = ctypes.c_size_t
            lib.qlm_search_moves.argtypes = [P, PL, i32, vp, ctypes.c_size_t, vp, vp]
            lib.qlm_search_screen.argtypes = [P, PL, i32, vp, ctypes.c_size_t, vp, vp, vp]
            lib.qlm_place_group.argtypes = [P, PL, ctypes.POINTER(PlansOut), i32, vp,
                                            ctypes.c_size_t, vp, vp, vp]
            lib.qlm_seed_workspace_bytes.argtypes = [P, i32]
            lib.qlm_seed_workspace_bytes.restype = ctypes.c_size_t
            lib.qlm_seed_plans.argtypes = [P, i32, ctypes.POINTER(ctypes.c_int32),
                                           ctypes.POINTER(PlansOut), vp, ctypes.c_size_t, vp]
            lib.qlm_local_search.argtypes = [P, PL, ctypes.POINTER(PlansOut), i32, i32, vp,
                                             ctypes.c_size_t, vp, vp, vp, vp]
            sz = ctypes.c_size_t
            lib.qlm_fcfs_workspace_bytes.argtypes = [P, i64, i64, i64]
            lib.qlm_fcfs_workspace_bytes.restype = sz
            lib.qlm_fcfs_score.argtypes = [P, PL, vp, i64, vp, sz, vp, vp]
            lib.qlm_fcfs_score_exact.argtypes = [P, PL, vp, i64, vp, i64, vp, sz, vp, vp]
            lib.qlm_fcfs_best_plan.argtypes = [P, PL, vp, i64, vp, sz, vp, vp, vp]
            lib.qlm_apply_profile.argtypes = [P, ctypes.POINTER(Profile), vp, vp, vp, vp, vp, i64,
                                              vp, vp]
            lib.qlm_place_begin.argtypes = [P, PL, vp, sz, vp]
            lib.qlm_place_step.argtypes = [P, i64, i32, vp, sz, vp, vp, vp]
            lib.qlm_place_end.argtypes = [P, i64, ctypes.POINTER(PlansOut), vp, sz, vp, vp]
            for name in ("qlm_rwt_score", "qlm_rwt_score_exact", "qlm_best_plan", "qlm_best_plan_static",
                         "qlm_score_form",
                         "qlm_validate_plans", "qlm_validate_problem", "qlm_timing_enable",
                         "qlm_timing_read", "qlm_search_moves", "qlm_search_screen",
                         "qlm_local_search", "qlm_seed_plans", "qlm_place_group",
                         "qlm_fcfs_score", "qlm_fcfs_score_exact", "qlm_fcfs_best_plan",
                         "qlm_apply_profile", "qlm_place_begin", "qlm_place_step",
                         "qlm_place_end"):
                getattr(lib, name).restype = ctypes.c_int
            _lib = lib
    return _lib


def _check(rc: int):
    if rc != QLM_OK:
        lib = library()
        raise QlmError(rc, lib.qlm_last_error().decode())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else t.data_ptr()


class DeviceProblem:
    """Problem tables in device memory (torch tensors) plus the C struct."""

    def __init__(self, problem, device="cuda"):
        import torch

        def dev(x, dt):
            if x is None:
                return None
            return torch.as_tensor(np.ascontiguousarray(x)).to(device=device, dtype=dt)

        self.n_groups = int(problem["n_groups"])
        self.n_instances = int(problem["n_instances"])
        self.n_models = int(problem["n_models"])
        self.n_classes = int(problem["n_classes"])
        self.grp_count = dev(problem["grp_count"], torch.int32)
        self.grp_mu = dev(problem["grp_mu"], torch.float32)
        self.grp_var = dev(problem["grp_var"], torch.float32)
        self.grp_model = dev(problem["grp_model"], torch.int32)
        self.grp_slo = dev(problem["grp_slo"], torch.float32)
        self.inst_tput = dev(problem["inst_tput"], torch.float32)
        self.inst_class = dev(problem["inst_class"], torch.int32)
        self.inst_model0 = dev(problem.get("inst_model0"), torch.int32)
        self.swap_cost = dev(problem.get("swap_cost"), torch.float32)
        self.evict_cost = float(problem.get("evict_cost", 0.0))
        self.total_requests = int(np.asarray(problem["grp_count"], np.int64).sum())
        self.struct = Problem(self.n_groups, self.n_instances, self.n_models, self.n_classes,
                              _ptr(self.grp_count), _ptr(self.grp_mu), _ptr(self.grp_var),
                              _ptr(self.grp_model), _ptr(self.grp_slo), _ptr(self.inst_tput),
                              _ptr(self.inst_class), _ptr(self.inst_model0),
                              _ptr(self.swap_cost), self.evict_cost)


class DevicePlans:
    """A slot-major plan batch in device memory plus the C struct.  ``perm`` is
    [G, stride] int32, ``qoff`` [I+1, stride] int32, ``evict_bits``
    [ceil(G/32), stride] int32 (bit patterns) or None."""

    def __init__(self, perm, qoff, evict_bits=None, n_plans=None):
        self.perm = perm
        self.qoff = qoff
        self.evict_bits = evict_bits
        stride = int(perm.shape[1])
        self.n_plans = stride if n_plans is None else int(n_plans)
        self.struct = Plans(self.n_plans, stride, _ptr(perm), _ptr(qoff), _ptr(evict_bits))

    @classmethod
    def from_host(cls, plans, device="cuda"):
        import torch
        perm = torch.from_numpy(np.ascontiguousarray(plans["perm"])).to(device)
        qoff = torch.from_numpy(np.ascontiguousarray(plans["qoff"])).to(device)
        ev = plans.get("evict_bits")
        if ev is not None:
            ev = torch.from_numpy(np.ascontiguousarray(ev).view(np.int32)).to(device)
        return cls(perm, qoff, ev, plans.get("n_plans"))


def rwt_score(problem: DeviceProblem, plans: DevicePlans, penalty: bool = False,
              detail: tuple[int, int] | None = None, stream=None, out=None):
    """Screening scores (and optionally penalties and per-slot detail for plans
    [begin, begin+count)).  Returns dict of device tensors."""
    import torch
    dev = plans.perm.device
    P = plans.n_plans
    # outputs start as NaN, so that an entry the library failed to write shows
    score = out if out is not None else torch.full((P,), float("nan"), dtype=torch.float64,
                                                   device=dev)
    pen = torch.full((P,), float("nan"), dtype=torch.float64, device=dev) if penalty else None
    det = None
    res = {"score": score, "penalty": pen}
    if detail is not None:
        b, c = detail
        G = problem.n_groups
        wm = torch.full((G, c), float("nan"), dtype=torch.float32, device=dev)
        ws = torch.full((G, c), float("nan"), dtype=torch.float32, device=dev)
        pr = torch.full((G, c), float("nan"), dtype=torch.float32, device=dev)
        det = Detail(b, c, _ptr(wm), _ptr(ws), _ptr(pr))
        res.update(wait_mean=wm, wait_sd=ws, prob=pr)
    _check(library().qlm_rwt_score(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                   _ptr(score), _ptr(pen),
                                   ctypes.byref(det) if det is not None else None,
                                   _stream(stream)))
    return res


def rwt_score_exact(problem: DeviceProblem, plans: DevicePlans, plan_index, stream=None):
    import torch
    idx = torch.as_tensor(plan_index, dtype=torch.int64).to(plans.perm.device)
    out = torch.full((idx.numel(),), float("nan"), dtype=torch.float64, device=plans.perm.device)
    _check(library().qlm_rwt_score_exact(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                         _ptr(idx), idx.numel(), _ptr(out), _stream(stream)))
    return out


def best_plan_workspace_bytes(problem: DeviceProblem, n_plans: int) -> int:
    return int(library().qlm_best_plan_workspace_bytes(ctypes.byref(problem.struct), n_plans))


def workspace(problem: DeviceProblem, n_plans: int, device="cuda"):
    import torch
    nbytes = best_plan_workspace_bytes(problem, n_plans)
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def best_plan(problem: DeviceProblem, plans: DevicePlans, ws=None, stream=None, out=None):
    """(best_index, best_score) as device tensors of shape [1]."""
    import torch
    dev = plans.perm.device
    if ws is None:
        ws = workspace(problem, plans.n_plans, dev)
    if out is None:
        bi = torch.full((1,), -2, dtype=torch.int64, device=dev)
        bs = torch.full((1,), float("nan"), dtype=torch.float64, device=dev)
    else:
        bi, bs = out
    _check(library().qlm_best_plan(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                   _ptr(ws), ws.numel(), _ptr(bi), _ptr(bs), _stream(stream)))
    return bi, bs


def best_plan_static(problem: DeviceProblem, plans: DevicePlans, stream=None, out=None):
    """qlm_best_plan_static: (best_index, best_score) as device tensors of
    shape [1], with the library's static scratch as the workspace."""
    import torch
    dev = plans.perm.device
    if out is None:
        bi = torch.full((1,), -2, dtype=torch.int64, device=dev)
        bs = torch.full((1,), float("nan"), dtype=torch.float64, device=dev)
    else:
        bi, bs = out
    _check(library().qlm_best_plan_static(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                          _ptr(bi), _ptr(bs), _stream(stream)))
    return bi, bs


def score_form(problem: DeviceProblem, with_eviction: bool, stream=None) -> int:
    """1 when qlm_rwt_score / qlm_best_plan take their fast path for this
    problem, 0 when they take the general exact walk (synchronizes)."""
    import torch
    f = torch.full((1,), -1, dtype=torch.int32, device=problem.grp_count.device)
    _check(library().qlm_score_form(ctypes.byref(problem.struct), int(bool(with_eviction)),
                                    _ptr(f), _stream(stream)))
    return int(f.item())


def validate_plans(problem: DeviceProblem, plans: DevicePlans, stream=None):
    """(n_invalid tensor [1], per-plan status tensor [P])."""
    import torch
    dev = plans.perm.device
    n = torch.empty(1, dtype=torch.int64, device=dev)
    st = torch.empty(max(plans.n_plans, 1), dtype=torch.int32, device=dev)
    _check(library().qlm_validate_plans(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                        _ptr(n), _ptr(st), _stream(stream)))
    return n, st[:plans.n_plans]


def validate_problem(problem: DeviceProblem, stream=None):
    import torch
    n = torch.empty(1, dtype=torch.int64, device=problem.grp_count.device)
    _check(library().qlm_validate_problem(ctypes.byref(problem.struct), _ptr(n), _stream(stream)))
    return n


def max_groups(n_models: int, n_classes: int, n_instances: int, with_eviction: bool) -> int:
    return int(library().qlm_max_groups(n_models, n_classes, n_instances, int(with_eviction)))


def timing_enable(on: bool = True):
    _check(library().qlm_timing_enable(int(on)))


def timing_read():
    """(number of scoring launches, total milliseconds) since the last read."""
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0.0)
    _check(library().qlm_timing_read(ctypes.byref(n), ctypes.byref(ms)))
    return int(n.value), float(ms.value)


# -- plan search --------------------------------------------------------------

def plans_like(plans: DevicePlans, n_groups: int) -> DevicePlans:
    """Output plans shaped like `plans`, always with eviction words (a
    relocation sets flags even in plans that had none)."""
    import torch
    ev = plans.evict_bits
    ev = torch.empty_like(ev) if ev is not None else torch.empty(
        ((n_groups + 31) // 32, plans.perm.shape[1]), dtype=torch.int32, device=plans.perm.device)
    return DevicePlans(torch.empty_like(plans.perm), torch.empty_like(plans.qoff), ev,
                       plans.n_plans)


def search_n_moves(n_groups: int, n_instances: int, window: int) -> int:
    return int(library().qlm_search_n_moves(n_groups, n_instances, window))


def search_workspace_bytes(problem: DeviceProblem, n_plans: int, window: int) -> int:
    return int(library().qlm_search_workspace_bytes(ctypes.byref(problem.struct), n_plans,
                                                    window))


def search_workspace(problem: DeviceProblem, n_plans: int, window: int, device="cuda"):
    import torch
    nbytes = search_workspace_bytes(problem, n_plans, window)
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def search_moves(problem: DeviceProblem, plans: DevicePlans, window: int, ws=None, stream=None,
                 out=None):
    """Exact score of every move of every plan: device tensor [P, n_moves]
    (+inf where a move number names no move)."""
    import torch
    dev = plans.perm.device
    nm = search_n_moves(problem.n_groups, problem.n_instances, window)
    if ws is None:
        ws = search_workspace(problem, plans.n_plans, window, dev)
    if out is None:
        # NaN until written: an entry the library leaves unwritten shows
        out = torch.full((plans.n_plans, nm), float("nan"), dtype=torch.float64, device=dev)
    _check(library().qlm_search_moves(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                      window, _ptr(ws), ws.numel(), _ptr(out), _stream(stream)))
    return out


def search_screen(problem: DeviceProblem, plans: DevicePlans, window: int, ws=None, stream=None):
    """Screened score and its error bound for every move of every plan: two
    device tensors [P, n_moves] (score +inf, bound 0 where a move number names
    no move; bound +inf where the screen cannot bound the move)."""
    import torch
    dev = plans.perm.device
    nm = search_n_moves(problem.n_groups, problem.n_instances, window)
    if ws is None:
        ws = search_workspace(problem, plans.n_plans, window, dev)
    score = torch.full((plans.n_plans, nm), float("nan"), dtype=torch.float64, device=dev)
    bound = torch.full((plans.n_plans, nm), float("nan"), dtype=torch.float64, device=dev)
    _check(library().qlm_search_screen(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                       window, _ptr(ws), ws.numel(), _ptr(score), _ptr(bound),
                                       _stream(stream)))
    return score, bound


def local_search(problem: DeviceProblem, plans: DevicePlans, window: int, max_steps: int,
                 trace: bool = False, ws=None, stream=None, out: DevicePlans | None = None):
    """Steepest-descent search from every plan.  Returns a dict with the final
    plans (a DevicePlans), their exact scores [P] f64, the steps applied [P]
    int32 and, when asked, the trace [P, max_steps] int64."""
    import torch
    dev = plans.perm.device
    P = plans.n_plans
    if ws is None:
        ws = search_workspace(problem, P, window, dev)
    if out is None:
        out = plans_like(plans, problem.n_groups)
    o = PlansOut(int(out.perm.shape[1]), _ptr(out.perm), _ptr(out.qoff), _ptr(out.evict_bits))
    # sentinels until written: NaN scores, -2 steps and moves
    score = torch.full((P,), float("nan"), dtype=torch.float64, device=dev)
    steps = torch.full((P,), -2, dtype=torch.int32, device=dev)
    tr = torch.full((P, max(max_steps, 1)), -2, dtype=torch.int64, device=dev) if trace else None
    _check(library().qlm_local_search(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                      ctypes.byref(o), window, max_steps, _ptr(ws), ws.numel(),
                                      _ptr(score), _ptr(steps), _ptr(tr), _stream(stream)))
    res = {"plans": out, "score": score, "steps": steps}
    if trace:
        res["trace"] = tr[:, :max_steps]
    return res


EDF, GROUPED = 0, 1


def seed_workspace_bytes(problem: DeviceProblem, n_seeds: int) -> int:
    return int(library().qlm_seed_workspace_bytes(ctypes.byref(problem.struct), n_seeds))


def seed_plans(problem: DeviceProblem, policies=(EDF, GROUPED), evict: bool = False, ws=None,
               stream=None, device="cuda"):
    """Seed plans (one per policy: EDF = 0, GROUPED = 1) as a DevicePlans; with
    evict=True the plans carry (cleared) eviction bits."""
    import torch
    n = len(policies)
    G, I = problem.n_groups, problem.n_instances
    perm = torch.empty((G, max(n, 1)), dtype=torch.int32, device=device)
    qoff = torch.empty((I + 1, max(n, 1)), dtype=torch.int32, device=device)
    ev = torch.empty(((G + 31) // 32, max(n, 1)), dtype=torch.int32, device=device) if evict else None
    if ws is None:
        ws = torch.empty(max(seed_workspace_bytes(problem, n), 1), dtype=torch.uint8, device=device)
    pol = (ctypes.c_int32 * max(n, 1))(*policies)
    o = PlansOut(int(perm.shape[1]), _ptr(perm), _ptr(qoff), _ptr(ev))
    _check(library().qlm_seed_plans(ctypes.byref(problem.struct), n, pol, ctypes.byref(o),
                                    _ptr(ws), ws.numel(), _stream(stream)))
    return DevicePlans(perm, qoff, ev, n)


def place_group(problem: DeviceProblem, plans: DevicePlans, group: int, ws=None, stream=None,
                out: DevicePlans | None = None):
    """Every plan with `group` moved to its best place: the EDF position after
    the head of queue c, or (c >= I) the head of queue c - I with its eviction
    flag set; a group at its queue's head stays.  Returns a dict with the
    placed plans (DevicePlans, with eviction words), their exact scores [P] f64
    and the chosen places c [P] int32."""
    import torch
    dev = plans.perm.device
    P = plans.n_plans
    if ws is None:
        ws = search_workspace(problem, P, 0, dev)
    if out is None:
        out = plans_like(plans, problem.n_groups)
    o = PlansOut(int(out.perm.shape[1]), _ptr(out.perm), _ptr(out.qoff), _ptr(out.evict_bits))
    score = torch.full((P,), float("nan"), dtype=torch.float64, device=dev)
    queue = torch.full((P,), -2, dtype=torch.int32, device=dev)
    _check(library().qlm_place_group(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                     ctypes.byref(o), int(group), _ptr(ws), ws.numel(),
                                     _ptr(score), _ptr(queue), _stream(stream)))
    return {"plans": out, "score": score, "queue": queue}


# -- per-request (first come, first served) variant ---------------------------

def device_requests(req_slo, device="cuda"):
    """Per-request SLOs (group by group, each group's in arrival order) as a
    float32 device tensor."""
    import torch
    return torch.as_tensor(np.ascontiguousarray(req_slo, dtype=np.float32)).to(device)


def fcfs_workspace_bytes(problem: DeviceProblem, n_plans: int, n_requests: int,
                         chunk_plans: int = 0) -> int:
    return int(library().qlm_fcfs_workspace_bytes(ctypes.byref(problem.struct), int(n_plans),
                                                  int(n_requests), int(chunk_plans)))


def fcfs_workspace(problem: DeviceProblem, n_plans: int, n_requests: int, device="cuda",
                   chunk_plans: int = 0):
    """A workspace for chunks of chunk_plans plans (0 = the default size)."""
    import torch
    nbytes = fcfs_workspace_bytes(problem, n_plans, n_requests, chunk_plans)
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def fcfs_score(problem: DeviceProblem, plans: DevicePlans, req_slo, ws=None, stream=None,
               out=None):
    """Screened per-request scores of every plan: device tensor [P] f64."""
    import torch
    dev = plans.perm.device
    if ws is None:
        ws = fcfs_workspace(problem, plans.n_plans, req_slo.numel(), dev)
    if out is None:
        out = torch.full((max(plans.n_plans, 1),), float("nan"), dtype=torch.float64, device=dev)
    _check(library().qlm_fcfs_score(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                    _ptr(req_slo), req_slo.numel(), _ptr(ws), ws.numel(),
                                    _ptr(out), _stream(stream)))
    return out[:plans.n_plans]


def fcfs_score_exact(problem: DeviceProblem, plans: DevicePlans, req_slo, plan_index, ws=None,
                     stream=None):
    """Exact per-request scores of the listed plans: device tensor [n] f64."""
    import torch
    dev = plans.perm.device
    idx = torch.as_tensor(plan_index, dtype=torch.int64).to(dev)
    if ws is None:
        ws = fcfs_workspace(problem, plans.n_plans, req_slo.numel(), dev)
    out = torch.full((max(idx.numel(), 1),), float("nan"), dtype=torch.float64, device=dev)
    _check(library().qlm_fcfs_score_exact(ctypes.byref(problem.struct),
                                          ctypes.byref(plans.struct), _ptr(req_slo),
                                          req_slo.numel(), _ptr(idx), idx.numel(), _ptr(ws),
                                          ws.numel(), _ptr(out), _stream(stream)))
    return out[:idx.numel()]


def fcfs_best_plan(problem: DeviceProblem, plans: DevicePlans, req_slo, ws=None, stream=None,
                   out=None):
    """(best_index, best_score) of the per-request score, device tensors [1]."""
    import torch
    dev = plans.perm.device
    if ws is None:
        ws = fcfs_workspace(problem, plans.n_plans, req_slo.numel(), dev)
    if out is None:
        bi = torch.full((1,), -2, dtype=torch.int64, device=dev)
        bs = torch.full((1,), float("nan"), dtype=torch.float64, device=dev)
    else:
        bi, bs = out
    _check(library().qlm_fcfs_best_plan(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                        _ptr(req_slo), req_slo.numel(), _ptr(ws), ws.numel(),
                                        _ptr(bi), _ptr(bs), _stream(stream)))
    return bi, bs


# -- problem tables from a hardware profile -----------------------------------

def apply_profile(problem: DeviceProblem, profile, inst_model=None, req_slo=None, stream=None):
    """The problem with the profile's prefill, drain and throughput folded into
    its SLO, swap and throughput tables (a new DeviceProblem sharing the other
    arrays), and the per-request SLOs less the prefill when req_slo is given.
    ``profile`` maps the qlm_profile field names to arrays (or None)."""
    import copy
    import torch
    dev = problem.grp_count.device
    M, C = problem.n_models, problem.n_classes
    keep = {}
    for f in PROFILE_FIELDS:
        x = profile.get(f)
        keep[f] = None if x is None else torch.as_tensor(
            np.ascontiguousarray(x, dtype=np.float32).reshape(-1)).to(dev)
    sizes = {"prefill": M, "decode_time": C * M, "ineff": C * M, "max_tokens": M,
             "kv_tokens": C * M, "mean_tokens": M}
    for f, x in keep.items():
        if x is not None and x.numel() != sizes[f]:
            raise ValueError(f + " has the wrong size")
    im = None if inst_model is None else torch.as_tensor(
        np.ascontiguousarray(inst_model, dtype=np.int32)).to(dev)
    if im is not None and im.numel() != problem.n_instances:
        raise ValueError("inst_model must have n_instances entries")
    pf = Profile(*[_ptr(keep[f]) for f in PROFILE_FIELDS])
    out = copy.copy(problem)
    out.swap_cost = torch.empty(C * M * M, dtype=torch.float32, device=dev)
    out.grp_slo = torch.empty(problem.n_groups, dtype=torch.float32, device=dev)
    out.inst_tput = torch.empty(problem.n_instances, dtype=torch.float32, device=dev)
    rs = None
    if req_slo is not None:
        rs = torch.empty_like(req_slo)
    _check(library().qlm_apply_profile(ctypes.byref(problem.struct), ctypes.byref(pf), _ptr(im),
                                       _ptr(out.swap_cost), _ptr(out.grp_slo),
                                       _ptr(out.inst_tput), _ptr(req_slo),
                                       0 if req_slo is None else req_slo.numel(), _ptr(rs),
                                       _stream(stream)))
    out._profile_keep = (keep, im)
    out.struct = Problem(out.n_groups, out.n_instances, out.n_models, out.n_classes,
                         _ptr(out.grp_count), _ptr(out.grp_mu), _ptr(out.grp_var),
                         _ptr(out.grp_model), _ptr(out.grp_slo), _ptr(out.inst_tput),
                         _ptr(out.inst_class), _ptr(out.inst_model0), _ptr(out.swap_cost),
                         out.evict_cost)
    return out, rs


class PlaceSession:
    """A placement session (qlm_place_begin / step / end): the plans stay in
    the workspace while groups are placed one after another, on one stream
    (`stream`, or the current stream when the session begins)."""

    def __init__(self, problem: DeviceProblem, plans: DevicePlans, ws=None, stream=None):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream()
        self.problem = problem
        self.n_plans = plans.n_plans
        self.has_evict = plans.evict_bits is not None
        self.like = plans
        self.dev = plans.perm.device
        self.ws = ws if ws is not None else search_workspace(problem, plans.n_plans, 0, self.dev)
        self.stream = stream
        _check(library().qlm_place_begin(ctypes.byref(problem.struct), ctypes.byref(plans.struct),
                                         _ptr(self.ws), self.ws.numel(), _stream(stream)))
        self.score = torch.full((max(self.n_plans, 1),), float("nan"), dtype=torch.float64,
                                device=self.dev)
        self.queue = torch.full((max(self.n_plans, 1),), -2, dtype=torch.int32, device=self.dev)
        # a step's arguments but the group, formed once (a step is a few tens of
        # microseconds of GPU work; marshalling them per call would add as much)
        self._fn = library().qlm_place_step
        self._args = (ctypes.byref(problem.struct), self.n_plans)
        self._rest = (_ptr(self.ws), self.ws.numel(), _ptr(self.score), _ptr(self.queue),
                      _stream(stream))
        self._out = (self.score[:self.n_plans], self.queue[:self.n_plans])

    def step(self, group: int):
        """Places `group` in every plan; returns (scores [P], places [P]) (device)."""
        _check(self._fn(*self._args, int(group), *self._rest))
        return self._out

    def end(self, out: DevicePlans | None = None):
        """The plans as they stand (DevicePlans) and their exact scores."""
        import torch
        if out is None:
            out = plans_like(self.like, self.problem.n_groups)
        o = PlansOut(int(out.perm.shape[1]), _ptr(out.perm), _ptr(out.qoff), _ptr(out.evict_bits))
        score = torch.empty(max(self.n_plans, 1), dtype=torch.float64, device=self.dev)
        _check(library().qlm_place_end(ctypes.byref(self.problem.struct), self.n_plans,
                                       ctypes.byref(o), _ptr(self.ws), self.ws.numel(),
                                       _ptr(score), _stream(self.stream)))
        return out, score[:self.n_plans]
