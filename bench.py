#!/usr/bin/env python3
"""Benchmark: candidate plans scored per second (RWT + SLO-violation
probability + exact argmin) on one MI355X, with the HBM roofline of the
scoring kernel and the fp64 CPU oracle timed beside it.

One step = one qlm_best_plan call over the whole plan batch, inputs already
resident in HBM: stage the tables, stream every plan, gather group statistics,
transitions and costs, running prefix sums, normal tail, per-plan reduction,
then the exact re-score of the screened candidates and the argmin.

Prints one JSON line (the last line of stdout).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "candidate plans scored/sec (RWT + SLO prob) and % of HBM roofline, 1 GPU"
SEARCH_METRIC = "plan-search moves scored/sec (screened + exact best) and % of VALU roofline, 1 GPU"
# MI355X vector issue: 256 CUs x 4 SIMDs, one wave64 VALU instruction per SIMD
# every 4 cycles (16 lanes a cycle) at 2.4 GHz.
PEAK_VALU_LANES = 256 * 4 * 16 * 2.4e9
# VALU instructions per slot in k_score's unrolled 32-slot block (gfx950 code of
# the benchmarked variant, eviction words on; the queue-head path and the
# per-block work excluded); the measured count per slot, those included, comes
# from the committed SQ counter summary when it matches the kernel source
VALU_PER_SLOT = 21
# VALU instructions per visited position in the main loop of the screen of
# moves into another queue (k_fmove), counted in its compiled loop body: margin
# (v_add_f64, v_cvt_f32_f64), variance (v_add_f32), v_rsq_f32, cell coordinate
# (v_fma_f32, v_med3_f32), cell address (v_lshrrev_b32, v_and_b32), the cell's
# line and the weighted sum (two v_fma_f32)
VALU_PER_VISIT = 10


def spin_up(call, seconds):
    """Calls `call` back to back for at least `seconds` (and ten times) before
    the warm-up steps.  Started from idle, the device raises its clock over
    the first tens of milliseconds of sustained load (k_score at large: 1.10,
    0.96, 0.91, 0.90 ms averaged over its first four tens of launches, then
    0.87-0.90 ms): the timed steps are to see the clock it holds under load.
    Returns what the JSON line reports of it."""
    import torch
    n, t0 = 0, time.perf_counter()
    while seconds > 0:
        for _ in range(10):
            call()
        n += 10
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= seconds:
            break
    return {"calls": n, "s": round(time.perf_counter() - t0, 3)}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes_per_plan(problem) -> int:
    """What the method must move per plan: every slot's group id, the queue
    offsets, the eviction bits (when present), and the plan's score."""
    G, I = problem["n_groups"], problem["n_instances"]
    ev = 4 * ((G + 31) // 32) if problem.get("n_evict", 0) > 0 else 0
    return 4 * G + 4 * (I + 1) + ev + 8


def kernel_source_hash() -> str:
    with open(os.path.join(ROOT, "paper_2407_00047_amd", "csrc", "qlm.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(config: str, plans: int):
    """HBM bytes per scoring launch from the committed rocprofv3 counter summary,
    when it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "k_score_%s_traffic.json" % config)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha256") != kernel_source_hash() or t.get("plans") != plans:
        return None
    return float(t["hbm_bytes_per_launch"])


COPY_BYTES = 1 << 30


def copy_calibration():
    """A plain 1 GiB device-to-device copy (three times), for scaling the HBM
    counters: rocprofv3's FETCH_SIZE / WRITE_SIZE of this copy, against its
    known size, give the bytes each counter unit stands for."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "copies": 3}), flush=True)


def _counter_rows(path, counter):
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no counter_collection.csv under %s" % path)
    out = []
    for r in csv.DictReader(open(files[0])):
        if r["Counter_Name"] == counter:
            out.append((r["Kernel_Name"], int(r["Dispatch_Id"]), float(r["Counter_Value"])))
    return out


def summarize_counters(args):
    """Per-launch HBM bytes of the scoring kernel from two rocprofv3 --pmc runs
    of bench.py (FETCH_SIZE, then WRITE_SIZE) and two of --copy-calibration;
    writes profiles/k_score_<config>_traffic.json and prints a summary."""
    fetch_dir, write_dir, cfetch_dir, cwrite_dir = args.summarize_counters

    def per_dispatch(rows, pred):
        vals = {}
        for name, d, v in rows:
            if pred(name):
                vals[d] = vals.get(d, 0.0) + v
        return list(vals.values())

    def is_score(n):
        return "k_score" in n

    def is_copy(n):
        return "copy" in n.lower()

    kf = per_dispatch(_counter_rows(fetch_dir, "FETCH_SIZE"), is_score)
    kw = per_dispatch(_counter_rows(write_dir, "WRITE_SIZE"), is_score)
    cf = per_dispatch(_counter_rows(cfetch_dir, "FETCH_SIZE"), is_copy)
    cw = per_dispatch(_counter_rows(cwrite_dir, "WRITE_SIZE"), is_copy)
    if not (kf and kw and cf and cw):
        raise SystemExit("missing dispatches: k_score %d/%d, copy %d/%d" % (len(kf), len(kw), len(cf), len(cw)))
    # counters are in KiB per dispatch; the largest copy dispatches are the 1 GiB copies
    cf_k, cw_k = max(cf), max(cw)
    f_scale = COPY_BYTES / (cf_k * 1024.0)
    w_scale = COPY_BYTES / (cw_k * 1024.0)
    kf_avg = sum(kf) / len(kf)
    kw_avg = sum(kw) / len(kw)
    fetch_b = kf_avg * 1024.0 * f_scale
    write_b = kw_avg * 1024.0 * w_scale
    from paper_2407_00047_amd import workload
    cfg = workload.CONFIGS[args.config]
    P = cfg["P"] if args.plans is None else args.plans
    pr = workload.make_problem(args.config)
    alg = algorithmic_bytes_per_plan(pr) * P
    out = {"config": args.config, "plans": P, "source_sha256": kernel_source_hash(),
           "fetch_kib_per_launch": kf_avg, "write_kib_per_launch": kw_avg,
           "copy_fetch_kib": cf_k, "copy_write_kib": cw_k,
           "fetch_scale": f_scale, "write_scale": w_scale,
           "hbm_bytes_per_launch": fetch_b + write_b,
           "algorithmic_bytes_per_launch": alg,
           "traffic_over_algorithmic": (fetch_b + write_b) / alg}
    path = os.path.join(ROOT, "profiles", "k_score_%s_traffic.json" % args.config)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


def summarize_sq(args):
    """SQ and read-request counters of the scoring kernel from rocprofv3 --pmc
    runs of bench.py (SQ_WAVES, SQ_INSTS_VALU, ...; and TCC_EA0_RDREQ_*_sum
    of bench.py and of --copy-calibration): VALU instructions per slot, LDS
    conflict cycles per slot, and the HBM read bytes from the request counts
    (32, 64 and 128-byte requests) against the copy's known size.  Writes
    profiles/k_score_<config>_counters.json and prints it."""
    sq_dir, rd_dir, crd_dir = args.summarize_sq
    from paper_2407_00047_amd import workload
    cfg = workload.CONFIGS[args.config]
    P = cfg["P"] if args.plans is None else args.plans
    pr = workload.make_problem(args.config)

    def avg(path, counter, pred):
        vals = {}
        for name, d, v in _counter_rows(path, counter):
            if pred(name):
                vals[d] = vals.get(d, 0.0) + v
        return sum(vals.values()) / len(vals) if vals else None

    def is_score(n):
        return "k_score" in n

    def is_copy(n):
        return "copy" in n.lower()

    out = {"config": args.config, "plans": P, "source_sha256": kernel_source_hash()}
    names = ("SQ_WAVES", "SQ_INSTS_VALU", "SQ_ACTIVE_INST_VALU", "SQ_INSTS_LDS",
             "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_WAVE_CYCLES", "GRBM_GUI_ACTIVE")
    for c in names:
        out[c] = avg(sq_dir, c, is_score)
    wave_slots = P * pr["n_groups"] / 64.0          # one wave instruction covers 64 plans
    out["valu_per_slot"] = out["SQ_INSTS_VALU"] / wave_slots
    out["lds_insts_per_slot"] = out["SQ_INSTS_LDS"] / wave_slots
    out["lds_conflict_cycles_per_slot"] = out["SQ_LDS_BANK_CONFLICT"] / wave_slots
    reqs = ("TCC_EA0_RDREQ_sum", "TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum",
            "TCC_EA0_RDREQ_128B_sum")

    def read_bytes(path, pred):
        v = {c: avg(path, c, pred) for c in reqs}
        v["bytes"] = (32.0 * v["TCC_EA0_RDREQ_32B_sum"] + 64.0 * v["TCC_EA0_RDREQ_64B_sum"] +
                      128.0 * v["TCC_EA0_RDREQ_128B_sum"])
        return v

    def max_copy(path):
        vals = {}
        for c in reqs:
            for name, d, val in _counter_rows(path, c):
                if is_copy(name):
                    vals.setdefault(d, {})[c] = vals.get(d, {}).get(c, 0.0) + val
        best = max(vals.values(), key=lambda x: x["TCC_EA0_RDREQ_sum"])
        best["bytes"] = (32.0 * best["TCC_EA0_RDREQ_32B_sum"] + 64.0 * best["TCC_EA0_RDREQ_64B_sum"] +
                         128.0 * best["TCC_EA0_RDREQ_128B_sum"])
        return best

    k = read_bytes(rd_dir, is_score)
    c = max_copy(crd_dir)
    alg = algorithmic_bytes_per_plan(pr) * P
    out["read_requests"] = k
    out["copy_read_requests"] = c
    out["copy_read_bytes_over_size"] = c["bytes"] / COPY_BYTES
    out["read_bytes_per_launch"] = k["bytes"]
    out["read_bytes_over_algorithmic_reads"] = k["bytes"] / (alg - 8 * P)
    path = os.path.join(ROOT, "profiles", "k_score_%s_counters.json" % args.config)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


def cpu_baseline(problem, plans, seconds: float, threads: int = 0):
    """The oracle on a prefix of the same batch, sized to about `seconds` of
    work: all host threads (threads=0) or the given count."""
    import oracle
    orc = oracle.default()
    P = plans["n_plans"]
    used = orc.max_threads() if threads <= 0 else threads
    n0 = min(P, max(16, 4 * used))
    t0 = time.perf_counter()
    orc.score_plans(problem, plans, 0, n0, threads=threads)
    dt = max(time.perf_counter() - t0, 1e-6)
    count = int(min(P, max(n0, seconds * n0 / dt)))
    t0 = time.perf_counter()
    orc.score_plans(problem, plans, 0, count, threads=threads)
    dt = time.perf_counter() - t0
    N = sum(int(x) for x in problem["grp_count"])
    return {"value": count / dt, "unit": "plans/s", "requests_per_s": count * N / dt,
            "cores": used, "kind": "oracle",
            "sample": "plans 0..%d of the same batch (%d of %d), %d host thread%s, fp64 C oracle,"
                      " %.1f s" % (count - 1, count, P, used, "" if used == 1 else "s", dt)}


def measured_counters(config: str, plans: int):
    """SQ counter summary of the scoring kernel (VALU instructions per slot and
    the like) when it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "k_score_%s_counters.json" % config)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha256") != kernel_source_hash() or t.get("plans") != plans:
        return None
    return t


def move_counts(problem, plans, p, window):
    """Valid moves of plan p by kind (swaps within a queue, reassignments,
    relocations to a queue's head) and the positions the screen of moves into
    another queue (k_fmove) visits for them: for a group moving to queue h,
    itself at its insertion point after h's head and every position of h from
    there on (one position when it goes to the end or into an empty queue);
    for a group relocated to the head of another queue h, itself and every
    position of h; for a group relocated to the head of its own queue, every
    position of it.  A queue's head (its running group) takes part in no
    move."""
    import numpy as np
    G, I = problem["n_groups"], problem["n_instances"]
    perm = plans["perm"][:, p]
    qoff = plans["qoff"][:, p]
    slo = np.asarray(problem["grp_slo"], np.float32)
    lens = np.diff(qoff)
    swaps = int(sum(max(int(L) - 1 - d, 0) for L in lens for d in range(1, window + 1)))
    busy = int(np.sum(lens > 0))
    movable = G - busy
    moves = movable * (I - 1)
    relocations = movable * busy
    owner = np.repeat(np.arange(I), lens)
    g_of = np.empty(G, np.int64)
    g_of[perm] = owner
    head = np.zeros(G, bool)
    head[perm[qoff[:-1][lens > 0]]] = True
    visits = 0
    for h in range(I):
        b, e = int(qoff[h]), int(qoff[h + 1])
        x = slo[(g_of != h) & ~head]
        if e == b:
            visits += x.size
            continue
        L = e - b
        pmax = np.maximum.accumulate(slo[perm[b + 1:e]]) if L > 1 else np.zeros(0, np.float32)
        pos = 1 + np.searchsorted(pmax, x, side="right")       # first later SLO after the head
        visits += int(np.sum(np.where(pos == L, 1, L - pos + 1)))
        visits += int(x.size) * (L + 1)                        # relocations to its head
        visits += (L - 1) * L                                  # relocations within h
    return {"valid": swaps + moves + relocations, "swaps": swaps, "moves": moves,
            "relocations": relocations, "visits": visits}


def cpu_search_baseline(problem, plans, window, seconds: float):
    import numpy as np
    import oracle
    orc = oracle.default()
    ms = np.arange(orc.n_moves(problem["n_groups"], problem["n_instances"], window))
    rng = np.random.default_rng(0)
    n0 = 64
    t0 = time.perf_counter()
    orc.move_scores(problem, plans, 0, window, ks=rng.choice(ms, n0, replace=False))
    dt = max(time.perf_counter() - t0, 1e-6)
    n = int(min(ms.size, max(n0, seconds * n0 / dt)))
    ks = rng.choice(ms, n, replace=False)
    t0 = time.perf_counter()
    sc = orc.move_scores(problem, plans, 0, window, ks=ks)
    dt = time.perf_counter() - t0
    valid = int(np.sum(np.isfinite(sc)))
    return {"value": valid / dt, "unit": "moves/s", "cores": orc.max_threads(), "kind": "oracle",
            "sample": "%d move numbers drawn at random from plan 0's neighbourhood (%d valid "
                      "moves), each moved plan built and scored from scratch by the fp64 C oracle, "
                      "all host threads, %.1f s" % (n, valid, dt)}


def bench_search(args):
    """One step = one step of the local search on every chain: cache the plan,
    screen every move (removals, swaps, reassignments, relocations), re-score
    exactly the moves that can still be the best, pick and apply."""
    import numpy as np
    import torch
    from paper_2407_00047_amd import qlm, workload
    dev = torch.device("cuda:0")
    B, W, K = args.chains, args.window, args.steps
    pr = workload.make_problem(args.config)
    pl = workload.make_plans(pr, 0, B)
    G, I = pr["n_groups"], pr["n_instances"]
    dpr = qlm.DeviceProblem(pr, device=dev)
    dpl = qlm.DevicePlans.from_host(pl, device=dev)
    ws = qlm.search_workspace(dpr, B, W, device=dev)
    nm = qlm.search_n_moves(G, I, W)
    counts = [move_counts(pr, pl, p, W) for p in range(B)]
    valid = sum(c["valid"] for c in counts)
    visits = sum(c["visits"] for c in counts)
    kinds = {k: sum(c[k] for c in counts) // B for k in ("swaps", "moves", "relocations")}
    log("search %s: G=%d I=%d chains=%d window=%d, %d valid moves per step %s" % (
        args.config, G, I, B, W, valid, kinds))
    out = qlm.plans_like(dpl, G)
    spin = spin_up(lambda: qlm.local_search(dpr, dpl, W, K, ws=ws, out=out), args.spinup)
    for _ in range(max(args.warmup, 1)):
        r = qlm.local_search(dpr, dpl, W, K, ws=ws, out=out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    qlm.timing_enable(True)
    qlm.timing_read()
    e0.record(stream)
    r = qlm.local_search(dpr, dpl, W, K, ws=ws, out=out)
    e1.record(stream)
    torch.cuda.synchronize()
    n_search, ms_search = qlm.timing_read()
    total_ms = e0.elapsed_time(e1)
    steps = r["steps"].cpu().numpy()
    applied = int(steps.sum())
    # the same search again, untimed, for the kinds of the moves it applied
    tr = qlm.local_search(dpr, dpl, W, K, trace=True, ws=ws, out=out)["trace"].cpu().numpy()
    relocs = int(np.sum(tr >= G * W + G * I))
    # the reassignment screen on the start plans (the positions it visits are
    # known exactly there), timed over repeated launches
    reps = 10
    qlm.search_screen(dpr, dpl, W, ws=ws)
    torch.cuda.synchronize()
    qlm.timing_read()
    for _ in range(reps):
        qlm.search_screen(dpr, dpl, W, ws=ws)
    torch.cuda.synchronize()
    n_launch, k_ms = qlm.timing_read()
    qlm.timing_enable(False)
    k_avg = k_ms / max(n_launch, 1)
    achieved = visits / (k_avg / 1e3) / 1e9
    peak = PEAK_VALU_LANES / VALU_PER_VISIT / 1e9
    roofline = {"bound": "alu", "achieved": round(achieved, 1), "peak": round(peak, 1),
                "unit": "Gvisits/s", "frac": round(achieved / peak, 4), "traffic": None,
                "kernel": "k_fmove", "kernel_avg_ms": round(k_avg, 4),
                "kernel_avg_ms_in_search": round(ms_search / max(n_search, 1), 4),
                "visits_per_launch": visits, "valu_per_visit": VALU_PER_VISIT}
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        cpu = cpu_search_baseline(pr, pl, W, args.cpu_seconds)
    ms_step = total_ms / K
    N = workload.total_requests(pr)
    res = {
        "metric": SEARCH_METRIC, "value": round(valid * K / (total_ms / 1e3), 1),
        "unit": "moves/s", "n_gpus": 1, "steps": K, "warmup": args.warmup, "spinup": spin,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32+f64", "data": "synthetic",
        "config": {"workload": "plan search on %s: %d groups (%d requests), %d instances, "
                               "%d start plans, window %d, %d valid moves per plan and step "
                               "(%d swaps, %d reassignments, %d relocations)"
                               % (args.config, G, N, I, B, W, valid // B, kinds["swaps"],
                                  kinds["moves"], kinds["relocations"]),
                   "chains": B, "window": W, "groups": G, "instances": I,
                   "moves_per_step": valid, "moves_per_plan_by_kind": kinds},
        "moves_applied": applied,
        "relocations_applied": relocs,
        "score_start_to_end": [float(x) for x in r["score"].cpu().numpy()[:4]],
        "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


FCFS_METRIC = "plans scored per second, per-request FCFS variant (exact argmin), 1 GPU"
FCFS_PLANS = 16384
# VALU instructions per request in k_fbscreen's unrolled loop (compiled code):
# margin (v_add_f64, v_fmac_f64, v_cvt_f32_f64), variance (v_fmamk_f32),
# v_rsq_f32, cell coordinate (v_fma_f32, v_med3_f32), cell address
# (v_lshrrev_b32, v_and_b32), the line (v_fmac_f32), the sum (v_add_f32)
VALU_PER_REQUEST = 11


def cpu_fcfs_baseline(problem, plans, req, seconds: float):
    import oracle
    orc = oracle.default()
    threads = orc.max_threads()
    P = plans["n_plans"]
    n, dt, t0 = 0, 0.0, time.perf_counter()
    while n < P and (n == 0 or dt < seconds):
        c = min(threads, P - n)
        orc.score_plans_fcfs(problem, plans, req, n, c)
        n += c
        dt = time.perf_counter() - t0
    N = int(req.size)
    return {"value": n / dt, "unit": "plans/s", "requests_per_s": n * N / dt, "cores": threads,
            "kind": "oracle",
            "sample": "the first %d plans of the same batch, exact fp64 per-request scores by the "
                      "C oracle on %d threads, %.1f s" % (n, threads, dt)}


def bench_fcfs(args):
    """One step = qlm_fcfs_best_plan over the batch: every plan screened (each
    group's start once per plan, each request's tail), the plans within the
    bound re-scored exactly, the lowest exact score."""
    import torch
    from paper_2407_00047_amd import qlm, workload
    dev = torch.device("cuda:0")
    K = args.steps
    P = args.plans or FCFS_PLANS
    pr = workload.make_problem(args.config)
    pl = workload.make_plans(pr, 0, P)
    req = workload.make_request_slos(pr)
    G, I, N = pr["n_groups"], pr["n_instances"], int(req.size)
    dpr = qlm.DeviceProblem(pr, device=dev)
    dpl = qlm.DevicePlans.from_host(pl, device=dev)
    dreq = qlm.device_requests(req, device=dev)
    ws = qlm.fcfs_workspace(dpr, P, N, device=dev, chunk_plans=args.chunk)
    log("fcfs %s: G=%d I=%d requests=%d plans=%d chunk=%d" % (args.config, G, I, N, P, args.chunk))
    spin = spin_up(lambda: qlm.fcfs_best_plan(dpr, dpl, dreq, ws=ws), args.spinup)
    for _ in range(max(args.warmup, 1)):
        bi, bs = qlm.fcfs_best_plan(dpr, dpl, dreq, ws=ws)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    qlm.timing_enable(True)
    qlm.timing_read()
    e0.record(stream)
    for _ in range(K):
        bi, bs = qlm.fcfs_best_plan(dpr, dpl, dreq, ws=ws, out=(bi, bs))
    e1.record(stream)
    torch.cuda.synchronize()
    n_launch, k_ms = qlm.timing_read()
    qlm.timing_enable(False)
    ms = e0.elapsed_time(e1) / K
    k_avg = k_ms / max(n_launch, 1)
    per_launch = N * P * K / max(n_launch, 1)          # requests screened per launch
    achieved = per_launch / (k_avg / 1e3) / 1e9
    peak = PEAK_VALU_LANES / VALU_PER_REQUEST / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        cpu = cpu_fcfs_baseline(pr, pl, req, args.cpu_seconds)
    res = {
        "metric": FCFS_METRIC, "value": round(P / (ms / 1e3), 1), "unit": "plans/s",
        "requests_per_s": round(P * N / (ms / 1e3), 1),
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "spinup": spin, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32+f64",
        "data": "synthetic",
        "config": {"workload": "per-request FCFS scoring on %s: %d groups, %d requests (each with "
                               "its own SLO), %d instances, %d plans" % (args.config, G, N, I, P),
                   "plans": P, "groups": G, "requests": N, "instances": I},
        "best": [int(bi.item()), float(bs.item())],
        "roofline": {"bound": "alu", "achieved": round(achieved, 1), "peak": round(peak, 1),
                     "unit": "Grequests/s", "frac": round(achieved / peak, 4), "traffic": None,
                     "kernel": "k_fbscreen", "kernel_avg_ms": round(k_avg, 4),
                     "requests_per_launch": int(per_launch),
                     "valu_per_request": VALU_PER_REQUEST},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


PLACE_METRIC = "group placements per second (arrival / violation re-score, exact), 1 GPU"


def cpu_place_baseline(problem, plans, groups, seconds: float):
    import oracle
    orc = oracle.default()
    G = problem["n_groups"]
    t0 = time.perf_counter()
    n = 0
    while n == 0 or time.perf_counter() - t0 < seconds:
        orc.place_group(problem, plans, 0, groups[n % len(groups)] % G)
        n += 1
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "updates/s", "cores": 1, "kind": "oracle",
            "sample": "%d placements of the timed groups into plan 0 of the same batch, each "
                      "candidate plan built and scored from scratch by the fp64 C oracle (one "
                      "thread), %.1f s" % (n, dt)}


def bench_place(args):
    """One update = one qlm_place_step of a placement session on every plan:
    the group scored exactly in every queue, the best placement applied, the
    cache of the changed queues formed again (the plans stay in the
    workspace).  The single-call form (qlm_place_group: load, place, write
    back) is timed beside it."""
    import torch
    from paper_2407_00047_amd import qlm, workload
    dev = torch.device("cuda:0")
    B, K = args.chains, args.steps
    pr = workload.make_problem(args.config)
    pl = workload.make_plans(pr, 0, B)
    G, I = pr["n_groups"], pr["n_instances"]
    dpr = qlm.DeviceProblem(pr, device=dev)
    dpl = qlm.DevicePlans.from_host(pl, device=dev)
    ws = qlm.search_workspace(dpr, B, 0, device=dev)
    groups = [(g * 7919) % G for g in range(K + args.warmup + 1)]
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    # the session
    ses = qlm.PlaceSession(dpr, dpl, ws=ws)
    for g in groups[:max(args.warmup, 1)]:
        ses.step(g)
    torch.cuda.synchronize()
    e0.record(stream)
    for g in groups[max(args.warmup, 1):max(args.warmup, 1) + K]:
        ses.step(g)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / K
    # the candidate kernel's own duration, in further steps (the events the
    # library then records around it are kept out of the timed steps above)
    qlm.timing_enable(True)
    qlm.timing_read()
    for g in groups[:K]:
        ses.step(g)
    torch.cuda.synchronize()
    n_launch, k_ms = qlm.timing_read()
    qlm.timing_enable(False)
    ses.end()
    # the single call, for comparison
    K1 = min(K, 20)
    qlm.place_group(dpr, dpl, groups[0], ws=ws)
    torch.cuda.synchronize()
    e0.record(stream)
    for g in groups[:K1]:
        qlm.place_group(dpr, dpl, g, ws=ws)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_call = e0.elapsed_time(e1) / K1
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        cpu = cpu_place_baseline(pr, pl, groups, args.cpu_seconds)
    N = workload.total_requests(pr)
    res = {
        "metric": PLACE_METRIC, "value": round(B / (ms / 1e3), 1), "unit": "updates/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "us_per_update": round(1e3 * ms, 2), "us_per_call_with_load": round(1e3 * ms_call, 2),
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "placement session, one group per update in %d plan(s) of %s: %d "
                               "groups (%d requests), %d instances" % (B, args.config, G, N, I),
                   "plans": B, "groups": G, "instances": I},
        "candidate_kernel_avg_ms": round(k_ms / max(n_launch, 1), 4),
        "roofline": {"bound": "latency", "achieved": round(1e3 * ms, 2), "peak": None,
                     "unit": "us/update", "frac": None, "traffic": None,
                     "kernel": "k_place_eval",
                     "note": "a chain of dependent launches; the latency, not a rate, bounds it"},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--spinup", type=float, default=0.15,
                    help="seconds of back-to-back calls before the warm-up steps (0: none)")
    ap.add_argument("--config", default="large",
                    help="workload: tiny, mixed, hetero, heavy, large (default)")
    ap.add_argument("--plans", type=int, default=None, help="override the plan count")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--all-configs", action="store_true",
                    help="best-plan benchmark of every workload in turn, one JSON line each "
                         "(large last)")
    ap.add_argument("--clock-check", action="store_true",
                    help="time the scoring kernel from a cold start (every ten launches) and "
                         "after idle gaps (the clock's ramp), print one JSON line and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 1 GiB device copy (for HBM counter scaling) and exit")
    ap.add_argument("--search", action="store_true",
                    help="benchmark the plan search (local search steps) instead")
    ap.add_argument("--place", action="store_true",
                    help="benchmark the placement of one group (arrival re-score) instead")
    ap.add_argument("--fcfs", action="store_true",
                    help="benchmark the per-request FCFS variant instead")
    ap.add_argument("--chunk", type=int, default=0,
                    help="--fcfs: plans per screening chunk (0 = the library's default)")
    ap.add_argument("--with-profile", action="store_true",
                    help="fold a synthetic hardware profile (prefill, drain, throughput) into "
                         "the problem tables first")
    ap.add_argument("--chains", type=int, default=1, help="--search / --place: plans")
    ap.add_argument("--window", type=int, default=16, help="--search: swap window")
    ap.add_argument("--summarize-counters", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="rocprofv3 --pmc output folders: write the traffic summary and exit")
    ap.add_argument("--summarize-sq", nargs=3, metavar=("SQ", "READS", "COPY_READS"),
                    help="rocprofv3 --pmc output folders (SQ counters of bench.py, read requests "
                         "of bench.py and of --copy-calibration): write the counter summary and exit")
    args = ap.parse_args()

    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.summarize_sq:
        summarize_sq(args)
        return

    if args.gpus != 1:
        print("bench.py: this build scores plans on one GPU; --gpus %d is not supported "
              "(plans shard across GPUs by range, see the design notes)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2407_00047_amd import qlm, workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration()
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    qlm.library()
    if args.search:
        bench_search(args)
        return
    if args.place:
        bench_place(args)
        return
    if args.fcfs:
        bench_fcfs(args)
        return

    if args.clock_check:
        bench_clock(args, args.config, dev)
        return
    if args.all_configs:
        for name in ("tiny", "mixed", "hetero", "heavy", "large"):
            bench_best(args, name, dev)
        return
    bench_best(args, args.config, dev)


def bench_clock(args, config, dev):
    """k_score's launch time as the device warms up: qlm_best_plan called back
    to back from the start (the average of each ten launches; the first ten
    include the first launch), then with the device idle 5 ms before each
    call.  Started from idle, the device raises its clock over the first tens
    of milliseconds of sustained load and lowers it again in idle gaps; the
    benchmark's spin-up (`--spinup`) is for that.  Prints one JSON line."""
    import statistics

    import torch

    from paper_2407_00047_amd import qlm, workload

    cfg = workload.CONFIGS[config]
    P = cfg["P"] if args.plans is None else args.plans
    pr = workload.make_problem(config)
    pl = workload.make_plans(pr, 0, P)
    dpr = qlm.DeviceProblem(pr, device=dev)
    dpl = qlm.DevicePlans.from_host(pl, device=dev)
    ws = qlm.workspace(dpr, P, device=dev)
    bi = torch.empty(1, dtype=torch.int64, device=dev)
    bs = torch.empty(1, dtype=torch.float64, device=dev)
    torch.cuda.synchronize()
    ramp = []
    qlm.timing_enable(True)
    qlm.timing_read()
    for _ in range(30):
        for _ in range(10):
            qlm.best_plan(dpr, dpl, ws=ws, out=(bi, bs))
        torch.cuda.synchronize()
        n, ms = qlm.timing_read()
        ramp.append(round(ms / max(n, 1), 4))
    for _ in range(args.steps):
        torch.cuda.synchronize()
        time.sleep(0.005)
        qlm.best_plan(dpr, dpl, ws=ws, out=(bi, bs))
    torch.cuda.synchronize()
    n, ms = qlm.timing_read()
    qlm.timing_enable(False)
    after_idle = ms / max(n, 1)
    steady = statistics.median(ramp[-10:])
    bpp = algorithmic_bytes_per_plan(pr)
    frac = lambda t: round(bpp * P / (t / 1e3) / 1e9 / PEAK_HBM_GBS, 4)
    print(json.dumps({"kernel": "k_score", "config": config, "plans": P,
                      "ramp_ms_per_10_launches": ramp, "steady_ms": round(steady, 4),
                      "after_idle_ms": round(after_idle, 4), "idle_gap_ms": 5.0,
                      "after_idle_launches": args.steps,
                      "frac_first_10": frac(ramp[0]), "frac_steady": frac(steady),
                      "frac_after_idle": frac(after_idle)}), flush=True)


def bench_best(args, config, dev):
    """One step = one qlm_best_plan over the whole batch of `config`; prints
    its JSON line."""
    import torch

    from paper_2407_00047_amd import qlm, workload

    cfg = workload.CONFIGS[config]
    P = cfg["P"] if args.plans is None else args.plans
    t0 = time.perf_counter()
    pr = workload.make_problem(config)
    pl = workload.make_plans(pr, 0, P)
    log("generated %s: G=%d I=%d P=%d in %.1f s" % (config, pr["n_groups"],
                                                     pr["n_instances"], P,
                                                     time.perf_counter() - t0))
    dpr = qlm.DeviceProblem(pr, device=dev)
    profile_ms = None
    if args.with_profile:
        # the estimator's prefill, drain and throughput terms folded into the
        # tables (instance g profiled for model g mod M); timed once
        pf = workload.make_profile(pr)
        im = [g % pr["n_models"] for g in range(pr["n_instances"])]
        p0 = torch.cuda.Event(enable_timing=True)
        p1 = torch.cuda.Event(enable_timing=True)
        qlm.apply_profile(dpr, pf, inst_model=im)
        torch.cuda.synchronize()
        p0.record()
        dpr, _ = qlm.apply_profile(dpr, pf, inst_model=im)
        p1.record()
        torch.cuda.synchronize()
        profile_ms = p0.elapsed_time(p1)
        if not args.no_cpu_baseline:
            import oracle
            pr = oracle.apply_profile(pr, pf, inst_model=im)[0]
    dpl = qlm.DevicePlans.from_host(pl, device=dev)
    ws = qlm.workspace(dpr, P, device=dev)
    bi = torch.empty(1, dtype=torch.int64, device=dev)
    bs = torch.empty(1, dtype=torch.float64, device=dev)
    torch.cuda.synchronize()

    spin = spin_up(lambda: qlm.best_plan(dpr, dpl, ws=ws, out=(bi, bs)), args.spinup)
    for _ in range(args.warmup):
        qlm.best_plan(dpr, dpl, ws=ws, out=(bi, bs))
    torch.cuda.synchronize()

    qlm.timing_enable(True)
    qlm.timing_read()                      # reset
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    e0.record(stream)
    ev[0].record(stream)
    for k in range(args.steps):
        qlm.best_plan(dpr, dpl, ws=ws, out=(bi, bs))
        ev[k + 1].record(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    step_ms = sorted(ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps))
    qlm.timing_enable(False)
    n_launch, k_ms = qlm.timing_read()
    total_ms = e0.elapsed_time(e1)
    ms_step = total_ms / args.steps
    plans_per_s = P / (ms_step / 1e3)
    best_index = int(bi.item())
    best_score = float(bs.item())

    bpp = algorithmic_bytes_per_plan(pr)
    k_avg_ms = k_ms / max(n_launch, 1)
    achieved = bpp * P / (k_avg_ms / 1e3) / 1e9
    traffic = measured_traffic(config, P)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": traffic, "kernel": "k_score", "kernel_avg_ms": round(k_avg_ms, 4),
                "algorithmic_bytes_per_launch": bpp * P}
    # the same kernel against its VALU issue bound (slot visits per second):
    # one wave64 instruction per SIMD every 4 cycles, at the measured VALU
    # count per slot when the counter summary matches the source, else the
    # unrolled block's count
    slots = P * pr["n_groups"]
    ctr = measured_counters(config, P)
    vps = float(ctr["valu_per_slot"]) if ctr else float(VALU_PER_SLOT)
    s_achieved = slots / (k_avg_ms / 1e3) / 1e9
    s_peak = PEAK_VALU_LANES / vps / 1e9
    valu_issue = {"bound": "alu", "achieved": round(s_achieved, 1), "peak": round(s_peak, 1),
                  "unit": "Gslots/s", "frac": round(s_achieved / s_peak, 4), "kernel": "k_score",
                  "slots_per_launch": slots, "valu_per_slot": round(vps, 2),
                  "valu_per_slot_from": "SQ counters" if ctr else "unrolled block"}

    # context, outside the timed steps: the same kernel launched after the
    # device has idled 5 ms (the clock it holds then, against the sustained
    # clock of the timed steps)
    idle_ms = []
    for _ in range(5):
        torch.cuda.synchronize()
        time.sleep(0.005)
        qlm.timing_enable(True)
        qlm.timing_read()
        qlm.best_plan(dpr, dpl, ws=ws, out=(bi, bs))
        torch.cuda.synchronize()
        n_i, ms_i = qlm.timing_read()
        qlm.timing_enable(False)
        idle_ms.append(ms_i / max(n_i, 1))
    idle_ms = sorted(idle_ms)[len(idle_ms) // 2]
    roofline["after_idle"] = {"kernel_ms": round(idle_ms, 4),
                              "frac": round(bpp * P / (idle_ms / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
                              "note": "median of 5 launches each after 5 ms idle; not the timed steps"}

    cpu = cpu1 = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (all host threads, then one) ...")
        cpu = cpu_baseline(pr, pl, args.cpu_seconds)
        cpu1 = cpu_baseline(pr, pl, args.cpu_seconds, threads=1)

    N = workload.total_requests(pr)
    out = {
        "metric": METRIC, "value": round(plans_per_s, 1), "unit": "plans/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "spinup": spin,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_median": round(step_ms[len(step_ms) // 2], 4),
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32+f64", "data": "synthetic",
        "config": {"workload": "%s: %d groups (%d requests), %d instances in %d classes, "
                               "%d models, %d plans" % (config, pr["n_groups"], N,
                                                        pr["n_instances"], pr["n_classes"],
                                                        pr["n_models"], P),
                   "plans": P, "groups": pr["n_groups"], "instances": pr["n_instances"],
                   "requests": N},
        "requests_per_s": round(plans_per_s * N, 1),
        "best_index": best_index, "best_score": best_score,
        "roofline": roofline, "valu_issue": valu_issue, "cpu_baseline": cpu,
        "cpu_baseline_1core": cpu1,
    }
    if args.with_profile:
        out["config"]["workload"] += ", tables from a hardware profile"
        out["profile_ms"] = round(profile_ms, 4)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
