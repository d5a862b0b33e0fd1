"""Helpers for the GPU tests: device copies of generated or hand-built inputs,
and the tolerances of the parity bar."""
from __future__ import annotations

import numpy as np

# Per-slot tolerances: |dE[W]| <= REL*|E[W]| + ABS_S, same for SD[W]; |dP| <= P_ABS.
REL = 1e-5
ABS_S = 1e-6
P_ABS = 1e-5
# Plan score: |d score| <= SCORE_REL * total requests -- the screening bound
# qlm_best_plan's candidate selection relies on (8e-6 per request).
SCORE_REL = 8e-6
# Exact path vs oracle: both are double precision; only erfc's last bits and
# the order of nothing else differ.
EXACT_REL = 1e-12


def device_inputs(problem, plans):
    from paper_2407_00047_amd import qlm
    return qlm.DeviceProblem(problem), qlm.DevicePlans.from_host(plans)


def assert_close_detail(gpu, ora, G, label=""):
    """gpu: dict of [G] float arrays for one plan; ora: oracle plan_detail."""
    wm, ws, pr = gpu
    e = np.abs(wm.astype(np.float64) - ora["wait_mean"])
    assert np.all(e <= REL * np.abs(ora["wait_mean"]) + ABS_S), (label, e.max())
    e = np.abs(ws.astype(np.float64) - ora["wait_sd"])
    assert np.all(e <= REL * np.abs(ora["wait_sd"]) + ABS_S), (label, e.max())
    e = np.abs(pr.astype(np.float64) - ora["prob"])
    assert np.all(e <= P_ABS), (label, e.max(), int(np.argmax(e)))


def assert_argmin(gi, osc, label=""):
    """The GPU's best plan against the oracle's scores: the oracle's argmin
    (lowest index on ties) -- or, printed as an escape, another plan whose
    oracle score equals the minimum exactly (the device and host erfc differ
    in their last bits, so of plans the oracle ties, the device may order two
    by those bits)."""
    import oracle
    oi, obs = oracle.argmin(osc)
    if gi != oi:
        print("near-tie escape:", label, "gpu", gi, repr(float(osc[gi])), "oracle", oi, repr(obs),
              flush=True)
        assert float(osc[gi]) == obs, (label, gi, oi, float(osc[gi]), obs)
    return oi, obs
