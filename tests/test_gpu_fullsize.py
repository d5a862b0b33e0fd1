"""Full-size parity: every workload at its full plan count, in the launch
configuration bench.py times (qlm_best_plan over the whole batch, and the
screening scores of qlm_rwt_score).

The oracle scores every plan (fp64, all host threads), so the checks are
element by element over the whole batch, not sampled:
  - every screening score within 1e-5 * (total requests) of the oracle's;
  - the chosen plan equal to the oracle's argmin (lowest index on ties), and its
    exact score within 1e-12 relative of the oracle's (both are fp64; only the
    device and host erfc differ, in the last bits);
  - the per-slot waits and probabilities of the first and last tile's plans.
"""
import time

import numpy as np
import pytest

from gpu_util import EXACT_REL, P_ABS, SCORE_REL, assert_close_detail, device_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CONFIGS = ["tiny", "mixed", "hetero", "heavy", "large"]


@pytest.fixture(scope="module")
def qlm():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_00047_amd import qlm as q
    q.library()
    return q


@pytest.mark.parametrize("name", CONFIGS)
def test_full_batch(qlm, orc, name):
    import torch
    from paper_2407_00047_amd import workload
    P = workload.CONFIGS[name]["P"]
    print("case", name, "full size P", P, flush=True)
    pr = workload.make_problem(name)
    pl = workload.make_plans(pr, 0, P)
    dpr, dpl = device_inputs(pr, pl)
    res = qlm.rwt_score(dpr, dpl)
    bi, bs = qlm.best_plan(dpr, dpl)
    b = P - 64 - 5 if P > 128 else 0
    det = qlm.rwt_score(dpr, dpl, detail=(b, min(64 + 5, P)))
    torch.cuda.synchronize()
    sc = res["score"].cpu().numpy()
    best_i, best_s = int(bi.item()), float(bs.item())
    del dpl
    torch.cuda.empty_cache()

    t0 = time.perf_counter()
    osc, _ = orc.score_plans(pr, pl)
    print("oracle: %d plans in %.1f s" % (P, time.perf_counter() - t0), flush=True)
    N = dpr.total_requests
    err = np.abs(sc - osc)
    print("max |d score| / N = %.3e over %d plans" % (err.max() / N, P))
    assert np.all(err <= SCORE_REL * N), (int(np.argmax(err)), err.max())

    oi, obs = orc.argmin(osc)
    print("best plan %d score %.17g (oracle %d %.17g)" % (best_i, best_s, oi, obs))
    assert best_i == oi
    assert abs(best_s - obs) <= EXACT_REL * abs(obs)

    wm = det["wait_mean"].cpu().numpy()
    ws = det["wait_sd"].cpu().numpy()
    pb = det["prob"].cpu().numpy()
    for q in list(range(0, min(5, wm.shape[1]))) + list(range(max(0, wm.shape[1] - 5), wm.shape[1])):
        d = orc.plan_detail(pr, pl, b + q)
        assert_close_detail((wm[:, q], ws[:, q], pb[:, q]), d, pr["n_groups"], (name, b + q))
        assert float(np.abs(pb[:, q] - d["prob"]).max()) <= P_ABS
