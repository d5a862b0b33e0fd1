"""qlm_best_plan_static, the entry point that allocates nothing (its workspace
is the library's static device scratch), against qlm_best_plan with a
caller's workspace, through the C interface: the same best index and score,
bit for bit, both equal to the oracle's argmin (lowest index on ties) and
its score, on calls in a row whose plan counts shrink (the scratch keeps each
call's contents for the next)."""
import numpy as np
import pytest

from gpu_util import EXACT_REL, device_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qlm():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_00047_amd import qlm as q
    q.library()
    return q


@pytest.mark.parametrize("name,sizes", [("hetero", (6000 + 17, 1300 + 3)),
                                        ("large", (2048 + 5, 300 + 1))])
def test_static_scratch_matches_workspace(qlm, orc, name, sizes):
    import torch
    from paper_2407_00047_amd import workload
    pr = workload.make_problem(name)
    for P in sizes:
        print("case", name, "plans", P, flush=True)
        pl = workload.make_plans(pr, 0, P)
        dpr, dpl = device_inputs(pr, pl)
        bi, bs = qlm.best_plan(dpr, dpl)
        si, ss = qlm.best_plan_static(dpr, dpl)
        torch.cuda.synchronize()
        b_i, s_i = int(bi.item()), int(si.item())
        b_s = np.float64(bs.item())
        s_s = np.float64(ss.item())
        assert s_i == b_i, (name, P, s_i, b_i)
        assert s_s.view(np.int64) == b_s.view(np.int64), (name, P, s_s, b_s)
        osc, _ = orc.score_plans(pr, pl)
        oi, obs = orc.argmin(osc)
        assert s_i == oi, (name, P, s_i, oi)
        assert abs(float(s_s) - obs) <= EXACT_REL * abs(obs)
