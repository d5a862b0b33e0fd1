"""Parity of the problem tables derived from a hardware profile
(qlm_apply_profile) with the oracle's, and of the scores computed from them.

  - the derived SLOs, swap table, throughputs and per-request SLOs equal the
    oracle's bit for bit (both form each value in double precision in the same
    order and store it in single precision);
  - the best plan and the per-request best plan of the derived problems equal
    the oracle's on hand-built cases and generated workloads.
"""
import numpy as np
import pytest

from cases import hand_case
from gpu_util import device_inputs

pytestmark = pytest.mark.gpu

EXACT_REL = 1e-12


@pytest.fixture(scope="module")
def qlm():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2407_00047_amd import qlm as q
    q.library()
    return q


def _profile(rng, C, M, drop=()):
    pf = {"prefill": rng.uniform(0.05, 2.0, M), "decode_time": rng.uniform(0.005, 0.05, C * M),
          "ineff": rng.uniform(1.0, 1.7, C * M), "max_tokens": rng.uniform(64, 4096, M),
          "kv_tokens": rng.uniform(2e4, 5e5, C * M), "mean_tokens": rng.uniform(100, 1500, M)}
    pf = {k: v.astype(np.float32) for k, v in pf.items()}
    for k in drop:
        pf[k] = None
    return pf


def _derive(qlm, pr, pf, inst_model, req=None):
    import torch
    dpr = qlm.DeviceProblem(pr)
    dreq = None if req is None else qlm.device_requests(req)
    out, rs = qlm.apply_profile(dpr, pf, inst_model=inst_model, req_slo=dreq)
    torch.cuda.synchronize()
    return out, (None if rs is None else rs.cpu().numpy())


@pytest.mark.parametrize("drop", [(), ("prefill",), ("kv_tokens",), ("max_tokens", "mean_tokens"),
                                  tuple(["prefill", "decode_time", "ineff", "max_tokens",
                                         "kv_tokens", "mean_tokens"])])
def test_tables_bit_exact(qlm, orc, drop):
    rng = np.random.default_rng(len(drop) + 3)
    pr, _ = hand_case(rng, G=37, I=9, M=3, C=2, P=1)
    if "kv_tokens" in drop:
        pr["swap_cost"] = None                 # drain onto an absent swap table
    pf = _profile(rng, 2, 3, drop)
    im = [int(x) for x in rng.integers(-1, 3, 9)]
    N = int(pr["grp_count"].sum())
    req = rng.uniform(0, 100, N).astype(np.float32)
    out, rs = _derive(qlm, pr, pf, im, req)
    want, wrs = orc.apply_profile(pr, pf, inst_model=im, req_slo=req)
    assert np.array_equal(out.swap_cost.cpu().numpy(), want["swap_cost"])
    assert np.array_equal(out.grp_slo.cpu().numpy(), want["grp_slo"])
    assert np.array_equal(out.inst_tput.cpu().numpy(), want["inst_tput"])
    assert np.array_equal(rs, wrs)


def test_no_instance_models(qlm, orc):
    rng = np.random.default_rng(11)
    pr, _ = hand_case(rng, G=20, I=4, M=2, C=2, P=1)
    pf = _profile(rng, 2, 2)
    out, _ = _derive(qlm, pr, pf, None)
    assert np.array_equal(out.inst_tput.cpu().numpy(), pr["inst_tput"])
    want, _ = orc.apply_profile(pr, pf)
    assert np.array_equal(out.swap_cost.cpu().numpy(), want["swap_cost"])


@pytest.mark.parametrize("name,P", [("hetero", 4096), ("heavy", 2048)])
def test_best_plan_with_profile(qlm, orc, name, P):
    """Scores of a generated workload with the profile's terms folded in: the
    best plan and its exact score, and the per-request best plan."""
    import torch
    from paper_2407_00047_amd import workload
    pr = workload.make_problem(name)
    pl = workload.make_plans(pr, 0, P)
    pf = workload.make_profile(pr)
    im = list(range(pr["n_instances"]))
    im = [m % pr["n_models"] for m in im]
    req = workload.make_request_slos(pr)
    out, rs = _derive(qlm, pr, pf, im, req)
    dpl = qlm.DevicePlans.from_host(pl)
    bi, bs = qlm.best_plan(out, dpl)
    torch.cuda.synchronize()
    opr, ors = orc.apply_profile(pr, pf, inst_model=im, req_slo=req)
    oi, os_ = orc.best_plan(opr, pl)
    assert int(bi.item()) == oi and abs(float(bs.item()) - os_) <= EXACT_REL * (abs(os_) + 1)
    # the terms change the answer's score (they are not a no-op here)
    _, plain = orc.best_plan(pr, pl)
    assert plain != os_
    # the per-request variant on the derived SLOs (a sample of the plans)
    sub = {"n_plans": 256, "perm": np.ascontiguousarray(pl["perm"][:, :256]),
           "qoff": np.ascontiguousarray(pl["qoff"][:, :256]),
           "evict_bits": None if pl["evict_bits"] is None
           else np.ascontiguousarray(pl["evict_bits"][:, :256])}
    dsub = qlm.DevicePlans.from_host(sub)
    fi, fs = qlm.fcfs_best_plan(out, dsub, torch.as_tensor(rs).cuda())
    torch.cuda.synchronize()
    oi, os_ = orc.best_plan_fcfs(opr, sub, ors)
    assert int(fi.item()) == oi and abs(float(fs.item()) - os_) <= EXACT_REL * (abs(os_) + 1)
