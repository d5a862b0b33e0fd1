"""The C interface without a GPU: the library loads, exports every function
include/qlm.h declares, and its host-side argument checks reject bad calls
before anything reaches the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qlm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(qlm_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    from paper_2407_00047_amd import qlm
    return qlm.library()


def test_header_declares_entry_points():
    names = declared_functions()
    for must in ("qlm_rwt_score", "qlm_best_plan", "qlm_best_plan_workspace_bytes",
                 "qlm_rwt_score_exact", "qlm_validate_plans", "qlm_validate_problem",
                 "qlm_status_string", "qlm_last_error", "qlm_search_n_moves",
                 "qlm_search_workspace_bytes", "qlm_search_moves", "qlm_search_screen",
                 "qlm_local_search", "qlm_seed_workspace_bytes", "qlm_seed_plans",
                 "qlm_place_group", "qlm_fcfs_workspace_bytes", "qlm_fcfs_score",
                 "qlm_fcfs_score_exact", "qlm_fcfs_best_plan", "qlm_apply_profile",
                 "qlm_place_begin", "qlm_place_step", "qlm_place_end"):
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(lib):
    from paper_2407_00047_amd import qlm
    for code in range(5):
        assert lib.qlm_status_string(code)
    assert lib.qlm_status_string(99) == b"unknown status"
    assert qlm.QLM_ERR_CAPACITY == 2


def _problem(qlm, G=4, I=1, M=1, C=1):
    # pointers are never dereferenced by the host-side checks that fail first
    fake = 0x1000
    return qlm.Problem(G, I, M, C, fake, fake, fake, fake, fake, fake, fake, None, None, 0.0)


def test_argument_errors_before_launch(lib):
    from paper_2407_00047_amd import qlm
    pr = _problem(qlm)
    pl = qlm.Plans(4, 4, 0x1000, 0x1000, None)
    P, PL = ctypes.byref, ctypes.byref
    assert lib.qlm_rwt_score(None, PL(pl), 0x1000, None, None, None) == qlm.QLM_ERR_ARG
    assert b"NULL" in lib.qlm_last_error()
    assert lib.qlm_rwt_score(P(pr), None, 0x1000, None, None, None) == qlm.QLM_ERR_ARG
    assert lib.qlm_rwt_score(P(pr), PL(pl), None, None, None, None) == qlm.QLM_ERR_ARG
    bad = _problem(qlm, G=0)
    assert lib.qlm_rwt_score(P(bad), PL(pl), 0x1000, None, None, None) == qlm.QLM_ERR_ARG
    bad = _problem(qlm, M=256)
    assert lib.qlm_rwt_score(P(bad), PL(pl), 0x1000, None, None, None) == qlm.QLM_ERR_ARG
    stride_bad = qlm.Plans(8, 4, 0x1000, 0x1000, None)
    assert lib.qlm_rwt_score(P(pr), PL(stride_bad), 0x1000, None, None, None) == qlm.QLM_ERR_ARG
    neg = qlm.Plans(-1, 4, 0x1000, 0x1000, None)
    assert lib.qlm_rwt_score(P(pr), PL(neg), 0x1000, None, None, None) == qlm.QLM_ERR_ARG
    det = qlm.Detail(2, 5, 0x1000, None, None)                 # beyond n_plans
    assert lib.qlm_rwt_score(P(pr), PL(pl), 0x1000, None, ctypes.byref(det), None) == qlm.QLM_ERR_ARG
    # zero plans: nothing to do, no device work
    zero = qlm.Plans(0, 1, None, None, None)
    assert lib.qlm_rwt_score(P(pr), PL(zero), None, None, None, None) == qlm.QLM_OK


def test_workspace_checks(lib):
    from paper_2407_00047_amd import qlm
    pr = _problem(qlm)
    pl = qlm.Plans(1000, 1000, 0x1000, 0x1000, None)
    need = lib.qlm_best_plan_workspace_bytes(ctypes.byref(pr), 1000)
    assert need >= 8 * 1000
    assert lib.qlm_best_plan_workspace_bytes(ctypes.byref(pr), 2000) > need
    P = ctypes.byref
    assert lib.qlm_best_plan(P(pr), P(pl), None, need, 0x1000, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    assert lib.qlm_best_plan(P(pr), P(pl), 0x1010, need, 0x1000, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    assert lib.qlm_best_plan(P(pr), P(pl), 0x1000, need - 1, 0x1000, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    assert lib.qlm_best_plan(P(pr), P(pl), 0x1000, need, None, 0x1000, None) == qlm.QLM_ERR_ARG


def test_static_best_plan_capacity(lib):
    """qlm_best_plan_static refuses, on the host, a batch whose workspace would
    not fit its 64 MiB static scratch, and takes the usual argument checks."""
    from paper_2407_00047_amd import qlm
    pr = _problem(qlm)
    P = ctypes.byref
    big = qlm.Plans(4000000, 4000000, 0x1000, 0x1000, None)
    assert lib.qlm_best_plan_workspace_bytes(P(pr), 4000000) > 64 << 20
    assert lib.qlm_best_plan_static(P(pr), P(big), 0x1000, 0x1000, None) == qlm.QLM_ERR_CAPACITY
    assert b"static scratch" in lib.qlm_last_error()
    pl = qlm.Plans(4, 4, 0x1000, 0x1000, None)
    assert lib.qlm_best_plan_static(None, P(pl), 0x1000, 0x1000, None) == qlm.QLM_ERR_ARG
    assert lib.qlm_best_plan_static(P(pr), P(qlm.Plans(-1, 4, 0x1000, 0x1000, None)),
                                    0x1000, 0x1000, None) == qlm.QLM_ERR_ARG


def test_max_groups(lib):
    # LDS budget 160 KiB: 16-byte group records plus cost and instance tables
    # (the eviction twins 8 KiB on); the large workload's 8192 groups fit
    mg = lib.qlm_max_groups(8, 4, 64, 1)
    assert 8192 <= mg < 10240
    assert lib.qlm_max_groups(1, 1, 1, 0) > mg
    assert lib.qlm_max_groups(0, 1, 1, 0) == 0
    assert lib.qlm_max_groups(256, 1, 1, 0) == 0


def test_search_argument_checks(lib):
    """The plan search rejects bad windows, sizes, workspaces and outputs on
    the host, before any launch."""
    from paper_2407_00047_amd import qlm
    P = ctypes.byref
    pr = _problem(qlm, G=8, I=2)
    pl = qlm.Plans(3, 3, 0x1000, 0x1000, None)
    assert lib.qlm_search_n_moves(8, 2, 3) == 8 * 3 + 2 * 8 * 2     # SWAP, MOVE, RELOCATE
    assert lib.qlm_search_n_moves(8, 2, -1) == 0
    need = lib.qlm_search_workspace_bytes(P(pr), 3, 4)
    assert need > 0 and lib.qlm_search_workspace_bytes(P(pr), 6, 4) > need
    assert lib.qlm_search_workspace_bytes(P(pr), 3, -1) == 0
    ws = 0x10000
    out = qlm.PlansOut(3, 0x1000, 0x1000, 0x1000)
    ms = lib.qlm_search_moves
    assert ms(P(pr), P(pl), -1, ws, need, 0x1000, None) == qlm.QLM_ERR_ARG
    assert ms(P(pr), P(pl), 1025, ws, need, 0x1000, None) == qlm.QLM_ERR_ARG
    assert ms(P(pr), P(pl), 4, ws, need, None, None) == qlm.QLM_ERR_ARG
    assert ms(P(pr), P(pl), 4, None, need, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    assert ms(P(pr), P(pl), 4, ws + 16, need, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    assert ms(P(pr), P(pl), 4, ws, need - 1, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    big = _problem(qlm, G=65537, I=2)
    assert ms(P(big), P(pl), 4, ws, need, 0x1000, None) == qlm.QLM_ERR_ARG
    many = _problem(qlm, G=8, I=4097)
    assert ms(P(many), P(pl), 4, ws, need, 0x1000, None) == qlm.QLM_ERR_ARG
    ls = lib.qlm_local_search
    assert ls(P(pr), P(pl), None, 4, 5, ws, need, None, None, None, None) == qlm.QLM_ERR_ARG
    assert ls(P(pr), P(pl), P(out), 4, -1, ws, need, None, None, None, None) == qlm.QLM_ERR_ARG
    short = qlm.PlansOut(2, 0x1000, 0x1000, 0x1000)
    assert ls(P(pr), P(pl), P(short), 4, 5, ws, need, None, None, None, None) == qlm.QLM_ERR_ARG
    # the eviction words of the output are required, with or without start ones
    noev = qlm.PlansOut(3, 0x1000, 0x1000, None)
    plev = qlm.Plans(3, 3, 0x1000, 0x1000, 0x1000)
    assert ls(P(pr), P(plev), P(noev), 4, 5, ws, need, None, None, None, None) == qlm.QLM_ERR_ARG
    assert ls(P(pr), P(pl), P(noev), 4, 5, ws, need, None, None, None, None) == qlm.QLM_ERR_ARG
    assert ls(P(pr), P(pl), P(out), 4, 5, ws, need - 1, None, None, None, None) == \
        qlm.QLM_ERR_WORKSPACE
    sc = lib.qlm_search_screen
    assert sc(P(pr), P(pl), 4, ws, need, 0x1000, None, None) == qlm.QLM_ERR_ARG
    assert sc(P(pr), P(pl), 4, ws, need - 1, 0x1000, 0x1000, None) == qlm.QLM_ERR_WORKSPACE
    assert sc(P(pr), P(pl), -2, ws, need, 0x1000, 0x1000, None) == qlm.QLM_ERR_ARG
    # no plans: nothing to do
    zero = qlm.Plans(0, 1, None, None, None)
    assert ms(P(pr), P(zero), 4, ws, need, 0x1000, None) == qlm.QLM_OK
    assert sc(P(pr), P(zero), 4, ws, need, 0x1000, 0x1000, None) == qlm.QLM_OK


def test_seed_argument_checks(lib):
    """Seed plans: policy, count, output and workspace are checked on the host."""
    from paper_2407_00047_amd import qlm
    P = ctypes.byref
    pr = _problem(qlm, G=8, I=2)
    need = lib.qlm_seed_workspace_bytes(P(pr), 2)
    assert need > 0 and lib.qlm_seed_workspace_bytes(P(pr), -1) == 0
    out = qlm.PlansOut(2, 0x1000, 0x1000, None)
    pol = (ctypes.c_int32 * 2)(0, 1)
    bad = (ctypes.c_int32 * 2)(0, 2)
    ws = 0x10000
    sp = lib.qlm_seed_plans
    assert sp(P(pr), 2, bad, P(out), ws, need, None) == qlm.QLM_ERR_ARG
    assert sp(P(pr), 65, pol, P(out), ws, need, None) == qlm.QLM_ERR_ARG
    assert sp(P(pr), 2, None, P(out), ws, need, None) == qlm.QLM_ERR_ARG
    assert sp(P(pr), 2, pol, None, ws, need, None) == qlm.QLM_ERR_ARG
    short = qlm.PlansOut(1, 0x1000, 0x1000, None)
    assert sp(P(pr), 2, pol, P(short), ws, need, None) == qlm.QLM_ERR_ARG
    assert sp(P(pr), 2, pol, P(out), ws, need - 1, None) == qlm.QLM_ERR_WORKSPACE
    assert sp(P(pr), 2, pol, P(out), ws + 8, need, None) == qlm.QLM_ERR_WORKSPACE
    assert sp(P(pr), 0, pol, P(out), ws, need, None) == qlm.QLM_OK


def test_place_argument_checks(lib):
    from paper_2407_00047_amd import qlm
    P = ctypes.byref
    pr = _problem(qlm, G=8, I=2)
    pl = qlm.Plans(3, 3, 0x1000, 0x1000, None)
    need = lib.qlm_search_workspace_bytes(P(pr), 3, 0)
    out = qlm.PlansOut(3, 0x1000, 0x1000, 0x1000)
    pg = lib.qlm_place_group
    noev = qlm.PlansOut(3, 0x1000, 0x1000, None)
    assert pg(P(pr), P(pl), P(noev), 1, 0x10000, need, None, None, None) == qlm.QLM_ERR_ARG
    assert pg(P(pr), P(pl), None, 0, 0x10000, need, None, None, None) == qlm.QLM_ERR_ARG
    assert pg(P(pr), P(pl), P(out), 8, 0x10000, need, None, None, None) == qlm.QLM_ERR_ARG
    assert pg(P(pr), P(pl), P(out), -1, 0x10000, need, None, None, None) == qlm.QLM_ERR_ARG
    assert pg(P(pr), P(pl), P(out), 1, 0x10000, need - 1, None, None, None) == qlm.QLM_ERR_WORKSPACE
    zero = qlm.Plans(0, 1, None, None, None)
    assert pg(P(pr), P(zero), P(out), 1, 0x10000, need, None, None, None) == qlm.QLM_OK


def test_fcfs_argument_checks(lib):
    from paper_2407_00047_amd import qlm
    P = ctypes.byref
    pr = _problem(qlm, G=8, I=2)
    pl = qlm.Plans(3, 3, 0x1000, 0x1000, None)
    need = lib.qlm_fcfs_workspace_bytes(P(pr), 3, 40, 0)
    assert need > 0 and need % 256 == 0
    assert lib.qlm_fcfs_workspace_bytes(P(pr), 3, 4000, 0) > need
    assert lib.qlm_fcfs_workspace_bytes(None, 3, 40, 0) == 0
    assert lib.qlm_fcfs_workspace_bytes(P(pr), 3, 40, 64) == need     # 3 plans: one chunk of 64
    big = qlm.Problem(8192, 64, 1, 1, 1, 1, 1, 1, 1, 1, 1, None, None, 0.0)
    full = lib.qlm_fcfs_workspace_bytes(P(big), 20000, 100, 0)
    small = lib.qlm_fcfs_workspace_bytes(P(big), 20000, 100, 100)
    assert small < full and lib.qlm_fcfs_workspace_bytes(P(big), 20000, 100, 128) == small
    ws, slo, out = 0x10000, 0x2000, 0x3000
    fs, fx, fb = lib.qlm_fcfs_score, lib.qlm_fcfs_score_exact, lib.qlm_fcfs_best_plan
    assert fs(P(pr), P(pl), None, 40, ws, need, out, None) == qlm.QLM_ERR_ARG
    assert fs(P(pr), P(pl), slo, -1, ws, need, out, None) == qlm.QLM_ERR_ARG
    assert fs(P(pr), P(pl), slo, 1 << 31, ws, need, out, None) == qlm.QLM_ERR_ARG
    assert fs(P(pr), P(pl), slo, 40, ws, need, None, None) == qlm.QLM_ERR_ARG
    assert fs(P(pr), P(pl), slo, 40, ws, need - 1, out, None) == qlm.QLM_ERR_WORKSPACE
    assert fs(P(pr), P(pl), slo, 40, ws + 8, need, out, None) == qlm.QLM_ERR_WORKSPACE
    assert fs(P(pr), P(pl), slo, 40, None, need, out, None) == qlm.QLM_ERR_WORKSPACE
    assert fs(None, P(pl), slo, 40, ws, need, out, None) == qlm.QLM_ERR_ARG
    idx = 0x4000
    assert fx(P(pr), P(pl), slo, 40, None, 2, ws, need, out, None) == qlm.QLM_ERR_ARG
    assert fx(P(pr), P(pl), slo, 40, idx, -1, ws, need, out, None) == qlm.QLM_ERR_ARG
    assert fx(P(pr), P(pl), slo, 40, idx, 4, ws, need, out, None) == qlm.QLM_ERR_ARG
    assert fx(P(pr), P(pl), slo, 40, idx, 2, ws, need - 1, out, None) == qlm.QLM_ERR_WORKSPACE
    assert fx(P(pr), P(pl), slo, 40, idx, 0, ws, need, out, None) == qlm.QLM_OK
    assert fb(P(pr), P(pl), slo, 40, ws, need, None, out, None) == qlm.QLM_ERR_ARG
    assert fb(P(pr), P(pl), None, 40, ws, need, idx, out, None) == qlm.QLM_ERR_ARG
    zero = qlm.Plans(0, 1, None, None, None)
    need0 = lib.qlm_fcfs_workspace_bytes(P(pr), 0, 40, 0)
    assert fs(P(pr), P(zero), slo, 40, ws, need0, None, None) == qlm.QLM_OK


def test_profile_argument_checks(lib):
    from paper_2407_00047_amd import qlm
    P = ctypes.byref
    pr = _problem(qlm, G=8, I=2, M=2, C=1)
    pf = qlm.Profile(None, None, None, None, None, None)
    out = 0x5000
    ap = lib.qlm_apply_profile
    assert ap(P(pr), None, None, out, out, out, None, 0, None, None) == qlm.QLM_ERR_ARG
    assert ap(P(pr), P(pf), None, None, out, out, None, 0, None, None) == qlm.QLM_ERR_ARG
    assert ap(P(pr), P(pf), None, out, None, out, None, 0, None, None) == qlm.QLM_ERR_ARG
    assert ap(P(pr), P(pf), None, out, out, None, None, 0, None, None) == qlm.QLM_ERR_ARG
    assert ap(P(pr), P(pf), None, out, out, out, 0x6000, -1, out, None) == qlm.QLM_ERR_ARG
    assert ap(P(pr), P(pf), None, out, out, out, 0x6000, 4, None, None) == qlm.QLM_ERR_ARG
    assert ap(P(pr), P(pf), None, out, out, out, None, 4, out, None) == qlm.QLM_ERR_ARG
    assert ap(None, P(pf), None, out, out, out, None, 0, None, None) == qlm.QLM_ERR_ARG


def test_place_session_argument_checks(lib):
    from paper_2407_00047_amd import qlm
    P = ctypes.byref
    pr = _problem(qlm, G=8, I=2)
    pl = qlm.Plans(3, 3, 0x1000, 0x1000, None)
    need = lib.qlm_search_workspace_bytes(P(pr), 3, 0)
    ws = 0x10000
    assert lib.qlm_place_begin(P(pr), P(pl), ws, need - 1, None) == qlm.QLM_ERR_WORKSPACE
    assert lib.qlm_place_begin(P(pr), P(pl), ws + 8, need, None) == qlm.QLM_ERR_WORKSPACE
    assert lib.qlm_place_begin(P(pr), None, ws, need, None) == qlm.QLM_ERR_ARG
    st = lib.qlm_place_step
    assert st(P(pr), 3, 8, ws, need, None, None, None) == qlm.QLM_ERR_ARG
    assert st(P(pr), 3, -1, ws, need, None, None, None) == qlm.QLM_ERR_ARG
    assert st(P(pr), 3, 1, ws, need - 1, None, None, None) == qlm.QLM_ERR_WORKSPACE
    assert st(P(pr), -1, 1, ws, need, None, None, None) == qlm.QLM_ERR_ARG
    assert st(P(pr), 0, 1, ws, need, None, None, None) == qlm.QLM_OK
    out = qlm.PlansOut(3, 0x1000, 0x1000, 0x1000)
    en = lib.qlm_place_end
    assert en(P(pr), 3, None, ws, need, None, None) == qlm.QLM_ERR_ARG
    assert en(P(pr), 3, P(out), ws, need - 1, None, None) == qlm.QLM_ERR_WORKSPACE
    noev = qlm.PlansOut(3, 0x1000, 0x1000, None)
    assert en(P(pr), 3, P(noev), ws, need, None, None) == qlm.QLM_ERR_ARG
    short = qlm.PlansOut(2, 0x1000, 0x1000, 0x1000)
    assert en(P(pr), 3, P(short), ws, need, None, None) == qlm.QLM_ERR_ARG

