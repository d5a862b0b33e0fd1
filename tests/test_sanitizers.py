"""The host C code under AddressSanitizer and UndefinedBehaviorSanitizer: the
oracle (oracle/qlm_oracle.c) and the plan generator (csrc/qlm_gen.c) built
with -fsanitize=address,undefined, then every oracle pin and a generated
batch of every workload scored by the oracle, in a child process with the
sanitizer runtime preloaded.  Any out-of-bounds access, use after free or
undefined operation ends the child with a report, and the test fails."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "qlm_oracle.c")
GEN_SRC = os.path.join(ROOT, "paper_2407_00047_amd", "csrc", "qlm_gen.c")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]

BATCH = r'''
import sys
sys.path.insert(0, sys.argv[1])
import numpy as np
import oracle
from paper_2407_00047_amd import workload
orc = oracle.default()
for name, P in (("tiny", 256), ("mixed", 300), ("hetero", 200), ("heavy", 200), ("large", 40)):
    pr = workload.make_problem(name)
    pl = workload.make_plans(pr, 0, P)
    s, pe = orc.score_plans(pr, pl)
    assert np.all(np.isfinite(s)) and np.all(np.isfinite(pe)), name
    orc.plan_detail(pr, pl, P - 1)
    orc.argmin(s)
print("sanitized batch ok", flush=True)
'''


def _runtime():
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if p.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_and_generator_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    asan = _runtime()
    if asan is None:
        pytest.skip("no AddressSanitizer runtime")
    olib = str(tmp_path / "libqlm_oracle_san.so")
    glib = str(tmp_path / "libqlm_gen_san.so")
    subprocess.run(["gcc", *SAN, "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
                    "-shared", "-fPIC", "-o", olib, ORACLE_SRC, "-lm"], check=True)
    subprocess.run(["gcc", *SAN, "-fopenmp", "-std=c11", "-shared", "-fPIC", "-o", glib, GEN_SRC],
                   check=True)
    env = dict(os.environ)
    env.update(QLM_ORACLE_LIB=olib, QLM_GEN_LIB=glib, LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="4")
    pins = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = pins.stdout + pins.stderr
    assert pins.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    batch = subprocess.run([sys.executable, "-c", BATCH, ROOT], cwd=ROOT, env=env,
                           capture_output=True, text=True, timeout=900)
    out = batch.stdout + batch.stderr
    assert batch.returncode == 0 and "sanitized batch ok" in out, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
