"""The host runtime (schedule ingestion, batch plans, bookkeeping, Eq. 7
helpers, the Sec. 3.2 search) built with AddressSanitizer and
UndefinedBehaviorSanitizer by the host C++ compiler alone (no HIP code in
the build) and driven by tests/host_sanitize/host_driver.cpp; a memory or
undefined-behaviour error aborts the driver.  The integer bookkeeping it
prints is compared with the oracle's.  CPU only."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import evo_oracle as O
from paper_2607_20293_amd import inputs as I

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_20293_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    out = str(tmp_path_factory.mktemp("san") / "host_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host_sanitize", "host_driver.cpp"),
           os.path.join(CSRC, "evo_host.cpp"), os.path.join(CSRC, "evo_ga.cpp"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out


def test_host_runtime_clean_under_sanitizers(driver):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([driver], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host driver ok" in r.stdout
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
    # the fixed bookkeeping case the driver prints, from the oracle
    s = I.PUSHT
    U, T = 3 * s.n_layers, s.n_steps
    lat = np.array([[((7 * b + 3 * t) % 10) < 3 for t in range(T)] for b in range(U)], np.uint8)
    full = np.ones((s.n_layers, T), np.uint8)
    st0 = O.bookkeeping(s, [lat], np.zeros(2, np.int32), O.GRAN_UNIT, O.COLD_COMPUTE)
    st1 = O.bookkeeping(s, [full], np.zeros(2, np.int32), O.GRAN_LAYER, O.COLD_COMPUTE)
    line = [ln for ln in r.stdout.splitlines() if ln.startswith("stats ")][0]
    got = [int(v) for v in line.split()[1:]]
    want = [st0[k] + st1[k] for k in ("refreshes_requested", "refreshes_effective", "flops_cacheable",
                                      "flops_always", "flops_full")]
    assert got == want
