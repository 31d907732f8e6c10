"""The C ABI used from C++ alone (paper_2607_20293_amd/examples/evo_demo.cpp,
built by build_lib.build()): the program creates a policy, registers a layer
lattice, runs the loop on a stream of its own and checks the bookkeeping
against evo_schedule_stats; here its JSON line is checked as well."""
import json
import os
import subprocess

import pytest

from paper_2607_20293_amd import build_lib

pytestmark = pytest.mark.gpu


def test_c_abi_demo_runs():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(build_lib.DEMO):
        pytest.skip("evo_demo not built (run __graft_entry__.build())")
    r = subprocess.run([build_lib.DEMO, "8", "5"], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stderr
    res = json.loads(r.stdout.strip().splitlines()[-1])
    assert res["finite"] and res["stats_match_host"]
    # every fourth step of 100, all 8 layers x 3 units, 8 samples
    assert res["refreshes_effective"] == 8 * 3 * 8 * 25
    assert res["chunks_per_s"] > 0
