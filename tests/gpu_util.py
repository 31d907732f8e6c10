"""Helpers shared by the GPU tests: run the HIP path through the C ABI and
the fp64 oracle on the same seeded inputs."""
import sys

import numpy as np
import pytest

from oracle import evo_oracle as O
from paper_2607_20293_amd import inputs as I

# Tolerances: fp32 max-abs, bf16 normwise relative (max-abs error over the
# max-abs of the oracle chunk), both on the final action chunk x_0.
TOL_FP32 = 1e-4
TOL_BF16 = 3e-2


def device():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(pol, inp_obs, inp_noise, ids):
    import torch
    dev = device()
    obs = torch.from_numpy(np.ascontiguousarray(inp_obs)).to(dev)
    noise = torch.from_numpy(np.ascontiguousarray(inp_noise)).to(dev)
    out = pol.denoise(obs, noise, ids)
    pol.synchronize()
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), pol.stats()


def run_oracle(shape, weights, obs, noise, lattices, ids, gran, cold, dtype, samples=None, clip=True):
    return O.denoise(shape, I.split_weights(shape, weights), obs, noise, lattices, ids,
                     granularity=gran, cold_policy=cold, clip=clip, dtype=dtype, samples=samples)


def compare(got, ref, dtype, what=""):
    """what=None: check quietly (the caller reports)."""
    err = float(np.max(np.abs(got - ref)))
    if dtype == "fp32":
        if what is not None:
            say(f"  {what}: max-abs err {err:.3e} (tol {TOL_FP32})")
        assert err <= TOL_FP32, f"{what}: max-abs {err} > {TOL_FP32}"
        return err
    rel = err / max(float(np.max(np.abs(ref))), 1e-6)
    if what is not None:
        say(f"  {what}: rel err {rel:.3e} (max-abs {err:.3e}, tol {TOL_BF16})")
    assert rel <= TOL_BF16, f"{what}: relative {rel} > {TOL_BF16}"
    return rel


def load_stored(name):
    """The oracle's chunks of a full-size workload written by
    tests/golden/make_oracle_outputs.py (samples, chunks, workload, seed,
    source_sha)."""
    import os
    p = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", f"oracle_{name}.npz")
    with np.load(p, allow_pickle=False) as z:
        g = {k: z[k] for k in z.files}
    assert str(g["workload"]) == name and int(g["seed"]) == 0
    return g


def check_stats(got, want):
    for k, v in want.items():
        assert got[k] == v, (k, got[k], v)
