"""Writes the fp64 oracle's action chunks for the full-size workloads into
tests/golden/oracle_<workload>.npz, so that the GPU parity tests can check
every sample of a batch (or a large spread subset) without running the slow
CPU oracle while the GPU waits.

Only the oracle (oracle/evo_oracle.py) and the seeded input generators
(paper_2607_20293_amd/inputs.py) are called; nothing here touches the HIP
library.  Each file records the samples, their chunks [n][H][A] (float64),
the workload name, the input seed, the SHA-256 of the oracle module and of
the seeded inputs; tests/test_golden_outputs.py checks both hashes against
the current tree and re-derives a sample of every file with the oracle on
the CPU.

Run from the repository root:  python tests/golden/make_oracle_outputs.py
[workload ...]  (about 30 CPU-minutes for all of them, spread over a
process pool).
"""
from __future__ import annotations

import hashlib
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))

SEED = 0


def spread(n_total: int, n: int) -> list:
    """n sample indices spread over [0, n_total) with every residue mod 8
    (the tile-to-XCD order) and mod 4 represented."""
    step = n_total // n
    if step <= 1:
        return list(range(n))
    per = max(1, 8 // step)          # consecutive picks that share an offset
    return sorted({i * step + (i // per) % step for i in range(n)})


# workload -> the samples whose chunks are stored (None: all of them)
CASES = {
    "pusht_fp32_b64_d25": None,
    "pusht_bf16_b64_d25": None,
    "pusht_bf16_b64_all": None,
    "image_bf16_b256_d12": None,
    "population_bf16_b512": None,
    "bimanual_bf16_b128_d20": None,
    "bimanual_bf16_b128_all": spread(128, 32),
}


def oracle_sha() -> str:
    """SHA-256 (16 hex digits) of the oracle module the chunks came from."""
    with open(os.path.join(ROOT, "oracle", "evo_oracle.py"), "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


def inputs_sha(inp) -> str:
    """SHA-256 (16 hex digits) of a workload's seeded inputs: weights,
    observations, noise, lattices and schedule ids, as stored bytes."""
    h = hashlib.sha256()
    for a in [inp.weights, inp.obs, inp.noise, *inp.lattices, inp.ids]:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode() + str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()[:16]


def _one(args):
    name, j = args
    from threadpoolctl import threadpool_limits
    from oracle import evo_oracle as O
    from paper_2607_20293_amd import inputs as I
    w = I.WORKLOADS[name]
    inp = I.make_inputs(w, seed=SEED)
    with threadpool_limits(1):
        out, _ = O.denoise(w.shape, I.split_weights(w.shape, inp.weights), inp.obs, inp.noise, inp.lattices,
                           inp.ids, dtype=w.dtype, samples=[j])
    return j, out[0]


def path_for(name: str) -> str:
    return os.path.join(HERE, f"oracle_{name}.npz")


def make(name: str, workers: int) -> str:
    from paper_2607_20293_amd import inputs as I
    w = I.WORKLOADS[name]
    samples = list(range(w.batch)) if CASES[name] is None else CASES[name]
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=workers) as ex:
        res = dict(ex.map(_one, [(name, j) for j in samples]))
    chunks = np.stack([res[j] for j in samples]).astype(np.float64)
    p = path_for(name)
    np.savez_compressed(p, samples=np.asarray(samples, np.int32), chunks=chunks, workload=np.str_(name),
                        seed=np.int64(SEED), oracle_sha=np.str_(oracle_sha()),
                        inputs_sha=np.str_(inputs_sha(I.make_inputs(w, seed=SEED))))
    print(f"{name}: {len(samples)} samples in {time.perf_counter() - t0:.1f} s -> {os.path.relpath(p, ROOT)}",
          flush=True)
    return p


if __name__ == "__main__":
    names = sys.argv[1:] or list(CASES)
    nw = min(8, os.cpu_count() or 1)
    for n in names:
        make(n, nw)
