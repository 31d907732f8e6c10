import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_printed_schedules(tag):
    """{method: {unit_name: [steps]}} from tests/golden/schedules_<tag>.txt."""
    out = {"BAC": {}, "EVO": {}}
    with open(os.path.join(GOLDEN, f"schedules_{tag}.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            steps = [int(x) for x in parts[2].split(",")] if len(parts) > 2 else []
            out[parts[1]][parts[0]] = steps
    return out


def printed_unit_lattice(tag, method, n_layers=8, T=100):
    """Unit-granular lattice [3L][T] (rows ordered layer-major SA, CA, FFN)."""
    import numpy as np
    sch = load_printed_schedules(tag)[method]
    lat = np.zeros((3 * n_layers, T), np.uint8)
    for l in range(n_layers):
        for u, nm in enumerate(("SA", "CA", "FFN")):
            for t in sch[f"layers.{l}.{nm}"]:
                lat[3 * l + u, t] = 1
    return lat
