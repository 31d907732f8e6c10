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
    from paper_2607_20293_amd import inputs as I
    out = {"BAC": {}, "EVO": {}}
    out.update(I.read_printed_schedules(os.path.join(GOLDEN, f"schedules_{tag}.txt")))
    return out


def printed_unit_lattice(tag, method, n_layers=8, T=100):
    """Unit-granular lattice [3L][T] (rows ordered layer-major SA, CA, FFN)."""
    from paper_2607_20293_amd import inputs as I
    return I.printed_lattice(os.path.join(GOLDEN, f"schedules_{tag}.txt"), method, n_layers, T)
