import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def read_golden(name):
    """Rows of a '|'-separated golden file, comments stripped."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append([c.strip() for c in line.split("|")])
    return rows


def _ensure_built():
    """Tests use the in-tree library as built; they build it only if nothing is there."""
    lib = os.path.join(ROOT, "paper_2607_02461_amd", "liborbitquant.so")
    if not os.path.exists(lib):
        from paper_2607_02461_amd.build import build
        build()


_ensure_built()
