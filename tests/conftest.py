import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def read_golden(name):
    """Parse a tests/golden fixture: '# ...' comment lines, then 'key v1 v2 ...' rows
    (or a bare row of numbers)."""
    path = os.path.join(ROOT, "tests", "golden", name)
    rows = {}
    bare = []
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            try:
                bare.append([float(p) for p in parts])
            except ValueError:
                rows[parts[0]] = [float(p) for p in parts[1:]]
    return rows, bare


def ensure_library():
    """Build libscaleqlora.so if it is not there yet (hipcc cross-compiles without a GPU)."""
    from paper_2609_04526_amd import build as _build, sq as _sq
    if not os.path.exists(_sq.LIB_PATH):
        _build.build()
    return _sq.load()


def gpu_ready():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False
