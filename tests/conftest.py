import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def parse_values(spec):
    """'1.0*32' or '1.0,-0x1p-3,...' -> 32 floats (rest zero)."""
    vals = []
    for tok in spec.split(","):
        tok = tok.strip()
        if "*" in tok:
            v, n = tok.split("*")
            vals += [float.fromhex(v) if "0x" in v else float(v)] * int(n)
        else:
            vals.append(float.fromhex(tok) if "0x" in tok else float(tok))
    return vals + [0.0] * (32 - len(vals))


def load_golden(name):
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([p.strip() for p in line.split("|")])
    return rows
