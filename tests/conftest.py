import json
import math
import os
import re
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size parity case (minutes of oracle time)")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


_LN = re.compile(r"ln(\d+)")


def golden_value(expr):
    """Evaluate a fixture expression such as '-2/9*ln2 - 30/169*ln3', '2**0.5/5'
    or '3*cos(1) + sin(1)' in float64."""
    names = {f"ln{n}": math.log(int(n)) for n in _LN.findall(expr)}
    names.update({"cos": math.cos, "sin": math.sin})
    if not re.fullmatch(r"([0-9+\-*/(). ]|ln\d+|cos|sin)*", expr):
        raise ValueError(f"unexpected token in fixture expression {expr!r}")
    return float(eval(expr, {"__builtins__": {}}, names))  # fixture-local arithmetic only


def rel_f(x, ref):
    """Relative Frobenius error ||x - ref|| / ||ref|| in float64."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(x - ref) / (den if den > 0 else 1.0))


def row_err(x, ref):
    """Largest row error norm relative to the RMS row norm of ``ref``.

    x, ref: [rows, features].  max_i ||x_i - ref_i|| / sqrt(mean_i ||ref_i||^2):
    a per-row bound that a single wrong row cannot dilute, and that stays
    meaningful for rows whose reference is exactly zero."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = math.sqrt(float(np.mean(np.sum(ref * ref, axis=1))))
    worst = float(np.max(np.linalg.norm(x - ref, axis=1)))
    return worst / (rms if rms > 0 else 1.0)
