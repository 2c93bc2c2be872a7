"""Element-wise comparison of GPU results with reference values, recording the
achieved error of every comparison.

Every comparison appends one row (test, case, output, max abs error, tolerance,
largest reference magnitude) to ``RECORD``. When the environment variable
``QL_PARITY_JSON`` names a file, the session writes the rows there at its end
(``conftest.pytest_sessionfinish``), so the margins under the tolerances are on
record, not only the pass/fail outcome.
"""

from __future__ import annotations

import json
import os

import numpy as np

RECORD: list[dict] = []
CURRENT = {"test": ""}


def close(got, want, tol, what, output=""):
    """Assert max |got - want| <= tol (absolute, element-wise) and record it."""
    a, b = np.asarray(got), np.asarray(want)
    assert a.shape == b.shape, f"{what} {output}: shape {a.shape} vs {b.shape}"
    if np.iscomplexobj(a) or np.iscomplexobj(b):
        a, b = a.astype(np.complex128), b.astype(np.complex128)
    else:
        a, b = a.astype(np.float64), b.astype(np.float64)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    ref = float(np.max(np.abs(b))) if b.size else 0.0
    RECORD.append({"test": CURRENT["test"], "case": what, "output": output, "max_abs_err": err,
                   "tol": float(tol), "max_abs_ref": ref, "size": int(a.size)})
    assert err <= tol, f"{what} {output}: max abs err {err:.3e} > {tol:.0e}"
    return err


def check(got, want, tol, what, keys=("expz", "grad_inputs", "grad_weights")):
    """``close`` on each named output of two result dicts."""
    for k in keys:
        close(got[k], want[k], tol, what, k)


def write(path):
    os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
    with open(path, "w") as f:
        json.dump(RECORD, f, indent=0)
