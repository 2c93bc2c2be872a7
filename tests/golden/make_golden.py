"""Write oracle reference values for the large workloads (calls only ``oracle/``).

For the 24- and 30-qubit workloads the CPU oracle takes minutes to an hour, far
too long for a GPU test run, so its results are computed once here and stored
as ``<workload>.npz`` (plain arrays, no pickle):

  rows          sampled batch rows
  expz          <Z_i> of those rows                       [len(rows), n]
  grad_inputs   VJP w.r.t. the inputs of those rows       [len(rows), F]
  grad_weights  VJP w.r.t. the weights with grad_out zeroed outside `rows`  [P]
  digest        sha256 of the workload's inputs, weights and grad_out

``16q`` holds the whole batch (all 1024 rows, so ``grad_weights`` is the
batch sum of the workload itself). ``24q_c128`` and ``30q_c128`` are the 24-
and 30-qubit workloads in complex128: the same circuits with their inputs
drawn and kept in fp64.

Usage: python tests/golden/make_golden.py 24q 30q 16q 24q_c128 30q_c128
"""

from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as W  # noqa: E402

ROWS = {"24q": [0, 7, 15], "30q": [0], "16q": list(range(1024)), "24q_c128": [0, 7, 15], "30q_c128": [0]}


def workload(name: str):
    """The workload a golden file is for: ``<name>`` or ``<name>_c128``."""
    if name.endswith("_c128"):
        return W.scaled(W.get(name[:-5]), dtype="c128")
    return W.get(name)


def digest(x, w, g) -> str:
    h = hashlib.sha256()
    for a in (x, w, g):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def make(name: str):
    wl = workload(name)
    x, w, g = wl.inputs()
    rows = ROWS[name]
    t0 = time.time()
    r = oracle.run(wl.n, wl.gates(), x[rows], w, grad_out=g[rows])
    shown = rows if len(rows) <= 8 else f"0..{rows[-1]}"
    print(f"{name}: oracle on rows {shown} took {time.time() - t0:.1f}s", flush=True)
    out = os.path.join(HERE, f"{name}.npz")
    np.savez(out, rows=np.asarray(rows, dtype=np.int64), expz=r["expz"],
             grad_inputs=r["grad_inputs"], grad_weights=r["grad_weights"],
             digest=np.asarray(digest(x, w, g)))
    print("wrote", out, flush=True)


if __name__ == "__main__":
    for name in sys.argv[1:]:
        make(name)
