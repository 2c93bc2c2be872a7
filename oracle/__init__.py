"""CPU oracle for the batched quantum-layer path -- TEST INFRASTRUCTURE ONLY.

Plain gate-by-gate complex128 simulation (``oracle.c``) with the adjoint VJP
and a parameter-shift cross-check. Only ``tests/``, ``__graft_entry__.smoke``
and the benchmark's CPU-baseline leg may import this package; the HIP product
path never does, and the two share no code.

Angles are consumed as float64. For complex64 workloads callers pass the
float32 values the GPU receives, upcast exactly.

Gate kinds: H 0, RX 1, RY 2, RZ 3, CNOT 4, CZ 5, CRX 6, CRY 7, CRZ 8 (q0 control,
q1 target) and PAULI 9 (a Pauli-channel trajectory: its uniform is input
feature ``index``, its probabilities the next row of ``pauli_p``). Embeddings
``embed = (kind, first)``: kind 0 none (|0...0>), 1 basis, 2 amplitude.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_default = None


def compile_source(src: str, out: str) -> str:
    """Compile an oracle C source with gcc (-O2, OpenMP) into a shared library."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                           "-Wall", "-o", tmp, src, "-lm"])
    os.replace(tmp, out)
    return out


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` (always when ``force``)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        compile_source(_SRC, _LIB)
    return _LIB


def _bind(path):
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.oracle_run.argtypes = [ctypes.c_int, P, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                               ctypes.c_int, P, P, P, P, P, P, P, P, P]
    lib.oracle_run.restype = ctypes.c_int
    lib.oracle_param_shift.argtypes = [ctypes.c_int, P, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, P, P, P, P, P]
    lib.oracle_param_shift.restype = ctypes.c_int
    ci = ctypes.c_int
    lib.oracle_run_ext.argtypes = [ci, P, ci, ci, ci, ci, ci, ci, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_run_ext.restype = ci
    lib.oracle_param_shift_ext.argtypes = [ci, P, ci, ci, ci, ci, ci, ci, P, P, P, P, P, P]
    lib.oracle_param_shift_ext.restype = ci
    lib.oracle_sample.argtypes = [ctypes.c_int, ctypes.c_int, P, ctypes.c_int64, P, P]
    lib.oracle_sample.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    return lib


def _load():
    global _default
    if _default is None:
        build()
        _default = Oracle(_LIB)
    return _default.lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _prep(gates, inputs, weights, B):
    gates = np.ascontiguousarray(gates, dtype=np.int32).reshape(-1, 5)
    x = np.ascontiguousarray(np.asarray(inputs, dtype=np.float64).reshape(B, -1))
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float64).reshape(-1))
    return gates, x, w


class Oracle:
    """Handle on one compiled oracle library (the default one, or a test copy)."""

    def __init__(self, path):
        self.lib = _bind(path)

    def run(self, n, gates, inputs, weights, grad_out=None, want_state=False, want_back=False,
            embed=None, pauli_p=None):
        return _run(self.lib, n, gates, inputs, weights, grad_out, want_state, want_back, embed,
                    pauli_p)

    def param_shift(self, n, gates, inputs, weights, grad_out, embed=None, pauli_p=None):
        return _param_shift(self.lib, n, gates, inputs, weights, grad_out, embed, pauli_p)

    def sample(self, n, states, uniforms):
        return _sample(self.lib, n, states, uniforms)


def default() -> "Oracle":
    _load()
    return _default


def run(n, gates, inputs, weights, grad_out=None, want_state=False, want_back=False, embed=None,
        pauli_p=None):
    """See ``_run``; uses the default oracle library."""
    return _run(_load(), n, gates, inputs, weights, grad_out, want_state, want_back, embed, pauli_p)


def param_shift(n, gates, inputs, weights, grad_out, embed=None, pauli_p=None):
    """See ``_param_shift``; uses the default oracle library."""
    return _param_shift(_load(), n, gates, inputs, weights, grad_out, embed, pauli_p)


def _ext(embed, pauli_p):
    kind, first = (0, 0) if embed is None else (int(embed[0]), int(embed[1]))
    pp = None if pauli_p is None else np.ascontiguousarray(np.asarray(pauli_p, np.float64).reshape(-1, 3))
    return kind, first, pp


def _run(lib, n, gates, inputs, weights, grad_out=None, want_state=False, want_back=False,
         embed=None, pauli_p=None):
    """Forward (+ adjoint VJP when ``grad_out`` is given) over a batch.

    Returns a dict with ``expz[B,n]`` and, with ``grad_out``, ``grad_inputs[B,F]``
    and ``grad_weights[P]``; ``state[B,2^n]`` (complex128) with ``want_state``;
    ``back_psi[B,2^n]`` and ``back_lam0[B]`` (psi and lambda[0] after the
    reverse sweep un-applied every gate) with ``want_back``. ``embed`` and
    ``pauli_p`` as in the module docstring.
    """
    inputs = np.asarray(inputs)
    B = inputs.shape[0]
    gates, x, w = _prep(gates, inputs, weights, B)
    F = x.shape[1]
    P = w.shape[0]
    dim = 1 << n
    expz = np.zeros((B, n), dtype=np.float64)
    out = {"expz": expz}
    g = gi = gw = None
    if grad_out is not None:
        g = np.ascontiguousarray(np.asarray(grad_out, dtype=np.float64).reshape(B, n))
        gi = np.zeros((B, F), dtype=np.float64)
        gw = np.zeros(P, dtype=np.float64)
        out["grad_inputs"], out["grad_weights"] = gi, gw
    st = np.zeros((B, dim), dtype=np.complex128) if want_state else None
    bp = bl = None
    if want_back and g is not None:
        bp = np.zeros((B, dim), dtype=np.complex128)
        bl = np.zeros(B, dtype=np.complex128)
        out["back_psi"], out["back_lam0"] = bp, bl
    if st is not None:
        out["state"] = st
    kind, first, pp = _ext(embed, pauli_p)
    rc = lib.oracle_run_ext(n, _ptr(gates), gates.shape[0], B, F, P, kind, first, _ptr(pp), _ptr(x),
                            _ptr(w), _ptr(g), _ptr(expz), _ptr(gi), _ptr(gw), _ptr(st), _ptr(bp),
                            _ptr(bl))
    if rc != 0:
        raise ValueError(f"oracle_run failed with code {rc}")
    return out


def _param_shift(lib, n, gates, inputs, weights, grad_out, embed=None, pauli_p=None):
    """Parameter-shift VJP: ``(grad_inputs[B,F], grad_weights[P])`` (two-term rule,
    four-term for controlled rotations; amplitude-embedding features get none)."""
    inputs = np.asarray(inputs)
    B = inputs.shape[0]
    gates, x, w = _prep(gates, inputs, weights, B)
    F, P = x.shape[1], w.shape[0]
    g = np.ascontiguousarray(np.asarray(grad_out, dtype=np.float64).reshape(B, n))
    gi = np.zeros((B, F), dtype=np.float64)
    gw = np.zeros(P, dtype=np.float64)
    kind, first, pp = _ext(embed, pauli_p)
    rc = lib.oracle_param_shift_ext(n, _ptr(gates), gates.shape[0], B, F, P, kind, first, _ptr(pp),
                                    _ptr(x), _ptr(w), _ptr(g), _ptr(gi), _ptr(gw))
    if rc != 0:
        raise ValueError(f"oracle_param_shift failed with code {rc}")
    return gi, gw


def sample(n, states, uniforms):
    """See ``_sample``; uses the default oracle library."""
    return _sample(_load(), n, states, uniforms)


def _sample(lib, n, states, uniforms):
    """Shots by the inverse CDF: ``states[B, 2^n]`` (complex), ``uniforms[B, shots]``
    in [0, 1) -> amplitude indices ``[B, shots]`` (int64)."""
    st = np.ascontiguousarray(np.asarray(states, dtype=np.complex128).reshape(-1, 1 << n))
    B = st.shape[0]
    u = np.ascontiguousarray(np.asarray(uniforms, dtype=np.float64).reshape(B, -1))
    out = np.zeros(u.shape, dtype=np.int64)
    rc = lib.oracle_sample(n, B, _ptr(st.view(np.float64)), u.shape[1], _ptr(u), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_sample failed with code {rc}")
    return out


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_load().oracle_num_threads())
