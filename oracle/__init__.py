"""CPU oracle for the batched quantum-layer path -- TEST INFRASTRUCTURE ONLY.

Plain gate-by-gate complex128 simulation (``oracle.c``) with the adjoint VJP
and a parameter-shift cross-check. Only ``tests/``, ``__graft_entry__.smoke``
and the benchmark's CPU-baseline leg may import this package; the HIP product
path never does, and the two share no code.

Angles are consumed as float64. For complex64 workloads callers pass the
float32 values the GPU receives, upcast exactly.
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

    def run(self, n, gates, inputs, weights, grad_out=None, want_state=False, want_back=False):
        return _run(self.lib, n, gates, inputs, weights, grad_out, want_state, want_back)

    def param_shift(self, n, gates, inputs, weights, grad_out):
        return _param_shift(self.lib, n, gates, inputs, weights, grad_out)

    def sample(self, n, states, uniforms):
        return _sample(self.lib, n, states, uniforms)


def default() -> "Oracle":
    _load()
    return _default


def run(n, gates, inputs, weights, grad_out=None, want_state=False, want_back=False):
    """See ``_run``; uses the default oracle library."""
    return _run(_load(), n, gates, inputs, weights, grad_out, want_state, want_back)


def param_shift(n, gates, inputs, weights, grad_out):
    """See ``_param_shift``; uses the default oracle library."""
    return _param_shift(_load(), n, gates, inputs, weights, grad_out)


def _run(lib, n, gates, inputs, weights, grad_out=None, want_state=False, want_back=False):
    """Forward (+ adjoint VJP when ``grad_out`` is given) over a batch.

    Returns a dict with ``expz[B,n]`` and, with ``grad_out``, ``grad_inputs[B,F]``
    and ``grad_weights[P]``; ``state[B,2^n]`` (complex128) with ``want_state``;
    ``back_psi[B,2^n]`` and ``back_lam0[B]`` (psi and lambda[0] after the
    reverse sweep un-applied every gate) with ``want_back``.
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
    rc = lib.oracle_run(n, _ptr(gates), gates.shape[0], B, F, P, _ptr(x), _ptr(w), _ptr(g),
                        _ptr(expz), _ptr(gi), _ptr(gw), _ptr(st), _ptr(bp), _ptr(bl))
    if rc != 0:
        raise ValueError(f"oracle_run failed with code {rc}")
    return out


def _param_shift(lib, n, gates, inputs, weights, grad_out):
    """Parameter-shift VJP: ``(grad_inputs[B,F], grad_weights[P])``."""
    inputs = np.asarray(inputs)
    B = inputs.shape[0]
    gates, x, w = _prep(gates, inputs, weights, B)
    F, P = x.shape[1], w.shape[0]
    g = np.ascontiguousarray(np.asarray(grad_out, dtype=np.float64).reshape(B, n))
    gi = np.zeros((B, F), dtype=np.float64)
    gw = np.zeros(P, dtype=np.float64)
    rc = lib.oracle_param_shift(n, _ptr(gates), gates.shape[0], B, F, P, _ptr(x), _ptr(w),
                                _ptr(g), _ptr(gi), _ptr(gw))
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
