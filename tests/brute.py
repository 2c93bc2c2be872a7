"""Brute-force dense-matrix model of a small circuit (n <= 4), used to pin the oracle.

Independent of the oracle's gate-by-gate loops: every gate is a full
2^n x 2^n matrix built from Kronecker products, rotations are the matrix
exponential exp(-i theta P / 2) of a Pauli generator (scipy.linalg.expm), and
the two-qubit gates are sums of projector products. Gradients are exact
derivatives of the full product of matrices, d U_k / d theta = -(i/2) P U_k,
inserted at gate k: no adjoint sweep and no parameter shift.

Controlled rotations are P0 (x) I + P1 (x) exp(-i theta P / 2), with derivative
-(i/2) (P1 (x) P) U. A Pauli-channel trajectory applies the Pauli matrix its
uniform selects. Embeddings give the initial state directly (a basis vector or
the normalised feature vector); amplitude-embedding gradients are not modelled
here (finite differences pin them).
"""

from __future__ import annotations

import numpy as np
from scipy.linalg import expm

import workloads as W

I2 = np.eye(2, dtype=np.complex128)
PX = np.array([[0, 1], [1, 0]], dtype=np.complex128)
PY = np.array([[0, -1j], [1j, 0]], dtype=np.complex128)
PZ = np.array([[1, 0], [0, -1]], dtype=np.complex128)
P0 = np.array([[1, 0], [0, 0]], dtype=np.complex128)
P1 = np.array([[0, 0], [0, 1]], dtype=np.complex128)
HAD = (PX + PZ) / np.sqrt(2.0)
GEN = {W.RX: PX, W.RY: PY, W.RZ: PZ}
CGEN = {W.CRX: PX, W.CRY: PY, W.CRZ: PZ}
PAULIS = [I2, PX, PY, PZ]


def pauli_choice(u: float, p) -> int:
    """Which Pauli (0 = none, 1 = X, 2 = Y, 3 = Z) a trajectory uniform selects."""
    edges = np.cumsum(np.asarray(p, dtype=np.float64))
    for k in range(3):
        if u < edges[k]:
            return k + 1
    return 0


def embed(n: int, ops: dict) -> np.ndarray:
    """Kronecker product with ``ops[q]`` on qubit q and identity elsewhere.

    Qubit q is bit q of the amplitude index, so the leftmost factor of the
    product is qubit n-1.
    """
    m = np.ones((1, 1), dtype=np.complex128)
    for q in reversed(range(n)):
        m = np.kron(m, ops.get(q, I2))
    return m


def gate_unitary(n: int, gate, theta: float) -> np.ndarray:
    kind, q0, q1 = int(gate[0]), int(gate[1]), int(gate[2])
    if kind == W.H:
        return embed(n, {q0: HAD})
    if kind in GEN:
        return embed(n, {q0: expm(-0.5j * theta * GEN[kind])})
    if kind == W.CNOT:
        return embed(n, {q0: P0}) + embed(n, {q0: P1, q1: PX})
    if kind == W.CZ:
        return np.eye(1 << n, dtype=np.complex128) - 2.0 * embed(n, {q0: P1, q1: P1})
    if kind in CGEN:
        return embed(n, {q0: P0}) + embed(n, {q0: P1, q1: expm(-0.5j * theta * CGEN[kind])})
    if kind == W.PAULI:  # theta carries the selected Pauli
        return embed(n, {q0: PAULIS[int(theta)]})
    raise ValueError(kind)


def gate_derivative(n: int, gate, theta: float) -> np.ndarray:
    """d/dtheta of a rotation's full unitary: -(i/2) P U (P = P1 (x) P_t when controlled)."""
    kind = int(gate[0])
    if kind in CGEN:
        P = embed(n, {int(gate[1]): P1, int(gate[2]): CGEN[kind]})
    else:
        P = embed(n, {int(gate[1]): GEN[kind]})
    return -0.5j * P @ gate_unitary(n, gate, theta)


def z_observable(n: int, q: int) -> np.ndarray:
    return embed(n, {q: PZ})


def angles(gates, x_b, w, pauli_p=None):
    """Angle of every gate; for a Pauli channel, the index of the selected Pauli."""
    th = []
    ch = 0
    for g in gates:
        src, idx = int(g[3]), int(g[4])
        if int(g[0]) == W.PAULI:
            th.append(float(pauli_choice(float(x_b[idx]), pauli_p[ch])))
            ch += 1
            continue
        th.append(float(x_b[idx]) if src == W.SRC_INPUT else
                  float(w[idx]) if src == W.SRC_WEIGHT else 0.0)
    return th


def initial_state(n: int, x_b, embed_kind=W.EMBED_NONE, first=0) -> np.ndarray:
    dim = 1 << n
    psi = np.zeros(dim, dtype=np.complex128)
    if embed_kind == W.EMBED_AMPLITUDE:
        v = np.asarray(x_b[first:first + dim], dtype=np.float64)
        r = np.linalg.norm(v)
        return psi if r == 0 else (v / r).astype(np.complex128)
    idx = 0
    if embed_kind == W.EMBED_BASIS:
        idx = sum(1 << q for q in range(n) if x_b[first + q] >= 0.5)
    psi[idx] = 1.0
    return psi


def unitary(n: int, gates, x_b, w) -> np.ndarray:
    U = np.eye(1 << n, dtype=np.complex128)
    for g, t in zip(gates, angles(gates, x_b, w)):
        U = gate_unitary(n, g, t) @ U
    return U


def run(n: int, gates, inputs, weights, grad_out=None, embed=None, pauli_p=None):
    """Dense reference: final states, <Z_i>, and the VJP gradients of the
    rotation angles (``embed = (kind, first)``, ``pauli_p[channels][3]``)."""
    inputs = np.asarray(inputs, dtype=np.float64)
    weights = np.asarray(weights, dtype=np.float64)
    B, F = inputs.shape
    P = weights.shape[0]
    dim = 1 << n
    Zs = [z_observable(n, q) for q in range(n)]
    states = np.zeros((B, dim), dtype=np.complex128)
    expz = np.zeros((B, n))
    gi = np.zeros((B, F))
    gw = np.zeros(P)
    ek, first = (W.EMBED_NONE, 0) if embed is None else embed
    for b in range(B):
        th = angles(gates, inputs[b], weights, pauli_p)
        mats = [gate_unitary(n, g, t) for g, t in zip(gates, th)]
        e0 = initial_state(n, inputs[b], ek, first)
        psi = e0.copy()
        for m in mats:
            psi = m @ psi
        states[b] = psi
        expz[b] = [np.real(np.vdot(psi, Z @ psi)) for Z in Zs]
        if grad_out is None:
            continue
        O = sum(float(grad_out[b][q]) * Zs[q] for q in range(n))
        for k, g in enumerate(gates):
            if int(g[0]) not in GEN and int(g[0]) not in CGEN:
                continue
            # d psi / d theta_k = U_G .. U_{k+1} (dU_k) U_{k-1} .. U_1 e0
            v = e0.copy()
            for j, m in enumerate(mats):
                v = (gate_derivative(n, g, th[k]) if j == k else m) @ v
            d = 2.0 * np.real(np.vdot(psi, O @ v))
            if int(g[3]) == W.SRC_WEIGHT:
                gw[int(g[4])] += d
            else:
                gi[b, int(g[4])] += d
    return {"state": states, "expz": expz, "grad_inputs": gi, "grad_weights": gw}
