"""Seeded synthetic workloads for the batched quantum-layer path.

This module only *describes* circuits and draws inputs; it holds none of the
simulation arithmetic. Both the CPU oracle (``oracle/``) and the HIP path
(``paper_2301_03251_amd``) consume what it returns, and neither imports the
other.

A circuit is an ``int32`` array of shape ``[G, 5]``; each row is one gate
``(kind, q0, q1, src, index)``:

* ``kind``  -- ``H=0, RX=1, RY=2, RZ=3, CNOT=4, CZ=5``, controlled rotations
  ``CRX=6, CRY=7, CRZ=8`` and Pauli-channel trajectories ``PAULI=9``;
* ``q0, q1`` -- qubits; ``q1 = -1`` for one-qubit gates, CNOT and the
  controlled rotations use ``q0 = control, q1 = target``;
* ``src``   -- where a rotation angle comes from: ``NONE=0`` (H, CNOT, CZ),
  ``INPUT=1`` (feature ``index`` of the sample), ``WEIGHT=2`` (trainable
  weight ``index``, shared by every sample). A Pauli channel reads its
  trajectory uniform from input feature ``index``; its probabilities
  ``(p_x, p_y, p_z)`` are given beside the circuit, one row per channel.

Initial-state embeddings: ``EMBED_NONE=0`` (|0...0>), ``EMBED_BASIS=1``
(qubit q is 1 where feature ``first + q`` is >= 0.5), ``EMBED_AMPLITUDE=2``
(the 2^n features from ``first`` on, normalised).

The gate set and the binding of rotation angles to input features or
trainable weights follow the quantum node of the paper (Sec. "Quantum Node":
a parameterised circuit with an encoding part and an evolution part, whose
parameters are trained by gradient descent), with angle encoding of features
(Sec. "Quantum Data", encoding into rotation angles).

The five standard workloads are hybrid-network-shaped circuits: an angle
encoding layer followed by layers of trainable rotations and an entangler.
Per layer: for each qubit ``q`` in ascending order, the listed rotations in
order; then the entangler. Weight index = ``(layer * n + q) * R + r`` with
``R`` rotations per qubit and ``r`` the position in the listed order.
Feature ``f`` is encoded on qubit ``f``.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np

H, RX, RY, RZ, CNOT, CZ = 0, 1, 2, 3, 4, 5
CRX, CRY, CRZ, PAULI = 6, 7, 8, 9
SRC_NONE, SRC_INPUT, SRC_WEIGHT = 0, 1, 2
EMBED_NONE, EMBED_BASIS, EMBED_AMPLITUDE = 0, 1, 2
KIND_NAMES = {H: "H", RX: "RX", RY: "RY", RZ: "RZ", CNOT: "CNOT", CZ: "CZ", CRX: "CRX",
              CRY: "CRY", CRZ: "CRZ", PAULI: "PAULI"}
ROTATIONS = (RX, RY, RZ)
CONTROLLED = (CRX, CRY, CRZ)


def _g(kind, q0, q1=-1, src=SRC_NONE, index=0):
    return (kind, q0, q1, src, index)


def entangler_pairs(n: int, pattern: str):
    """Ordered (q0, q1) pairs of one entangling layer.

    ``ring``   -- (0,1), (1,2), ..., (n-2,n-1), (n-1,0)
    ``linear`` -- (0,1), ..., (n-2,n-1)
    ``brick``  -- even pairs (0,1), (2,3), ... then odd pairs (1,2), (3,4), ...
    """
    if pattern == "linear":
        return [(q, q + 1) for q in range(n - 1)]
    if pattern == "ring":
        pairs = [(q, q + 1) for q in range(n - 1)]
        if n > 2:
            pairs.append((n - 1, 0))
        return pairs
    if pattern == "brick":
        return [(q, q + 1) for q in range(0, n - 1, 2)] + \
               [(q, q + 1) for q in range(1, n - 1, 2)]
    raise ValueError(f"unknown entangler pattern {pattern!r}")


def layered_circuit(n, encoding, layers, rotations, entangler, pattern):
    """Gate array for: encoding, then ``layers`` x (rotations per qubit, entangler).

    ``encoding`` is ``"ry"`` (RY(x_q) on qubit q) or ``"h_rz"`` (H on every
    qubit, then RZ(x_q) on qubit q). ``entangler`` is ``CNOT``, ``CZ`` or
    ``None``.
    """
    gates = []
    if encoding == "ry":
        gates += [_g(RY, q, -1, SRC_INPUT, q) for q in range(n)]
    elif encoding == "h_rz":
        gates += [_g(H, q) for q in range(n)]
        gates += [_g(RZ, q, -1, SRC_INPUT, q) for q in range(n)]
    else:
        raise ValueError(encoding)
    R = len(rotations)
    for layer in range(layers):
        for q in range(n):
            for r, kind in enumerate(rotations):
                gates.append(_g(kind, q, -1, SRC_WEIGHT, (layer * n + q) * R + r))
        if entangler is not None:
            gates += [_g(entangler, a, b) for a, b in entangler_pairs(n, pattern)]
    return np.asarray(gates, dtype=np.int32).reshape(-1, 5)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic quantum-layer workload (circuit + batch + dtype + seed)."""
    name: str
    n: int            # qubits
    batch: int        # samples
    dtype: str        # "c64" or "c128"
    encoding: str     # "ry" | "h_rz"
    input_dist: str   # "uniform_0_pi" | "normal"
    layers: int
    rotations: tuple
    entangler: int | None
    pattern: str
    seed: int

    @property
    def n_inputs(self) -> int:
        return self.n

    @property
    def n_weights(self) -> int:
        return self.layers * self.n * len(self.rotations)

    def gates(self) -> np.ndarray:
        return layered_circuit(self.n, self.encoding, self.layers, self.rotations,
                               self.entangler, self.pattern)

    @property
    def n_gates(self) -> int:
        return int(self.gates().shape[0])

    def updates(self) -> int:
        """Amplitude-gate updates of one fused forward + adjoint call.

        The forward applies every gate to psi; the backward un-applies every
        gate on psi and on lambda: 3 * G * B * 2^n.
        """
        return 3 * self.n_gates * self.batch * (1 << self.n)

    def inputs(self):
        """Seeded ``(inputs[B,F], weights[P], grad_out[B,n])``.

        Draw order: inputs, weights, then u ~ U[-1, 1]; grad_out = u / B (the
        upstream gradient of a batch-mean loss). Arrays are float32 for
        complex64 workloads (the values both sides consume) and float64 for
        complex128 ones.
        """
        rng = np.random.default_rng(self.seed)
        B, F, P, n = self.batch, self.n_inputs, self.n_weights, self.n
        if self.input_dist == "uniform_0_pi":
            x = rng.uniform(0.0, math.pi, size=(B, F))
        elif self.input_dist == "normal":
            x = rng.standard_normal(size=(B, F))
        else:
            raise ValueError(self.input_dist)
        w = rng.uniform(-math.pi, math.pi, size=P)
        u = rng.uniform(-1.0, 1.0, size=(B, n))
        g = u / B
        rdt = np.float32 if self.dtype == "c64" else np.float64
        return x.astype(rdt), w.astype(rdt), g.astype(rdt)


WORKLOADS = {
    "4q": Workload("4q_b8_c128", 4, 8, "c128", "ry", "uniform_0_pi", 2,
                   (RY, RZ), CNOT, "ring", 101),
    "10q": Workload("10q_b256_c64", 10, 256, "c64", "ry", "uniform_0_pi", 6,
                    (RX, RY, RZ), CNOT, "linear", 102),
    "16q": Workload("16q_b1024_c64", 16, 1024, "c64", "h_rz", "normal", 8,
                    (RY, RZ), CZ, "ring", 103),
    "24q": Workload("24q_b16_c64", 24, 16, "c64", "ry", "uniform_0_pi", 20,
                    (RX, RY, RZ), CNOT, "brick", 104),
    "30q": Workload("30q_b1_c64", 30, 1, "c64", "ry", "uniform_0_pi", 10,
                    (RY, RZ), CNOT, "linear", 105),
}


@dataclasses.dataclass(frozen=True)
class QAEWorkload:
    """The quantum-autoencoder layer of the paper's appendix ("Quantum
    Autoencoder"): 7 qubits = 4 training qubits (0..3), of which 2 are trash
    (2, 3), plus 1 auxiliary (4) and 2 reference (5, 6) qubits; 60 weights =
    a Rot on each training qubit (12), a controlled Rot on every ordered pair
    of training qubits (12 pairs, 36), and a Rot on each training qubit (12).
    Rot(a, b, c) is RZ(a), RY(b), RZ(c) in that order; the controlled Rot is
    CRZ, CRY, CRZ with the pair's first qubit as control.

    Input states: the paper compresses ground states of Hubbard and molecular
    Hamiltonians, which are not available; seeded random real 16-dimensional
    states on the training qubits stand in for them, given as an amplitude
    embedding of 2^7 features (zero off the training subspace). Output: <Z>
    of every qubit; the trash qubits' <Z> give the compression cost
    sum_t (1 - <Z_t>) / 2 (the swap test against |0> references measures the
    same populations)."""
    name: str = "qae7_b256_c64"
    n: int = 7
    batch: int = 256
    dtype: str = "c64"
    seed: int = 107
    n_train: int = 4

    @property
    def n_inputs(self) -> int:
        return 1 << self.n

    @property
    def n_weights(self) -> int:
        t = self.n_train
        return 3 * t + 3 * t * (t - 1) + 3 * t

    @property
    def embed(self):
        return (EMBED_AMPLITUDE, 0)

    def gates(self) -> np.ndarray:
        t = self.n_train
        gates, w = [], 0
        for rng_ in ("begin", "pairs", "end"):
            if rng_ == "pairs":
                for c in range(t):
                    for q in range(t):
                        if c == q:
                            continue
                        for kind in (CRZ, CRY, CRZ):
                            gates.append(_g(kind, c, q, SRC_WEIGHT, w))
                            w += 1
            else:
                for q in range(t):
                    for kind in (RZ, RY, RZ):
                        gates.append(_g(kind, q, -1, SRC_WEIGHT, w))
                        w += 1
        return np.asarray(gates, dtype=np.int32).reshape(-1, 5)

    @property
    def n_gates(self) -> int:
        return int(self.gates().shape[0])

    def updates(self) -> int:
        """3 * G * B * 2^n with G the gates as listed (a controlled rotation is one)."""
        return 3 * self.n_gates * self.batch * (1 << self.n)

    def inputs(self):
        """Seeded ``(inputs[B, 2^n], weights[60], grad_out[B, n])``: a standard
        normal 16-vector per sample in features 0..15 (normalised by the
        embedding), weights U[-pi, pi], grad_out = u / B with u ~ U[-1, 1]."""
        rng = np.random.default_rng(self.seed)
        B, n = self.batch, self.n
        x = np.zeros((B, 1 << n))
        x[:, :1 << self.n_train] = rng.standard_normal((B, 1 << self.n_train))
        w = rng.uniform(-math.pi, math.pi, size=self.n_weights)
        g = rng.uniform(-1.0, 1.0, size=(B, n)) / B
        rdt = np.float32 if self.dtype == "c64" else np.float64
        return x.astype(rdt), w.astype(rdt), g.astype(rdt)


def with_depolarizing(gates, n_qubits: int, n_inputs: int, p: float, every: int = 1):
    """Insert a depolarizing-channel trajectory (X, Y, Z with p/3 each) on every
    qubit after every ``every``-th gate. Channel c reads its uniform from input
    feature ``n_inputs + c``. Returns ``(gates, pauli_p, n_channels)``."""
    out, pp = [], []
    for i, g in enumerate(np.asarray(gates).tolist()):
        out.append(g)
        if (i + 1) % every == 0:
            for q in range(n_qubits):
                out.append(_g(PAULI, q, -1, SRC_INPUT, n_inputs + len(pp)))
                pp.append([p / 3, p / 3, p / 3])
    return np.asarray(out, dtype=np.int32).reshape(-1, 5), np.asarray(pp, dtype=np.float64).reshape(-1, 3), len(pp)


def get(name: str):
    if name == "qae":
        return QAEWorkload()
    return WORKLOADS[name]


def scaled(w: Workload, **changes) -> Workload:
    """Same circuit family with some fields replaced (e.g. fewer qubits)."""
    return dataclasses.replace(w, **changes)


def random_circuit(n: int, n_gates: int, n_inputs: int, n_weights: int, seed: int,
                   kinds=(H, RX, RY, RZ, CNOT, CZ)) -> np.ndarray:
    """Seeded random gate list over every gate kind, qubit and binding."""
    rng = np.random.default_rng(seed)
    gates = []
    for _ in range(n_gates):
        kind = int(kinds[rng.integers(len(kinds))])
        if kind in (CNOT, CZ) + CONTROLLED:
            if n < 2:
                kind = H
            else:
                a, b = rng.choice(n, size=2, replace=False)
                if kind in (CNOT, CZ):
                    gates.append(_g(kind, int(a), int(b)))
                elif n_inputs > 0 and (n_weights == 0 or rng.random() < 0.4):
                    gates.append(_g(kind, int(a), int(b), SRC_INPUT, int(rng.integers(n_inputs))))
                else:
                    gates.append(_g(kind, int(a), int(b), SRC_WEIGHT, int(rng.integers(n_weights))))
                continue
        q = int(rng.integers(n))
        if kind == H:
            gates.append(_g(H, q))
        elif kind == PAULI:
            gates.append(_g(PAULI, q, -1, SRC_INPUT, int(rng.integers(n_inputs))))
        else:
            use_input = n_inputs > 0 and (n_weights == 0 or rng.random() < 0.4)
            if use_input:
                gates.append(_g(kind, q, -1, SRC_INPUT, int(rng.integers(n_inputs))))
            else:
                gates.append(_g(kind, q, -1, SRC_WEIGHT, int(rng.integers(n_weights))))
    return np.asarray(gates, dtype=np.int32).reshape(-1, 5)


def random_inputs(B: int, F: int, P: int, n: int, seed: int, dtype: str = "c128"):
    """Seeded ``(inputs, weights, grad_out)`` with angles in [-pi, pi]."""
    rng = np.random.default_rng(seed)
    x = rng.uniform(-math.pi, math.pi, size=(B, F))
    w = rng.uniform(-math.pi, math.pi, size=P)
    g = rng.uniform(-1.0, 1.0, size=(B, n)) / max(B, 1)
    rdt = np.float32 if dtype == "c64" else np.float64
    return x.astype(rdt), w.astype(rdt), g.astype(rdt)
