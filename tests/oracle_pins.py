"""Pins of the CPU oracle against facts fixed outside the oracle.

Each ``pin_*`` takes an oracle handle (``oracle.Oracle``) and raises
AssertionError when the oracle disagrees with a closed form, a dense
brute-force model (``brute.py``), an invariant of unitary evolution, or a
derivative computed another way. ``test_oracle_pins.py`` runs them against the
real oracle; ``test_oracle_mutants.py`` runs them against deliberately broken
copies of the oracle to show each plausible mistake fails at least one pin.
"""

from __future__ import annotations

import math

import numpy as np

import brute
import workloads as W

TOL = 1e-12


def _g(kind, q0, q1=-1, src=W.SRC_NONE, index=0):
    return [kind, q0, q1, src, index]


def _arr(gs):
    return np.asarray(gs, dtype=np.int32).reshape(-1, 5)


def _close(a, b, tol=TOL, what=""):
    a = np.asarray(a, dtype=np.complex128)
    b = np.asarray(b, dtype=np.complex128)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.1e}"


THETAS = np.array([-2.9, -1.3, -0.4, 0.0, 0.35, 1.1, 2.2, 3.0])


# --------------------------------------------------------------------------
# one-qubit closed forms (Bloch-sphere rotations)

def pin_rotations_on_zero(orc):
    """RX(t)|0> and RY(t)|0> give <Z> = cos t, d<Z>/dt = -sin t; RZ leaves |0> alone."""
    for kind in (W.RX, W.RY, W.RZ):
        gates = _arr([_g(kind, 0, -1, W.SRC_WEIGHT, 0)])
        for t in THETAS:
            r = orc.run(1, gates, np.zeros((1, 0)), [t], grad_out=[[1.0]])
            want = 1.0 if kind == W.RZ else math.cos(t)
            dwant = 0.0 if kind == W.RZ else -math.sin(t)
            _close(r["expz"][0, 0], want, what=f"{W.KIND_NAMES[kind]} <Z>")
            _close(r["grad_weights"][0], dwant, what=f"{W.KIND_NAMES[kind]} grad")


def pin_rotation_axes(orc):
    """H, RZ(phi), then RX(t) or RY(t): Bloch vector (cos phi, sin phi, 0) rotated.

    About x: <Z> = sin(phi) sin(t). About y: <Z> = -cos(phi) sin(t). These fix
    the axis and sense of each rotation and the relative phase RZ applies.
    """
    for phi in (-1.0, 0.3, 2.0):
        for t in THETAS:
            for kind, want in ((W.RX, math.sin(phi) * math.sin(t)),
                               (W.RY, -math.cos(phi) * math.sin(t))):
                gates = _arr([_g(W.H, 0), _g(W.RZ, 0, -1, W.SRC_INPUT, 0),
                              _g(kind, 0, -1, W.SRC_WEIGHT, 0)])
                r = orc.run(1, gates, [[phi]], [t], grad_out=[[1.0]])
                _close(r["expz"][0, 0], want, what=f"axis {W.KIND_NAMES[kind]}")
                if kind == W.RX:
                    dphi, dt = math.cos(phi) * math.sin(t), math.sin(phi) * math.cos(t)
                else:
                    dphi, dt = math.sin(phi) * math.sin(t), -math.cos(phi) * math.cos(t)
                _close(r["grad_inputs"][0, 0], dphi, what="d/dphi")
                _close(r["grad_weights"][0], dt, what="d/dt")


def pin_h_rz_h(orc):
    """H RZ(t) H |0> is RX(t)|0> up to a phase: <Z> = cos t."""
    gates = _arr([_g(W.H, 0), _g(W.RZ, 0, -1, W.SRC_WEIGHT, 0), _g(W.H, 0)])
    for t in THETAS:
        r = orc.run(1, gates, np.zeros((1, 0)), [t], grad_out=[[1.0]])
        _close(r["expz"][0, 0], math.cos(t), what="H RZ H")
        _close(r["grad_weights"][0], -math.sin(t), what="H RZ H grad")


def pin_hybrid_node(orc):
    """The paper's hybrid network node (appendix on hybrid quantum-classical
    networks): one qubit, H then RY(input).

    <Z> = -sin t, so P(1) = (1 + sin t) / 2. The node's backward takes the
    difference of P(1) at t +- pi/2 without a 1/2 factor, which is cos t; the
    exact derivative d<Z>/dt is -cos t.
    """
    gates = _arr([_g(W.H, 0), _g(W.RY, 0, -1, W.SRC_INPUT, 0)])
    for t in THETAS:
        r = orc.run(1, gates, [[t]], [], grad_out=[[1.0]])
        _close(r["expz"][0, 0], -math.sin(t), what="hybrid node <Z>")
        _close(r["grad_inputs"][0, 0], -math.cos(t), what="hybrid node grad")
        p1 = [(1.0 - orc.run(1, gates, [[t + s]], [])["expz"][0, 0]) / 2.0
              for s in (math.pi / 2, -math.pi / 2)]
        _close(p1[0] - p1[1], math.cos(t), what="hybrid node shifted difference")


def pin_shared_parameter(orc):
    """The paper's compatibility example: H on every qubit, then RY(t) on every
    qubit with ONE shared parameter. <Z_i> = -sin t for all i and
    d/dt sum_i <Z_i> = -n cos t (every occurrence of the parameter adds up)."""
    for n in (1, 3, 5):
        gates = _arr([_g(W.H, q) for q in range(n)] +
                     [_g(W.RY, q, -1, W.SRC_WEIGHT, 0) for q in range(n)])
        for t in THETAS[::2]:
            r = orc.run(n, gates, np.zeros((1, 0)), [t], grad_out=np.ones((1, n)))
            _close(r["expz"][0], np.full(n, -math.sin(t)), what="shared <Z>")
            _close(r["grad_weights"][0], -n * math.cos(t), what="shared grad")


# --------------------------------------------------------------------------
# two-qubit gates: truth tables and entanglement

def _basis_prep(bits):
    """RY(pi) on each set bit: maps |0> to |1> (a real rotation, no phase issue)."""
    return [_g(W.RY, q, -1, W.SRC_INPUT, 0) for q, b in enumerate(bits) if b]


def pin_cnot_truth_table(orc):
    """CNOT(c, t) on every basis state of 3 qubits flips bit t iff bit c is 1."""
    n = 3
    for c in range(n):
        for t in range(n):
            if c == t:
                continue
            for v in range(1 << n):
                bits = [(v >> q) & 1 for q in range(n)]
                gates = _arr(_basis_prep(bits) + [_g(W.CNOT, c, t)])
                r = orc.run(n, gates, [[math.pi]], [])
                out = list(bits)
                out[t] ^= bits[c]
                _close(r["expz"][0], [1 - 2 * b for b in out], tol=1e-12,
                       what=f"CNOT({c},{t}) on {bits}")


def pin_cnot_chain_parity(orc):
    """A linear CNOT chain (0,1), (1,2), ... writes prefix parities into each bit."""
    n = 4
    for v in range(1 << n):
        bits = [(v >> q) & 1 for q in range(n)]
        gates = _arr(_basis_prep(bits) + [_g(W.CNOT, q, q + 1) for q in range(n - 1)])
        r = orc.run(n, gates, [[math.pi]], [])
        pref = np.cumsum(bits) % 2
        _close(r["expz"][0], 1 - 2 * pref, what=f"chain on {bits}")


def pin_cz_kickback(orc):
    """H(t) CZ(c, t) H(t) acts as CNOT(c, t) (truth table); CZ is symmetric."""
    n = 2
    for c, t in ((0, 1), (1, 0)):
        for v in range(4):
            bits = [(v >> q) & 1 for q in range(n)]
            for a, b in ((c, t), (t, c)):
                gates = _arr(_basis_prep(bits) + [_g(W.H, t), _g(W.CZ, a, b), _g(W.H, t)])
                r = orc.run(n, gates, [[math.pi]], [])
                out = list(bits)
                out[t] ^= bits[c]
                _close(r["expz"][0], [1 - 2 * x for x in out], what=f"CZ kickback {bits}")


def pin_bell(orc):
    """H(0) CNOT(0,1): (|00> + |11>)/sqrt2, so <Z0> = <Z1> = 0 and <Z0 Z1> = 1.
    RY(t) on 0 then CNOT(0,1): <Z0> = <Z1> = cos t. RY(t) on the target only:
    <Z0> = 1, <Z1> = cos t."""
    r = orc.run(2, _arr([_g(W.H, 0), _g(W.CNOT, 0, 1)]), np.zeros((1, 0)), [], want_state=True)
    _close(r["expz"][0], [0.0, 0.0], what="Bell <Z>")
    psi = r["state"][0]
    zz = np.sum(np.abs(psi) ** 2 * np.array([1, -1, -1, 1]))
    _close(zz, 1.0, what="Bell <ZZ>")
    _close(psi, np.array([1, 0, 0, 1]) / math.sqrt(2), what="Bell state")
    for t in THETAS:
        r = orc.run(2, _arr([_g(W.RY, 0, -1, W.SRC_WEIGHT, 0), _g(W.CNOT, 0, 1)]),
                    np.zeros((1, 0)), [t])
        _close(r["expz"][0], [math.cos(t)] * 2, what="RY then CNOT")
        r = orc.run(2, _arr([_g(W.RY, 1, -1, W.SRC_WEIGHT, 0), _g(W.CNOT, 0, 1)]),
                    np.zeros((1, 0)), [t])
        _close(r["expz"][0], [1.0, math.cos(t)], what="target-only RY then CNOT")


# --------------------------------------------------------------------------
# brute force and invariants

def _random_case(n, G, seed, B=2, F=3, P=4):
    gates = W.random_circuit(n, G, F, P, seed)
    x, w, g = W.random_inputs(B, F, P, n, seed + 1)
    return gates, x, w, g


def pin_brute_force(orc):
    """Random circuits on 1..4 qubits over every gate kind: states, <Z_i> and VJP
    gradients equal the dense Kronecker-product model within 1e-12."""
    for n in (1, 2, 3, 4):
        for seed in range(3):
            gates, x, w, g = _random_case(n, 14, 1000 * n + seed)
            r = orc.run(n, gates, x, w, grad_out=g, want_state=True)
            b = brute.run(n, gates, x, w, grad_out=g)
            _close(r["state"], b["state"], what=f"brute state n={n}")
            _close(r["expz"], b["expz"], what=f"brute expz n={n}")
            _close(r["grad_inputs"], b["grad_inputs"], what=f"brute grad_x n={n}")
            _close(r["grad_weights"], b["grad_weights"], what=f"brute grad_w n={n}")


def pin_unitarity(orc):
    """Norm is preserved, un-applying every gate returns psi to |0...0>, and
    lambda[0] at the end of the sweep equals sum_i g_i <Z_i> (because
    <e0| U^dag O U |e0> = <O>)."""
    for n in (3, 6):
        gates, x, w, g = _random_case(n, 40, 77 + n, B=3)
        r = orc.run(n, gates, x, w, grad_out=g, want_state=True, want_back=True)
        _close(np.sum(np.abs(r["state"]) ** 2, axis=1), np.ones(3), what="norm")
        e0 = np.zeros((3, 1 << n))
        e0[:, 0] = 1
        _close(r["back_psi"], e0, what="inverse sweep")
        _close(r["back_lam0"], np.sum(g * r["expz"], axis=1), what="lambda_0[0]")


def pin_param_shift(orc):
    """Adjoint VJP equals the two-term parameter-shift rule (exact for
    exp(-i t P / 2)), on random circuits and on the 4-qubit workload."""
    for n, seed in ((3, 5), (5, 6)):
        gates, x, w, g = _random_case(n, 30, seed)
        r = orc.run(n, gates, x, w, grad_out=g)
        gi, gw = orc.param_shift(n, gates, x, w, g)
        _close(r["grad_inputs"], gi, tol=1e-12, what="shift grad_x")
        _close(r["grad_weights"], gw, tol=1e-12, what="shift grad_w")
    wl = W.get("4q")
    x, w, g = wl.inputs()
    r = orc.run(wl.n, wl.gates(), x, w, grad_out=g)
    gi, gw = orc.param_shift(wl.n, wl.gates(), x, w, g)
    _close(r["grad_inputs"], gi, what="4q shift grad_x")
    _close(r["grad_weights"], gw, what="4q shift grad_w")


def pin_finite_difference(orc):
    """Central differences (h = 1e-5) of sum_i g_i <Z_i> match the VJP to ~1e-9."""
    n = 4
    gates, x, w, g = _random_case(n, 24, 31, B=2)
    r = orc.run(n, gates, x, w, grad_out=g)
    h = 1e-5

    def f(xx, ww):
        return float(np.sum(g * orc.run(n, gates, xx, ww)["expz"]))

    for p in range(w.size):
        wp, wm = w.astype(np.float64), w.astype(np.float64)
        wp[p] += h
        wm[p] -= h
        _close((f(x, wp) - f(x, wm)) / (2 * h), r["grad_weights"][p], tol=1e-8, what="fd w")
    for b in range(x.shape[0]):
        for k in range(x.shape[1]):
            xp, xm = x.astype(np.float64), x.astype(np.float64)
            xp[b, k] += h
            xm[b, k] -= h
            # only sample b depends on x[b]; the other rows cancel
            _close((f(xp, w) - f(xm, w)) / (2 * h), r["grad_inputs"][b, k], tol=1e-8, what="fd x")


def pin_vjp_structure(orc):
    """VJP is linear in grad_out; weight gradients add over the batch; one-hot
    grad_out gives one Jacobian row."""
    n = 4
    gates, x, w, g = _random_case(n, 30, 41, B=3)
    g2 = np.roll(g, 1, axis=1) * 0.7
    r1 = orc.run(n, gates, x, w, grad_out=g)
    r2 = orc.run(n, gates, x, w, grad_out=g2)
    r12 = orc.run(n, gates, x, w, grad_out=2.0 * g - 3.0 * g2)
    _close(r12["grad_weights"], 2 * r1["grad_weights"] - 3 * r2["grad_weights"], what="linear w")
    _close(r12["grad_inputs"], 2 * r1["grad_inputs"] - 3 * r2["grad_inputs"], what="linear x")
    acc = np.zeros_like(r1["grad_weights"])
    for b in range(3):
        rb = orc.run(n, gates, x[b:b + 1], w, grad_out=g[b:b + 1])
        acc += rb["grad_weights"]
        _close(rb["grad_inputs"][0], r1["grad_inputs"][b], what="per-sample x")
        _close(rb["expz"][0], r1["expz"][b], what="per-sample expz")
    _close(acc, r1["grad_weights"], what="batch additivity")
    # Jacobian row q from a one-hot grad_out vs the brute-force derivative
    for q in range(n):
        oh = np.zeros((1, n))
        oh[0, q] = 1.0
        ro = orc.run(n, gates, x[:1], w, grad_out=oh)
        bo = brute.run(n, gates, x[:1], w, grad_out=oh)
        _close(ro["grad_weights"], bo["grad_weights"], what="jacobian row")


# --------------------------------------------------------------------------
# product states at larger n: SO(3) closed form per qubit

def _so3(kind, t):
    c, s = math.cos(t), math.sin(t)
    if kind == W.RX:
        return np.array([[1, 0, 0], [0, c, -s], [0, s, c]])
    if kind == W.RY:
        return np.array([[c, 0, s], [0, 1, 0], [-s, 0, c]])
    if kind == W.RZ:
        return np.array([[c, -s, 0], [s, c, 0], [0, 0, 1]])
    if kind == W.H:  # x <-> z, y -> -y
        return np.array([[0, 0, 1], [0, -1, 0], [1, 0, 0]], dtype=float)
    raise ValueError(kind)


def _so3_gen(kind):
    return {W.RX: np.array([[0, 0, 0], [0, 0, -1], [0, 1, 0]]),
            W.RY: np.array([[0, 0, 1], [0, 0, 0], [-1, 0, 0]]),
            W.RZ: np.array([[0, -1, 0], [1, 0, 0], [0, 0, 0]])}[kind]


def product_state_reference(n, gates, x_b, w, g_b):
    """Closed form for circuits with no two-qubit gates: each qubit's Bloch
    vector starts at (0,0,1) and is rotated by SO(3) matrices; <Z_q> is its z
    component, and d<Z_q>/dt inserts the rotation generator at that gate."""
    F, P = len(x_b), len(w)
    expz = np.zeros(n)
    gx = np.zeros(F)
    gw = np.zeros(P)
    for q in range(n):
        seq = [(int(gg[0]), (x_b[gg[4]] if gg[3] == W.SRC_INPUT else w[gg[4]] if gg[3] == W.SRC_WEIGHT else 0.0),
                int(gg[3]), int(gg[4])) for gg in gates if int(gg[1]) == q]
        mats = [_so3(k, t) for k, t, _, _ in seq]
        v = np.array([0.0, 0.0, 1.0])
        for m in mats:
            v = m @ v
        expz[q] = v[2]
        for i, (k, t, src, idx) in enumerate(seq):
            if k == W.H:
                continue
            u = np.array([0.0, 0.0, 1.0])
            for j, m in enumerate(mats):
                u = (_so3_gen(k) @ m if j == i else m) @ u
            if src == W.SRC_WEIGHT:
                gw[idx] += g_b[q] * u[2]
            else:
                gx[idx] += g_b[q] * u[2]
    return expz, gx, gw


def pin_product_states(orc):
    """Workload-shaped circuits with the entanglers removed (n = 8 and 11)
    against the per-qubit SO(3) closed form."""
    for name, n in (("24q", 8), ("16q", 11), ("10q", 9)):
        wl = W.scaled(W.get(name), n=n, batch=2, layers=3, entangler=None, dtype="c128")
        x, w, g = wl.inputs()
        gates = wl.gates()
        r = orc.run(n, gates, x, w, grad_out=g)
        for b in range(2):
            e, gx, gw = product_state_reference(n, gates, x[b], w, g[b])
            _close(r["expz"][b], e, tol=1e-12, what=f"{name} product expz")
            _close(r["grad_inputs"][b], gx, tol=1e-12, what=f"{name} product grad_x")
        gw_all = sum(product_state_reference(n, gates, x[b], w, g[b])[2] for b in range(2))
        _close(r["grad_weights"], gw_all, tol=1e-12, what=f"{name} product grad_w")


def pin_cyclic_shift(orc):
    """The ring-CZ workload family is symmetric under relabelling q -> q+1 mod n:
    shifting features, per-qubit weights and grad_out shifts every output."""
    n = 6
    wl = W.scaled(W.get("16q"), n=n, batch=2, layers=2, dtype="c128")
    x, w, g = wl.inputs()
    gates = wl.gates()
    R = len(wl.rotations)
    r = orc.run(n, gates, x, w, grad_out=g)
    xs = np.roll(x, 1, axis=1)
    gs = np.roll(g, 1, axis=1)
    ws = np.roll(w.reshape(wl.layers, n, R), 1, axis=1).reshape(-1)
    rs = orc.run(n, gates, xs, ws, grad_out=gs)
    _close(rs["expz"], np.roll(r["expz"], 1, axis=1), tol=1e-12, what="shift expz")
    _close(rs["grad_inputs"], np.roll(r["grad_inputs"], 1, axis=1), tol=1e-12, what="shift gx")
    _close(rs["grad_weights"],
           np.roll(r["grad_weights"].reshape(wl.layers, n, R), 1, axis=1).reshape(-1),
           tol=1e-12, what="shift gw")


def pin_sampling(orc):
    """Shot sampling against what the definition of sampling fixes, without
    re-deriving the CDF: a basis state always returns itself; a uniform
    superposition with stratified uniforms (i + 1/2) / 2^n returns i; one RY(t)
    qubit returns 0 exactly for u < cos^2(t/2); u = 0 returns the first index of
    nonzero probability (never a zero-probability one); a state and twice that
    state give the same shots; and the frequencies of many shots of a random
    state match |psi|^2 within five standard errors."""
    n = 4
    dim = 1 << n
    for j in (0, 5, dim - 1):
        e = np.zeros((1, dim), np.complex128)
        e[0, j] = 1.0
        got = orc.sample(n, e, np.linspace(0.0, 0.999, 9)[None, :])
        assert np.all(got == j), f"basis state {j}: {got}"
    uni = np.full((1, dim), 1.0 / np.sqrt(dim), np.complex128)
    got = orc.sample(n, uni, ((np.arange(dim) + 0.5) / dim)[None, :])
    assert np.array_equal(got[0], np.arange(dim)), f"stratified uniform: {got}"
    for t in (0.3, 1.7, 2.9):
        st = orc.run(1, _arr([_g(W.RY, 0, src=W.SRC_WEIGHT)]), np.zeros((1, 0)), [t], want_state=True)["state"]
        p0 = np.cos(t / 2) ** 2
        u = np.array([[p0 - 1e-9, p0 + 1e-9, 0.0, 0.999999]])
        got = orc.sample(1, st, u)[0]
        assert list(got) == [0, 1, 0, 1], f"RY({t}) threshold: {got}"
    st = np.zeros((1, dim), np.complex128)
    st[0, 3] = 0.6
    st[0, 9] = 0.8j
    got = orc.sample(n, st, np.array([[0.0, 0.35, 0.36, 0.999]]))[0]
    assert list(got) == [3, 3, 9, 9], f"zero-probability skip: {got}"
    gates, x, w, _ = _random_case(n, 30, seed=44, B=1)
    psi = orc.run(n, gates, x, w, want_state=True)["state"]
    p = np.abs(psi[0]) ** 2
    rng = np.random.default_rng(45)
    shots = 200000
    got = orc.sample(n, psi, rng.random((1, shots)))[0]
    # scale invariance: sampling reads |psi|^2 relative to the state's norm
    us = rng.random((1, 64))
    assert np.array_equal(orc.sample(n, 2.0 * psi, us), orc.sample(n, psi, us)), "norm-dependent shots"
    freq = np.bincount(got, minlength=dim) / shots
    se = np.sqrt(p * (1 - p) / shots) + 1e-12
    assert np.all(np.abs(freq - p) <= 5 * se + 1e-9), "shot frequencies do not follow |psi|^2"


# --------------------------------------------------------------------------
# controlled rotations (the quantum autoencoder's controlled gates)

def _wrap_crz(kind):
    """CRZ acts on the phase; H before and after turns it into a population change."""
    return ([_g(W.H, 1)], [_g(W.H, 1)]) if kind == W.CRZ else ([], [])


def pin_controlled_rotation_closed_forms(orc):
    """Control |0>: the target keeps <Z> = 1 and the gradient is 0. Control |1>
    (prepared by RY(pi)): CRX(t), CRY(t) and H CRZ(t) H give <Z_t> = cos t with
    derivative -sin t. Control |+> (H): <Z_t> = (1 + cos t) / 2, derivative
    -sin(t) / 2, and the control keeps <Z> = 0."""
    for kind in W.CONTROLLED:
        pre, post = _wrap_crz(kind)
        cr = [_g(kind, 0, 1, W.SRC_WEIGHT, 0)]
        for t in THETAS:
            name = W.KIND_NAMES[kind]
            r = orc.run(2, _arr(pre + cr + post), np.zeros((1, 1)), [t], grad_out=[[0.0, 1.0]])
            _close(r["expz"][0, 1], 1.0, what=f"{name} control 0")
            _close(r["grad_weights"][0], 0.0, what=f"{name} control 0 grad")
            r = orc.run(2, _arr([_g(W.RY, 0, -1, W.SRC_INPUT, 0)] + pre + cr + post),
                        np.array([[math.pi]]), [t], grad_out=[[0.0, 1.0]])
            _close(r["expz"][0, 1], math.cos(t), what=f"{name} control 1")
            _close(r["grad_weights"][0], -math.sin(t), what=f"{name} control 1 grad")
            r = orc.run(2, _arr([_g(W.H, 0)] + pre + cr + post), np.zeros((1, 1)), [t],
                        grad_out=[[0.0, 1.0]])
            _close(r["expz"][0], [0.0, 0.5 * (1 + math.cos(t))], what=f"{name} control +")
            _close(r["grad_weights"][0], -0.5 * math.sin(t), what=f"{name} control + grad")


def pin_controlled_rotation_brute_force(orc):
    """Random circuits with controlled rotations on 2..4 qubits: states, <Z_i>
    and gradients equal the dense model P0 (x) I + P1 (x) exp(-i t P / 2)."""
    kinds = (W.H, W.RY, W.RZ, W.CNOT, W.CRX, W.CRY, W.CRZ)
    for n in (2, 3, 4):
        for seed in range(2):
            gates = W.random_circuit(n, 16, 3, 4, 500 * n + seed, kinds=kinds)
            x, w, g = W.random_inputs(2, 3, 4, n, 500 * n + seed + 7)
            r = orc.run(n, gates, x, w, grad_out=g, want_state=True)
            b = brute.run(n, gates, x, w, grad_out=g)
            _close(r["state"], b["state"], what=f"crot brute state n={n}")
            _close(r["expz"], b["expz"], what=f"crot brute expz n={n}")
            _close(r["grad_inputs"], b["grad_inputs"], what=f"crot brute grad_x n={n}")
            _close(r["grad_weights"], b["grad_weights"], what=f"crot brute grad_w n={n}")


def pin_controlled_rotation_decomposition(orc):
    """CRY(t) = RY(t/2) CNOT RY(-t/2) CNOT, CRZ likewise with RZ, and CRX(t) =
    RX(t/2) CZ RX(-t/2) CZ (X RY(a) X = RY(-a), X RZ(a) X = RZ(-a), Z RX(a) Z =
    RX(-a)): the same final states inside a random circuit, and the gradient of
    t equals (g(t/2) - g(-t/2)) / 2 from the two half-angle rotations."""
    n = 3
    for kind, rot, ent in ((W.CRX, W.RX, W.CZ), (W.CRY, W.RY, W.CNOT), (W.CRZ, W.RZ, W.CNOT)):
        pre = W.random_circuit(n, 8, 1, 2, 61 + kind, kinds=(W.H, W.RX, W.RY, W.CNOT)).tolist()
        post = W.random_circuit(n, 8, 1, 2, 71 + kind, kinds=(W.H, W.RZ, W.RY, W.CZ)).tolist()
        t = 1.234
        x, w, g = W.random_inputs(1, 1, 2, n, 81)
        wc = np.concatenate([w, [t]])
        full = _arr(pre + [_g(kind, 2, 0, W.SRC_WEIGHT, 2)] + post)
        wd = np.concatenate([w, [0.5 * t, -0.5 * t]])
        dec = _arr(pre + [_g(rot, 0, -1, W.SRC_WEIGHT, 2), _g(ent, 2, 0), _g(rot, 0, -1, W.SRC_WEIGHT, 3),
                          _g(ent, 2, 0)] + post)
        rc = orc.run(n, full, x, wc, grad_out=g, want_state=True)
        rd = orc.run(n, dec, x, wd, grad_out=g, want_state=True)
        _close(rc["state"], rd["state"], what=f"{W.KIND_NAMES[kind]} decomposition state")
        _close(rc["grad_weights"][2], 0.5 * (rd["grad_weights"][2] - rd["grad_weights"][3]),
               what=f"{W.KIND_NAMES[kind]} decomposition grad")
        _close(rc["grad_weights"][:2], rd["grad_weights"][:2], what="other weights")


def pin_controlled_rotation_shift_and_fd(orc):
    """Adjoint gradients of circuits with controlled rotations equal the
    four-term parameter-shift rule for generators with eigenvalues {0, +-1/2}
    (Anselmetti et al. 2021) and central differences (h = 1e-5)."""
    n = 3
    kinds = (W.H, W.RX, W.CNOT, W.CRX, W.CRY, W.CRZ)
    gates = W.random_circuit(n, 20, 2, 3, 91, kinds=kinds)
    x, w, g = W.random_inputs(2, 2, 3, n, 92)
    r = orc.run(n, gates, x, w, grad_out=g)
    gi, gw = orc.param_shift(n, gates, x, w, g)
    _close(r["grad_inputs"], gi, tol=1e-12, what="crot shift grad_x")
    _close(r["grad_weights"], gw, tol=1e-12, what="crot shift grad_w")
    h = 1e-5
    for p in range(w.size):
        wp, wm = w.copy(), w.copy()
        wp[p] += h
        wm[p] -= h
        fd = (np.sum(g * orc.run(n, gates, x, wp)["expz"]) - np.sum(g * orc.run(n, gates, x, wm)["expz"])) / (2 * h)
        _close(fd, r["grad_weights"][p], tol=1e-8, what="crot fd w")


# --------------------------------------------------------------------------
# initial-state embeddings (Sec. "Quantum Data")

def pin_basis_embedding(orc):
    """Basis embedding: qubit q is 1 where feature first + q is >= 0.5 (0.5
    itself counts as 1, just below does not); <Z_q> = 1 - 2 bit_q, and a
    circuit after it acts as on the basis state prepared by RY(pi) gates
    (RY(pi)|0> = |1> exactly)."""
    n = 4
    feats = np.array([[7.0, 0.5, 0.49999999, 1.0, 0.0, 3.0],
                      [7.0, 0.0, 1.0, 0.2, 0.7, 3.0]])
    bits = [[1, 0, 1, 0], [0, 1, 0, 1]]
    r = orc.run(n, _arr([]), feats, [], embed=(W.EMBED_BASIS, 1), want_state=True)
    for b in range(2):
        idx = sum(bits[b][q] << q for q in range(n))
        e = np.zeros(1 << n)
        e[idx] = 1
        _close(r["state"][b], e, what="basis state")
        _close(r["expz"][b], [1 - 2 * bits[b][q] for q in range(n)], what="basis <Z>")
    circ = W.random_circuit(n, 20, 1, 3, 33)
    x, w, g = W.random_inputs(2, 1, 3, n, 34)
    xe = np.concatenate([x, feats], axis=1)
    circ_e = circ.copy()
    r = orc.run(n, circ_e, xe, w, grad_out=g, embed=(W.EMBED_BASIS, 2), want_state=True)
    for b in range(2):
        prep = [_g(W.RY, q, -1, W.SRC_WEIGHT, 3) for q in range(n) if bits[b][q]]
        rb = orc.run(n, _arr(prep + circ.tolist()), x[b:b + 1], np.concatenate([w, [math.pi]]),
                     grad_out=g[b:b + 1], want_state=True)
        _close(r["state"][b], rb["state"][0], what="basis embedding then circuit")
        _close(r["grad_inputs"][b, :1], rb["grad_inputs"][0], what="basis embedding grad_x")
        _close(r["grad_inputs"][b, 1:], 0.0, what="no gradient for embedded bits")


def pin_amplitude_embedding(orc):
    """Amplitude embedding: psi_0 = x / |x| (so <Z_q> = sum x_j^2 (1 - 2 bit_q(j)) / |x|^2
    with no gates); with a circuit after it, states, <Z> and rotation gradients
    equal the dense model started from x / |x|; the zero vector gives <Z> = 0."""
    n = 3
    dim = 1 << n
    rng = np.random.default_rng(5)
    feats = rng.standard_normal((2, dim + 2))
    r = orc.run(n, _arr([]), feats, [], embed=(W.EMBED_AMPLITUDE, 1), want_state=True)
    for b in range(2):
        v = feats[b, 1:1 + dim]
        _close(r["state"][b], v / np.linalg.norm(v), what="amplitude state")
        want = [np.sum(v ** 2 * np.where((np.arange(dim) >> q) & 1, -1.0, 1.0)) / np.sum(v ** 2)
                for q in range(n)]
        _close(r["expz"][b], want, what="amplitude <Z>")
    circ = W.random_circuit(n, 24, 2, 3, 35)
    x, w, g = W.random_inputs(2, 2, 3, n, 36)
    xe = np.concatenate([x, feats], axis=1)
    r = orc.run(n, circ, xe, w, grad_out=g, embed=(W.EMBED_AMPLITUDE, 3), want_state=True)
    b_ = brute.run(n, circ, xe, w, grad_out=g, embed=(W.EMBED_AMPLITUDE, 3))
    _close(r["state"], b_["state"], what="amplitude brute state")
    _close(r["expz"], b_["expz"], what="amplitude brute expz")
    _close(r["grad_weights"], b_["grad_weights"], what="amplitude brute grad_w")
    _close(r["grad_inputs"][:, :2], b_["grad_inputs"][:, :2], what="amplitude brute grad_x (angles)")
    z = np.zeros((1, dim))
    r0 = orc.run(n, circ, np.concatenate([x[:1], z], axis=1), w, embed=(W.EMBED_AMPLITUDE, 2))
    _close(r0["expz"], 0.0, what="zero vector")


def pin_amplitude_embedding_gradient(orc):
    """Gradient with respect to the embedded features: central differences
    (h = 1e-6); f is invariant under x -> c x, so sum_j x_j df/dx_j = 0 (Euler)
    and the gradient of 3x is a third of that of x."""
    n = 3
    dim = 1 << n
    circ = W.random_circuit(n, 20, 1, 3, 37)
    x, w, g = W.random_inputs(2, 1, 3, n, 38)
    rng = np.random.default_rng(39)
    xe = np.concatenate([x, rng.standard_normal((2, dim))], axis=1)
    emb = (W.EMBED_AMPLITUDE, 1)
    r = orc.run(n, circ, xe, w, grad_out=g, embed=emb)
    h = 1e-6

    def f(xx):
        return float(np.sum(g * orc.run(n, circ, xx, w, embed=emb)["expz"]))

    for b in range(2):
        for j in range(1, 1 + dim):
            xp, xm = xe.copy(), xe.copy()
            xp[b, j] += h
            xm[b, j] -= h
            _close((f(xp) - f(xm)) / (2 * h), r["grad_inputs"][b, j], tol=1e-8, what="amplitude fd")
        _close(np.dot(xe[b, 1:], r["grad_inputs"][b, 1:]), 0.0, tol=1e-12, what="Euler homogeneity")
    x3 = xe.copy()
    x3[:, 1:] *= 3.0
    r3 = orc.run(n, circ, x3, w, grad_out=g, embed=emb)
    _close(r3["grad_inputs"][:, 1:], r["grad_inputs"][:, 1:] / 3.0, what="gradient of 3x")
    _close(r3["expz"], r["expz"], what="scale invariance")


# --------------------------------------------------------------------------
# Pauli-channel trajectories (noise-inclusive simulation)

def pin_pauli_trajectory_choices(orc):
    """With probabilities (1/8, 1/4, 3/8) a uniform below 1/8 applies X, [1/8, 3/8)
    Y, [3/8, 3/4) Z and the rest nothing (edges belong to the next bin): on |0>,
    X|0> = |1>, Y|0> = i|1>; on |+> (H), Z gives |->. The channel's uniform
    feature gets no gradient."""
    pp = [[0.125, 0.25, 0.375]]
    cases = [(0.0, 1), (0.124, 1), (0.125, 2), (0.374, 2), (0.375, 3), (0.749, 3), (0.75, 0), (0.99, 0)]
    for u, which in cases:
        r = orc.run(1, _arr([_g(W.PAULI, 0, -1, W.SRC_INPUT, 0)]), np.array([[u]]), [], want_state=True,
                    pauli_p=pp)
        want = {0: [1, 0], 1: [0, 1], 2: [0, 1j], 3: [1, 0]}[which]
        _close(r["state"][0], want, what=f"pauli u={u} on |0>")
        r = orc.run(1, _arr([_g(W.H, 0), _g(W.PAULI, 0, -1, W.SRC_INPUT, 0)]), np.array([[u]]), [],
                    want_state=True, pauli_p=pp)
        s2 = 1 / math.sqrt(2)
        want = {0: [s2, s2], 1: [s2, s2], 2: [-1j * s2, 1j * s2], 3: [s2, -s2]}[which]
        _close(r["state"][0], want, what=f"pauli u={u} on |+>")
    gates = _arr([_g(W.RY, 0, -1, W.SRC_WEIGHT, 0), _g(W.PAULI, 0, -1, W.SRC_INPUT, 0)])
    r = orc.run(1, gates, np.array([[0.2]]), [0.4], grad_out=[[1.0]], pauli_p=pp)
    _close(r["grad_inputs"], 0.0, what="no gradient for the uniform")
    _close(r["expz"][0, 0], -math.cos(0.4), what="Y flips <Z>")
    _close(r["grad_weights"][0], math.sin(0.4), what="gradient through the flip")


def _density_reference(n, gates, x_b, w, pauli_p):
    """<Z_q> of the channel-averaged state: rho -> U rho U^dag per gate and
    rho -> sum_k p_k P_k rho P_k + (1 - sum p) rho per channel."""
    dim = 1 << n
    rho = np.zeros((dim, dim), np.complex128)
    rho[0, 0] = 1
    ch = 0
    th = brute.angles(gates, x_b, w, [[0, 0, 0]] * len(pauli_p))
    for gt, t in zip(gates, th):
        if int(gt[0]) == W.PAULI:
            p = pauli_p[ch]
            ch += 1
            acc = (1 - sum(p)) * rho
            for k in range(3):
                P = brute.embed(n, {int(gt[1]): brute.PAULIS[k + 1]})
                acc = acc + p[k] * P @ rho @ P.conj().T
            rho = acc
        else:
            U = brute.gate_unitary(n, gt, t)
            rho = U @ rho @ U.conj().T
    return np.array([np.real(np.trace(brute.z_observable(n, q) @ rho)) for q in range(n)])


def pin_pauli_channel_average(orc):
    """Averaging the trajectories over every outcome of two channels, weighted by
    the outcome probabilities, gives the density-matrix expectation exactly."""
    n = 3
    base = W.random_circuit(n, 12, 1, 3, 95, kinds=(W.H, W.RX, W.RY, W.CNOT, W.CRY)).tolist()
    gates = _arr(base[:6] + [_g(W.PAULI, 1, -1, W.SRC_INPUT, 1)] + base[6:] +
                 [_g(W.PAULI, 2, -1, W.SRC_INPUT, 2)])
    pp = [[0.1, 0.05, 0.2], [0.02, 0.3, 0.08]]
    x, w, _ = W.random_inputs(1, 1, 3, n, 96)
    mid = []  # a uniform inside each outcome's bin, and the outcome probability
    for p in pp:
        e = np.cumsum([0.0] + list(p) + [1 - sum(p)])
        mid.append([(0.5 * (e[k] + e[k + 1]), e[k + 1] - e[k]) for k in range(4)])
    avg = np.zeros(n)
    for a in range(4):
        for b in range(4):
            u = np.array([[x[0, 0], mid[0][a][0], mid[1][b][0]]])
            avg += mid[0][a][1] * mid[1][b][1] * orc.run(n, gates, u, w, pauli_p=pp)["expz"][0]
    xb = np.array([x[0, 0], 0.0, 0.0])
    _close(avg, _density_reference(n, gates, xb, w, pp), what="trajectory average vs density matrix")


def pin_large_states(orc):
    """States of 2^16 and 2^18 amplitudes, where the oracle's amplitude loops run
    in parallel and its pairwise sums split into 4 and 16 chunks combined as a
    tree: workload-shaped circuits without entanglers against the per-qubit
    SO(3) closed form (expectations and gradients); a CNOT chain over a basis
    state gives prefix parities; H CZ H on qubits far apart acts as a CNOT;
    Pauli channels with probability 1 flip <Z> (X and Y on |0>, Z on |+>);
    un-applying a random entangled circuit returns |0...0> and lambda_0[0]
    equals sum_i g_i <Z_i>."""
    for name, n in (("24q", 16), ("30q", 18)):
        wl = W.scaled(W.get(name), n=n, batch=1, layers=1, entangler=None, dtype="c128")
        x, w, g = wl.inputs()
        gates = wl.gates()
        r = orc.run(n, gates, x, w, grad_out=g)
        e, gx, gw = product_state_reference(n, gates, x[0], w, g[0])
        _close(r["expz"][0], e, tol=1e-12, what=f"n={n} product expz")
        _close(r["grad_inputs"][0], gx, tol=1e-12, what=f"n={n} product grad_x")
        _close(r["grad_weights"], gw, tol=1e-12, what=f"n={n} product grad_w")
    n = 16
    rng = np.random.default_rng(16)
    bits = [int(v) for v in rng.integers(0, 2, n)]
    bits[0] = bits[n - 1] = 1
    r = orc.run(n, _arr(_basis_prep(bits) + [_g(W.CNOT, q, q + 1) for q in range(n - 1)]), [[math.pi]], [])
    _close(r["expz"][0], 1 - 2 * (np.cumsum(bits) % 2), what="n=16 chain parity")
    for c, t, a_, b_ in ((0, 15, 15, 0), (14, 1, 1, 14)):
        gates = _arr(_basis_prep(bits) + [_g(W.H, t), _g(W.CZ, a_, b_), _g(W.H, t)])
        out = list(bits)
        out[t] ^= bits[c]
        _close(orc.run(n, gates, [[math.pi]], [])["expz"][0], [1 - 2 * v for v in out], what="n=16 CZ kickback")
    pp = [[1.0, 0.0, 0.0], [0.0, 1.0, 0.0], [0.0, 0.0, 1.0]]
    gates = _arr([_g(W.PAULI, 15, -1, W.SRC_INPUT, 0), _g(W.PAULI, 3, -1, W.SRC_INPUT, 0),
                  _g(W.H, 9), _g(W.PAULI, 9, -1, W.SRC_INPUT, 0), _g(W.H, 9)])
    want = np.ones(n)
    want[[15, 3, 9]] = -1
    _close(orc.run(n, gates, [[0.5]], [], pauli_p=pp)["expz"][0], want, what="n=16 Pauli channels")
    gates, x, w, g = _random_case(n, 40, 1616, B=1)
    r = orc.run(n, gates, x, w, grad_out=g, want_state=True, want_back=True)
    _close(np.sum(np.abs(r["state"]) ** 2), 1.0, what="n=16 norm")
    e0 = np.zeros(1 << n)
    e0[0] = 1
    _close(r["back_psi"][0], e0, what="n=16 inverse sweep")
    _close(r["back_lam0"][0], np.sum(g[0] * r["expz"][0]), what="n=16 lambda_0[0]")


ALL_PINS = [
    pin_rotations_on_zero, pin_rotation_axes, pin_h_rz_h, pin_hybrid_node,
    pin_shared_parameter, pin_cnot_truth_table, pin_cnot_chain_parity, pin_cz_kickback,
    pin_bell, pin_brute_force, pin_unitarity, pin_param_shift, pin_finite_difference,
    pin_vjp_structure, pin_product_states, pin_cyclic_shift, pin_sampling,
    pin_controlled_rotation_closed_forms, pin_controlled_rotation_brute_force,
    pin_controlled_rotation_decomposition, pin_controlled_rotation_shift_and_fd,
    pin_basis_embedding, pin_amplitude_embedding, pin_amplitude_embedding_gradient,
    pin_pauli_trajectory_choices, pin_pauli_channel_average, pin_large_states,
]
