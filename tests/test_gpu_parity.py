"""HIP path vs the CPU oracle, through the C ABI (needs an MI355X).

Tolerances: 1e-5 absolute for complex64 and 1e-12 absolute for complex128, on
<Z_i>, input gradients and weight gradients. The oracle always runs in
complex128 on the exact (float32-rounded for complex64) values the GPU gets.
"""

from __future__ import annotations

import math
import os

import numpy as np
import pytest

import oracle
from parity import check, close
import oracle_pins
import workloads as W

torch = pytest.importorskip("torch")
import paper_2301_03251_amd as Q  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = {"c64": 1e-5, "c128": 1e-12}
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.load()


def _real(dtype):
    return torch.float32 if dtype == "c64" else torch.float64


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=_real(dtype))


def gpu_fb(circ, dtype, x, w, g, runner=None):
    r = runner or Q.Runner(circ, dtype)
    e, gx, gw = r.forward_backward(_dev(x, dtype), _dev(w, dtype), _dev(g, dtype))
    torch.cuda.synchronize()
    return {"expz": e.cpu().double().numpy(), "grad_inputs": gx.cpu().double().numpy(),
            "grad_weights": gw.cpu().double().numpy()}




# ---------------------------------------------------------------------------
# random circuits on every code path

TILED = [
    # n, G, B, dtype, options
    (9, 60, 3, "c64", dict(force_tiled=1, log_regs=3, log_threads=6)),
    (10, 80, 2, "c128", dict(force_tiled=1, log_regs=2, log_threads=6)),
    (11, 90, 3, "c64", dict(force_tiled=1, log_regs=4, log_threads=6, low_qubits=2)),
    (11, 90, 3, "c128", dict(force_tiled=1, log_regs=3, log_threads=7, low_qubits=3)),
    (12, 120, 2, "c64", dict(force_tiled=1, log_regs=5, log_threads=6)),
    (12, 120, 2, "c64", dict(force_tiled=1, log_regs=4, log_threads=6, max_gates_per_pass=1)),
    (13, 150, 3, "c64", dict()),
    (13, 150, 3, "c128", dict(force_tiled=1, log_regs=4, log_threads=8, max_gates_per_pass=7)),
    (14, 200, 2, "c64", dict()),
    (14, 200, 2, "c128", dict()),
    (14, 160, 3, "c64", dict(log_regs=2, log_threads=8, low_qubits=1)),
    (15, 160, 2, "c64", dict(log_regs=5, log_threads=7, wg_per_sample=3)),
]


@pytest.mark.parametrize("n,G,B,dtype,opts", TILED,
                         ids=[f"n{c[0]}-{c[3]}-{'-'.join(f'{k}{v}' for k, v in c[4].items()) or 'default'}"
                              for c in TILED])
def test_random_tiled(n, G, B, dtype, opts):
    F, P = 5, 7
    gates = W.random_circuit(n, G, F, P, seed=n * 100 + G)
    x, w, g = W.random_inputs(B, F, P, n, seed=n + G, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P, **opts)
    info = circ.plan_info(dtype)
    assert info["kernel"] == 1
    got = gpu_fb(circ, dtype, x, w, g)
    want = oracle.run(n, gates, x, w, grad_out=g)
    check(got, want, TOL[dtype], f"tiled n={n} {dtype} {opts} passes={info['n_passes']}")


@pytest.mark.parametrize("case", [1, 2, 5, 7, 9, 11])
def test_kept_states_and_plain(case):
    """forward_backward with the forward states kept in the workspace (the
    backward passes load them) and without (each backward pass stores its
    un-computed state): both against the oracle, and against each other."""
    n, G, B, dtype, opts = TILED[case]
    F, P = 5, 7
    gates = W.random_circuit(n, G, F, P, seed=n * 100 + G)
    x, w, g = W.random_inputs(B, F, P, n, seed=n + G, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P, **opts)
    m = circ.plan_info(dtype)["n_passes"]
    assert m > 1
    want = oracle.run(n, gates, x, w, grad_out=g)
    got = {}
    # two passes: the kept state has the plain path's size and is always used
    plain = Q.MODE_FWD_BWD if m > 2 else Q.MODE_FWD_BWD_KEEP
    for keep, mode in ((False, plain), (True, Q.MODE_FWD_BWD_KEEP)):
        r = Q.Runner(circ, dtype, keep_states=keep)
        assert r.backward_mode(B) == mode
        got[keep] = gpu_fb(circ, dtype, x, w, g, runner=r)
        check(got[keep], want, TOL[dtype], f"tiled n={n} {dtype} keep={keep}")
    check(got[True], got[False], TOL[dtype], f"kept vs plain n={n} {dtype}")


@pytest.mark.parametrize("dtype", ["c64", "c128"])
@pytest.mark.parametrize("n", [1, 2, 3, 5, 7, 8, 11, 12])
def test_random_whole_state(n, dtype):
    if dtype == "c128" and n == 12:
        n = 11
    F, P = 3, 4
    gates = W.random_circuit(n, 40 + 5 * n, F, P, seed=7 * n + 1)
    x, w, g = W.random_inputs(5, F, P, n, seed=n, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P, force_tiled=-1)
    assert circ.plan_info(dtype)["kernel"] == 0
    check(gpu_fb(circ, dtype, x, w, g), oracle.run(n, gates, x, w, grad_out=g), TOL[dtype],
          f"whole n={n} {dtype}")


@pytest.mark.parametrize("n,dtype", [(6, "c64"), (8, "c128")])
def test_whole_state_forward_large_batch(n, dtype):
    """Forward-only launches of many small circuits (the LDS whole-state
    kernel takes them over from the one-wavefront kernel): <Z> and final
    states against the oracle."""
    F, P, B = 3, 4, 2100
    gates = W.random_circuit(n, 40 + 5 * n, F, P, seed=500 + n)
    x, w, _ = W.random_inputs(B, F, P, n, seed=501 + n, dtype=dtype)
    r = Q.Runner(Q.Circuit(n, gates, F, P), dtype)
    e = r.forward(_dev(x, dtype), _dev(w, dtype))
    psi = r.state(_dev(x, dtype), _dev(w, dtype))
    torch.cuda.synchronize()
    want = oracle.run(n, gates, x, w, want_state=True)
    close(e.cpu().double().numpy(), want["expz"], TOL[dtype], f"forward n={n} B={B} {dtype}", "expz")
    close(psi.cpu().numpy(), want["state"], TOL[dtype], f"forward n={n} B={B} {dtype}", "state")


@pytest.mark.parametrize("dtype", ["c64", "c128"])
def test_degenerate_circuits(dtype):
    """No gates, no rotations, inputs only, weights only."""
    n, B = 13, 2
    cases = [
        (np.zeros((0, 5), np.int32), 0, 0),
        (np.array([[W.H, 0, -1, 0, 0], [W.CNOT, 0, 12, 0, 0], [W.CZ, 12, 3, 0, 0]], np.int32), 0, 0),
        (np.array([[W.RY, q, -1, W.SRC_INPUT, q % 2] for q in range(n)], np.int32), 2, 0),
        (np.array([[W.RX, q, -1, W.SRC_WEIGHT, 0] for q in range(n)], np.int32), 0, 1),
    ]
    for gates, F, P in cases:
        for opts in (dict(), dict(force_tiled=1)):
            x, w, g = W.random_inputs(B, F, P, n, seed=3, dtype=dtype)
            circ = Q.Circuit(n, gates, F, P, **opts)
            got = gpu_fb(circ, dtype, x, w, g)
            check(got, oracle.run(n, gates, x, w, grad_out=g), TOL[dtype], f"degenerate {gates.shape[0]} gates")


# ---------------------------------------------------------------------------
# the five workloads

@pytest.mark.parametrize("name", ["4q", "10q"])
def test_workload_full(name):
    wl = W.get(name)
    x, w, g = wl.inputs()
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    got = gpu_fb(circ, wl.dtype, x, w, g)
    want = oracle.run(wl.n, wl.gates(), x, w, grad_out=g)
    check(got, want, TOL[wl.dtype], name)


@pytest.mark.parametrize("name", ["10q", "16q"])
def test_workload_in_c128(name):
    """The same circuits in complex128: separates logic errors from fp32 rounding."""
    wl = W.scaled(W.get(name), dtype="c128")
    x, w, g = wl.inputs()
    rows = [0, 1, wl.batch - 1] if wl.batch > 64 else list(range(wl.batch))
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    got = gpu_fb(circ, "c128", x, w, g)
    want = oracle.run(wl.n, wl.gates(), x[rows], w, grad_out=g[rows])
    gm = np.zeros_like(g)
    gm[rows] = g[rows]
    got_m = gpu_fb(circ, "c128", x, w, gm)
    check({"expz": got["expz"][rows], "grad_inputs": got["grad_inputs"][rows],
           "grad_weights": got_m["grad_weights"]}, want, 1e-12, name + " c128")


def test_workload_16q_sampled():
    """Full batch of 1024 on the GPU; the oracle checks sampled rows. Weight
    gradients are batch sums, so a second call zeroes grad_out outside the
    sampled rows (the VJP is linear in grad_out)."""
    wl = W.get("16q")
    x, w, g = wl.inputs()
    rows = [0, 1, 2, 255, 511, 777, 1022, 1023]
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    r = Q.Runner(circ, wl.dtype)
    got = gpu_fb(circ, wl.dtype, x, w, g, r)
    gm = np.zeros_like(g)
    gm[rows] = g[rows]
    got_m = gpu_fb(circ, wl.dtype, x, w, gm, r)
    want = oracle.run(wl.n, wl.gates(), x[rows], w, grad_out=g[rows])
    check({"expz": got["expz"][rows], "grad_inputs": got["grad_inputs"][rows],
           "grad_weights": got_m["grad_weights"]}, want, TOL[wl.dtype], "16q")
    assert np.all(np.abs(got["expz"]) <= 1 + 1e-5)


@pytest.mark.parametrize("keep", [True, False], ids=["kept", "plain"])
@pytest.mark.parametrize("name", ["16q", "24q", "24q_c128", "30q", "30q_c128"])
def test_workload_golden(name, keep):
    """Full workload on the GPU vs oracle values stored by tests/golden/make_golden.py,
    with and without the kept forward states: 16q over its whole batch (so the
    weight gradients are the batch sums of the workload itself), 24q and 30q on
    sampled rows, and 24q and 30q in complex128 (inputs drawn in fp64) at 1e-12
    (30q complex128 with kept states: a 176 GiB workspace)."""
    path = os.path.join(GOLDEN, f"{name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    gold = np.load(path, allow_pickle=False)
    import sys
    sys.path.insert(0, GOLDEN)
    import make_golden  # noqa: E402  (digest and workload only)
    wl = make_golden.workload(name)
    x, w, g = wl.inputs()
    assert str(gold["digest"]) == make_golden.digest(x, w, g), "golden file is stale"
    rows = [int(v) for v in gold["rows"]]
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    r = Q.Runner(circ, wl.dtype, keep_states=keep)
    got = gpu_fb(circ, wl.dtype, x, w, g, r)
    if len(rows) < wl.batch:
        gm = np.zeros_like(g)
        gm[rows] = g[rows]
        gw = gpu_fb(circ, wl.dtype, x, w, gm, r)["grad_weights"]
    else:
        gw = got["grad_weights"]
    check({"expz": got["expz"][rows], "grad_inputs": got["grad_inputs"][rows], "grad_weights": gw},
          {"expz": gold["expz"], "grad_inputs": gold["grad_inputs"],
           "grad_weights": gold["grad_weights"]}, TOL[wl.dtype], name)
    assert np.all(np.abs(got["expz"]) <= 1 + 1e-5)


def sweep_circuit(n, kind, F, P, seed):
    """A generic state (RY then RZ on every qubit), then `kind` on every qubit
    (one-qubit kinds) or on pairs that put the operands low/high, high/low,
    high/high, at the ends of the register and at qubit n-1 (two-qubit
    kinds), then a closing RX layer."""
    rng = np.random.default_rng(seed)

    def rot(k, q):
        if rng.random() < 0.4:
            return (k, q, -1, W.SRC_INPUT, int(rng.integers(F)))
        return (k, q, -1, W.SRC_WEIGHT, int(rng.integers(P)))
    g = [rot(W.RY, q) for q in range(n)] + [rot(W.RZ, q) for q in range(n)]
    if kind in (W.CNOT, W.CZ):
        pairs = [(0, n - 1), (n - 1, 0), (1, 12), (12, 1), (11, 12), (12, 11), (12, 13), (13, n - 1),
                 (n - 1, 13), (n - 2, n - 1), (2, 3), (3, 2), (5, 16), (16, 5), (9, 17), (17, 9)]
        for a, b in pairs:
            g.append((kind, a, b, 0, 0))
            g.append(rot(W.RY, b))
    elif kind == W.H:
        g += [(W.H, q, -1, 0, 0) for q in range(n)]
    else:
        g += [rot(kind, q) for q in range(n)]
    g += [rot(W.RX, q) for q in range(n)]
    return np.array(g, np.int32)


SWEEP_OPTS = [dict(), dict(max_gates_per_pass=5), dict(log_regs=3, log_threads=7, low_qubits=2)]


@pytest.mark.parametrize("opts", SWEEP_OPTS, ids=["default", "five-per-pass", "r3-t7-low2"])
@pytest.mark.parametrize("kind", [W.H, W.RX, W.RY, W.RZ, W.CNOT, W.CZ], ids=["H", "RX", "RY", "RZ", "CNOT", "CZ"])
def test_gate_sweep_n20(kind, opts):
    """Every gate kind on every qubit of a 20-qubit state (two-qubit kinds on
    pairs across the tile edges and the top qubit), in complex128 against the
    oracle at 1e-12, under three plans that put the operands on different
    register, lane, wavefront and fixed bits."""
    n, F, P, B = 20, 4, 9, 2
    gates = sweep_circuit(n, kind, F, P, seed=2000 + kind)
    x, w, g = W.random_inputs(B, F, P, n, seed=2100 + kind, dtype="c128")
    circ = Q.Circuit(n, gates, F, P, **opts)
    assert circ.plan_info("c128")["kernel"] == 1
    want = _sweep_oracle(n, kind, gates, x, w, g)
    check(gpu_fb(circ, "c128", x, w, g), want, 1e-12, f"sweep n={n} kind={kind} {opts}")


_SWEEP_CACHE = {}


def _sweep_oracle(n, kind, gates, x, w, g):
    if kind not in _SWEEP_CACHE:
        _SWEEP_CACHE[kind] = oracle.run(n, gates, x, w, grad_out=g)
    return _SWEEP_CACHE[kind]


def test_batch_edges():
    """B = 1 and a B that is not a multiple of anything, on the tiled path."""
    n, F, P = 14, 4, 6
    gates = W.random_circuit(n, 120, F, P, seed=11)
    circ = Q.Circuit(n, gates, F, P)
    for B in (1, 7):
        x, w, g = W.random_inputs(B, F, P, n, seed=B, dtype="c64")
        check(gpu_fb(circ, "c64", x, w, g), oracle.run(n, gates, x, w, grad_out=g), 1e-5, f"B={B}")


def test_forward_only_and_null_grads():
    n, F, P, B = 14, 3, 5, 3
    gates = W.random_circuit(n, 100, F, P, seed=5)
    circ = Q.Circuit(n, gates, F, P)
    x, w, g = W.random_inputs(B, F, P, n, seed=9, dtype="c64")
    r = Q.Runner(circ, "c64")
    e = r.forward(_dev(x, "c64"), _dev(w, "c64"))
    e2, gx, gw = r.forward_backward(_dev(x, "c64"), _dev(w, "c64"), _dev(g, "c64"),
                                    want_inputs=False, want_weights=True)
    torch.cuda.synchronize()
    assert gx is None
    want = oracle.run(n, gates, x, w, grad_out=g)
    close(e.cpu().double().numpy(), want["expz"], 1e-5, "forward only", "expz")
    assert np.array_equal(e.cpu().numpy(), e2.cpu().numpy())
    close(gw.cpu().double().numpy(), want["grad_weights"], 1e-5, "weights only", "grad_weights")


def test_destroy_right_after_a_call():
    """A handle destroyed while its call may still be queued: the outputs are
    still right (the table upload reads the handle's pinned copy, and
    destruction waits for the device first)."""
    import gc
    n, F, P, B = 14, 3, 5, 2
    gates = W.random_circuit(n, 120, F, P, seed=33)
    x, w, g = W.random_inputs(B, F, P, n, seed=34, dtype="c64")
    circ = Q.Circuit(n, gates, F, P)
    r = Q.Runner(circ, "c64")
    e, gx, gw = r.forward_backward(_dev(x, "c64"), _dev(w, "c64"), _dev(g, "c64"))
    r.c = None
    del r, circ
    gc.collect()
    torch.cuda.synchronize()
    got = {"expz": e.cpu().double().numpy(), "grad_inputs": gx.cpu().double().numpy(),
           "grad_weights": gw.cpu().double().numpy()}
    check(got, oracle.run(n, gates, x, w, grad_out=g), 1e-5, "destroyed handle")


def test_timing_classes():
    """Only the selected kernel classes are bracketed by events."""
    n, F, P, B = 14, 3, 5, 2
    gates = W.random_circuit(n, 120, F, P, seed=35)
    x, w, g = W.random_inputs(B, F, P, n, seed=36, dtype="c64")
    circ = Q.Circuit(n, gates, F, P)
    r = Q.Runner(circ, "c64")
    for mask, want in ((1, (True, False, False, False)), (12, (False, False, True, True)),
                       (15, (True, False, True, True))):
        circ.timing(True, mask)
        r.forward_backward(_dev(x, "c64"), _dev(w, "c64"), _dev(g, "c64"))
        ms, cnt = circ.timing_read()
        circ.timing(False)
        assert tuple(c > 0 for c in cnt) == want, (mask, cnt)
        assert all((m > 0) == (c > 0) for m, c in zip(ms, cnt))


def test_deterministic():
    """Two calls give bit-identical outputs (fixed-order fp64 reductions, no atomics)."""
    wl = W.get("16q")
    x, w, g = wl.inputs()
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    r = Q.Runner(circ, wl.dtype)
    a = gpu_fb(circ, wl.dtype, x, w, g, r)
    b = gpu_fb(circ, wl.dtype, x, w, g, r)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_plans_agree():
    """Different tilings of one circuit agree to rounding (c128: 1e-12)."""
    n, F, P, B = 14, 4, 6, 2
    gates = W.random_circuit(n, 150, F, P, seed=21)
    x, w, g = W.random_inputs(B, F, P, n, seed=22, dtype="c128")
    ref = None
    for opts in (dict(), dict(log_regs=2, log_threads=6), dict(max_gates_per_pass=3),
                 dict(log_regs=3, log_threads=7, low_qubits=1)):
        got = gpu_fb(Q.Circuit(n, gates, F, P, **opts), "c128", x, w, g)
        if ref is None:
            ref = got
        else:
            check(got, ref, 1e-12, f"plan {opts}")


def prefix_circuit(n, F, P, seed, body=60):
    """One to three one-qubit gates (H, RX, RY, RZ) on every qubit, then a
    random circuit of `body` gates: every qubit starts with a product-state
    prefix of mixed kinds."""
    rng = np.random.default_rng(seed)
    g = []
    for q in range(n):
        for _ in range(int(rng.integers(1, 4))):
            k = int(rng.choice([W.H, W.RX, W.RY, W.RZ]))
            if k == W.H:
                g.append((W.H, q, -1, 0, 0))
            elif rng.random() < 0.4:
                g.append((k, q, -1, W.SRC_INPUT, int(rng.integers(F))))
            else:
                g.append((k, q, -1, W.SRC_WEIGHT, int(rng.integers(P))))
    pre = np.array(g, np.int32).reshape(-1, 5)
    if body == 0:
        return pre
    return np.concatenate([pre, W.random_circuit(n, body, F, P, seed=seed + 1)])


PREFIX_CASES = [
    # n, body gates, planner options
    (8, 60, {}),                                      # one tile per sample; environment: 4 amplitudes per lane
    (9, 60, {}),                                      # environment: 8 amplitudes per lane
    (11, 80, dict(log_regs=2, log_threads=6)),        # small tiles, several per sample
    (14, 120, {}),
    (16, 120, dict(max_gates_per_pass=7)),            # many passes
    (12, 0, {}),                                      # prefix gates only: one pass with no ops
]


@pytest.mark.parametrize("n,body,opts", PREFIX_CASES,
                         ids=[f"n{c[0]}-g{c[1]}-{'-'.join(f'{k}{v}' for k, v in c[2].items()) or 'default'}"
                              for c in PREFIX_CASES])
def test_product_prefix(n, body, opts):
    """The product-state prefix (first pass from the per-qubit factors, prefix
    gradients from lambda's environment) against the oracle and against the
    same plan with the prefix run as tile ops (product_prefix=-1): c128 at
    1e-12, c64 at 1e-5. Weight 0 is exactly zero, so some factors have a zero
    component (an RY(0) or RX(0) leaves |0>), which the environment sums must
    handle without dividing by a factor."""
    F, P, B = 4, 6, 3
    gates = prefix_circuit(n, F, P, seed=400 + n + body, body=body)
    on = Q.Circuit(n, gates, F, P, product_prefix=1, **opts)
    off = Q.Circuit(n, gates, F, P, product_prefix=-1, **opts)
    assert on.plan_info("c64")["n_prefix_gates"] > 0 and off.plan_info("c64")["n_prefix_gates"] == 0
    for dtype in ("c128", "c64"):
        x, w, g = W.random_inputs(B, F, P, n, seed=401 + n, dtype=dtype)
        w[0] = 0.0
        want = oracle.run(n, gates, x, w, grad_out=g)
        got = gpu_fb(on, dtype, x, w, g)
        check(got, want, TOL[dtype], f"prefix n={n} {opts} {dtype} vs oracle")
        check(got, gpu_fb(off, dtype, x, w, g), 2 * TOL[dtype], f"prefix n={n} {opts} {dtype} on vs off")


@pytest.mark.parametrize("name", ["24q", "30q"])
def test_product_state_full_size(name):
    """Workload circuit with its entanglers removed, at full size: every qubit
    evolves alone, so <Z_q> and the gradients have the SO(3) closed form."""
    wl = W.scaled(W.get(name), entangler=None)
    x, w, g = wl.inputs()
    gates = wl.gates()
    circ = Q.Circuit(wl.n, gates, wl.n_inputs, wl.n_weights)
    got = gpu_fb(circ, wl.dtype, x, w, g)
    xs, ws, gs = (a.astype(np.float64) for a in (x, w, g))
    gw = np.zeros(wl.n_weights)
    for b in range(wl.batch):
        e, gx, gwb = oracle_pins.product_state_reference(wl.n, gates, xs[b], ws, gs[b])
        gw += gwb
        close(got["expz"][b], e, 1e-5, f"{name} product state row {b}", "expz")
        close(got["grad_inputs"][b], gx, 1e-5, f"{name} product state row {b}", "grad_inputs")
    close(got["grad_weights"], gw, 1e-5, f"{name} product state", "grad_weights")


@pytest.mark.parametrize("prefix", [1, -1], ids=["prefix", "ops"])
@pytest.mark.parametrize("n,dtype,keep", [(32, "c64", False), (31, "c128", True)],
                         ids=["n32-c64-plain", "n31-c128-kept"])
def test_maximum_qubits(n, dtype, keep, prefix):
    """The largest state each dtype allows (32 GiB), one sample: rotation layers
    around CNOT and CZ pairs that cancel (on qubits 0, 3, n-2 and n-1, so the
    top amplitude-index bits take part), against the SO(3) closed form of the
    product state; with the first rotation layer as the product-state prefix
    (one tile pass left), and with every gate as a tile op (several passes)."""
    torch.cuda.empty_cache()
    P = 2 * n
    ry = [(W.RY, q, -1, W.SRC_WEIGHT, q) for q in range(n)]
    rest = [(W.RZ, q, -1, W.SRC_WEIGHT, n + q) for q in range(n)] + \
        [(W.RX, q, -1, W.SRC_INPUT, 0) for q in (0, n - 1)]
    pairs = [(W.CNOT, n - 1, 0, 0, 0), (W.CZ, 3, n - 2, 0, 0)]
    gates = np.array(ry + pairs + pairs + rest, np.int32)
    x, w, g = W.random_inputs(1, 1, P, n, seed=n, dtype=dtype)
    circ = Q.Circuit(n, gates, 1, P, product_prefix=prefix)
    if prefix == 1:
        assert circ.plan_info(dtype)["n_prefix_gates"] >= n
    else:
        assert circ.plan_info(dtype)["n_passes"] > 1
    r = Q.Runner(circ, dtype, keep_states=keep)
    got = gpu_fb(circ, dtype, x, w, g, r)
    del r
    torch.cuda.empty_cache()
    one_qubit = np.array(ry + rest, np.int32)
    e, gx, gw = oracle_pins.product_state_reference(n, one_qubit, x[0].astype(np.float64), w.astype(np.float64),
                                                    g[0].astype(np.float64))
    check(got, {"expz": e[None], "grad_inputs": gx[None], "grad_weights": gw}, TOL[dtype], f"n={n} {dtype}")


def test_hybrid_node_closed_form():
    """The paper's one-qubit hybrid node (H, then RY(input)): <Z> = -sin t and
    d<Z>/dt = -cos t, on a batch of angles."""
    t = np.linspace(-3.0, 3.0, 33)
    gates = np.array([[W.H, 0, -1, 0, 0], [W.RY, 0, -1, W.SRC_INPUT, 0]], np.int32)
    circ = Q.Circuit(1, gates, 1, 0)
    got = gpu_fb(circ, "c128", t[:, None], np.zeros(0), np.ones((t.size, 1)))
    close(got["expz"][:, 0], -np.sin(t), 1e-12, "hybrid node", "expz")
    close(got["grad_inputs"][:, 0], -np.cos(t), 1e-12, "hybrid node", "grad_inputs")


def test_autograd_function():
    """The torch.autograd.Function wrapper returns the library's VJP."""
    wl = W.get("10q")
    x, w, g = wl.inputs()
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    r = Q.Runner(circ, wl.dtype)
    fn = Q.quantum_layer_function()
    xt = _dev(x, "c64").requires_grad_(True)
    wt = _dev(w, "c64").requires_grad_(True)
    out = fn.apply(r, xt, wt)
    (out * _dev(g, "c64")).sum().backward()
    torch.cuda.synchronize()
    want = oracle.run(wl.n, wl.gates(), x, w, grad_out=g)
    check({"expz": out.detach().cpu().numpy(), "grad_inputs": xt.grad.cpu().numpy(),
           "grad_weights": wt.grad.cpu().numpy()}, want, 1e-5, "autograd function")


def test_quantum_layer_module():
    """The nn.Module form: weights are its parameter, autograd gives the
    library's VJP, and an optimizer step moves them."""
    wl = W.get("10q")
    x, w, g = wl.inputs()
    layer = Q.QuantumLayer(wl.gates(), wl.n, wl.n_inputs, wl.n_weights, dtype="c64", weights=w)
    assert [p.shape for p in layer.parameters()] == [torch.Size([wl.n_weights])]
    xt = _dev(x, "c64").requires_grad_(True)
    out = layer(xt)
    (out * _dev(g, "c64")).sum().backward()
    torch.cuda.synchronize()
    want = oracle.run(wl.n, wl.gates(), x, w, grad_out=g)
    check({"expz": out.detach().cpu().numpy(), "grad_inputs": xt.grad.cpu().numpy(),
           "grad_weights": layer.weights.grad.cpu().numpy()}, want, 1e-5, "QuantumLayer")
    opt = torch.optim.SGD(layer.parameters(), lr=0.1)
    w0 = layer.weights.detach().clone()
    opt.step()
    assert torch.allclose(layer.weights.detach(), w0 - 0.1 * layer.weights.grad)


def test_shared_parameter_closed_form():
    """The paper's compatibility example at 14 qubits (tiled path): H on every
    qubit, RY with one shared weight; d/dt of the mean of <Z_i> is -cos t
    (grad_out = 1/n, the mean-reduced loss of the harness), and of the sum
    -n cos t (grad_out = 1: the VJP is linear in grad_out, so its value and
    its rounding both scale by n, and so does the bound)."""
    n = 14
    gates = np.array([[W.H, q, -1, 0, 0] for q in range(n)] +
                     [[W.RY, q, -1, W.SRC_WEIGHT, 0] for q in range(n)], np.int32)
    circ = Q.Circuit(n, gates, 0, 1)
    for t in (-1.2, 0.4, 2.5):
        got = gpu_fb(circ, "c128", np.zeros((1, 0)), np.array([t]), np.full((1, n), 1.0 / n))
        close(got["expz"][0], np.full(n, -math.sin(t)), 1e-12, f"shared parameter t={t}", "expz")
        close(got["grad_weights"], [-math.cos(t)], 1e-12, f"shared parameter t={t} mean", "grad_weights")
        got = gpu_fb(circ, "c128", np.zeros((1, 0)), np.array([t]), np.ones((1, n)))
        close(got["grad_weights"], [-n * math.cos(t)], n * 1e-12, f"shared parameter t={t} sum", "grad_weights")


# ---------------------------------------------------------------------------
# parameter-shift gradients (the paper's rule, shifted circuits batched)

def gpu_shift(circ, dtype, x, w, g, max_chunk=0, runner=None):
    r = runner or Q.Runner(circ, dtype)
    e, gx, gw = r.param_shift(_dev(x, dtype), _dev(w, dtype), _dev(g, dtype), max_chunk=max_chunk)
    torch.cuda.synchronize()
    return {"expz": e.cpu().double().numpy(), "grad_inputs": gx.cpu().double().numpy(),
            "grad_weights": gw.cpu().double().numpy()}


SHIFT_CASES = [
    # n, G, B, dtype, options, max_chunk
    (5, 40, 3, "c128", dict(), 0),
    (8, 60, 2, "c64", dict(), 7),
    (11, 70, 2, "c128", dict(), 0),
    (13, 80, 2, "c64", dict(), 0),
    (14, 90, 2, "c64", dict(), 33),
    (14, 60, 2, "c128", dict(), 0),
]


@pytest.mark.parametrize("n,G,B,dtype,opts,chunk", SHIFT_CASES,
                         ids=[f"n{c[0]}-{c[3]}-chunk{c[5]}" for c in SHIFT_CASES])
def test_param_shift_vs_oracle(n, G, B, dtype, opts, chunk):
    """GPU parameter shift against the oracle's parameter shift (expz from the
    unshifted circuits against the oracle forward)."""
    F, P = 4, 6
    gates = W.random_circuit(n, G, F, P, seed=500 + n * 7 + G)
    x, w, g = W.random_inputs(B, F, P, n, seed=600 + n, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P, **opts)
    got = gpu_shift(circ, dtype, x, w, g, max_chunk=chunk)
    gx, gw = oracle.param_shift(n, gates, x, w, g)
    want = {"expz": oracle.run(n, gates, x, w)["expz"], "grad_inputs": gx, "grad_weights": gw}
    check(got, want, TOL[dtype], f"shift n={n} {dtype} chunk={chunk}")


@pytest.mark.parametrize("name", ["4q", "10q"])
def test_param_shift_equals_adjoint_on_workloads(name):
    """Two gradient methods, one answer: parameter shift and the adjoint sweep
    on the small workloads at full batch."""
    wl = W.get(name)
    x, w, g = wl.inputs()
    circ = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    r = Q.Runner(circ, wl.dtype)
    adj = gpu_fb(circ, wl.dtype, x, w, g, r)
    sh = gpu_shift(circ, wl.dtype, x, w, g, max_chunk=4096, runner=r)
    check(sh, adj, 2 * TOL[wl.dtype], f"{name} shift vs adjoint")


def test_param_shift_chunks_agree():
    """Chunk size only changes how the shifted circuits are grouped."""
    n, F, P, B = 14, 3, 5, 2
    gates = W.random_circuit(n, 70, F, P, seed=77)
    x, w, g = W.random_inputs(B, F, P, n, seed=78, dtype="c128")
    circ = Q.Circuit(n, gates, F, P)
    ref = gpu_shift(circ, "c128", x, w, g, max_chunk=0)
    for chunk in (1, 5, 64):
        check(gpu_shift(circ, "c128", x, w, g, max_chunk=chunk), ref, 1e-12, f"chunk {chunk}")


def test_param_shift_hybrid_node():
    """The paper's one-qubit hybrid node (H, then RY(input)) differentiated by
    the paper's own rule: d<Z>/dt = -cos t."""
    t = np.linspace(-3.0, 3.0, 17)
    gates = np.array([[W.H, 0, -1, 0, 0], [W.RY, 0, -1, W.SRC_INPUT, 0]], np.int32)
    circ = Q.Circuit(1, gates, 1, 0)
    got = gpu_shift(circ, "c128", t[:, None], np.zeros(0), np.ones((t.size, 1)))
    close(got["expz"][:, 0], -np.sin(t), 1e-12, "hybrid node shift", "expz")
    close(got["grad_inputs"][:, 0], -np.cos(t), 1e-12, "hybrid node shift", "grad_inputs")


# ---------------------------------------------------------------------------
# final states and shot sampling (the paper's Monte Carlo measurement)

STATE_CASES = [(3, "c128"), (6, "c64"), (9, "c64"), (10, "c128"), (13, "c64"), (14, "c128"), (16, "c64")]


@pytest.mark.parametrize("n,dtype", STATE_CASES, ids=[f"n{c[0]}-{c[1]}" for c in STATE_CASES])
def test_state_vs_oracle(n, dtype):
    F, P, B = 3, 5, 3
    gates = W.random_circuit(n, 12 * n, F, P, seed=900 + n)
    x, w, _ = W.random_inputs(B, F, P, n, seed=901 + n, dtype=dtype)
    r = Q.Runner(Q.Circuit(n, gates, F, P), dtype)
    psi = r.state(_dev(x, dtype), _dev(w, dtype))
    torch.cuda.synchronize()
    want = oracle.run(n, gates, x, w, want_state=True)["state"]
    close(psi.cpu().numpy(), want, TOL[dtype], f"state n={n} {dtype}", "state")


def rz_layer_circuit(n, layers, F, P, seed):
    """RY on every qubit, then RZ on every qubit (bound to inputs and shared
    weights), then a CNOT ring, per layer: the RZs of each tile layout commute
    into one place, so the planner groups them."""
    rng = np.random.default_rng(seed)
    g = []
    for _ in range(layers):
        for kind in (W.RY, W.RZ):
            for q in range(n):
                if rng.random() < 0.3:
                    g.append((kind, q, -1, W.SRC_INPUT, int(rng.integers(F))))
                else:
                    g.append((kind, q, -1, W.SRC_WEIGHT, int(rng.integers(P))))
        for q in range(n):
            g.append((W.CNOT, q, (q + 1) % n, 0, 0))
    return np.array(g, np.int32)


def staircase_circuit(n, layers, F, P, seed):
    """RY then RZ on each qubit, then a CNOT chain, per layer (the workloads'
    shape): most RZs commute back to their qubit's RY and run in one op with
    it, the rest form groups."""
    rng = np.random.default_rng(seed)
    g = []
    for _ in range(layers):
        for q in range(n):
            for kind in (W.RY, W.RZ):
                if rng.random() < 0.3:
                    g.append((kind, q, -1, W.SRC_INPUT, int(rng.integers(F))))
                else:
                    g.append((kind, q, -1, W.SRC_WEIGHT, int(rng.integers(P))))
        for q in range(n - 1):
            g.append((W.CNOT, q, q + 1, 0, 0))
    return np.array(g, np.int32)


RZ_GROUP_CASES = [(13, "c64", dict()), (14, "c128", dict()), (12, "c64", dict(log_regs=3, log_threads=6)),
                  (11, "c128", dict(force_tiled=1, log_regs=4, log_threads=6, max_gates_per_pass=20))]


@pytest.mark.parametrize("shape", ["layers", "staircase"])
@pytest.mark.parametrize("n,dtype,opts", RZ_GROUP_CASES,
                         ids=[f"n{c[0]}-{c[1]}-{'-'.join(f'{k}{v}' for k, v in c[2].items()) or 'default'}"
                              for c in RZ_GROUP_CASES])
def test_rz_groups(n, dtype, opts, shape):
    """RZ groups (one phase op for several RZs) and RY-RZ pair ops against the
    oracle and against the plan without them: forward + adjoint VJP, and exact
    final states."""
    F, P, B = 4, 6, 3
    build = rz_layer_circuit if shape == "layers" else staircase_circuit
    gates = build(n, 3, F, P, seed=70 + n)
    x, w, g = W.random_inputs(B, F, P, n, seed=71 + n, dtype=dtype)
    x[0, 0] = 9.0      # angles well outside [-pi, pi]
    w[1] = -7.5
    # the first layer runs as tile ops too (not as the product-state prefix),
    # so that its RZs form groups and pairs
    grouped = Q.Circuit(n, gates, F, P, product_prefix=-1, **opts)
    single = Q.Circuit(n, gates, F, P, rz_groups=-1, product_prefix=-1, **opts)
    assert grouped.plan_info(dtype)["n_rz_groups"] > 0
    if shape == "staircase":
        assert grouped.plan_info(dtype)["n_ryz_pairs"] > 0
    assert single.plan_info(dtype)["n_rz_groups"] == 0 and single.plan_info(dtype)["n_ryz_pairs"] == 0
    want = oracle.run(n, gates, x, w, grad_out=g)
    got = gpu_fb(grouped, dtype, x, w, g)
    check(got, want, TOL[dtype], f"rz groups n={n} {dtype}")
    check(got, gpu_fb(single, dtype, x, w, g), TOL[dtype], "grouped vs single")
    psi = Q.Runner(grouped, dtype).state(_dev(x, dtype), _dev(w, dtype))
    torch.cuda.synchronize()
    ref = oracle.run(n, gates, x, w, want_state=True)["state"]
    close(psi.cpu().numpy(), ref, TOL[dtype], f"rz groups n={n} {dtype}", "state")


def cz_circuit(n, layers, F, P, seed, extra=6):
    """Per layer: RY on every qubit, RZ on some, a ring of CZs, `extra` CZs on
    random pairs (long-range ones reach the fixed qubits of a tile pass) and one
    pair twice (the two cancel); a CNOT now and then closes a CZ group early."""
    rng = np.random.default_rng(seed)
    g = []
    for layer in range(layers):
        for q in range(n):
            src = W.SRC_INPUT if rng.random() < 0.3 else W.SRC_WEIGHT
            g.append((W.RY, q, -1, src, int(rng.integers(F if src == W.SRC_INPUT else P))))
            if rng.random() < 0.5:
                g.append((W.RZ, q, -1, W.SRC_WEIGHT, int(rng.integers(P))))
        for q in range(n):
            g.append((W.CZ, q, (q + 1) % n, 0, 0))
            if layer % 2 and q == n // 2:
                g.append((W.CNOT, q, (q + 3) % n, 0, 0))
        for _ in range(extra):
            a, b = rng.choice(n, 2, replace=False)
            g.append((W.CZ, int(a), int(b), 0, 0))
        a, b = rng.choice(n, 2, replace=False)
        g += [(W.CZ, int(a), int(b), 0, 0)] * 2
    return np.array(g, np.int32)


CZ_GROUP_CASES = [(16, "c64", dict()), (15, "c128", dict()), (12, "c64", dict(log_regs=3, log_threads=6)),
                  (14, "c64", dict(log_regs=5, log_threads=7)),
                  (11, "c128", dict(force_tiled=1, log_regs=4, log_threads=6, max_gates_per_pass=30))]


@pytest.mark.parametrize("n,dtype,opts", CZ_GROUP_CASES,
                         ids=[f"n{c[0]}-{c[1]}-{'-'.join(f'{k}{v}' for k, v in c[2].items()) or 'default'}"
                              for c in CZ_GROUP_CASES])
def test_cz_groups(n, dtype, opts):
    """CZ groups (one sign op for the CZs of a layout) against the oracle and
    against the plan without them: forward + adjoint VJP (the two-tile forward
    and the backward kernel), and exact final states."""
    F, P, B = 4, 6, 3
    gates = cz_circuit(n, 3, F, P, seed=170 + n)
    x, w, g = W.random_inputs(B, F, P, n, seed=171 + n, dtype=dtype)
    grouped = Q.Circuit(n, gates, F, P, **opts)
    single = Q.Circuit(n, gates, F, P, cz_groups=-1, **opts)
    assert grouped.plan_info(dtype)["n_cz_groups"] > 0
    assert single.plan_info(dtype)["n_cz_groups"] == 0
    want = oracle.run(n, gates, x, w, grad_out=g)
    got = gpu_fb(grouped, dtype, x, w, g)
    check(got, want, TOL[dtype], f"cz groups n={n} {dtype}")
    check(got, gpu_fb(single, dtype, x, w, g), TOL[dtype], "grouped vs single")
    psi = Q.Runner(grouped, dtype).state(_dev(x, dtype), _dev(w, dtype))
    torch.cuda.synchronize()
    ref = oracle.run(n, gates, x, w, want_state=True)["state"]
    close(psi.cpu().numpy(), ref, TOL[dtype], f"cz groups n={n} {dtype}", "state")


def test_cz_groups_split():
    """100 CZs on random pairs after a product-state prefix, all in one pass
    and one layout: more pairs without a register operand than one group
    record holds, so the planner splits the collection into several groups."""
    n, dtype, F, P, B = 16, "c64", 2, 3, 4
    rng = np.random.default_rng(33)
    g = [(W.H, q, -1, 0, 0) for q in range(n)] + [(W.RY, q, -1, W.SRC_WEIGHT, q % P) for q in range(n)]
    for _ in range(100):
        a, b = rng.choice(n, 2, replace=False)
        g.append((W.CZ, int(a), int(b), 0, 0))
    gates = np.array(g, np.int32)
    x, w, gout = W.random_inputs(B, F, P, n, seed=34, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P)
    info = circ.plan_info(dtype)
    assert info["n_passes"] == 1 and info["n_transposes"] + info["n_lane_swaps"] == 0
    assert info["n_cz_groups"] >= 3
    check(gpu_fb(circ, dtype, x, w, gout), oracle.run(n, gates, x, w, grad_out=gout), TOL[dtype], "cz split")


def test_cz_groups_param_shift():
    """The shifted circuits of a parameter-shift chunk run the same CZ groups
    (two-tile forward launches): shift gradients against the oracle's rule."""
    n, dtype, F, P, B = 14, "c128", 4, 6, 2
    gates = cz_circuit(n, 2, F, P, seed=190)
    x, w, g = W.random_inputs(B, F, P, n, seed=191, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P)
    assert circ.plan_info(dtype)["n_cz_groups"] > 0
    e, gx, gw = Q.Runner(circ, dtype).param_shift(_dev(x, dtype), _dev(w, dtype), _dev(g, dtype), max_chunk=41)
    torch.cuda.synchronize()
    got = {"expz": e.cpu().numpy(), "grad_inputs": gx.cpu().numpy(), "grad_weights": gw.cpu().numpy()}
    ox, ow = oracle.param_shift(n, gates, x, w, g)
    want = {"expz": oracle.run(n, gates, x, w)["expz"], "grad_inputs": ox, "grad_weights": ow}
    check(got, want, 1e-12, "cz groups shift")


def test_rz_groups_param_shift():
    """The shifted circuits of a parameter-shift chunk shift one member of an
    RZ group's phase table at a time."""
    n, dtype, F, P, B = 13, "c128", 3, 5, 2
    gates = np.concatenate([rz_layer_circuit(n, 1, F, P, seed=90), staircase_circuit(n, 1, F, P, seed=92)])
    x, w, g = W.random_inputs(B, F, P, n, seed=91, dtype=dtype)
    circ = Q.Circuit(n, gates, F, P, product_prefix=-1)  # the first layer as tile ops
    assert circ.plan_info(dtype)["n_rz_groups"] > 0 and circ.plan_info(dtype)["n_ryz_pairs"] > 0
    e, gx, gw = Q.Runner(circ, dtype).param_shift(_dev(x, dtype), _dev(w, dtype), _dev(g, dtype), max_chunk=37)
    torch.cuda.synchronize()
    got = {"expz": e.cpu().numpy(), "grad_inputs": gx.cpu().numpy(), "grad_weights": gw.cpu().numpy()}
    check(got, oracle.run(n, gates, x, w, grad_out=g), 1e-12, "rz groups shift")


def _valid_near_tie(psi_row, u, idx, tol=1e-12):
    """A shot that differs from the oracle must sit on a CDF boundary of the same state."""
    p = np.abs(psi_row) ** 2
    cdf = np.cumsum(p)
    r = u * cdf[-1]
    lo = cdf[idx - 1] if idx > 0 else 0.0
    return p[idx] > 0 and lo - tol * cdf[-1] <= r <= cdf[idx] + tol * cdf[-1]


SAMPLE_CASES = [(3, "c64"), (7, "c128"), (10, "c64"), (14, "c64"), (16, "c128")]


@pytest.mark.parametrize("n,dtype", SAMPLE_CASES, ids=[f"n{c[0]}-{c[1]}" for c in SAMPLE_CASES])
def test_sample_vs_oracle(n, dtype):
    """Shots from the GPU's own states: the kernel's indices against the
    oracle sampler on the same states and uniforms (integers, so exact; a
    uniform on a CDF boundary within rounding may pick the neighbour, which is
    then checked to be valid). zhat equals the count formula of the indices."""
    F, P, B, shots = 3, 5, 2, 4096
    gates = W.random_circuit(n, 10 * n, F, P, seed=950 + n)
    x, w, _ = W.random_inputs(B, F, P, n, seed=951 + n, dtype=dtype)
    r = Q.Runner(Q.Circuit(n, gates, F, P), dtype)
    psi = r.state(_dev(x, dtype), _dev(w, dtype))
    u = np.random.default_rng(952 + n).random((B, shots))
    idx, zhat = Q.sample(psi, torch.from_numpy(u).to("cuda"))
    torch.cuda.synchronize()
    st = psi.cpu().numpy().astype(np.complex128)
    got = idx.cpu().numpy()
    want = oracle.sample(n, st, u)
    bad = np.argwhere(got != want)
    assert len(bad) <= 2, f"{len(bad)} shots differ from the oracle"
    for b, s_ in bad:
        assert _valid_near_tie(st[b], u[b, s_], int(got[b, s_])), f"invalid shot {b},{s_}"
    bits = (got[:, :, None] >> np.arange(n)) & 1
    zc = (shots - 2 * bits.sum(axis=1)) / shots
    assert np.array_equal(zhat.cpu().double().numpy(), zc.astype(np.float32 if dtype == "c64" else np.float64).astype(np.float64))


def test_sample_statistics_and_scale():
    """Many shots estimate <Z_q> within five standard errors of the exact value;
    scaling the state leaves the shots unchanged; zero shots writes nothing."""
    wl = W.scaled(W.get("16q"), batch=2, layers=2)
    x, w, _ = wl.inputs()
    r = Q.Runner(Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights), wl.dtype)
    psi = r.state(_dev(x, wl.dtype), _dev(w, wl.dtype))
    exact = oracle.run(wl.n, wl.gates(), x, w)["expz"]
    shots = 200000
    u = torch.from_numpy(np.random.default_rng(5).random((wl.batch, shots))).to("cuda")
    idx, zhat = Q.sample(psi, u)
    idx2, _ = Q.sample((psi * 2).contiguous(), u)  # a power of two scales every sum exactly
    torch.cuda.synchronize()
    se = np.sqrt(np.maximum(1 - exact ** 2, 1e-12) / shots)
    assert np.all(np.abs(zhat.cpu().double().numpy() - exact) <= 5 * se + 1e-6)
    assert torch.equal(idx, idx2)
    empty, ez = Q.sample(psi, torch.empty((wl.batch, 0), dtype=torch.float64, device="cuda"))
    assert empty.shape == (wl.batch, 0)
