"""Host-side checks of the C ABI (no GPU): exports, validation, planner invariants,
workspace arithmetic. Nothing here launches a kernel."""

from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qlayer.h")

Q = pytest.importorskip("paper_2301_03251_amd")


@pytest.fixture(scope="module")
def lib():
    return Q.load()


def test_exports_every_declared_symbol(lib):
    decl = re.findall(r"\b(ql_[a-z_0-9]+)\s*\(", open(HEADER).read())
    names = sorted(set(decl))
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), f"{name} declared in qlayer.h but not exported"


def test_static_scratch_size_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define QL_STATIC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == Q.STATIC_SCRATCH_BYTES


def test_product_package_never_uses_the_oracle():
    pkg = os.path.join(ROOT, "paper_2301_03251_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".hpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text, f"{f} mentions the oracle"


def _err(fn):
    with pytest.raises(Q.QLError) as e:
        fn()
    return e.value.code


G1 = [[W.RY, 0, -1, W.SRC_WEIGHT, 0]]


@pytest.mark.parametrize("gates,n,F,P,code", [
    ([[W.RY, 3, -1, W.SRC_WEIGHT, 0]], 3, 0, 1, -1),     # qubit out of range
    ([[W.CNOT, 1, 1, 0, 0]], 3, 0, 0, -1),               # q0 == q1
    ([[W.CZ, 0, 5, 0, 0]], 3, 0, 0, -1),                 # q1 out of range
    ([[W.H, 0, -1, W.SRC_WEIGHT, 0]], 3, 0, 1, -1),      # H with a source
    ([[W.RX, 0, -1, W.SRC_NONE, 0]], 3, 0, 1, -1),       # rotation without source
    ([[W.RZ, 0, -1, W.SRC_INPUT, 2]], 3, 2, 0, -1),      # input index out of range
    ([[W.RZ, 0, -1, W.SRC_WEIGHT, -1]], 3, 0, 1, -1),    # negative weight index
    ([[10, 0, -1, 0, 0]], 3, 0, 0, -1),                  # unknown kind
    ([[W.CRY, 1, 1, W.SRC_WEIGHT, 0]], 3, 0, 1, -1),     # controlled rotation with q0 == q1
    ([[W.CRX, 0, 1, W.SRC_NONE, 0]], 3, 0, 1, -1),       # controlled rotation without source
    ([[W.CRZ, 0, -1, W.SRC_WEIGHT, 0]], 3, 0, 1, -1),    # controlled rotation without target
    ([[W.PAULI, 0, -1, W.SRC_WEIGHT, 0]], 3, 0, 1, -1),  # channel uniform must be an input
    ([[W.RY, 0, 1, W.SRC_WEIGHT, 0]], 3, 0, 1, -1),      # one-qubit gate with q1
    (G1, 0, 0, 1, -1),                                   # n = 0
    (G1, 33, 0, 1, -1),                                  # n = 33
])
def test_create_rejects(lib, gates, n, F, P, code):
    assert _err(lambda: Q.Circuit(n, np.array(gates, np.int32), F, P)) == code


@pytest.mark.parametrize("opts", [dict(log_regs=1), dict(log_regs=6), dict(log_threads=5),
                                  dict(log_threads=10), dict(low_qubits=9), dict(wg_per_sample=-1),
                                  dict(rz_groups=2), dict(cz_groups=1), dict(cz_groups=-2)])
def test_create_rejects_options(lib, opts):
    assert _err(lambda: Q.Circuit(14, np.array(G1, np.int32), 0, 1, **opts)) == -3


def test_create_null_pointers(lib):
    h = ctypes.c_void_p()
    assert lib.ql_circuit_create(3, None, 2, 0, 0, ctypes.byref(h)) == -1
    assert lib.ql_circuit_create(3, None, 0, 0, 0, None) == -1
    assert lib.ql_last_error()


def test_call_validation_before_launch(lib):
    """Errors that are caught before anything touches a GPU."""
    c = Q.Circuit(14, np.array(G1, np.int32), 0, 1)
    need = c.workspace_bytes("c64", 2)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    # NULL workspace, workspace too small, NULL expz, NULL weights, bad batch, bad dtype
    assert _err(lambda: c.forward_backward_raw("c64", 2, None, fake, fake, fake, None, None,
                                               None, need, None)) == -1
    assert _err(lambda: c.forward_backward_raw("c64", 2, None, fake, fake, fake, None, None,
                                               fake, need - 1, None)) == -2
    assert _err(lambda: c.forward_backward_raw("c64", 2, None, fake, fake, None, None, None,
                                               fake, need, None)) == -1
    assert _err(lambda: c.forward_raw("c64", 2, None, None, fake, fake, need, None)) == -1
    assert _err(lambda: c.forward_backward_raw("c64", 2, None, fake, None, fake, None, None,
                                               fake, need, None)) == -1
    assert _err(lambda: c.forward_raw("c64", 0, None, fake, fake, fake, need, None)) == -1
    assert _err(lambda: c.forward_raw(7, 2, None, fake, fake, fake, need, None)) == -1
    assert _err(lambda: c.workspace_bytes("c64", 1 << 31)) == -1


def test_param_shift_validation_and_workspace(lib):
    """Parameter-shift entry point: errors before launch and workspace size
    (one chunk's forward layout + its <Z> values + one fp64 per circuit)."""
    wl = W.get("10q")
    c = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    S = c.plan_info("c64")["n_param_gates"]
    B = 4
    total = B * (2 * S + 1)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    need = c.param_shift_workspace_bytes("c64", B, 64)
    assert _err(lambda: c.param_shift_raw("c64", B, fake, fake, None, fake, None, None, 64, fake,
                                          need, None)) == -1           # grad_out NULL
    assert _err(lambda: c.param_shift_raw("c64", B, fake, fake, fake, fake, None, None, 64, fake,
                                          need - 1, None)) == -2       # workspace too small
    assert _err(lambda: c.param_shift_raw("c64", B, fake, fake, fake, fake, None, None, -1, fake,
                                          need, None)) == -1           # negative chunk
    assert _err(lambda: c.param_shift_workspace_bytes("c64", 0, 0)) == -1
    chunk64 = c.workspace_bytes("c64", 64, Q.MODE_FWD)
    assert chunk64 + 64 * wl.n * 4 + total * 8 <= need <= chunk64 + 64 * wl.n * 4 + total * 8 + 512
    # chunk 0 means all circuits at once
    assert c.param_shift_workspace_bytes("c64", B, 0) == c.param_shift_workspace_bytes("c64", B, total)
    assert c.param_shift_workspace_bytes("c64", B, 10 * total) == c.param_shift_workspace_bytes("c64", B, 0)


def test_state_and_sample_validation(lib):
    """ql_state / ql_sample: errors before launch and workspace sizes."""
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    c = Q.Circuit(14, W.random_circuit(14, 40, 0, 1, seed=3), 0, 1, max_gates_per_pass=5)
    need = c.state_workspace_bytes("c64", 2)
    # the caller's state buffer is the working state: the workspace holds none
    assert need + 2 * (1 << 14) * 8 == c.workspace_bytes("c64", 2, Q.MODE_FWD)
    assert _err(lambda: c.state_raw("c64", 2, None, fake, None, fake, need, None)) == -1
    assert _err(lambda: c.state_raw("c64", 2, None, fake, fake, fake, need - 1, None)) == -2
    # per block of 4096 amplitudes: the prefix of block totals and 64 chunk sums
    assert Q.sample_workspace_bytes(30, 3) == 3 * (1 << 18) * 8 * 65
    assert Q.sample_workspace_bytes(5, 1) == 256 + 64 * 8
    assert _err(lambda: Q.sample_workspace_bytes(0, 1)) == -1
    assert _err(lambda: Q.sample_workspace_bytes(33, 1)) == -1
    ws = Q.sample_workspace_bytes(10, 2)
    raw = Q.qlayer.sample_raw
    assert _err(lambda: raw("c64", 10, 2, None, 4, fake, fake, None, fake, ws, None)) == -1  # psi NULL
    assert _err(lambda: raw("c64", 10, 2, fake, 4, None, fake, None, fake, ws, None)) == -1  # uniforms NULL
    assert _err(lambda: raw("c64", 10, 2, fake, -1, fake, fake, None, fake, ws, None)) == -1  # shots < 0
    assert _err(lambda: raw("c64", 10, 2, fake, 4, fake, fake, None, fake, ws - 1, None)) == -2
    assert _err(lambda: raw("c128", 32, 1, fake, 4, fake, fake, None, fake, 1 << 30, None)) == -3


def test_workspace_arithmetic(lib):
    wl = W.get("30q")
    c = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    S = (1 << 30) * 8
    fb = c.workspace_bytes("c64", 1)
    fw = c.workspace_bytes("c64", 1, Q.MODE_FWD)
    assert 2 * S <= fb < 2 * S + (64 << 20)      # psi + lambda + small tables/partials
    assert S <= fw < S + (64 << 20)              # psi only
    assert c.workspace_bytes("c128", 1) >= 4 * S
    m = c.plan_info("c64")["n_passes"]
    # with a product prefix the last backward pass also stores lambda (the
    # environment of the prefix gates is read from it)
    assert c.plan_info("c64")["n_prefix_gates"] == 90
    assert c.state_bytes("c64", 1) == (6 * m - 5) * S
    assert c.state_bytes("c64", 1, Q.MODE_FWD) == (2 * m - 2) * S
    off = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights, product_prefix=-1)
    m2 = off.plan_info("c64")["n_passes"]
    assert off.plan_info("c64")["n_prefix_gates"] == 0
    assert off.state_bytes("c64", 1) == (6 * m2 - 6) * S
    small = Q.Circuit(4, W.get("4q").gates(), 4, 16)
    assert small.state_bytes("c128", 8) == 0.0   # whole state in LDS: no HBM state traffic
    # kept forward states: lambda plus one state per pass but the last (no
    # separate psi buffer), one state write fewer per backward pass
    keep = c.workspace_bytes("c64", 1, Q.MODE_FWD_BWD_KEEP)
    assert m * S <= keep < m * S + (64 << 20)
    assert keep - fb == (m - 2) * S
    assert c.state_bytes("c64", 1, Q.MODE_FWD_BWD_KEEP) == (5 * m - 4) * S
    assert small.workspace_bytes("c64", 8, Q.MODE_FWD_BWD_KEEP) == small.workspace_bytes("c64", 8)
    assert _err(lambda: c.workspace_bytes("c64", 1, 3)) == -1


@pytest.mark.parametrize("name", ["16q", "24q", "30q"])
def test_rz_groups_in_workload_plans(lib, name):
    """The workloads' RZs on register bits form groups; the option turns them off."""
    wl = W.get(name)
    on = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    off = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights, rz_groups=-1)
    for dt in ("c64", "c128"):
        assert on.plan_info(dt)["n_rz_groups"] > 0 and on.plan_info(dt)["n_ryz_pairs"] > 0
        assert off.plan_info(dt)["n_rz_groups"] == 0 and off.plan_info(dt)["n_ryz_pairs"] == 0
        assert on.plan_info(dt)["n_passes"] == off.plan_info(dt)["n_passes"]
        # grouping moves ops within a pass, never between passes
        assert np.array_equal(on.schedule(dt)[0], off.schedule(dt)[0])
    assert _err(lambda: Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights, rz_groups=1)) == -3


def test_timing_mask(lib):
    """ql_timing_enable takes a mask of kernel classes (0..15)."""
    c = Q.Circuit(14, np.array(G1, np.int32), 0, 1)
    for m in (0, 1, 2, 15):
        assert lib.ql_timing_enable(c.handle, m) == 0
    for m in (-1, 16):
        assert lib.ql_timing_enable(c.handle, m) == -1
    c.timing(True, 1)
    c.timing(False)


def test_keep_mode_embeddings_and_single_pass(lib):
    # an embedded initial state keeps its own buffer; a one-pass tiled circuit
    # has nothing to keep
    n = 12
    gates = W.random_circuit(n, 40, 2 ** n, 6, seed=3)
    emb = Q.Circuit(n, gates, 2 ** n, 6, embed=(W.EMBED_AMPLITUDE, 0), log_regs=2, log_threads=6,
                    max_gates_per_pass=8)
    m = emb.plan_info("c64")["n_passes"]
    assert m > 2
    S = (1 << n) * 8 * 3
    assert emb.workspace_bytes("c64", 3, Q.MODE_FWD_BWD_KEEP) - emb.workspace_bytes("c64", 3) == (m - 1) * S
    one = Q.Circuit(n, gates[:1], 2 ** n, 6, force_tiled=1)
    assert one.plan_info("c64")["n_passes"] == 1
    assert one.workspace_bytes("c64", 3, Q.MODE_FWD_BWD_KEEP) == one.workspace_bytes("c64", 3)


def _check_schedule(c, gates, dtype):
    pog, order = c.schedule(dtype)
    G = gates.shape[0]
    assert sorted(order.tolist()) == list(range(G)), "every gate scheduled exactly once"
    assert np.all(pog >= 0)
    pos = np.empty(G, dtype=np.int64)
    pos[order] = np.arange(G)
    # passes are contiguous in the execution order
    assert np.all(np.diff(pog[order]) >= 0)
    # gates that share a qubit keep their relative order
    last = {}
    for i, g in enumerate(gates):
        qs = [int(g[1])] + ([int(g[2])] if g[0] in (W.CNOT, W.CZ) + W.CONTROLLED else [])
        for q in qs:
            if q in last:
                assert pos[last[q]] < pos[i], f"gate {i} overtakes gate {last[q]} on qubit {q}"
            last[q] = i


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_workload_plans(lib, name):
    wl = W.get(name)
    c = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    for dt in ("c64", "c128"):
        _check_schedule(c, wl.gates(), dt)
        info = c.plan_info(dt)
        assert info["n_param_gates"] == sum(1 for g in wl.gates() if g[0] in W.ROTATIONS)
        if wl.n < 8:  # below one minimal register tile: whole state in LDS
            assert info["kernel"] == 0 and info["n_passes"] == 1
        else:
            assert info["kernel"] == 1 and info["tile_qubits"] == info["log_regs"] + info["log_threads"]
        whole = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights, force_tiled=-1).plan_info(dt)
        assert whole["kernel"] == (0 if wl.n <= (12 if dt == "c64" else 11) else 1)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("opts", [dict(force_tiled=1), dict(force_tiled=1, max_gates_per_pass=1),
                                  dict(log_regs=2, log_threads=6, low_qubits=1),
                                  dict(log_regs=3, log_threads=7, max_gates_per_pass=5)])
def test_random_plans(lib, seed, opts):
    n = 10 + seed % 5
    gates = W.random_circuit(n, 150, 4, 6, seed=seed)
    c = Q.Circuit(n, gates, 4, 6, **opts)
    for dt in ("c64", "c128"):
        _check_schedule(c, gates, dt)
        info = c.plan_info(dt)
        if opts.get("max_gates_per_pass") == 1:  # one pass per gate outside the product prefix
            assert info["n_passes"] == gates.shape[0] - info["n_prefix_gates"]


def test_cz_groups_plan(lib):
    """The 16-qubit workload's rings of CZs run as sign ops: with groups on,
    the CZs of each layout between rotations form one op (128 CZs: 17 groups
    and one CZ on its own at c64); off, none. Passes and layout changes are
    the same either way, and the schedule stays valid."""
    wl = W.get("16q")
    on = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    off = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights, cz_groups=-1)
    for dt in ("c64", "c128"):
        a, b = on.plan_info(dt), off.plan_info(dt)
        assert a["n_cz_groups"] > 0 and b["n_cz_groups"] == 0
        for key in ("n_passes", "n_transposes", "n_lane_swaps", "n_prefix_gates"):
            assert a[key] == b[key], key
        pog, order = on.schedule(dt)
        assert sorted(order.tolist()) == list(range(len(wl.gates())))
    assert on.plan_info("c64")["n_cz_groups"] == 17
    # a circuit without CZs has no groups
    w30 = W.get("30q")
    assert Q.Circuit(w30.n, w30.gates(), w30.n_inputs, w30.n_weights).plan_info("c64")["n_cz_groups"] == 0


def test_product_prefix_plan(lib):
    """The product-state prefix: every qubit's one-qubit gates before any
    two-qubit gate or Pauli channel touches it; none with an embedding or when
    turned off; a circuit of one-qubit gates only is one pass of no ops. The
    prefix gates are reported in pass 0, first, and every schedule stays
    valid."""
    wl = W.get("30q")
    c = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
    for dt in ("c64", "c128"):
        assert c.plan_info(dt)["n_prefix_gates"] == 90  # RY encoding, RY and RZ of layer 1
        pog, order = c.schedule(dt)
        assert np.all(pog[order[:90]] == 0)
        assert sorted(order[:90].tolist()) == [i for i, g in enumerate(wl.gates())
                                               if i < 30 or (30 <= i and g[0] in (W.RY, W.RZ) and i < 90)]
    g = np.array([[W.RY, 0, -1, W.SRC_WEIGHT, 0], [W.RX, 1, -1, W.SRC_WEIGHT, 1], [W.H, 2, -1, 0, 0],
                  [W.CNOT, 0, 1, 0, 0], [W.RY, 0, -1, W.SRC_WEIGHT, 2],
                  [W.PAULI, 2, -1, W.SRC_INPUT, 0], [W.RZ, 2, -1, W.SRC_WEIGHT, 3],
                  [W.RY, 9, -1, W.SRC_WEIGHT, 4]], np.int32)
    c = Q.Circuit(10, g, 1, 5, pauli_p=[[0.1, 0.1, 0.1]], product_prefix=1)
    assert c.plan_info("c64")["n_prefix_gates"] == 4   # RY q0, RX q1, H q2, RY q9
    _check_schedule(c, g, "c64")
    assert Q.Circuit(10, g, 1, 5, pauli_p=[[0.1, 0.1, 0.1]], product_prefix=-1).plan_info("c64")["n_prefix_gates"] == 0
    only = np.array([[W.RY, q, -1, W.SRC_WEIGHT, q % 3] for q in range(12)] + [[W.H, 3, -1, 0, 0]], np.int32)
    c = Q.Circuit(12, only, 0, 3, product_prefix=1)
    assert c.plan_info("c64")["n_prefix_gates"] == 13 and c.plan_info("c64")["n_passes"] == 1
    _check_schedule(c, only, "c64")
    emb = W.get("qae")
    assert Q.Circuit(emb.n, emb.gates(), emb.n_inputs, emb.n_weights, embed=emb.embed,
                     force_tiled=1).plan_info("c64")["n_prefix_gates"] == 0
    assert _err(lambda: Q.Circuit(10, g, 1, 5, pauli_p=[[0.1, 0.1, 0.1]], product_prefix=2)) == -3


def test_pass_counts_are_small(lib):
    """Fusion budget of the light-cone planner on the large workloads: far fewer
    passes than layers x qubits."""
    for name, limit in (("16q", 8), ("24q", 20), ("30q", 16)):
        wl = W.get(name)
        c = Q.Circuit(wl.n, wl.gates(), wl.n_inputs, wl.n_weights)
        assert c.plan_info("c64")["n_passes"] <= limit, name


def test_pass_search(lib):
    """The three tile choices on the 30-qubit CNOT staircase: the look-ahead
    (pass_search=1) needs fewer passes than the widest-pass greedy (-1) and
    leaves no nearly empty pass at the end of the chains; the default (0)
    takes the beam search's plan, fewer passes still (9 in complex64). All
    plans are valid. The option takes -1, 0 or 1 only."""
    wl = W.get("30q")
    gates = wl.gates()
    best = Q.Circuit(wl.n, gates, wl.n_inputs, wl.n_weights)
    look = Q.Circuit(wl.n, gates, wl.n_inputs, wl.n_weights, pass_search=1)
    greedy = Q.Circuit(wl.n, gates, wl.n_inputs, wl.n_weights, pass_search=-1)
    for dt in ("c64", "c128"):
        for c in (best, look, greedy):
            _check_schedule(c, gates, dt)
        n0, n1, n2 = (c.plan_info(dt)["n_passes"] for c in (best, look, greedy))
        assert n0 < n1 < n2, (dt, n0, n1, n2)
        sizes = np.bincount(look.schedule(dt)[0])
        assert sizes.min() >= 30, (dt, sizes)
        assert np.bincount(greedy.schedule(dt)[0]).min() < 30
    assert best.plan_info("c64")["n_passes"] == 9
    for bad in (2, -2):
        assert _err(lambda: Q.Circuit(wl.n, gates, wl.n_inputs, wl.n_weights, pass_search=bad)) == -3
    # on every workload: default <= look-ahead <= greedy in passes, all valid
    for name in W.WORKLOADS:
        w2 = W.get(name)
        cs = [Q.Circuit(w2.n, w2.gates(), w2.n_inputs, w2.n_weights, pass_search=ps) for ps in (0, 1, -1)]
        for dt in ("c64", "c128"):
            n = [c.plan_info(dt)["n_passes"] for c in cs]
            assert n[0] <= n[1] <= n[2], (name, dt, n)
            _check_schedule(cs[0], w2.gates(), dt)


# ---------------------------------------------------------------------------
# controlled rotations, embeddings, Pauli channels (host side)

def _desc_err(n, gates, F, P, **kw):
    return _err(lambda: Q.Circuit(n, np.asarray(gates, np.int32), F, P, **kw))


def test_extension_validation(lib):
    pauli = [[W.PAULI, 0, -1, W.SRC_INPUT, 0]]
    assert _desc_err(2, pauli, 1, 0) == -1                                  # no probabilities
    assert _desc_err(2, pauli, 1, 0, pauli_p=[[-0.1, 0, 0]]) == -1          # negative
    assert _desc_err(2, pauli, 1, 0, pauli_p=[[0.5, 0.4, 0.2]]) == -1       # sum above 1
    Q.Circuit(2, np.asarray(pauli, np.int32), 1, 0, pauli_p=[[0.5, 0.25, 0.25]])
    assert _desc_err(3, G1, 2, 1, embed=(W.EMBED_BASIS, 0)) == -1           # 3 features needed
    assert _desc_err(3, G1, 5, 1, embed=(W.EMBED_BASIS, 3)) == -1
    Q.Circuit(3, np.asarray(G1, np.int32), 5, 1, embed=(W.EMBED_BASIS, 2))
    assert _desc_err(3, G1, 8, 1, embed=(W.EMBED_AMPLITUDE, 1)) == -1       # 2^3 from feature 1
    assert _desc_err(3, G1, 9, 1, embed=(W.EMBED_AMPLITUDE, -1)) == -1
    Q.Circuit(3, np.asarray(G1, np.int32), 9, 1, embed=(W.EMBED_AMPLITUDE, 1))
    assert _desc_err(3, G1, 9, 1, embed=(7, 0)) == -1                       # unknown embedding


def test_extension_slot_counts(lib):
    """A controlled rotation is two trainable half-angle rotations; Pauli
    channels add no trainable slot."""
    gates = np.asarray([[W.CRX, 0, 1, W.SRC_WEIGHT, 0], [W.CRY, 1, 2, W.SRC_INPUT, 0],
                        [W.CRZ, 2, 0, W.SRC_WEIGHT, 1], [W.RX, 1, -1, W.SRC_WEIGHT, 1],
                        [W.PAULI, 2, -1, W.SRC_INPUT, 1], [W.PAULI, 0, -1, W.SRC_INPUT, 2]], np.int32)
    c = Q.Circuit(3, gates, 3, 2, pauli_p=[[0.1, 0.0, 0.2], [0.0, 0.0, 0.0]])
    for dt in ("c64", "c128"):
        assert c.plan_info(dt)["n_param_gates"] == 7
        pog, order = c.schedule(dt)
        assert pog[5] == -1 and order[0] == 5          # a channel with all p = 0 applies nothing
        assert sorted(order.tolist()) == list(range(6))
    qae = W.get("qae")
    cq = Q.Circuit(qae.n, qae.gates(), qae.n_inputs, qae.n_weights, embed=qae.embed)
    assert qae.n_weights == 60 and cq.plan_info("c64")["n_param_gates"] == 24 + 2 * 36


@pytest.mark.parametrize("seed", range(4))
def test_extension_schedules(lib, seed):
    n = 9 + seed
    kinds = (W.H, W.RX, W.RY, W.RZ, W.CNOT, W.CZ, W.CRX, W.CRY, W.CRZ)
    gates = W.random_circuit(n, 120, 4, 6, seed=300 + seed, kinds=kinds)
    gates, pp, nch = W.with_depolarizing(gates, n, 4, 0.05, every=17)
    for opts in (dict(), dict(force_tiled=1, log_regs=3, log_threads=6)):
        c = Q.Circuit(n, gates, 4 + nch, 6, pauli_p=pp, **opts)
        for dt in ("c64", "c128"):
            _check_schedule(c, gates, dt)


def test_param_shift_rejects_amplitude_input_grads(lib):
    n, F = 3, 8
    c = Q.Circuit(n, np.asarray(G1, np.int32), F, 1, embed=(W.EMBED_AMPLITUDE, 0))
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    need = c.param_shift_workspace_bytes("c64", 2, 0)
    assert _err(lambda: c.param_shift_raw("c64", 2, fake, fake, fake, fake, fake, None, 0, fake,
                                          need, None)) == -3
