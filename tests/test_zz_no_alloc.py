"""The allocation-free entry point (ql_forward_backward_static) against
ql_forward_backward on the same inputs, through the C ABI (needs an MI355X).

Two calls in a row, the second with a smaller batch, so that the second reads
a static scratch buffer that still holds the first call's contents; plus the
refusal of a call whose scratch would exceed the static maximum.
"""

from __future__ import annotations

import ctypes

import numpy as np
import pytest

import workloads as W
from parity import check

torch = pytest.importorskip("torch")
import paper_2301_03251_amd as Q  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = {"c64": 1e-5, "c128": 1e-12}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.load()


def _dev(a, dtype):
    real = torch.float32 if dtype == "c64" else torch.float64
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=real)


def _host(t):
    return t.cpu().double().numpy()


def _static(circ, dtype, x, w, g):
    """ql_forward_backward_static called directly through ctypes."""
    lib = Q.load()
    B = x.shape[0]
    real = torch.float32 if dtype == "c64" else torch.float64
    xt, wt, gt = _dev(x, dtype), _dev(w, dtype), _dev(g, dtype)
    e = torch.full((B, circ.n), float("nan"), dtype=real, device="cuda")
    gx = torch.full((B, circ.n_inputs), float("nan"), dtype=real, device="cuda")
    gw = torch.full((circ.n_weights,), float("nan"), dtype=real, device="cuda")
    p = lambda t: ctypes.c_void_p(t.data_ptr()) if t.numel() else None  # noqa: E731
    rc = lib.ql_forward_backward_static(circ.handle, Q.C64 if dtype == "c64" else Q.C128, B, p(xt), p(wt),
                                        p(gt), p(e), p(gx), p(gw),
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, lib.ql_last_error()
    torch.cuda.synchronize()
    return {"expz": _host(e), "grad_inputs": _host(gx), "grad_weights": _host(gw)}


def _workspace(circ, dtype, x, w, g):
    r = Q.Runner(circ, dtype)
    e, gx, gw = r.forward_backward(_dev(x, dtype), _dev(w, dtype), _dev(g, dtype))
    torch.cuda.synchronize()
    return {"expz": _host(e), "grad_inputs": _host(gx), "grad_weights": _host(gw)}


CASES = [
    # name, n, gates, batch (first call), batch (second call), dtype, options
    ("10q tile", 10, None, 64, 5, "c64", {}),
    ("14q tiles", 14, 120, 6, 1, "c64", {}),
    ("13q tiles c128", 13, 90, 4, 3, "c128", {}),
    ("6q whole state", 6, 50, 40, 7, "c128", {}),
]


@pytest.mark.parametrize("name,n,G,B1,B2,dtype,opts", CASES, ids=[c[0].replace(" ", "-") for c in CASES])
def test_static_matches_workspace_call(name, n, G, B1, B2, dtype, opts):
    if G is None:
        wl = W.scaled(W.get("10q"), batch=B1)
        gates, F, P = wl.gates(), wl.n_inputs, wl.n_weights
    else:
        F, P = 4, 6
        gates = W.random_circuit(n, G, F, P, seed=n * 31 + G)
    circ = Q.Circuit(n, gates, F, P, **opts)
    for call, B in enumerate((B1, B2)):
        x, w, g = W.random_inputs(B, F, P, n, seed=100 * call + n, dtype=dtype)
        want = _workspace(circ, dtype, x, w, g)
        got = _static(circ, dtype, x, w, g)
        check(got, want, TOL[dtype], f"static vs workspace {name} call {call} B={B}")


def test_static_refuses_beyond_its_maximum():
    n, F, P = 20, 2, 3
    gates = W.random_circuit(n, 30, F, P, seed=5)
    circ = Q.Circuit(n, gates, F, P)
    B = 64  # 64 samples of 2^20 amplitudes: 512 MiB of states
    assert circ.workspace_bytes("c64", B, Q.MODE_FWD_BWD) > Q.STATIC_SCRATCH_BYTES
    x, w, g = W.random_inputs(B, F, P, n, seed=6, dtype="c64")
    with pytest.raises(Q.QLError) as e:
        Q.Runner(circ, "c64").forward_backward_static(_dev(x, "c64"), _dev(w, "c64"), _dev(g, "c64"))
    assert e.value.code == -2
