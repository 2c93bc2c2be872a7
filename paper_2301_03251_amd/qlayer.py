"""ctypes binding of ``libqlayer.so`` (C ABI in ``include/qlayer.h``).

Argument marshalling only: every step of the forward pass, the adjoint sweep
and the reductions runs in the library's HIP kernels. PyTorch supplies device
memory and the current stream. There is no CPU fallback: if the library is
missing the import of the entry points raises.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqlayer.so")

C64, C128 = 0, 1
MODE_FWD, MODE_FWD_BWD, MODE_FWD_BWD_KEEP = 0, 1, 2
STATIC_SCRATCH_BYTES = 64 << 20  # QL_STATIC_SCRATCH_BYTES of qlayer.h
H, RX, RY, RZ, CNOT, CZ, CRX, CRY, CRZ, PAULI = range(10)
SRC_NONE, SRC_INPUT, SRC_WEIGHT = 0, 1, 2
EMBED_NONE, EMBED_BASIS, EMBED_AMPLITUDE = 0, 1, 2
DTYPES = {"c64": C64, "c128": C128}
ERRORS = {-1: "QL_EINVAL", -2: "QL_ENOMEM", -3: "QL_EUNSUPPORTED", -4: "QL_EHIP"}


class QLError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class _Options(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("log_regs", "log_threads", "low_qubits",
                                              "max_gates_per_pass", "force_tiled",
                                              "wg_per_sample", "rz_groups", "pass_search",
                                              "product_prefix", "cz_groups")]


class _Desc(ctypes.Structure):
    _fields_ = [("embedding", ctypes.c_int32), ("embed_first", ctypes.c_int32),
                ("pauli_p", ctypes.c_void_p)]


class _PlanInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("kernel", "n_passes", "tile_qubits", "log_regs",
                                              "log_threads", "low_qubits", "n_transposes",
                                              "n_param_gates", "n_lane_swaps", "n_rz_groups",
                                              "n_ryz_pairs", "n_prefix_gates", "n_cz_groups")]


_lib = None
EXPORTS = ("ql_circuit_create", "ql_circuit_create_ex", "ql_circuit_create_desc", "ql_circuit_destroy",
           "ql_workspace_bytes", "ql_forward", "ql_forward_backward", "ql_last_error",
           "ql_param_shift_workspace_bytes", "ql_param_shift", "ql_state_workspace_bytes",
           "ql_state", "ql_sample_workspace_bytes", "ql_sample",
           "ql_plan_info_get", "ql_plan_schedule", "ql_plan_state_bytes",
           "ql_timing_enable", "ql_timing_read")


def load():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python paper_2301_03251_amd/build.py` (no CPU fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.ql_circuit_create.argtypes = [I32, P, I32, I32, I32, ctypes.POINTER(P)]
    lib.ql_circuit_create_ex.argtypes = [I32, P, I32, I32, I32, ctypes.POINTER(_Options),
                                         ctypes.POINTER(P)]
    lib.ql_circuit_create_desc.argtypes = [I32, P, I32, I32, I32, ctypes.POINTER(_Desc),
                                           ctypes.POINTER(_Options), ctypes.POINTER(P)]
    lib.ql_circuit_destroy.argtypes = [P]
    lib.ql_circuit_destroy.restype = None
    lib.ql_workspace_bytes.argtypes = [P, ctypes.c_int, I64, ctypes.c_int, ctypes.POINTER(SZ)]
    lib.ql_forward.argtypes = [P, ctypes.c_int, I64, P, P, P, P, SZ, P]
    lib.ql_forward_backward.argtypes = [P, ctypes.c_int, I64, P, P, P, P, P, P, P, SZ, P]
    lib.ql_forward_backward_static.argtypes = [P, ctypes.c_int, I64, P, P, P, P, P, P, P]
    lib.ql_param_shift_workspace_bytes.argtypes = [P, ctypes.c_int, I64, I64, ctypes.POINTER(SZ)]
    lib.ql_param_shift.argtypes = [P, ctypes.c_int, I64, P, P, P, P, P, P, I64, P, SZ, P]
    lib.ql_state_workspace_bytes.argtypes = [P, ctypes.c_int, I64, ctypes.POINTER(SZ)]
    lib.ql_state.argtypes = [P, ctypes.c_int, I64, P, P, P, P, SZ, P]
    lib.ql_sample_workspace_bytes.argtypes = [I32, I64, ctypes.POINTER(SZ)]
    lib.ql_sample.argtypes = [ctypes.c_int, I32, I64, P, I64, P, P, P, P, SZ, P]
    lib.ql_last_error.argtypes = []
    lib.ql_last_error.restype = ctypes.c_char_p
    lib.ql_plan_info_get.argtypes = [P, ctypes.c_int, ctypes.POINTER(_PlanInfo)]
    lib.ql_plan_schedule.argtypes = [P, ctypes.c_int, P, P]
    lib.ql_plan_state_bytes.argtypes = [P, ctypes.c_int, I64, ctypes.c_int,
                                        ctypes.POINTER(ctypes.c_double)]
    lib.ql_timing_enable.argtypes = [P, ctypes.c_int]
    lib.ql_timing_read.argtypes = [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I32)]
    for name in ("ql_circuit_create", "ql_circuit_create_ex", "ql_circuit_create_desc",
                 "ql_workspace_bytes", "ql_forward",
                 "ql_forward_backward", "ql_param_shift_workspace_bytes", "ql_param_shift",
                 "ql_state_workspace_bytes", "ql_state", "ql_sample_workspace_bytes", "ql_sample",
                 "ql_plan_info_get", "ql_plan_schedule",
                 "ql_plan_state_bytes", "ql_timing_enable", "ql_timing_read"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc):
    if rc != 0:
        raise QLError(rc, load().ql_last_error().decode())


def _dt(dtype):
    return DTYPES[dtype] if isinstance(dtype, str) else int(dtype)


class Circuit:
    """A validated gate list with its pass plans (``ql_circuit_create_desc``).

    ``embed = (kind, first)`` selects an initial-state embedding (``EMBED_*``)
    reading features from ``first`` on; ``pauli_p[c] = (p_x, p_y, p_z)`` are
    the probabilities of the c-th ``PAULI`` gate. Other keyword arguments are
    planning options (``ql_options`` fields).
    """

    def __init__(self, n_qubits, gates, n_inputs, n_weights, embed=None, pauli_p=None, **options):
        lib = load()
        g = np.ascontiguousarray(np.asarray(gates, dtype=np.int32).reshape(-1, 5))
        self.n = int(n_qubits)
        self.gates = g
        self.n_inputs, self.n_weights = int(n_inputs), int(n_weights)
        opts = _Options(**{k: int(v) for k, v in options.items()})
        pp = None
        if pauli_p is not None:
            pp = np.ascontiguousarray(np.asarray(pauli_p, dtype=np.float64).reshape(-1, 3))
        kind, first = (EMBED_NONE, 0) if embed is None else (int(embed[0]), int(embed[1]))
        self.embed = (kind, first)
        desc = _Desc(kind, first, None if pp is None else pp.ctypes.data_as(ctypes.c_void_p))
        h = ctypes.c_void_p()
        _check(lib.ql_circuit_create_desc(self.n, g.ctypes.data_as(ctypes.c_void_p), g.shape[0],
                                          self.n_inputs, self.n_weights, ctypes.byref(desc),
                                          ctypes.byref(opts), ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            load().ql_circuit_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def workspace_bytes(self, dtype, batch, mode=MODE_FWD_BWD) -> int:
        out = ctypes.c_size_t()
        _check(load().ql_workspace_bytes(self._h, _dt(dtype), int(batch), int(mode), ctypes.byref(out)))
        return out.value

    def plan_info(self, dtype) -> dict:
        info = _PlanInfo()
        _check(load().ql_plan_info_get(self._h, _dt(dtype), ctypes.byref(info)))
        return {f: getattr(info, f) for f, _ in _PlanInfo._fields_}

    def schedule(self, dtype):
        G = self.gates.shape[0]
        pog = np.zeros(max(G, 1), dtype=np.int32)
        order = np.zeros(max(G, 1), dtype=np.int32)
        _check(load().ql_plan_schedule(self._h, _dt(dtype), pog.ctypes.data_as(ctypes.c_void_p),
                                       order.ctypes.data_as(ctypes.c_void_p)))
        return pog[:G], order[:G]

    def state_bytes(self, dtype, batch, mode=MODE_FWD_BWD) -> float:
        out = ctypes.c_double()
        _check(load().ql_plan_state_bytes(self._h, _dt(dtype), int(batch), int(mode), ctypes.byref(out)))
        return out.value

    def timing(self, enable: bool, classes: int = 0xF):
        """Bracket the launches of the kernel classes in the mask `classes`
        (bit 0 tile passes, 1 whole-state kernel, 2 binding, 3 reductions)."""
        _check(load().ql_timing_enable(self._h, int(classes) & 0xF if enable else 0))

    def timing_read(self):
        ms = (ctypes.c_double * 4)()
        cnt = (ctypes.c_int32 * 4)()
        _check(load().ql_timing_read(self._h, ms, cnt))
        return list(ms), list(cnt)

    def param_shift_workspace_bytes(self, dtype, batch, max_chunk=0) -> int:
        out = ctypes.c_size_t()
        _check(load().ql_param_shift_workspace_bytes(self._h, _dt(dtype), int(batch), int(max_chunk),
                                                     ctypes.byref(out)))
        return out.value

    def state_workspace_bytes(self, dtype, batch) -> int:
        out = ctypes.c_size_t()
        _check(load().ql_state_workspace_bytes(self._h, _dt(dtype), int(batch), ctypes.byref(out)))
        return out.value

    def state_raw(self, dtype, batch, inputs, weights, psi, ws, ws_bytes, stream):
        _check(load().ql_state(self._h, _dt(dtype), int(batch), inputs, weights, psi, ws,
                               int(ws_bytes), stream))

    # raw entry points: device pointers as ints, stream as int (hipStream_t)
    def forward_raw(self, dtype, batch, inputs, weights, expz, ws, ws_bytes, stream):
        _check(load().ql_forward(self._h, _dt(dtype), int(batch), inputs, weights, expz, ws,
                                 int(ws_bytes), stream))

    def forward_backward_raw(self, dtype, batch, inputs, weights, grad_out, expz, grad_inputs,
                             grad_weights, ws, ws_bytes, stream):
        _check(load().ql_forward_backward(self._h, _dt(dtype), int(batch), inputs, weights,
                                          grad_out, expz, grad_inputs, grad_weights, ws,
                                          int(ws_bytes), stream))

    def forward_backward_static_raw(self, dtype, batch, inputs, weights, grad_out, expz, grad_inputs,
                                    grad_weights, stream):
        _check(load().ql_forward_backward_static(self._h, _dt(dtype), int(batch), inputs, weights,
                                                 grad_out, expz, grad_inputs, grad_weights, stream))

    def param_shift_raw(self, dtype, batch, inputs, weights, grad_out, expz, grad_inputs,
                        grad_weights, max_chunk, ws, ws_bytes, stream):
        _check(load().ql_param_shift(self._h, _dt(dtype), int(batch), inputs, weights, grad_out,
                                     expz, grad_inputs, grad_weights, int(max_chunk), ws,
                                     int(ws_bytes), stream))


# ---------------------------------------------------------------------------
# torch plumbing (device memory and streams only)

def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


class Runner:
    """Holds a circuit, a dtype and a reusable device workspace.

    keep_states: forward_backward keeps the state after every tile pass in the
    workspace (QL_MODE_FWD_BWD_KEEP: fewer HBM bytes, m - 2 more states of
    memory for m passes) when True, never when False, and when None whenever
    the larger workspace fits in 80 % of the device's free memory. With two
    passes the sizes are equal and the library always keeps the state.

    The memory cost of the default can be large: with m tile passes the kept
    workspace holds m - 1 states of batch * 2^n amplitudes instead of 2. For
    the 30-qubit workload (9 passes, 8 GiB per state) that is a 72 GiB
    workspace against 16 GiB, for a step about 4 % faster (the backward passes then store no
    state). Pass keep_states=False when the device memory is needed for
    anything else (for example several layers of a model in one step)."""

    def __init__(self, circuit: Circuit, dtype="c64", device="cuda", keep_states=None):
        torch = _torch()
        self.c = circuit
        self.dtype = dtype
        self.real = torch.float32 if _dt(dtype) == C64 else torch.float64
        self.device = torch.device(device)
        self.keep_states = keep_states
        self._ws = None
        self._modes = {}
        self._sizes = {}

    def backward_mode(self, batch) -> int:
        """MODE_FWD_BWD_KEEP or MODE_FWD_BWD, as forward_backward will run (the
        first answer for a batch size is kept)."""
        mode = self._modes.get(batch)
        if mode is None:
            mode = self._modes[batch] = self._choose_mode(batch)
        return mode

    def _choose_mode(self, batch) -> int:
        info = self.c.plan_info(self.dtype)
        if info["kernel"] == 0 or info["n_passes"] < 2:
            return MODE_FWD_BWD  # whole state, or one tile pass: nothing to keep
        need = self.c.workspace_bytes(self.dtype, batch, MODE_FWD_BWD_KEEP)
        if need == self.c.workspace_bytes(self.dtype, batch, MODE_FWD_BWD):
            return MODE_FWD_BWD_KEEP  # two passes: the kept state replaces the psi buffer
        if self.keep_states is False:
            return MODE_FWD_BWD
        if self.keep_states:
            return MODE_FWD_BWD_KEEP
        have = self._ws.numel() if self._ws is not None else 0
        if need <= have:
            return MODE_FWD_BWD_KEEP
        free, _ = _torch().cuda.mem_get_info(self.device)
        return MODE_FWD_BWD_KEEP if need - have <= 0.8 * free else MODE_FWD_BWD

    def _need(self, batch, mode) -> int:
        key = (batch, mode)
        if key not in self._sizes:
            self._sizes[key] = self.c.workspace_bytes(self.dtype, batch, mode)
        return self._sizes[key]

    def workspace(self, batch, mode):
        torch = _torch()
        need = self._need(batch, mode)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        return self._ws

    def _args(self, inputs, weights, B):
        torch = _torch()
        x = inputs if inputs is not None else torch.empty((B, 0), dtype=self.real, device=self.device)
        w = weights if weights is not None else torch.empty(0, dtype=self.real, device=self.device)
        for t in (x, w):
            if t.dtype != self.real or t.device.type != "cuda" or not t.is_contiguous():
                raise ValueError("inputs/weights must be contiguous CUDA tensors of the layer's real dtype")
        return x, w

    def forward(self, inputs, weights, out=None):
        torch = _torch()
        B = int(inputs.shape[0])
        x, w = self._args(inputs, weights, B)
        expz = out if out is not None else torch.empty((B, self.c.n), dtype=self.real, device=self.device)
        ws = self.workspace(B, MODE_FWD)
        self.c.forward_raw(self.dtype, B, _ptr(x) if self.c.n_inputs else None,
                           _ptr(w) if self.c.n_weights else None, _ptr(expz), _ptr(ws), ws.numel(),
                           ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream))
        return expz

    def forward_backward(self, inputs, weights, grad_out, want_inputs=True, want_weights=True,
                         outs=None):
        torch = _torch()
        B = int(inputs.shape[0])
        x, w = self._args(inputs, weights, B)
        if grad_out.dtype != self.real or not grad_out.is_contiguous():
            raise ValueError("grad_out must be a contiguous tensor of the layer's real dtype")
        if outs is None:
            expz = torch.empty((B, self.c.n), dtype=self.real, device=self.device)
            gx = torch.empty((B, self.c.n_inputs), dtype=self.real, device=self.device) if want_inputs else None
            gw = torch.empty(self.c.n_weights, dtype=self.real, device=self.device) if want_weights else None
        else:
            expz, gx, gw = outs
        mode = self.backward_mode(B)
        ws = self.workspace(B, mode)
        # the library keeps the states whenever the workspace it is given holds
        # them, so the plain path is handed exactly its own size
        ws_bytes = ws.numel() if mode == MODE_FWD_BWD_KEEP else self._need(B, mode)
        self.c.forward_backward_raw(
            self.dtype, B, _ptr(x) if self.c.n_inputs else None, _ptr(w) if self.c.n_weights else None,
            _ptr(grad_out), _ptr(expz), _ptr(gx) if (gx is not None and self.c.n_inputs) else None,
            _ptr(gw) if (gw is not None and self.c.n_weights) else None, _ptr(ws), ws_bytes,
            ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream))
        return expz, gx, gw


    def forward_backward_static(self, inputs, weights, grad_out, outs=None):
        """forward_backward through the allocation-free entry point: the
        library's static per-GPU scratch instead of this runner's workspace
        (small circuits and batches only; calls on one GPU must not overlap)."""
        torch = _torch()
        B = int(inputs.shape[0])
        x, w = self._args(inputs, weights, B)
        if outs is None:
            outs = (torch.empty((B, self.c.n), dtype=self.real, device=self.device),
                    torch.empty((B, self.c.n_inputs), dtype=self.real, device=self.device),
                    torch.empty(self.c.n_weights, dtype=self.real, device=self.device))
        expz, gx, gw = outs
        self.c.forward_backward_static_raw(
            self.dtype, B, _ptr(x) if self.c.n_inputs else None, _ptr(w) if self.c.n_weights else None,
            _ptr(grad_out), _ptr(expz), _ptr(gx) if (gx is not None and self.c.n_inputs) else None,
            _ptr(gw) if (gw is not None and self.c.n_weights) else None,
            ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream))
        return expz, gx, gw

    def param_shift(self, inputs, weights, grad_out, max_chunk=0, want_inputs=True, want_weights=True,
                    outs=None):
        """The VJP of forward_backward by the two-term parameter-shift rule
        (shifted circuits folded into the batch, in chunks of max_chunk)."""
        torch = _torch()
        B = int(inputs.shape[0])
        x, w = self._args(inputs, weights, B)
        if grad_out.dtype != self.real or not grad_out.is_contiguous():
            raise ValueError("grad_out must be a contiguous tensor of the layer's real dtype")
        if outs is None:
            expz = torch.empty((B, self.c.n), dtype=self.real, device=self.device)
            gx = torch.empty((B, self.c.n_inputs), dtype=self.real, device=self.device) if want_inputs else None
            gw = torch.empty(self.c.n_weights, dtype=self.real, device=self.device) if want_weights else None
        else:
            expz, gx, gw = outs
        need = self.c.param_shift_workspace_bytes(self.dtype, B, max_chunk)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        ws = self._ws
        self.c.param_shift_raw(
            self.dtype, B, _ptr(x) if self.c.n_inputs else None, _ptr(w) if self.c.n_weights else None,
            _ptr(grad_out), _ptr(expz), _ptr(gx) if (gx is not None and self.c.n_inputs) else None,
            _ptr(gw) if (gw is not None and self.c.n_weights) else None, max_chunk, _ptr(ws), ws.numel(),
            ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream))
        return expz, gx, gw


    def state(self, inputs, weights):
        """Final states [B, 2^n] (complex64 / complex128) of the batch."""
        torch = _torch()
        B = int(inputs.shape[0])
        x, w = self._args(inputs, weights, B)
        cdt = torch.complex64 if self.real == torch.float32 else torch.complex128
        psi = torch.empty((B, 1 << self.c.n), dtype=cdt, device=self.device)
        need = self.c.state_workspace_bytes(self.dtype, B)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        self.c.state_raw(self.dtype, B, _ptr(x) if self.c.n_inputs else None,
                         _ptr(w) if self.c.n_weights else None, _ptr(psi), _ptr(self._ws),
                         self._ws.numel(), ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream))
        return psi


def sample_workspace_bytes(n_qubits, batch) -> int:
    out = ctypes.c_size_t()
    _check(load().ql_sample_workspace_bytes(int(n_qubits), int(batch), ctypes.byref(out)))
    return out.value


def sample_raw(dtype, n_qubits, batch, psi, shots, uniforms, samples, zhat, ws, ws_bytes, stream):
    _check(load().ql_sample(_dt(dtype), int(n_qubits), int(batch), psi, int(shots), uniforms, samples,
                            zhat, ws, int(ws_bytes), stream))


def sample(psi, uniforms, want_z=True):
    """Shots from states ``psi[B, 2^n]`` (complex CUDA tensor) with uniforms
    ``[B, shots]`` (float64 CUDA tensor): returns (indices[B, shots] int64,
    <Z_q> shot estimates [B, n] or None)."""
    torch = _torch()
    B, dim = int(psi.shape[0]), int(psi.shape[1])
    n = dim.bit_length() - 1
    if dim != 1 << n or not psi.is_contiguous() or psi.dtype not in (torch.complex64, torch.complex128):
        raise ValueError("psi must be a contiguous complex tensor [B, 2^n]")
    if uniforms.dtype != torch.float64 or not uniforms.is_contiguous() or int(uniforms.shape[0]) != B:
        raise ValueError("uniforms must be a contiguous float64 tensor [B, shots]")
    shots = int(uniforms.shape[1])
    dtype = "c64" if psi.dtype == torch.complex64 else "c128"
    real = torch.float32 if dtype == "c64" else torch.float64
    out = torch.empty((B, shots), dtype=torch.int64, device=psi.device)
    zhat = torch.empty((B, n), dtype=real, device=psi.device) if want_z else None
    ws = torch.empty(max(sample_workspace_bytes(n, B), 256), dtype=torch.uint8, device=psi.device)
    sample_raw(dtype, n, B, _ptr(psi), shots, _ptr(uniforms), _ptr(out), _ptr(zhat), _ptr(ws), ws.numel(),
               ctypes.c_void_p(torch.cuda.current_stream(psi.device).cuda_stream))
    return out, zhat


def quantum_layer_function():
    """``torch.autograd.Function`` whose forward returns <Z_i> and whose
    backward runs one fused forward + adjoint call for the VJP."""
    torch = _torch()

    class QuantumLayerFn(torch.autograd.Function):
        @staticmethod
        def forward(ctx, runner, inputs, weights):
            ctx.runner = runner
            ctx.save_for_backward(inputs, weights)
            return runner.forward(inputs.contiguous(), weights.contiguous())

        @staticmethod
        def backward(ctx, grad_expz):
            inputs, weights = ctx.saved_tensors
            _, gx, gw = ctx.runner.forward_backward(
                inputs.contiguous(), weights.contiguous(), grad_expz.contiguous(),
                want_inputs=ctx.needs_input_grad[1], want_weights=ctx.needs_input_grad[2])
            return None, gx, gw

    return QuantumLayerFn


_QL_MODULE = None


def _ql_module_class():
    global _QL_MODULE
    if _QL_MODULE is None:
        torch = _torch()

        class QuantumLayerModule(torch.nn.Module):
            def __init__(self, circuit, dtype, device, weights, keep_states):
                super().__init__()
                self.circuit = circuit
                self.runner = Runner(circuit, dtype, device, keep_states=keep_states)
                real = self.runner.real
                if weights is None:
                    w = (torch.rand(circuit.n_weights, dtype=torch.float64) * 2.0 - 1.0) * np.pi
                else:
                    w = torch.as_tensor(weights, dtype=torch.float64).reshape(circuit.n_weights)
                self.weights = torch.nn.Parameter(w.to(device=self.runner.device, dtype=real))
                self._fn = quantum_layer_function()

            def forward(self, inputs):
                return self._fn.apply(self.runner, inputs, self.weights)

        _QL_MODULE = QuantumLayerModule
    return _QL_MODULE


def QuantumLayer(gates, n_qubits, n_inputs, n_weights, dtype="c64", device="cuda", weights=None,
                 keep_states=None, embed=None, pauli_p=None, **options):
    """A quantum node as a ``torch.nn.Module`` (the paper's quantum layer:
    section "Pipeline of VQNet 2.0", quantum node, and the simulator choice in
    "Unification of Classical and Quantum Machine"): the circuit's trainable
    angles are the module's ``weights`` parameter (initialised uniformly in
    [-pi, pi) from torch's generator unless given), ``forward(inputs)`` returns
    <Z_i> per sample and autograd's backward runs the library's fused forward +
    adjoint call. With ``pauli_p`` the circuit holds Pauli channels (the
    noise-inclusive simulator's trajectories: each channel reads its uniform
    from an input feature)."""
    circ = Circuit(n_qubits, gates, n_inputs, n_weights, embed=embed, pauli_p=pauli_p, **options)
    return _ql_module_class()(circ, dtype, device, weights, keep_states)

