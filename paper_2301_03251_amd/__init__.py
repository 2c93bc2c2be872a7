"""Batched quantum-layer simulation on MI355X (gfx950): forward <Z_i> and adjoint
VJP gradients of parameterised circuits, in hand-written HIP kernels behind a
C ABI (``include/qlayer.h``). See ``qlayer.py`` for the Python binding."""

from .qlayer import (C64, C128, MODE_FWD, MODE_FWD_BWD, MODE_FWD_BWD_KEEP, STATIC_SCRATCH_BYTES, Circuit, QLError, Runner,  # noqa: F401
                     sample, sample_workspace_bytes,
                     load, quantum_layer_function, QuantumLayer)

__all__ = ["C64", "C128", "MODE_FWD", "MODE_FWD_BWD", "MODE_FWD_BWD_KEEP", "STATIC_SCRATCH_BYTES", "Circuit", "QLError", "Runner", "load", "sample", "sample_workspace_bytes",
           "quantum_layer_function", "QuantumLayer"]
