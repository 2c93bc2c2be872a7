"""Benchmark: one fused forward + adjoint call of the batched quantum layer.

A step is one ``ql_forward_backward`` call over one batch of synthetic inputs
already resident in HBM: angle binding, every forward tile pass, the fused
<Z>/seed/first-backward pass, every backward pass and the reductions. The
metric is amplitude-gate updates per second, U = 3 * G * B * 2^n per step (the
forward applies G gates to psi, the adjoint sweep un-applies G gates on psi and
on lambda), plus the dominant kernel's achieved HBM bandwidth against the
MI355X peak.

Prints one JSON line. ``--gpus`` above 1 is not supported (one GPU holds the
whole state; the batch/state sharding design is documented separately).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as W  # noqa: E402

METRIC = "amplitude-gate updates/s (batched fwd+adjoint grad); % of HBM peak BW"
HBM_PEAK_GBS = 8000.0
# MI355X published vector peaks (TFLOP/s): fp32 157.3 (reached only with packed
# two-wide fp32 instructions), fp64 78.6.
ALU_PEAK_TFLOPS = {"c64": 157.3, "c128": 78.6}
# The issue ceiling of the arithmetic this library emits: one fp32 (or fp64)
# FMA per lane per cycle, no packed fp32: 256 CUs x 4 SIMDs x 16 lanes x 2 flop
# x 2.4 GHz.
ISSUE_PEAK_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12
# Algorithmic flops per amplitude, each gate in its cheapest exact form: RX/RY
# rotate a real plane per pair of components, 6 flops per amplitude; RZ is, up
# to a global phase, a complex multiply of the bit-1 half of the amplitudes,
# 3 flops per amplitude; H is 4; CNOT/CZ are permutations/signs (0); a
# controlled rotation is its rotation on the control-1 half; a Pauli-channel
# outcome is a permutation/sign (0). One step applies every gate once
# (forward) and un-applies it on psi and lambda (backward); each rotation also
# takes a gradient term Im<lambda|P|psi> (4 flops per amplitude, 2 for a
# controlled one).
FLOPS_FWD = {W.H: 4, W.RX: 6, W.RY: 6, W.RZ: 3, W.CNOT: 0, W.CZ: 0, W.CRX: 3, W.CRY: 3, W.CRZ: 1.5,
             W.PAULI: 0}
FLOPS_GRAD = {W.RX: 4, W.RY: 4, W.RZ: 4, W.CRX: 2, W.CRY: 2, W.CRZ: 2}


def algorithmic_flops(gates, batch, n) -> float:
    per_amp = 0
    for g in gates:
        k = int(g[0])
        per_amp += 3 * FLOPS_FWD[k] + FLOPS_GRAD.get(k, 0)
    return float(per_amp) * batch * (1 << n)


def shift_circuits(gates, batch) -> int:
    """Circuits one parameter-shift VJP runs: per sample the unshifted circuit
    and two shifted copies per rotation occurrence (a controlled rotation is
    two half-angle rotations)."""
    rot = sum(1 if int(g[0]) in W.ROTATIONS else 2 if int(g[0]) in W.CONTROLLED else 0 for g in gates)
    return batch * (2 * rot + 1)


def shift_flops(gates, batch, n, ops=None) -> float:
    """Algorithmic flops of one parameter-shift VJP: forward passes only, over
    the gates that run as ops (all of them unless `ops` says otherwise)."""
    per_amp = sum(FLOPS_FWD[int(g[0])] for g in (gates if ops is None else ops))
    return float(per_amp) * shift_circuits(gates, batch) * (1 << n)


def profiled_traffic(wl):
    """Calibrated HBM bytes per step of the tile kernel from the committed
    rocprofv3 summary (None unless it was taken with the current kernel
    source), and the bandwidth of the plain 1 GiB copy kernel measured in the
    same runs (the achievable line), in GB/s."""
    path = os.path.join(ROOT, "profiles", f"k_tile_{wl.name}.txt")
    if not os.path.exists(path):
        return None, None
    text = open(path).read()
    fields = dict(l.split(": ", 1) for l in text.splitlines() if ": " in l and not l.startswith("#"))
    m = re.search(r"copy duration ([0-9.]+) ms", text)
    copy_gbs = 2 * 2 ** 30 / (float(m.group(1)) * 1e-3) / 1e9 if m else None
    # the counters hold only for the tile kernel's source and the planner that
    # made the passes they were taken on
    digests = source_digests()
    for key in ("tile_sha256", "plan_sha256"):
        if fields.get(key) != digests[key]:
            return None, copy_gbs
    return float(fields["traffic_bytes_per_step"]), copy_gbs


def source_digests():
    """sha256 of the tile kernel's sources (tile.hip, kcommon.hpp, launch.hpp,
    plan.hpp) and of the planner (plan.cpp), which key the committed rocprofv3
    summaries."""
    csrc = os.path.join(ROOT, "paper_2301_03251_amd", "csrc")
    h = hashlib.sha256()
    for name in ("tile.hip", "kcommon.hpp", "launch.hpp", "plan.hpp"):
        h.update(open(os.path.join(csrc, name), "rb").read())
    return {"tile_sha256": h.hexdigest(),
            "plan_sha256": hashlib.sha256(open(os.path.join(csrc, "plan.cpp"), "rb").read()).hexdigest()}


def host_info():
    """CPU model, CPUs this process may run on, and installed RAM."""
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    ram = None
    try:
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal:"):
                ram = round(int(line.split()[1]) / 2 ** 20, 1)
                break
    except OSError:
        pass
    return {"cpu_model": model, "affinity_cpus": len(os.sched_getaffinity(0)), "ram_gib": ram}


def cpu_baseline(wl, gates, x, w, g, pauli_p, prefixes):
    """The CPU oracle (complex128, all host threads) on a bounded sample of the
    same workload: one sample at full size, forward + adjoint, over two
    prefixes of the gate list (k1 < k2 gates). The rate is the slope: the
    amplitude-gate updates of the k2 - k1 extra gates over the extra time, so
    that the costs that do not depend on the gate count (allocating and
    clearing the states, the <Z> sums, the lambda seed) are reported apart
    (``fixed_s``) instead of diluting the per-gate rate."""
    import oracle
    oracle.build()
    times = []
    for k in prefixes:
        sub = gates[:k]
        n_ch = int(sum(1 for gg in sub if int(gg[0]) == W.PAULI))
        pp = None if pauli_p is None else pauli_p[:max(n_ch, 1)]
        t0 = time.perf_counter()
        oracle.run(wl.n, sub, x[:1], w, grad_out=g[:1], embed=getattr(wl, "embed", None), pauli_p=pp)
        times.append(time.perf_counter() - t0)
    (k1, k2), (t1, t2) = prefixes, times
    upd = 3.0 * (k2 - k1) * (1 << wl.n)
    dt = max(t2 - t1, 1e-9)
    fixed = max(t1 - k1 * dt / (k2 - k1), 0.0)
    return {"value": upd / dt, "unit": "amplitude-gate updates/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{wl.name} batch row 0 of {wl.batch}, n={wl.n}, complex128, forward + adjoint "
                      f"over the first {k1} and the first {k2} of {len(gates)} gates: {t1:.2f} s and "
                      f"{t2:.2f} s; value = 3*({k2}-{k1})*2^{wl.n} updates / {dt:.2f} s",
            "fixed_s": fixed, "prefix_gates": [k1, k2], "prefix_s": [t1, t2],
            "whole_prefix_rate": 3.0 * k2 * (1 << wl.n) / t2, **host_info()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="30q", choices=sorted(W.WORKLOADS) + ["qae"])
    ap.add_argument("--noise", type=float, default=0.0,
                    help="depolarizing probability p: a Pauli-channel trajectory on every qubit "
                         "after every --noise-every gates, one trajectory per sample")
    ap.add_argument("--noise-every", type=int, default=1)
    ap.add_argument("--cpu-gates", default="8,32",
                    help="the two gate-list prefixes the CPU oracle times, k1,k2 (0 disables it)")
    ap.add_argument("--no-timing", action="store_true",
                    help="time only the whole step (no per-kernel events)")
    ap.add_argument("--calibrate", action="store_true",
                    help="run one 1 GiB device-to-device copy first (a plain copy kernel of known "
                         "size, to scale hardware byte counters)")
    ap.add_argument("--grad", choices=("adjoint", "shift"), default="adjoint",
                    help="gradient method timed: the adjoint sweep (the headline metric) or the "
                         "batched parameter-shift rule")
    ap.add_argument("--shots", type=int, default=0,
                    help="time measurement by shots instead of a gradient step: final states "
                         "(ql_state) plus this many shots per sample (ql_sample)")
    ap.add_argument("--shift-chunk", type=int, default=0,
                    help="shifted circuits per chunk (0: as many as 8 GiB of states hold)")
    ap.add_argument("--states", choices=("auto", "kept", "plain"), default="auto",
                    help="backward workspace: kept forward states when they fit (auto), always "
                         "(kept), or never (plain: each backward pass stores psi for the next)")
    ap.add_argument("--opt", action="append", default=[],
                    help="planner option key=value (log_regs, log_threads, low_qubits, "
                         "max_gates_per_pass, wg_per_sample)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported; this build runs on one GPU "
              "(every workload fits one MI355X).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2301_03251_amd as Q

    wl = W.get(args.workload)
    x, w, g = wl.inputs()
    gates, pauli_p, n_in = wl.gates(), None, wl.n_inputs
    if args.noise > 0:
        gates, pauli_p, n_ch = W.with_depolarizing(gates, wl.n, wl.n_inputs, args.noise, args.noise_every)
        u = np.random.default_rng(wl.seed + 1000).random((wl.batch, n_ch)).astype(x.dtype)
        x = np.concatenate([x, u], axis=1)
        n_in = x.shape[1]
    opts = {kv.split("=")[0]: int(kv.split("=")[1]) for kv in args.opt}
    circ = Q.Circuit(wl.n, gates, n_in, wl.n_weights, embed=getattr(wl, "embed", None), pauli_p=pauli_p,
                     **opts)
    runner = Q.Runner(circ, wl.dtype, keep_states={"auto": None, "kept": True, "plain": False}[args.states])
    real = torch.float32 if wl.dtype == "c64" else torch.float64
    dev = torch.device("cuda")
    xt = torch.from_numpy(x).to(dev, real)
    wt = torch.from_numpy(w).to(dev, real)
    gt = torch.from_numpy(g).to(dev, real)
    outs = (torch.empty((wl.batch, wl.n), dtype=real, device=dev),
            torch.empty((wl.batch, n_in), dtype=real, device=dev),
            torch.empty(wl.n_weights, dtype=real, device=dev))
    shift = args.grad == "shift"
    if shift and getattr(wl, "embed", (W.EMBED_NONE, 0))[0] == W.EMBED_AMPLITUDE:
        outs = (outs[0], None, outs[2])  # the shift rule gives no amplitude gradient
    amp = 8 if wl.dtype == "c64" else 16
    n_shift = shift_circuits(gates, wl.batch)
    chunk = args.shift_chunk or max(1, min(n_shift, (8 << 30) // ((1 << wl.n) * amp)))
    if args.shots > 0:
        uni = torch.from_numpy(np.random.default_rng(7).random((wl.batch, args.shots))).to(dev)
        step = lambda: Q.sample(runner.state(xt, wt), uni)  # noqa: E731
    elif shift:
        step = lambda: runner.param_shift(xt, wt, gt, max_chunk=chunk, outs=outs)  # noqa: E731
    else:
        runner.workspace(wl.batch, runner.backward_mode(wl.batch))
        step = lambda: runner.forward_backward(xt, wt, gt, outs=outs)  # noqa: E731
    if args.calibrate:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    timing = not args.no_timing
    # events around the dominant kernel's launches only: each event pair costs
    # host time, which would show in the step time of launch-bound workloads
    dominant = 1 if circ.plan_info(wl.dtype)["kernel"] == 1 else 2
    circ.timing(timing, dominant)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    kms, kcnt = circ.timing_read() if timing else ([0.0] * 4, [0] * 4)
    circ.timing(False)

    info = circ.plan_info(wl.dtype)
    G = int(gates.shape[0])
    U = 3 * G * wl.batch * (1 << wl.n)
    if shift:
        # amplitude-gate updates the parameter-shift VJP performs
        U = n_shift * G * (1 << wl.n)
    if args.shots > 0:
        U = G * wl.batch * (1 << wl.n)  # forward only
    line = {
        "metric": ("amplitude-gate updates/s (final states + shot sampling)" if args.shots > 0 else
                   "amplitude-gate updates/s (batched parameter-shift grad)" if shift else METRIC),
        "value": U / (ms_step / 1e3),
        "unit": "amplitude-gate updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "n_qubits": wl.n, "batch": wl.batch,
                   "gates": G, "weights": wl.n_weights,
                   "updates_per_step": U, "tile_passes": info["n_passes"],
                   "tile_qubits": info["tile_qubits"], "planner_options": opts},
    }
    if getattr(wl, "embed", None):
        line["config"]["embedding"] = {W.EMBED_BASIS: "basis", W.EMBED_AMPLITUDE: "amplitude"}[wl.embed[0]]
    if args.noise > 0:
        line["config"]["noise"] = {"model": "depolarizing trajectories", "p": args.noise,
                                   "every": args.noise_every, "channels": int(pauli_p.shape[0])}
    if args.shots > 0:
        line["config"].update({"measurement": "shots", "shots": args.shots})
        line["shots_per_s"] = args.shots * wl.batch * 1e3 / ms_step
    elif shift:
        line["config"].update({"grad": "parameter shift", "circuits_per_step": n_shift,
                               "chunk": chunk})
    else:
        line["config"]["kept_states"] = runner.backward_mode(wl.batch) == Q.MODE_FWD_BWD_KEEP
        line["vjp_per_s"] = 1e3 / ms_step
    if timing and kcnt[0] > 0:
        tile_ms = kms[0] / args.steps
        # the tile kernel's own work: the gates of the product-state prefix are
        # not tile ops (the first pass writes their state from per-qubit
        # factors; their gradients come from the environment kernels)
        n_pre = circ.plan_info(wl.dtype)["n_prefix_gates"]
        tile_gates = gates
        if n_pre:
            tile_gates = np.delete(gates, circ.schedule(wl.dtype)[1][:n_pre], axis=0)
        if args.shots > 0:
            state_bytes = circ.state_bytes(wl.dtype, wl.batch, Q.MODE_FWD) + (1 << wl.n) * wl.batch * amp
            flops = sum(FLOPS_FWD[int(g_[0])] for g_ in tile_gates) * wl.batch * float(1 << wl.n)
            traffic = None
        elif shift:
            state_bytes = circ.state_bytes(wl.dtype, n_shift, Q.MODE_FWD)
            flops = shift_flops(gates, wl.batch, wl.n, tile_gates)
            traffic = None
        else:
            state_bytes = circ.state_bytes(wl.dtype, wl.batch, runner.backward_mode(wl.batch))
            flops = algorithmic_flops(tile_gates, wl.batch, wl.n)
            # the committed summaries were taken on the default plan with kept states
            same_run = (args.noise == 0 and not opts
                        and runner.backward_mode(wl.batch) == Q.MODE_FWD_BWD_KEEP)
            traffic = profiled_traffic(wl)[0] if same_run else None
        copy_gbs = profiled_traffic(wl)[1]
        hbm = state_bytes / (tile_ms / 1e3) / 1e9
        alu = flops / (tile_ms / 1e3) / 1e12
        launches = kcnt[0] / args.steps
        peak = ALU_PEAK_TFLOPS[wl.dtype]
        line["roofline"] = {"bound": "alu", "kernel": "k_tile", "achieved": alu,
                            "peak": peak, "unit": "TFLOP/s", "frac": alu / peak,
                            "traffic": None if traffic is None else traffic / launches,
                            "traffic_unit": "bytes per launch",
                            "launches_per_step": launches,
                            "kernel_ms_per_step": tile_ms,
                            "algorithmic_flops_per_step": flops,
                            "prefix_gates": n_pre,
                            "algorithmic_bytes_per_step": state_bytes,
                            "issue_peak": ISSUE_PEAK_TFLOPS,
                            "frac_of_issue_peak": alu / ISSUE_PEAK_TFLOPS,
                            "hbm": {"achieved": hbm, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                    "frac": hbm / HBM_PEAK_GBS, "copy_kernel": copy_gbs}}
        line["alu_frac"] = alu / peak
        line["hbm_frac"] = hbm / HBM_PEAK_GBS
        line["kernel_ms_per_step"] = {"k_tile": kms[0] / args.steps}
    elif timing and kcnt[1] > 0:
        whole_ms = kms[1] / args.steps
        alu = (shift_flops(gates, wl.batch, wl.n) if shift else
               algorithmic_flops(gates, wl.batch, wl.n)) / (whole_ms / 1e3) / 1e12
        peak = ALU_PEAK_TFLOPS[wl.dtype]
        line["roofline"] = {"bound": "alu", "kernel": "k_whole", "achieved": alu,
                            "peak": peak, "unit": "TFLOP/s", "frac": alu / peak,
                            "traffic": None, "kernel_ms_per_step": whole_ms,
                            "issue_peak": ISSUE_PEAK_TFLOPS, "frac_of_issue_peak": alu / ISSUE_PEAK_TFLOPS}
        line["alu_frac"] = alu / peak
    pre = [int(v) for v in str(args.cpu_gates).split(",") if v.strip()]
    if pre and pre[0] > 0:
        k2 = min(pre[-1], G)
        k1 = min(pre[0], k2 - 1) if len(pre) > 1 else max(1, k2 // 4)
        if k1 >= 1:
            line["cpu_baseline"] = cpu_baseline(wl, gates, x, w, g, pauli_p, (k1, k2))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
