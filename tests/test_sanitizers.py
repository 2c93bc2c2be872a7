"""Sanitizer runs of the host code (CPU only, no GPU).

- The circuit intake and tile-pass planner (``plan.cpp``, plain C++) built with
  AddressSanitizer and UndefinedBehaviorSanitizer (g++), run over every
  workload, random circuits of every gate kind, embeddings, Pauli channels,
  several planner options, and invalid circuits that must be rejected.
- The CPU oracle built with ThreadSanitizer (clang, LLVM OpenMP with the
  Archer annotations), run on a 16-qubit circuit where its amplitude loops run
  in parallel and its pairwise sums split into chunks; its results with four
  threads must equal those with one thread bit for bit. A copy of the oracle
  with a planted race (the chunk sums added into one word from every thread)
  must be reported, which shows the ThreadSanitizer run is live.
"""

from __future__ import annotations

import os
import shutil
import subprocess

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2301_03251_amd", "csrc")
LLVM = "/opt/rocm/llvm"


def _record(f, n, gates, F, P, embed=(0, 0), pauli_p=None, ok=True):
    gates = np.ascontiguousarray(gates, np.int32).reshape(-1, 5)
    pp = np.zeros((0, 3)) if pauli_p is None else np.asarray(pauli_p, np.float64).reshape(-1, 3)
    np.array([n, gates.shape[0], F, P, embed[0], embed[1], pp.shape[0], int(ok)], np.int32).tofile(f)
    gates.tofile(f)
    np.ascontiguousarray(pp, np.float64).tofile(f)


def _circuits(path):
    with open(path, "wb") as f:
        for name in list(W.WORKLOADS) + ["qae"]:
            wl = W.get(name)
            emb = getattr(wl, "embed", None) or (0, 0)
            _record(f, wl.n, wl.gates(), wl.n_inputs, wl.n_weights, embed=emb)
        for seed in range(12):
            n = [3, 6, 9, 12, 14, 17][seed % 6]
            F, P = 4, 6
            g = W.random_circuit(n, 80 + 10 * seed, F, P, seed=seed)
            rng = np.random.default_rng(seed)
            extra = []
            for _ in range(6):  # controlled rotations
                a, b = rng.choice(n, 2, replace=False)
                extra.append([int(rng.choice([W.CRX, W.CRY, W.CRZ])), int(a), int(b), W.SRC_WEIGHT,
                              int(rng.integers(P))])
            chans = [[W.PAULI, int(rng.integers(n)), -1, W.SRC_INPUT, F + c] for c in range(3)]
            gates = np.concatenate([g, np.array(extra + chans, np.int32)])
            pp = rng.random((3, 3)) / 3
            _record(f, n, gates, F + 3, P, pauli_p=pp)
            if n <= 12:
                _record(f, n, g, 2 ** n + 1, P, embed=(W.EMBED_AMPLITUDE, 1))
            _record(f, n, g, n + F, P, embed=(W.EMBED_BASIS, F))
        bad = [
            (3, [[W.RY, 3, -1, W.SRC_WEIGHT, 0]], 0, 1),    # qubit out of range
            (3, [[W.CNOT, 1, 1, 0, 0]], 0, 0),              # q0 == q1
            (3, [[W.RX, 0, -1, W.SRC_INPUT, 5]], 2, 0),     # input index out of range
            (3, [[W.H, 0, -1, W.SRC_WEIGHT, 0]], 0, 1),     # H with a source
            (3, [[99, 0, -1, 0, 0]], 0, 0),                 # unknown kind
            (40, [[W.H, 0, -1, 0, 0]], 0, 0),               # too many qubits
            (0, [[W.H, 0, -1, 0, 0]], 0, 0),                # no qubits
        ]
        for n, gates, F, P in bad:
            _record(f, n, gates, F, P, ok=False)
        _record(f, 3, [[W.PAULI, 0, -1, W.SRC_INPUT, 0]], 1, 0, pauli_p=[[0.6, 0.5, 0.0]], ok=False)


def _run(cmd, env=None, timeout=300):
    return subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not found")
def test_planner_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "planner")
    b = _run(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
              "-fsanitize=address,undefined", "-fno-sanitize-recover=all", f"-I{CSRC}",
              os.path.join(HERE, "planner_driver.cpp"), os.path.join(CSRC, "plan.cpp"), "-o", exe])
    assert b.returncode == 0, b.stderr[-2000:]
    data = str(tmp_path / "circuits.bin")
    _circuits(data)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = _run([exe, data], env=env)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
    assert r.stdout.startswith("cases "), r.stdout


def _tsan_build(src, exe):
    return _run([os.path.join(LLVM, "bin", "clang"), "-O1", "-g", "-fopenmp", "-fsanitize=thread", src,
                 os.path.join(HERE, "oracle_threads.c"), "-lm", "-o", exe])


def _tsan_env(threads):
    return dict(os.environ, OMP_NUM_THREADS=str(threads), LD_LIBRARY_PATH=os.path.join(LLVM, "lib"),
                OMP_TOOL_LIBRARIES=os.path.join(LLVM, "lib", "libarcher.so"),
                TSAN_OPTIONS="halt_on_error=1 ignore_noninstrumented_modules=1")


@pytest.mark.skipif(not os.path.exists(os.path.join(LLVM, "lib", "libarcher.so")),
                    reason="LLVM OpenMP with Archer not found")
def test_oracle_under_tsan(tmp_path):
    exe = str(tmp_path / "oracle_tsan")
    b = _tsan_build(os.path.join(ROOT, "oracle", "oracle.c"), exe)
    assert b.returncode == 0, b.stderr[-2000:]
    outs = {}
    for threads in (1, 4):
        r = _run([exe], env=_tsan_env(threads))
        assert r.returncode == 0 and "ThreadSanitizer" not in r.stderr, r.stderr[-4000:]
        outs[threads] = r.stdout
    assert outs[1] == outs[4] and len(outs[1].split()) == 32


@pytest.mark.skipif(not os.path.exists(os.path.join(LLVM, "lib", "libarcher.so")),
                    reason="LLVM OpenMP with Archer not found")
def test_tsan_reports_a_planted_race(tmp_path):
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    old = "for (int i = 0; i < nch; i++) part[i] = psum_real(c, f, (int64_t)i * len, (int64_t)(i + 1) * len);"
    assert src.count(old) == 1
    racy = tmp_path / "oracle_racy.c"
    racy.write_text(src.replace(old, "for (int i = 0; i < nch; i++) part[0] += "
                                     "psum_real(c, f, (int64_t)i * len, (int64_t)(i + 1) * len);"))
    exe = str(tmp_path / "oracle_racy")
    b = _tsan_build(str(racy), exe)
    assert b.returncode == 0, b.stderr[-2000:]
    r = _run([exe], env=_tsan_env(4))
    assert "WARNING: ThreadSanitizer: data race" in r.stderr
