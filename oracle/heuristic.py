"""CPU oracle of the decentralized GWTF flow heuristic (paper Sec. V-C).

TEST INFRASTRUCTURE ONLY: the tests and the benchmark's CPU-baseline leg are
the only callers; the GPU library never imports, links or runs anything in
this directory.

``simulate(batch, ...)`` runs ``gwtf_heuristic.c`` (synchronous rounds of
Request Flow, then Request Change / Request Redirect under simulated
annealing, Philox4x64-10 random numbers; every reading of the paper is listed
at the top of the C file) over a batch in the canonical layout of the exact
solver and returns the routed microbatches and their cost.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "gwtf_heuristic.c")
_LIB_PATH = os.path.join(_HERE, "libheuristic.so")
_lib = None
_lock = threading.Lock()

OBJECTIVES = {"sum": 0, "max": 1}
T0 = 1.7      # initial temperature (Sec. VI setup)
ALPHA = 0.95  # cooling factor (Sec. VI setup)


def build(src: str = SRC, out: str = _LIB_PATH) -> str:
    """Compile the simulator with gcc into ``out``."""
    tmp = out + f".tmp{os.getpid()}"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC", "-pthread",
                           src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


def bind(path: str):
    lib = ctypes.CDLL(path)
    p32, p64, pd, pu = (ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64),
                        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_uint64))
    i32 = ctypes.c_int32
    lib.heur_simulate_batch.restype = ctypes.c_int
    lib.heur_simulate_batch.argtypes = [i32, i32, i32] + [p32] * 7 + [i32, i32, i32, ctypes.c_double,
                                                                    ctypes.c_double, ctypes.c_uint64, i32,
                                                                    p64, p64, p32, p32, p32, p32, p32, pd,
                                                                    p64, i32]
    lib.heur_philox4x64_10.restype = None
    lib.heur_philox4x64_10.argtypes = [pu, pu, pu]
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                build()
            _lib = bind(_LIB_PATH)
    return _lib


def philox4x64_10(counter, key, lib=None):
    """The simulator's generator: four 64-bit words for a counter and key."""
    lib = _load() if lib is None else lib
    c = (ctypes.c_uint64 * 4)(*[int(x) for x in counter])
    k = (ctypes.c_uint64 * 2)(*[int(x) for x in key])
    o = (ctypes.c_uint64 * 4)()
    lib.heur_philox4x64_10(c, k, o)
    return [int(x) for x in o]


def _p(a, ctype):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctype))


def simulate(batch, rounds: int = 120, objective: str = "sum", seed: int = 0, T0: float = T0,
             alpha: float = ALPHA, max_slots: int = 1024, paths=None, nthreads: int | None = None,
             lib=None) -> dict:
    """Simulate every instance of ``batch`` for ``rounds`` rounds.

    ``paths`` (optional int32 [B][P][S], node index per stage, rows starting
    with -1 unused) gives complete paths the flow starts from.  Returns numpy
    arrays: F, cost (int64 [B]), status (int32 [B]), node_flow [B][S][n] and
    arc_flow [B][S-1][n][n] of the routed microbatches, used slots and
    accepted moves [B][S][n], final temperatures [B][S][n] (float64),
    counters [B][4] (paths paired by the data node, Request Flow approvals,
    accepted moves, dangling slots) and the thread count.
    """
    lib = _load() if lib is None else lib
    S, n = int(batch.S), int(batch.n)
    i32 = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.int32)
    cap, cost, supply = i32(batch.node_cap), i32(batch.node_cost), i32(batch.supply)
    arc = i32(batch.arc_cost) if S > 1 else None
    src, snk = i32(batch.src_cost), i32(batch.snk_cost)
    B = int(supply.shape[0])
    P = 0
    if paths is not None:
        paths = i32(paths)
        assert paths.ndim == 3 and paths.shape[0] == B and paths.shape[2] == S
        P = int(paths.shape[1])
    out = {"F": np.zeros(B, np.int64), "cost": np.zeros(B, np.int64), "status": np.zeros(B, np.int32),
           "node_flow": np.zeros((B, S, n), np.int32), "arc_flow": np.zeros((B, max(S - 1, 0), n, n), np.int32),
           "used": np.zeros((B, S, n), np.int32), "accepted": np.zeros((B, S, n), np.int32),
           "temperature": np.zeros((B, S, n), np.float64), "counters": np.zeros((B, 4), np.int64)}
    if nthreads is None:
        nthreads = os.cpu_count() or 1
    p32, p64 = ctypes.c_int32, ctypes.c_int64
    used = lib.heur_simulate_batch(
        B, S, n, _p(cap, p32), _p(cost, p32), _p(arc, p32), _p(src, p32), _p(snk, p32), _p(supply, p32),
        _p(paths, p32), P, int(rounds), OBJECTIVES[objective], float(T0), float(alpha), int(seed) & (2**64 - 1),
        int(max_slots), _p(out["F"], p64), _p(out["cost"], p64), _p(out["status"], p32),
        _p(out["node_flow"], p32), _p(out["arc_flow"], p32), _p(out["used"], p32), _p(out["accepted"], p32),
        _p(out["temperature"], ctypes.c_double), _p(out["counters"], p64), int(nthreads))
    if used < 0:
        raise ValueError("heuristic oracle: bad shape or arguments")
    out["threads"] = int(used)
    return out
