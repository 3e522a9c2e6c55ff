"""CPU oracle for the layered min-cost max-flow problem.

TEST INFRASTRUCTURE ONLY: the tests, the package smoke check and the
benchmark's CPU-baseline leg are the only callers.  The GPU library never
imports, links or runs anything in this directory, and this directory never
imports the GPU package.

``solve(batch)`` runs ``mcf_oracle.c`` (successive shortest paths with a
binary-heap Dijkstra on Johnson-reduced costs, in 64-bit integers) over a
batch given in the canonical layout (any object with the attributes S, n,
node_cap, node_cost, arc_cost, src_cost, snk_cost, supply as int32 numpy
arrays).  The method and the flow network are described at the top of the C
file; the objective is the paper's Eq. 2 (Sec. V-A): among integral flows of
maximum value (capped by the data node's supply) minimise the sum over arcs
of flow times delay.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mcf_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()

STATUS_OK = 0
STATUS_BAD_INPUT = 1
STATUS_SELFCHECK = 99


def build() -> str:
    """Compile the oracle with gcc into oracle/liboracle.so, and the
    decentralized-heuristic simulator (oracle/heuristic.py) beside it."""
    tmp = _LIB_PATH + f".tmp{os.getpid()}"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                           "-pthread", _SRC, "-o", tmp])
    os.replace(tmp, _LIB_PATH)
    from . import heuristic

    heuristic.build()
    return _LIB_PATH


def bind(path: str):
    """Load a compiled oracle library from ``path`` and declare its entry."""
    lib = ctypes.CDLL(path)
    p32 = ctypes.POINTER(ctypes.c_int32)
    p64 = ctypes.POINTER(ctypes.c_int64)
    lib.oracle_solve_batch.restype = ctypes.c_int
    lib.oracle_solve_batch.argtypes = [ctypes.c_int32] * 3 + [p32] * 6 + [p64, p64, p32] + \
        [p32] * 4 + [p64, p64, ctypes.c_int32]
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                build()
            _lib = bind(_LIB_PATH)
    return _lib


def _ptr(a, ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a


def solve(batch, nthreads: int | None = None, flows: bool = True, potentials: bool = True,
          lib=None) -> dict:
    """Solve every instance of ``batch``; returns a dict of numpy arrays.

    Keys: F, cost (int64 [B]); status (int32 [B]); augmentations,
    arc_scans (int64 [B]); threads (int); and, when requested, node_flow
    [B][S][n], arc_flow [B][S-1][n][n], src_flow [B][n], snk_flow [B][n]
    (int32) and potential [B][V] (int64, vertex order s0, s, t, then
    in/out of each node stage-major).  ``lib`` selects another compiled
    copy of the oracle (the mutation tests pass one).
    """
    lib = _load() if lib is None else lib
    S, n = int(batch.S), int(batch.n)
    cap, ncost, supply = _i32(batch.node_cap), _i32(batch.node_cost), _i32(batch.supply)
    B = int(supply.shape[0])
    acost = _i32(batch.arc_cost) if S > 1 else None
    src = None if batch.src_cost is None else _i32(batch.src_cost)
    snk = None if batch.snk_cost is None else _i32(batch.snk_cost)
    V = 3 + 2 * S * n
    out = {
        "F": np.zeros(B, np.int64), "cost": np.zeros(B, np.int64),
        "status": np.zeros(B, np.int32), "stats": np.zeros((B, 2), np.int64),
    }
    if flows:
        out["node_flow"] = np.zeros((B, S, n), np.int32)
        out["arc_flow"] = np.zeros((B, max(S - 1, 0), n, n), np.int32)
        out["src_flow"] = np.zeros((B, n), np.int32)
        out["snk_flow"] = np.zeros((B, n), np.int32)
    if potentials:
        out["potential"] = np.zeros((B, V), np.int64)
    if nthreads is None:
        nthreads = os.cpu_count() or 1
    p32, p64 = ctypes.c_int32, ctypes.c_int64
    used = lib.oracle_solve_batch(
        B, S, n, _ptr(cap, p32), _ptr(ncost, p32), _ptr(acost, p32), _ptr(src, p32),
        _ptr(snk, p32), _ptr(supply, p32),
        _ptr(out["F"], p64), _ptr(out["cost"], p64), _ptr(out["status"], p32),
        _ptr(out.get("node_flow"), p32), _ptr(out.get("arc_flow"), p32),
        _ptr(out.get("src_flow"), p32), _ptr(out.get("snk_flow"), p32),
        _ptr(out.get("potential"), p64), _ptr(out["stats"], p64), int(nthreads))
    if used < 0:
        raise ValueError("oracle: bad shape")
    out["threads"] = int(used)
    out["augmentations"] = out["stats"][:, 0].copy()
    out["arc_scans"] = out["stats"][:, 1].copy()
    del out["stats"]
    return out
