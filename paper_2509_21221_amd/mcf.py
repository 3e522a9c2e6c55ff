"""Python binding of the C ABI in include/gwtf_mcf.h (ctypes; argument
marshalling only -- every step of the solve runs in the HIP library).

The functions carry the C names (``gwtf_mcf_create``, ``gwtf_mcf_solve_batch``,
``gwtf_mcf_get_flows``, ``gwtf_mcf_get_stats``, ``gwtf_mcf_get_passes``,
``gwtf_mcf_solve_batch_noalloc``,
``gwtf_mcf_solve_located``, ``gwtf_whatif_count``, ``gwtf_mcf_whatif_expand``, ``gwtf_mcf_whatif_best``,
``gwtf_mcf_resolve_churn``, ``gwtf_mcf_simulate_heuristic``,
``gwtf_mcf_destroy``, ``gwtf_mcf_last_error``); ``Solver`` wraps them for
torch device tensors.
PyTorch only provides device memory and the HIP stream.

There is no fallback: if ``libgwtf_mcf.so`` is missing or cannot be loaded,
every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libgwtf_mcf.so")

GWTF_OK = 0
GWTF_ERR_INVALID_ARG = 1
GWTF_ERR_OUT_OF_MEMORY = 2
GWTF_ERR_DEVICE = 3
GWTF_ERR_NOT_SOLVED = 4
GWTF_ERR_RANGE = 5
GWTF_INST_OK = 0
GWTF_INST_BAD_INPUT = 1
GWTF_INST_OVERFLOW = 2
GWTF_INST_NOT_CONVERGED = 3
CHURN_WORK_PER_INSTANCE = 4
GWTF_NO_ARC = -1
STATS_PER_INSTANCE = 10
GWTF_PASS_REGISTER = 1
GWTF_PASS_LDS = 2
GWTF_PASS_GRID = 3
GWTF_PASS_GLOBAL = 4
GWTF_PASS_PACKED = 5

STATUS_NAMES = {0: "GWTF_OK", 1: "GWTF_ERR_INVALID_ARG", 2: "GWTF_ERR_OUT_OF_MEMORY",
                3: "GWTF_ERR_DEVICE", 4: "GWTF_ERR_NOT_SOLVED", 5: "GWTF_ERR_RANGE"}


class gwtf_mcf_shape_t(ctypes.Structure):
    _fields_ = [("num_stages", ctypes.c_int32), ("nodes_per_stage", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("device", ctypes.c_int32)]


class gwtf_mcf_batch_t(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32),
                ("node_cap", ctypes.c_void_p), ("node_cost", ctypes.c_void_p),
                ("arc_cost", ctypes.c_void_p), ("src_cost", ctypes.c_void_p),
                ("snk_cost", ctypes.c_void_p), ("supply", ctypes.c_void_p),
                ("flow_value", ctypes.c_void_p), ("total_cost", ctypes.c_void_p),
                ("status", ctypes.c_void_p)]


class gwtf_mcf_located_batch_t(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_locations", ctypes.c_int32),
                ("node_cap", ctypes.c_void_p), ("node_cost", ctypes.c_void_p),
                ("location", ctypes.c_void_p), ("latency", ctypes.c_void_p),
                ("src_cost", ctypes.c_void_p), ("snk_cost", ctypes.c_void_p),
                ("supply", ctypes.c_void_p), ("flow_value", ctypes.c_void_p),
                ("total_cost", ctypes.c_void_p), ("status", ctypes.c_void_p)]


class gwtf_whatif_candidates_t(ctypes.Structure):
    _fields_ = [("num_candidates", ctypes.c_int32), ("slot", ctypes.c_int32),
                ("cap", ctypes.c_void_p), ("cost", ctypes.c_void_p), ("in_cost", ctypes.c_void_p),
                ("out_cost", ctypes.c_void_p), ("link_cost", ctypes.c_void_p),
                ("src_cost", ctypes.c_void_p), ("snk_cost", ctypes.c_void_p)]


class gwtf_mcf_instances_t(ctypes.Structure):
    _fields_ = [("node_cap", ctypes.c_void_p), ("node_cost", ctypes.c_void_p),
                ("arc_cost", ctypes.c_void_p), ("src_cost", ctypes.c_void_p),
                ("snk_cost", ctypes.c_void_p), ("supply", ctypes.c_void_p)]


class gwtf_mcf_flow_in_t(ctypes.Structure):
    _fields_ = [("node_flow", ctypes.c_void_p), ("arc_flow", ctypes.c_void_p),
                ("src_flow", ctypes.c_void_p), ("snk_flow", ctypes.c_void_p),
                ("per_instance", ctypes.c_int32)]


class gwtf_mcf_flow_out_t(ctypes.Structure):
    _fields_ = [("node_flow", ctypes.c_void_p), ("arc_flow", ctypes.c_void_p),
                ("src_flow", ctypes.c_void_p), ("snk_flow", ctypes.c_void_p)]


class gwtf_heur_config_t(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_int32), ("objective", ctypes.c_int32), ("t0", ctypes.c_double),
                ("alpha", ctypes.c_double), ("seed", ctypes.c_uint64), ("max_slots", ctypes.c_int32),
                ("num_paths", ctypes.c_int32), ("paths", ctypes.c_void_p)]


class gwtf_heur_out_t(ctypes.Structure):
    _fields_ = [("node_flow", ctypes.c_void_p), ("arc_flow", ctypes.c_void_p), ("used", ctypes.c_void_p),
                ("accepted", ctypes.c_void_p), ("temperature", ctypes.c_void_p), ("counters", ctypes.c_void_p)]


GWTF_HEUR_SUM = 0
GWTF_HEUR_MAX = 1
HEUR_COUNTERS_PER_INSTANCE = 4


class GwtfError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


_lib = None
_lock = threading.Lock()


def load_library(path: str = LIB_PATH):
    """Load libgwtf_mcf.so and declare its prototypes (raises if absent)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: build the HIP library first "
                "(python -m paper_2509_21221_amd.build_native or __graft_entry__.build())")
        lib = ctypes.CDLL(path)
        vp, i32, i64p = ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p
        lib.gwtf_mcf_create.argtypes = [ctypes.POINTER(gwtf_mcf_shape_t), vp, ctypes.POINTER(vp)]
        lib.gwtf_mcf_create.restype = ctypes.c_int
        lib.gwtf_mcf_solve_batch.argtypes = [vp, ctypes.POINTER(gwtf_mcf_batch_t)]
        lib.gwtf_mcf_solve_batch.restype = ctypes.c_int
        lib.gwtf_mcf_get_flows.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp]
        lib.gwtf_mcf_get_flows.restype = ctypes.c_int
        lib.gwtf_mcf_get_stats.argtypes = [vp, i32, i32, i64p]
        lib.gwtf_mcf_get_stats.restype = ctypes.c_int
        lib.gwtf_mcf_get_passes.argtypes = [vp, i32, i32, vp]
        lib.gwtf_mcf_get_passes.restype = ctypes.c_int
        lib.gwtf_mcf_solve_batch_noalloc.argtypes = [ctypes.POINTER(gwtf_mcf_shape_t), vp,
                                                     ctypes.POINTER(gwtf_mcf_batch_t)]
        lib.gwtf_mcf_solve_batch_noalloc.restype = ctypes.c_int
        lib.gwtf_mcf_solve_located.argtypes = [vp, ctypes.POINTER(gwtf_mcf_located_batch_t)]
        lib.gwtf_mcf_solve_located.restype = ctypes.c_int
        lib.gwtf_whatif_count.argtypes = [i32, i32, ctypes.POINTER(ctypes.c_int64)]
        lib.gwtf_whatif_count.restype = ctypes.c_int
        lib.gwtf_mcf_whatif_expand.argtypes = [vp, ctypes.POINTER(gwtf_mcf_batch_t),
                                               ctypes.POINTER(gwtf_whatif_candidates_t), ctypes.c_int64, i32,
                                               ctypes.POINTER(gwtf_mcf_instances_t)]
        lib.gwtf_mcf_whatif_expand.restype = ctypes.c_int
        lib.gwtf_mcf_whatif_best.argtypes = [vp, i32, vp, vp, vp, ctypes.c_int64, i32, vp]
        lib.gwtf_mcf_whatif_best.restype = ctypes.c_int
        lib.gwtf_mcf_resolve_churn.argtypes = [vp, ctypes.POINTER(gwtf_mcf_batch_t),
                                               ctypes.POINTER(gwtf_mcf_flow_in_t),
                                               ctypes.POINTER(gwtf_mcf_flow_out_t), vp]
        lib.gwtf_mcf_resolve_churn.restype = ctypes.c_int
        lib.gwtf_mcf_simulate_heuristic.argtypes = [vp, ctypes.POINTER(gwtf_mcf_batch_t),
                                                    ctypes.POINTER(gwtf_heur_config_t),
                                                    ctypes.POINTER(gwtf_heur_out_t)]
        lib.gwtf_mcf_simulate_heuristic.restype = ctypes.c_int
        lib.gwtf_mcf_calibrate_handoff.argtypes = [i32, vp, i32, ctypes.POINTER(ctypes.c_double)]
        lib.gwtf_mcf_calibrate_handoff.restype = ctypes.c_int
        lib.gwtf_mcf_destroy.argtypes = [vp]
        lib.gwtf_mcf_destroy.restype = None
        lib.gwtf_mcf_last_error.argtypes = [vp]
        lib.gwtf_mcf_last_error.restype = ctypes.c_char_p
        _lib = lib
        return lib


def gwtf_mcf_last_error(handle=None) -> str:
    return load_library().gwtf_mcf_last_error(handle).decode()


def _check(code, handle=None):
    if code != GWTF_OK:
        raise GwtfError(code, gwtf_mcf_last_error(handle))


def gwtf_mcf_create(num_stages: int, nodes_per_stage: int, max_batch: int, device: int = 0,
                    hip_stream: int = 0):
    """Returns an opaque handle (int) for solves of this shape on ``device``."""
    lib = load_library()
    shape = gwtf_mcf_shape_t(num_stages, nodes_per_stage, max_batch, device)
    out = ctypes.c_void_p()
    _check(lib.gwtf_mcf_create(ctypes.byref(shape), ctypes.c_void_p(hip_stream or None),
                               ctypes.byref(out)))
    return out.value


def gwtf_mcf_solve_batch(handle, batch: int, node_cap: int, node_cost: int, arc_cost: int,
                         src_cost: int, snk_cost: int, supply: int, flow_value: int,
                         total_cost: int, status: int) -> None:
    """All arguments after ``batch`` are device addresses (0 = NULL)."""
    b = gwtf_mcf_batch_t(batch, node_cap or None, node_cost or None, arc_cost or None,
                         src_cost or None, snk_cost or None, supply or None, flow_value or None,
                         total_cost or None, status or None)
    _check(load_library().gwtf_mcf_solve_batch(ctypes.c_void_p(handle), ctypes.byref(b)), handle)


def gwtf_mcf_solve_batch_noalloc(num_stages: int, nodes_per_stage: int, max_batch: int, device: int,
                                 hip_stream: int, batch: int, node_cap: int, node_cost: int, arc_cost: int,
                                 src_cost: int, snk_cost: int, supply: int, flow_value: int,
                                 total_cost: int, status: int) -> None:
    """The solve of ``gwtf_mcf_solve_batch`` without a handle, its workspace
    in the library's fixed per-device array (no allocation).  Arguments
    after ``batch`` are device addresses (0 = NULL)."""
    shape = gwtf_mcf_shape_t(num_stages, nodes_per_stage, max_batch, device)
    b = gwtf_mcf_batch_t(batch, node_cap or None, node_cost or None, arc_cost or None,
                         src_cost or None, snk_cost or None, supply or None, flow_value or None,
                         total_cost or None, status or None)
    _check(load_library().gwtf_mcf_solve_batch_noalloc(ctypes.byref(shape), ctypes.c_void_p(hip_stream or None),
                                                        ctypes.byref(b)))


def gwtf_mcf_solve_located(handle, batch: int, num_locations: int, node_cap: int, node_cost: int,
                           location: int, latency: int, src_cost: int, snk_cost: int, supply: int,
                           flow_value: int, total_cost: int, status: int) -> None:
    """All arguments after ``num_locations`` are device addresses (0 = NULL)."""
    b = gwtf_mcf_located_batch_t(batch, num_locations, node_cap or None, node_cost or None,
                                 location or None, latency or None, src_cost or None, snk_cost or None,
                                 supply or None, flow_value or None, total_cost or None, status or None)
    _check(load_library().gwtf_mcf_solve_located(ctypes.c_void_p(handle), ctypes.byref(b)), handle)


def gwtf_mcf_calibrate_handoff(device: int = 0, hip_stream: int = 0, block_distance: int = 4):
    """One-way hand-off latencies in ns: LDS wave to wave, device scope
    between workgroups 0 and ``block_distance``, and between workgroups 0
    and 8 (-1 where a bounded wait ran out)."""
    out = (ctypes.c_double * 3)()
    _check(load_library().gwtf_mcf_calibrate_handoff(device, ctypes.c_void_p(hip_stream or None), block_distance,
                                                     out))
    return {"lds_wave_ns": out[0], "device_neighbour_ns": out[1], "device_same_xcd_ns": out[2]}


def gwtf_mcf_get_flows(handle, first: int, count: int, node_flow: int = 0, arc_flow: int = 0,
                       src_flow: int = 0, snk_flow: int = 0, potential: int = 0) -> None:
    _check(load_library().gwtf_mcf_get_flows(
        ctypes.c_void_p(handle), first, count, node_flow or None, arc_flow or None,
        src_flow or None, snk_flow or None, potential or None), handle)


def gwtf_mcf_get_stats(handle, first: int, count: int, stats: int) -> None:
    _check(load_library().gwtf_mcf_get_stats(ctypes.c_void_p(handle), first, count,
                                             stats or None), handle)


def gwtf_mcf_get_passes(handle, first: int, count: int, passes: int) -> None:
    _check(load_library().gwtf_mcf_get_passes(ctypes.c_void_p(handle), first, count,
                                              passes or None), handle)


def gwtf_whatif_count(num_stages: int, num_candidates: int) -> int:
    """S!/(S-m)!: the number of placements of m candidates over S stages."""
    out = ctypes.c_int64()
    _check(load_library().gwtf_whatif_count(num_stages, num_candidates, ctypes.byref(out)))
    return out.value


def gwtf_mcf_whatif_expand(handle, base: dict, cand: dict, first: int, count: int, out: dict) -> None:
    """``base``, ``cand`` and ``out`` map the C struct field names to device
    addresses (0 = NULL); cand also carries num_candidates and slot."""
    b = gwtf_mcf_batch_t(1, base.get("node_cap") or None, base.get("node_cost") or None,
                         base.get("arc_cost") or None, base.get("src_cost") or None,
                         base.get("snk_cost") or None, base.get("supply") or None, None, None, None)
    c = gwtf_whatif_candidates_t(cand["num_candidates"], cand["slot"],
                                 *(cand.get(k) or None for k in ("cap", "cost", "in_cost", "out_cost",
                                                                  "link_cost", "src_cost", "snk_cost")))
    o = gwtf_mcf_instances_t(*(out.get(k) or None for k in ("node_cap", "node_cost", "arc_cost", "src_cost",
                                                             "snk_cost", "supply")))
    _check(load_library().gwtf_mcf_whatif_expand(ctypes.c_void_p(handle), ctypes.byref(b), ctypes.byref(c),
                                                 first, count, ctypes.byref(o)), handle)


def gwtf_mcf_whatif_best(handle, count: int, flow_value: int, total_cost: int, status: int, first: int,
                         merge: int, best: int) -> None:
    _check(load_library().gwtf_mcf_whatif_best(ctypes.c_void_p(handle), count, flow_value or None,
                                               total_cost or None, status or None, first, merge,
                                               best or None), handle)


def gwtf_mcf_resolve_churn(handle, batch: int, node_cap: int, node_cost: int, arc_cost: int,
                           src_cost: int, snk_cost: int, supply: int, flow_value: int,
                           total_cost: int, status: int, start: dict, per_instance: bool,
                           out: dict | None = None, work: int = 0) -> None:
    """Device addresses as for ``gwtf_mcf_solve_batch``; ``start`` (and
    ``out``, if given) map node_flow, arc_flow, src_flow, snk_flow to device
    addresses (0 = NULL)."""
    b = gwtf_mcf_batch_t(batch, node_cap or None, node_cost or None, arc_cost or None,
                         src_cost or None, snk_cost or None, supply or None, flow_value or None,
                         total_cost or None, status or None)
    keys = ("node_flow", "arc_flow", "src_flow", "snk_flow")
    st = gwtf_mcf_flow_in_t(*[start.get(k) or None for k in keys], int(bool(per_instance)))
    o = gwtf_mcf_flow_out_t(*[out.get(k) or None for k in keys]) if out is not None else None
    _check(load_library().gwtf_mcf_resolve_churn(ctypes.c_void_p(handle), ctypes.byref(b), ctypes.byref(st),
                                                 ctypes.byref(o) if o is not None else None,
                                                 ctypes.c_void_p(work or None)), handle)


def gwtf_mcf_simulate_heuristic(handle, batch: int, node_cap: int, node_cost: int, arc_cost: int,
                                src_cost: int, snk_cost: int, supply: int, flow_value: int, total_cost: int,
                                status: int, rounds: int, objective: int, t0: float, alpha: float, seed: int,
                                max_slots: int, num_paths: int = 0, paths: int = 0, out: dict | None = None) -> None:
    """Device addresses as for ``gwtf_mcf_solve_batch``; ``out`` maps the
    gwtf_heur_out_t field names to device addresses (0 = NULL)."""
    b = gwtf_mcf_batch_t(batch, node_cap or None, node_cost or None, arc_cost or None,
                         src_cost or None, snk_cost or None, supply or None, flow_value or None,
                         total_cost or None, status or None)
    c = gwtf_heur_config_t(rounds, objective, t0, alpha, seed & (2**64 - 1), max_slots, num_paths, paths or None)
    o = None
    if out is not None:
        o = gwtf_heur_out_t(*(out.get(k) or None for k in ("node_flow", "arc_flow", "used", "accepted",
                                                             "temperature", "counters")))
    _check(load_library().gwtf_mcf_simulate_heuristic(ctypes.c_void_p(handle), ctypes.byref(b), ctypes.byref(c),
                                                      ctypes.byref(o) if o is not None else None), handle)


def gwtf_mcf_destroy(handle) -> None:
    load_library().gwtf_mcf_destroy(ctypes.c_void_p(handle))


class Solver:
    """A solver handle bound to torch's current HIP stream on ``device``.

    ``solve`` takes int32 device tensors in the canonical layout
    ([B][S][n] caps and compute costs, [B][S-1][n][n] link delays or None
    when S == 1, optional [B][n] data-node delays, [B] supply) and returns
    int64 flow value, int64 cost and int32 status tensors on the device.
    """

    def __init__(self, num_stages: int, nodes_per_stage: int, max_batch: int, device: int = 0,
                 stream=None):
        import torch

        self.torch = torch
        self.S, self.n, self.max_batch, self.device = num_stages, nodes_per_stage, max_batch, device
        self.stream = stream if stream is not None else torch.cuda.current_stream(device)
        self.handle = gwtf_mcf_create(num_stages, nodes_per_stage, max_batch, device,
                                      self.stream.cuda_stream)
        self.last_batch = 0

    def _arg(self, t, shape, name):
        torch = self.torch
        if t is None:
            return 0
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name}: expected a torch tensor")
        if t.dtype != torch.int32 or not t.is_contiguous() or t.device.type != "cuda" \
                or t.device.index != self.device:
            raise ValueError(f"{name}: need a contiguous int32 tensor on cuda:{self.device}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name}: shape {tuple(t.shape)} != {tuple(shape)}")
        return t.data_ptr()

    def solve(self, node_cap, node_cost, arc_cost, supply, src_cost=None, snk_cost=None,
              out=None):
        torch = self.torch
        S, n = self.S, self.n
        B = int(supply.shape[0])
        args = [self._arg(node_cap, (B, S, n), "node_cap"), self._arg(node_cost, (B, S, n), "node_cost"),
                self._arg(arc_cost, (B, S - 1, n, n), "arc_cost") if S > 1 else 0,
                self._arg(src_cost, (B, n), "src_cost"), self._arg(snk_cost, (B, n), "snk_cost"),
                self._arg(supply, (B,), "supply")]
        if S > 1 and arc_cost is None:
            raise ValueError("arc_cost is required when S > 1")
        dev = torch.device("cuda", self.device)
        if out is None:
            out = (torch.empty(B, dtype=torch.int64, device=dev),
                   torch.empty(B, dtype=torch.int64, device=dev),
                   torch.empty(B, dtype=torch.int32, device=dev))
        F, cost, status = out
        gwtf_mcf_solve_batch(self.handle, B, *args, F.data_ptr(), cost.data_ptr(), status.data_ptr())
        self.last_batch = B
        return F, cost, status

    def solve_located(self, node_cap, node_cost, location, latency, supply, src_cost=None, snk_cost=None,
                      out=None):
        """Located batch: [B][S][n] capacities, compute costs and locations,
        [B][L][L] latencies, [B] supply, optional [B][n] data-node delays."""
        torch = self.torch
        S, n = self.S, self.n
        B = int(supply.shape[0])
        L = int(latency.shape[1]) if latency.dim() == 3 else -1
        args = [self._arg(node_cap, (B, S, n), "node_cap"), self._arg(node_cost, (B, S, n), "node_cost"),
                self._arg(location, (B, S, n), "location"), self._arg(latency, (B, L, L), "latency"),
                self._arg(src_cost, (B, n), "src_cost"), self._arg(snk_cost, (B, n), "snk_cost"),
                self._arg(supply, (B,), "supply")]
        dev = torch.device("cuda", self.device)
        if out is None:
            out = (torch.empty(B, dtype=torch.int64, device=dev),
                   torch.empty(B, dtype=torch.int64, device=dev),
                   torch.empty(B, dtype=torch.int32, device=dev))
        F, cost, status = out
        gwtf_mcf_solve_located(self.handle, B, L, *args, F.data_ptr(), cost.data_ptr(), status.data_ptr())
        self.last_batch = B
        return F, cost, status

    def resolve_churn(self, node_cap, node_cost, arc_cost, supply, start, src_cost=None, snk_cost=None,
                      flows=False, work=False):
        """Warm-started solve of a batch from ``start`` (a dict of int32 device
        tensors node_flow, arc_flow, src_flow, snk_flow with a leading
        dimension of 1 for one flow shared by the batch, or B).  Returns
        (F, cost, status) and, when asked, a dict of result flows and the
        [B][4] work counters."""
        torch = self.torch
        S, n = self.S, self.n
        B = int(supply.shape[0])
        args = [self._arg(node_cap, (B, S, n), "node_cap"), self._arg(node_cost, (B, S, n), "node_cost"),
                self._arg(arc_cost, (B, S - 1, n, n), "arc_cost") if S > 1 else 0,
                self._arg(src_cost, (B, n), "src_cost"), self._arg(snk_cost, (B, n), "snk_cost"),
                self._arg(supply, (B,), "supply")]
        if S > 1 and arc_cost is None:
            raise ValueError("arc_cost is required when S > 1")
        m = int(start["node_flow"].shape[0])
        if m not in (1, B):
            raise ValueError("start flow: leading dimension must be 1 or the batch size")
        shapes = {"node_flow": (m, S, n), "arc_flow": (m, S - 1, n, n), "src_flow": (m, n), "snk_flow": (m, n)}
        st = {k: (self._arg(start[k], shp, "start " + k) if (k != "arc_flow" or S > 1) else 0)
              for k, shp in shapes.items()}
        dev = torch.device("cuda", self.device)
        F = torch.empty(B, dtype=torch.int64, device=dev)
        cost = torch.empty(B, dtype=torch.int64, device=dev)
        status = torch.empty(B, dtype=torch.int32, device=dev)
        out = None
        if flows:
            out = {"node_flow": torch.empty((B, S, n), dtype=torch.int32, device=dev),
                   "arc_flow": torch.empty((B, max(S - 1, 0), n, n), dtype=torch.int32, device=dev),
                   "src_flow": torch.empty((B, n), dtype=torch.int32, device=dev),
                   "snk_flow": torch.empty((B, n), dtype=torch.int32, device=dev)}
        wk = torch.empty((B, CHURN_WORK_PER_INSTANCE), dtype=torch.int64, device=dev) if work else None
        gwtf_mcf_resolve_churn(self.handle, B, *args, F.data_ptr(), cost.data_ptr(), status.data_ptr(), st,
                               m == B and B > 1,
                               {k: (v.data_ptr() if (k != "arc_flow" or S > 1) else 0) for k, v in out.items()}
                               if out is not None else None,
                               wk.data_ptr() if wk is not None else 0)
        res = (F, cost, status)
        if flows:
            res = res + (out,)
        if work:
            res = res + (wk,)
        return res

    def simulate_heuristic(self, node_cap, node_cost, arc_cost, supply, src_cost=None, snk_cost=None,
                           rounds: int = 120, objective: str = "sum", t0: float = 1.7, alpha: float = 0.95,
                           seed: int = 0, max_slots: int = 1024, paths=None, details: bool = False):
        """Decentralized-heuristic simulation of a batch (one wave per
        instance).  Returns (F, cost, status) device tensors and, with
        ``details``, a dict of node_flow, arc_flow, used, accepted,
        temperature and counters tensors.  ``paths``: optional int32 device
        tensor [B][P][S] of initial complete paths."""
        torch = self.torch
        S, n = self.S, self.n
        B = int(supply.shape[0])
        args = [self._arg(node_cap, (B, S, n), "node_cap"), self._arg(node_cost, (B, S, n), "node_cost"),
                self._arg(arc_cost, (B, S - 1, n, n), "arc_cost") if S > 1 else 0,
                self._arg(src_cost, (B, n), "src_cost"), self._arg(snk_cost, (B, n), "snk_cost"),
                self._arg(supply, (B,), "supply")]
        if S > 1 and arc_cost is None:
            raise ValueError("arc_cost is required when S > 1")
        P = 0
        pp = 0
        if paths is not None:
            P = int(paths.shape[1])
            pp = self._arg(paths, (B, P, S), "paths")
        dev = torch.device("cuda", self.device)
        F = torch.empty(B, dtype=torch.int64, device=dev)
        cost = torch.empty(B, dtype=torch.int64, device=dev)
        status = torch.empty(B, dtype=torch.int32, device=dev)
        det = None
        if details:
            det = {"node_flow": torch.empty((B, S, n), dtype=torch.int32, device=dev),
                   "arc_flow": torch.empty((B, max(S - 1, 0), n, n), dtype=torch.int32, device=dev),
                   "used": torch.empty((B, S, n), dtype=torch.int32, device=dev),
                   "accepted": torch.empty((B, S, n), dtype=torch.int32, device=dev),
                   "temperature": torch.empty((B, S, n), dtype=torch.float64, device=dev),
                   "counters": torch.empty((B, HEUR_COUNTERS_PER_INSTANCE), dtype=torch.int64, device=dev)}
        obj = {"sum": GWTF_HEUR_SUM, "max": GWTF_HEUR_MAX}[objective]
        gwtf_mcf_simulate_heuristic(
            self.handle, B, *args, F.data_ptr(), cost.data_ptr(), status.data_ptr(), rounds, obj, t0, alpha,
            seed, max_slots, P, pp,
            {k: (v.data_ptr() if (k != "arc_flow" or S > 1) else 0) for k, v in det.items()} if det else None)
        return (F, cost, status, det) if details else (F, cost, status)

    def flows(self, first: int = 0, count: int | None = None):
        torch = self.torch
        count = self.last_batch - first if count is None else count
        S, n = self.S, self.n
        dev = torch.device("cuda", self.device)
        nf = torch.empty((count, S, n), dtype=torch.int32, device=dev)
        af = torch.empty((count, max(S - 1, 0), n, n), dtype=torch.int32, device=dev)
        sf = torch.empty((count, n), dtype=torch.int32, device=dev)
        tf = torch.empty((count, n), dtype=torch.int32, device=dev)
        pot = torch.empty((count, 2 * S * n + 3), dtype=torch.int32, device=dev)
        gwtf_mcf_get_flows(self.handle, first, count, nf.data_ptr(), af.data_ptr() if S > 1 else 0,
                           sf.data_ptr(), tf.data_ptr(), pot.data_ptr())
        return {"node_flow": nf, "arc_flow": af, "src_flow": sf, "snk_flow": tf, "potential": pot}

    def stats(self, first: int = 0, count: int | None = None):
        torch = self.torch
        count = self.last_batch - first if count is None else count
        st = torch.empty((count, STATS_PER_INSTANCE), dtype=torch.int64, device=torch.device("cuda", self.device))
        gwtf_mcf_get_stats(self.handle, first, count, st.data_ptr())
        return st

    def passes(self, first: int = 0, count: int | None = None):
        torch = self.torch
        count = self.last_batch - first if count is None else count
        out = torch.empty(count, dtype=torch.int32, device=torch.device("cuda", self.device))
        gwtf_mcf_get_passes(self.handle, first, count, out.data_ptr())
        return out

    def whatif_expand(self, base, cand, slot: int, first: int = 0, count: int | None = None, out=None):
        """Placements [first, first + count) of ``cand`` over the base instance
        as a batch of device tensors (keys node_cap, node_cost, arc_cost,
        src_cost, snk_cost, supply).  ``base`` maps those keys to one
        instance's int32 device tensors (src_cost / snk_cost optional);
        ``cand`` maps cap [m][S], cost [m][S], in_cost and out_cost [m][S][n],
        link_cost [m][m] and optional src_cost / snk_cost [m]."""
        torch = self.torch
        S, n = self.S, self.n
        m = 0 if cand.get("cap") is None else int(cand["cap"].shape[0])
        total = gwtf_whatif_count(S, m)
        count = total - first if count is None else count
        ba = {"node_cap": self._arg(base["node_cap"], (1, S, n), "node_cap"),
              "node_cost": self._arg(base["node_cost"], (1, S, n), "node_cost"),
              "arc_cost": self._arg(base.get("arc_cost"), (1, S - 1, n, n), "arc_cost") if S > 1 else 0,
              "src_cost": self._arg(base.get("src_cost"), (1, n), "src_cost"),
              "snk_cost": self._arg(base.get("snk_cost"), (1, n), "snk_cost"),
              "supply": self._arg(base["supply"], (1,), "supply")}
        links = S > 1 and m > 0
        ca = {"num_candidates": m, "slot": slot,
              "cap": self._arg(cand.get("cap"), (m, S), "cap") if m > 0 else 0,
              "cost": self._arg(cand.get("cost"), (m, S), "cost") if m > 0 else 0,
              "in_cost": self._arg(cand.get("in_cost"), (m, S, n), "in_cost") if links else 0,
              "out_cost": self._arg(cand.get("out_cost"), (m, S, n), "out_cost") if links else 0,
              "link_cost": self._arg(cand.get("link_cost"), (m, m), "link_cost") if links else 0,
              "src_cost": self._arg(cand.get("src_cost"), (m,), "src_cost") if m > 0 else 0,
              "snk_cost": self._arg(cand.get("snk_cost"), (m,), "snk_cost") if m > 0 else 0}
        dev = torch.device("cuda", self.device)
        if out is None:
            e = lambda *shape: torch.empty(shape, dtype=torch.int32, device=dev)
            out = {"node_cap": e(count, S, n), "node_cost": e(count, S, n),
                   "arc_cost": e(count, S - 1, n, n) if S > 1 else None,
                   "src_cost": e(count, n), "snk_cost": e(count, n), "supply": e(count)}
        oa = {"node_cap": self._arg(out["node_cap"], (count, S, n), "out node_cap"),
              "node_cost": self._arg(out["node_cost"], (count, S, n), "out node_cost"),
              "arc_cost": self._arg(out.get("arc_cost"), (count, S - 1, n, n), "out arc_cost") if S > 1 else 0,
              "src_cost": self._arg(out["src_cost"], (count, n), "out src_cost"),
              "snk_cost": self._arg(out["snk_cost"], (count, n), "out snk_cost"),
              "supply": self._arg(out["supply"], (count,), "out supply")}
        gwtf_mcf_whatif_expand(self.handle, ba, ca, first, count, oa)
        return out

    def whatif_best(self, F, cost, status, first: int = 0, best=None, merge: bool = False):
        """Best placement of a solved expanded batch: an int64 device tensor
        {first + index, F, cost} ({-1, 0, 0} if no instance is OK).  With
        ``merge`` the result is combined with what ``best`` holds."""
        torch = self.torch
        count = int(F.shape[0])
        for t, dt, name in ((F, torch.int64, "F"), (cost, torch.int64, "cost"), (status, torch.int32, "status")):
            if t.dtype != dt or not t.is_contiguous() or t.device.type != "cuda" or t.device.index != self.device \
                    or tuple(t.shape) != (count,):
                raise ValueError(f"{name}: need a contiguous {dt} tensor of shape ({count},) on cuda:{self.device}")
        if best is None:
            if merge:
                raise ValueError("merge needs an existing best tensor")
            best = torch.empty(3, dtype=torch.int64, device=torch.device("cuda", self.device))
        elif best.dtype != torch.int64 or tuple(best.shape) != (3,) or not best.is_contiguous() \
                or best.device.type != "cuda" or best.device.index != self.device:
            raise ValueError(f"best: need a contiguous int64 tensor of shape (3,) on cuda:{self.device}")
        gwtf_mcf_whatif_best(self.handle, count, F.data_ptr(), cost.data_ptr(), status.data_ptr(), first,
                             int(merge), best.data_ptr())
        return best

    def close(self):
        if self.handle:
            gwtf_mcf_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
