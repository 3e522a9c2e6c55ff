"""Seeded synthetic workloads for the layered min-cost max-flow problem.

This module only draws random numbers and lays them out; it performs none of
the flow method's arithmetic, so the HIP path and the CPU oracle can both be
fed from it without sharing any solver code.  It imports nothing from the rest
of the package.

Problem shape (paper Sec. III system model and Sec. IV, Eq. 1): S pipeline
stages with n relay nodes each.  Node i has a memory capacity cap_i (how many
microbatches it can hold at once) and a compute cost c_i; consecutive stages
are linked by delays d(i, j).  One data node injects ``supply`` microbatches
into stage 0 and receives them back from stage S-1 (Sec. V-A: the data node
is both source and sink).

Canonical layout of a batch of B instances (all int32, C-contiguous):

    node_cap  [B][S][n]        >= 0 (0 = node absent, e.g. crashed)
    node_cost [B][S][n]        >= 0 (compute cost, put on the node's split arc)
    arc_cost  [B][S-1][n][n]   arc_cost[b][k][i][j] = delay from node i of
                               stage k to node j of stage k+1, >= 0, or
                               NO_ARC (-1) when the two nodes share no link
    src_cost  [B][n]           data node -> stage-0 node delay, >= 0
    snk_cost  [B][n]           stage-(S-1) node -> data node delay, >= 0
    supply    [B]              microbatches the data node injects, >= 0

Seeding: instance ``i`` of preset ``c`` draws from
``np.random.SeedSequence(0, spawn_key=(c, i))``, so any subset of a batch
regenerates identically.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

NO_ARC = -1

# The ten simulated geographic locations of the paper's testbed (abstract,
# Sec. VI setup).
NUM_LOCATIONS = 10


@dataclass
class Batch:
    """A batch of independent layered instances in the canonical layout."""

    S: int
    n: int
    node_cap: np.ndarray
    node_cost: np.ndarray
    arc_cost: np.ndarray
    src_cost: np.ndarray
    snk_cost: np.ndarray
    supply: np.ndarray
    name: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return int(self.supply.shape[0])

    def subset(self, idx) -> "Batch":
        idx = np.asarray(idx, dtype=np.int64)
        return Batch(
            self.S, self.n,
            np.ascontiguousarray(self.node_cap[idx]),
            np.ascontiguousarray(self.node_cost[idx]),
            np.ascontiguousarray(self.arc_cost[idx]),
            np.ascontiguousarray(self.src_cost[idx]),
            np.ascontiguousarray(self.snk_cost[idx]),
            np.ascontiguousarray(self.supply[idx]),
            name=self.name, meta=dict(self.meta),
        )

    def instance(self, b: int) -> "Batch":
        return self.subset([b])

    def check_layout(self) -> None:
        B, S, n = self.B, self.S, self.n
        shapes = {
            "node_cap": (B, S, n), "node_cost": (B, S, n),
            "arc_cost": (B, max(S - 1, 0), n, n),
            "src_cost": (B, n), "snk_cost": (B, n), "supply": (B,),
        }
        for key, shp in shapes.items():
            a = getattr(self, key)
            if a.shape != shp:
                raise ValueError(f"{key}: shape {a.shape} != {shp}")
            if a.dtype != np.int32 or not a.flags.c_contiguous:
                raise ValueError(f"{key}: need C-contiguous int32")


def _empty(B: int, S: int, n: int, name: str) -> Batch:
    return Batch(
        S, n,
        np.zeros((B, S, n), np.int32),
        np.zeros((B, S, n), np.int32),
        np.zeros((B, max(S - 1, 0), n, n), np.int32),
        np.zeros((B, n), np.int32),
        np.zeros((B, n), np.int32),
        np.zeros((B,), np.int32),
        name=name,
    )


def _rng(preset: int, instance: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(0, spawn_key=(preset, instance)))


def _int_uniform(rng, lo, hi, size):
    """Integer uniform on the closed range [lo, hi]."""
    return rng.integers(lo, hi + 1, size=size, dtype=np.int64).astype(np.int32)


def _location_instance(rng, S, n, cap_hi, out, b):
    """Fill instance b of ``out`` with the location-latency recipe.

    Every node sits at one of NUM_LOCATIONS locations; a symmetric latency
    matrix has off-diagonal entries U[5, 300] and diagonal entries U[1, 5]
    (ms).  The delay of the arc between two nodes is the latency between
    their locations.  Compute costs are lognormal(3, 0.5) rounded to the
    nearest integer and clipped to [5, 200]; capacities are U[1, cap_hi].
    """
    L = _int_uniform(rng, 5, 300, (NUM_LOCATIONS, NUM_LOCATIONS)).astype(np.int64)
    L = np.triu(L, 1)
    L = L + L.T
    L[np.arange(NUM_LOCATIONS), np.arange(NUM_LOCATIONS)] = _int_uniform(rng, 1, 5, NUM_LOCATIONS)
    loc = rng.integers(0, NUM_LOCATIONS, size=(S, n))
    ncost = np.clip(np.rint(rng.lognormal(3.0, 0.5, size=(S, n))), 5, 200).astype(np.int32)
    cap = _int_uniform(rng, 1, cap_hi, (S, n))
    out.node_cap[b] = cap
    out.node_cost[b] = ncost
    if S > 1:
        out.arc_cost[b] = L[loc[:-1, :, None], loc[1:, None, :]].astype(np.int32)
    return loc, L


def config1(B: int = 1024, first: int = 0) -> Batch:
    """Tiny batch: S=4, n=4, caps U[1,4], node and arc costs U[1,100], supply 16."""
    S, n = 4, 4
    out = _empty(B, S, n, "c1: S=4 n=4 tiny batch")
    for b in range(B):
        rng = _rng(1, first + b)
        out.node_cap[b] = _int_uniform(rng, 1, 4, (S, n))
        out.node_cost[b] = _int_uniform(rng, 1, 100, (S, n))
        out.arc_cost[b] = _int_uniform(rng, 1, 100, (S - 1, n, n))
        out.supply[b] = 16
    return out


def config2(B: int = 16384, first: int = 0) -> Batch:
    """Heterogeneous geography: S=8, n=8, 10 locations, caps U[1,8], supply 64."""
    S, n = 8, 8
    out = _empty(B, S, n, "c2: S=8 n=8 10-location geography")
    for b in range(B):
        _location_instance(_rng(2, first + b), S, n, 8, out, b)
        out.supply[b] = 64
    return out


def config3(B: int = 16384, first: int = 0) -> Batch:
    """Churn re-solve variants of config-2 instance 0.

    Variant v draws p ~ U(0.1, 0.3), deletes (cap = 0) each node
    independently with probability p, and multiplies the delay of every arc
    whose two endpoints both survive by j/100, j an integer U[90, 130],
    rounded half up: (cost * j + 50) // 100.
    """
    base = config2(1, 0)
    S, n = base.S, base.n
    out = _empty(B, S, n, "c3: churn variants of c2 instance 0")
    for b in range(B):
        rng = _rng(3, first + b)
        p = rng.uniform(0.1, 0.3)
        alive = rng.random((S, n)) >= p
        cap = base.node_cap[0].copy()
        cap[~alive] = 0
        jit = _int_uniform(rng, 90, 130, (S - 1, n, n)).astype(np.int64)
        arc = base.arc_cost[0].astype(np.int64)
        both = alive[:-1, :, None] & alive[1:, None, :]
        arc = np.where(both, (arc * jit + 50) // 100, arc)
        out.node_cap[b] = cap
        out.node_cost[b] = base.node_cost[0]
        out.arc_cost[b] = arc.astype(np.int32)
        out.supply[b] = 64
    return out


def config4(B: int = 256, first: int = 0) -> Batch:
    """7B-scale pipeline: S=32, n=64, full bipartite, c2 recipe, supply 512."""
    S, n = 32, 64
    out = _empty(B, S, n, "c4: S=32 n=64 full bipartite")
    for b in range(B):
        _location_instance(_rng(4, first + b), S, n, 8, out, b)
        out.supply[b] = 512
    return out


def config5(B: int = 1, first: int = 0) -> Batch:
    """Single huge instance: S=64, n=512, caps U[1,16], supply 4096."""
    S, n = 64, 512
    out = _empty(B, S, n, "c5: S=64 n=512 single huge instance")
    for b in range(B):
        _location_instance(_rng(5, first + b), S, n, 16, out, b)
        out.supply[b] = 4096
    return out


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


def paper_flow_test(setting: int, B: int = 8, first: int = 0) -> Batch:
    """Single-source settings 1-4 of the paper's flow-test table (Sec. VI,
    ablation): 40 relays over 8 (or 10) stages, capacities floor(U(a, b)),
    link costs floor(U(a, b)) on every link including the data node's.
    Relays are split evenly over the stages; node compute costs are 0
    because the table lists link costs only; the data node's supply is the
    total relay capacity so that it is never the bottleneck."""
    spec = {
        1: (8, (1, 3), (1, 20)),
        2: (10, (1, 3), (1, 20)),
        3: (8, (5, 15), (1, 20)),
        4: (8, (1, 3), (5, 100)),
    }[setting]
    S, (clo, chi), (alo, ahi) = spec
    n = 40 // S
    out = _empty(B, S, n, f"paper flow-test setting {setting}")
    for b in range(B):
        rng = _rng(100 + setting, first + b)
        flo = lambda lo, hi, size: np.floor(rng.uniform(lo, hi, size=size)).astype(np.int32)
        out.node_cap[b] = flo(clo, chi, (S, n))
        out.arc_cost[b] = flo(alo, ahi, (S - 1, n, n))
        out.src_cost[b] = flo(alo, ahi, n)
        out.snk_cost[b] = flo(alo, ahi, n)
        out.supply[b] = int(out.node_cap[b].sum())
    return out


def random_small(B: int, S: int, n: int, seed: int, cap_hi: int = 3, cost_hi: int = 20,
                 supply_hi: int = 6, holes: float = 0.0, zero_cap: float = 0.0,
                 src_snk: bool = True) -> Batch:
    """Small random instances for exhaustive and cross-library checks.

    Capacities U[0 or 1, cap_hi], costs U[0, cost_hi], supply U[0, supply_hi];
    a fraction ``holes`` of inter-stage arcs is removed (NO_ARC) and a
    fraction ``zero_cap`` of nodes is deleted (cap = 0).
    """
    out = _empty(B, S, n, f"random S={S} n={n}")
    for b in range(B):
        rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(S, n, b)))
        cap = _int_uniform(rng, 1, cap_hi, (S, n))
        cap[rng.random((S, n)) < zero_cap] = 0
        out.node_cap[b] = cap
        out.node_cost[b] = _int_uniform(rng, 0, cost_hi, (S, n))
        arc = _int_uniform(rng, 0, cost_hi, (max(S - 1, 0), n, n))
        if holes > 0:
            arc[rng.random(arc.shape) < holes] = NO_ARC
        out.arc_cost[b] = arc
        if src_snk:
            out.src_cost[b] = _int_uniform(rng, 0, cost_hi, n)
            out.snk_cost[b] = _int_uniform(rng, 0, cost_hi, n)
        out.supply[b] = int(rng.integers(0, supply_hi + 1))
    return out


def concat(batches) -> Batch:
    """Concatenate batches of one shape."""
    batches = list(batches)
    S, n = batches[0].S, batches[0].n
    for x in batches:
        if (x.S, x.n) != (S, n):
            raise ValueError("concat needs one shape")
    cat = lambda key: np.ascontiguousarray(np.concatenate([getattr(x, key) for x in batches]))
    return Batch(S, n, cat("node_cap"), cat("node_cost"), cat("arc_cost"),
                 cat("src_cost"), cat("snk_cost"), cat("supply"), name=batches[0].name)


@dataclass
class Candidates:
    """m nodes that may join a pipeline, with their costs for every stage
    (paper Sec. VI, handling joining nodes: every candidate knows its costs
    for each stage).  All int32, C-contiguous:

        cap  [m][S]     memory capacity if it joins stage k
        cost [m][S]     compute cost if it joins stage k
        inn  [m][S][n]  delay from node i of stage k-1 to it in stage k
                        (row k = 0 unused)
        out  [m][S][n]  delay from it in stage k to node j of stage k+1
                        (row k = S-1 unused)
        link [m][m]     delay from candidate c (stage k) to d (stage k+1)
        src  [m]        data node -> it, when it joins stage 0
        snk  [m]        it -> data node, when it joins stage S-1
    """

    cap: np.ndarray
    cost: np.ndarray
    inn: np.ndarray
    out: np.ndarray
    link: np.ndarray
    src: np.ndarray
    snk: np.ndarray

    @property
    def m(self) -> int:
        return int(self.cap.shape[0])

    def permuted(self, order) -> "Candidates":
        """The same candidates listed in another order."""
        o = np.asarray(order, dtype=np.int64)
        return Candidates(*(np.ascontiguousarray(a[o]) for a in (self.cap, self.cost, self.inn,
                                                                 self.out)),
                          np.ascontiguousarray(self.link[o][:, o]),
                          np.ascontiguousarray(self.src[o]), np.ascontiguousarray(self.snk[o]))


# Node-addition settings of the paper's test table (Sec. VI): stages,
# capacity range, inter-stage (link) cost range, each floor(U(a, b)).
NODE_ADD_SETTINGS = {1: (8, (1, 20), (1, 100)), 2: (8, (1, 20), (20, 100)),
                     3: (8, (1, 5), (1, 100)), 4: (12, (1, 20), (1, 100))}


def node_addition(setting: int = 1, instance: int = 0, supply: int = 64):
    """One what-if problem of the paper's node-addition tests (Sec. VI):
    96 relays (97 nodes, one of them the data holder) split evenly over the
    stages, plus one empty position per stage (the last) for a joining node,
    and S candidates, one per stage in every placement.

    Capacities floor(U(a, b)); every link delay (between relays, with the
    data node, and of the candidates) floor(U(a, b)); a node's compute cost
    is phi + floor(U(50, 100)), phi being the largest delay of its links
    into and out of its stage (for a candidate, of the stage it would join).
    The empty position has capacity 0 and no links.  The data node's supply
    is not given by the paper; ``supply`` microbatches (64, as in the
    8 x 8 preset) are pushed.

    Returns (base Batch with B = 1, slot, Candidates)."""
    S, (clo, chi), (alo, ahi) = NODE_ADD_SETTINGS[setting]
    n0 = 96 // S
    n = n0 + 1
    slot = n - 1
    rng = _rng(200 + setting, instance)
    flo = lambda lo, hi, size: np.floor(rng.uniform(lo, hi, size=size)).astype(np.int32)
    base = _empty(1, S, n, f"node-addition setting {setting}")
    cap = np.zeros((S, n), np.int32)
    cap[:, :n0] = flo(clo, chi, (S, n0))
    arc = np.full((max(S - 1, 0), n, n), NO_ARC, np.int32)
    arc[:, :n0, :n0] = flo(alo, ahi, (S - 1, n0, n0))
    src = np.zeros(n, np.int32)
    snk = np.zeros(n, np.int32)
    src[:n0] = flo(alo, ahi, n0)
    snk[:n0] = flo(alo, ahi, n0)
    phi = np.zeros((S, n0), np.int32)
    for k in range(S):
        into = src[None, :n0] if k == 0 else arc[k - 1, :n0, :n0]
        outof = snk[None, :n0].T if k == S - 1 else arc[k, :n0, :n0].T
        phi[k] = np.maximum(into.max(axis=0), outof.max(axis=0))
    cost = np.zeros((S, n), np.int32)
    cost[:, :n0] = phi + flo(50, 100, (S, n0))
    base.node_cap[0], base.node_cost[0], base.arc_cost[0] = cap, cost, arc
    base.src_cost[0], base.snk_cost[0], base.supply[0] = src, snk, supply

    m = S
    ccap = np.repeat(flo(clo, chi, (m, 1)), S, axis=1)
    inn = flo(alo, ahi, (m, S, n))
    out = flo(alo, ahi, (m, S, n))
    inn[:, :, slot] = flo(alo, ahi, (m, S))
    inn[:, 0, :] = 0
    out[:, S - 1, :] = 0
    link = flo(alo, ahi, (m, m))
    csrc, csnk = flo(alo, ahi, m), flo(alo, ahi, m)
    cphi = np.maximum(inn[:, :, :n0].max(axis=2), out[:, :, :n0].max(axis=2))
    cphi[:, 0] = np.maximum(csrc, out[:, 0, :n0].max(axis=1))
    cphi[:, S - 1] = np.maximum(csnk, inn[:, S - 1, :n0].max(axis=1))
    ccost = (cphi + flo(50, 100, (m, S))).astype(np.int32)
    c = Candidates(ccap, ccost, inn, out, link, csrc, csnk)
    return base, slot, c


def random_candidates(S: int, n: int, m: int, seed: int, cap_hi: int = 3, cost_hi: int = 20,
                      holes: float = 0.0) -> Candidates:
    """Small random candidates for exhaustive and cross-library checks:
    capacities U[0, cap_hi], costs U[0, cost_hi], a fraction ``holes`` of
    their links missing (NO_ARC)."""
    rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(S, n, m, 7)))
    u = lambda lo, hi, size: _int_uniform(rng, lo, hi, size)
    inn, out, link = u(0, cost_hi, (m, S, n)), u(0, cost_hi, (m, S, n)), u(0, cost_hi, (m, m))
    if holes > 0:
        for a in (inn, out, link):
            a[rng.random(a.shape) < holes] = NO_ARC
    return Candidates(u(0, cap_hi, (m, S)), u(0, cost_hi, (m, S)), inn, out, link,
                      u(0, cost_hi, m), u(0, cost_hi, m))


@dataclass
class LocatedBatch:
    """A batch whose link delays are latencies between node locations (the
    paper's testbed of Sec. VI places every node at one of a few geographic
    locations).  All int32, C-contiguous:

        node_cap, node_cost  [B][S][n]
        location             [B][S][n]   in [0, L)
        latency              [B][L][L]   >= 0: delay between two locations
        src_cost, snk_cost   [B][n]
        supply               [B]

    The link from node i of stage k to node j of stage k+1 has delay
    latency[b][location[b][k][i]][location[b][k+1][j]]."""

    S: int
    n: int
    L: int
    node_cap: np.ndarray
    node_cost: np.ndarray
    location: np.ndarray
    latency: np.ndarray
    src_cost: np.ndarray
    snk_cost: np.ndarray
    supply: np.ndarray
    name: str = ""

    @property
    def B(self) -> int:
        return int(self.supply.shape[0])

    def subset(self, idx) -> "LocatedBatch":
        idx = np.asarray(idx, dtype=np.int64)
        take = lambda a: np.ascontiguousarray(a[idx])
        return LocatedBatch(self.S, self.n, self.L, take(self.node_cap), take(self.node_cost),
                            take(self.location), take(self.latency), take(self.src_cost),
                            take(self.snk_cost), take(self.supply), name=self.name)


def located(preset: int, B: int | None = None, first: int = 0) -> LocatedBatch:
    """The location-latency presets (2, 4 and 5) in located form: the same
    random draws as CONFIGS[preset], so the implied link delays equal that
    preset's arc_cost arrays element for element."""
    S, n, cap_hi, supply, default_B = {2: (8, 8, 8, 64, 16384), 4: (32, 64, 8, 512, 256),
                                       5: (64, 512, 16, 4096, 1)}[preset]
    B = default_B if B is None else B
    L = NUM_LOCATIONS
    out = LocatedBatch(S, n, L, np.zeros((B, S, n), np.int32), np.zeros((B, S, n), np.int32),
                       np.zeros((B, S, n), np.int32), np.zeros((B, L, L), np.int32),
                       np.zeros((B, n), np.int32), np.zeros((B, n), np.int32),
                       np.full(B, supply, np.int32), name=f"located preset {preset}")
    scratch = _empty(1, S, n, "")
    for b in range(B):
        loc, lat = _location_instance(_rng(preset, first + b), S, n, cap_hi, scratch, 0)
        out.node_cap[b] = scratch.node_cap[0]
        out.node_cost[b] = scratch.node_cost[0]
        out.location[b] = loc
        out.latency[b] = lat
    return out


def random_located(B: int, S: int, n: int, L: int, seed: int, cap_hi: int = 4, cost_hi: int = 30,
                   supply_hi: int = 12) -> LocatedBatch:
    """Small random located instances: locations U[0, L-1], latencies
    U[0, cost_hi] (not symmetric), capacities U[0, cap_hi]."""
    out = LocatedBatch(S, n, L, np.zeros((B, S, n), np.int32), np.zeros((B, S, n), np.int32),
                       np.zeros((B, S, n), np.int32), np.zeros((B, L, L), np.int32),
                       np.zeros((B, n), np.int32), np.zeros((B, n), np.int32),
                       np.zeros(B, np.int32), name=f"random located S={S} n={n} L={L}")
    for b in range(B):
        rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(S, n, L, b)))
        out.node_cap[b] = _int_uniform(rng, 0, cap_hi, (S, n))
        out.node_cost[b] = _int_uniform(rng, 0, cost_hi, (S, n))
        out.location[b] = _int_uniform(rng, 0, L - 1, (S, n))
        out.latency[b] = _int_uniform(rng, 0, cost_hi, (L, L))
        out.src_cost[b] = _int_uniform(rng, 0, cost_hi, n)
        out.snk_cost[b] = _int_uniform(rng, 0, cost_hi, n)
        out.supply[b] = int(rng.integers(0, supply_hi + 1))
    return out
