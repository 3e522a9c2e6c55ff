"""CPU oracle for location-factored instances (link delays given as
latencies between node locations; the paper's testbed of Sec. VI places
every node at one of ten geographic locations, and Eq. 1's link term is the
latency between the two nodes).

TEST INFRASTRUCTURE ONLY: the tests, the package smoke check and the
benchmark's CPU-baseline leg are the only callers.  Nothing here is shared
with the GPU library.

A located instance stands for the ordinary layered instance whose link from
node i of stage k to node j of stage k+1 has delay
latency[location[k][i]][location[k+1][j]].  ``to_dense`` writes that
instance out element by element; ``solve`` hands it to the oracle's solver,
so the optimum is Eq. 2's (Sec. V-A) by definition.  With S > 1 an
out-of-range location or a negative latency makes the instance invalid
(status 1); with one stage there are no links and neither is read.

parity: pinned by a network with one hub vertex per (stage boundary,
location) built and solved by networkx (equal optima because every link is
uncapacitated), by brute force on tiny instances, and by the generator's own
dense presets.
"""
from __future__ import annotations

from types import SimpleNamespace

import numpy as np

from . import solve as _solve


def to_dense(lb):
    """The located batch as an ordinary batch (int32 arrays)."""
    B, S, n, L = lb.B, int(lb.S), int(lb.n), int(lb.L)
    arc = np.zeros((B, max(S - 1, 0), n, n), np.int32)
    bad = np.zeros(B, bool)
    for b in range(B):
        loc, lat = lb.location[b], lb.latency[b]
        # with one stage there are no links, and neither array is read
        bad[b] = S > 1 and bool((loc < 0).any() or (loc >= L).any() or (lat < 0).any())
        if bad[b]:
            continue
        for k in range(S - 1):
            for i in range(n):  # row i: the latencies from i's location to each j's
                arc[b, k, i, :] = lat[loc[k, i], loc[k + 1, :]]
    return SimpleNamespace(S=S, n=n, node_cap=lb.node_cap, node_cost=lb.node_cost, arc_cost=arc,
                           src_cost=lb.src_cost, snk_cost=lb.snk_cost, supply=lb.supply), bad


def solve(lb, nthreads: int | None = None, flows: bool = True, potentials: bool = True) -> dict:
    """Optimum of every located instance; invalid ones report status 1 and
    F = cost = 0."""
    dense, bad = to_dense(lb)
    r = _solve(dense, nthreads=nthreads, flows=flows, potentials=potentials)
    r["status"][bad] = 1
    r["F"][bad] = 0
    r["cost"][bad] = 0
    return r
