"""CPU oracle for what-if node addition (paper Sec. VI, handling joining
nodes; the example of Sec. V-B).

TEST INFRASTRUCTURE ONLY: the tests, the package smoke check and the
benchmark's CPU-baseline leg are the only callers.  Nothing here is shared
with the GPU library.

The paper picks where joining nodes go by solving the flow problem once for
every way of assigning the candidate nodes to stages and keeping the best
assignment.  Written out:

* A base instance (one instance in the canonical layout) reserves one node
  position ``slot`` in every stage for a joining node.
* m candidates (0 <= m <= S).  Candidate c, if it joins stage k, has memory
  capacity ``cap[c][k]`` and compute cost ``cost[c][k]``; it receives from
  node i of stage k-1 over a link of delay ``inn[c][k][i]`` and sends to node
  j of stage k+1 over ``out[c][k][j]``; a link from candidate c in stage k to
  candidate d in stage k+1 has delay ``link[c][d]``; in stage 0 the data node
  reaches it with delay ``src[c]``, and from stage S-1 it returns to the data
  node with delay ``snk[c]`` (the paper lets every joining node know its
  costs for every stage).
* A placement sends every candidate to a different stage.  Placements are
  numbered in lexicographic order of (stage of candidate 0, stage of
  candidate 1, ...): there are S! / (S-m)! of them.
* Placement p turns the base instance into one instance of the same shape:
  in each stage that receives a candidate, the slot takes the candidate's
  capacity, compute cost, incoming and outgoing links (and data-node links
  at the two ends); stages without a candidate keep the base's slot as it
  is (an empty slot has capacity 0).  Where candidates sit in two
  consecutive stages, the link between the two slots is the candidates'
  own link.  Everything else is copied from the base.
* Each placement is solved for the optimum of Eq. 2 (Sec. V-A) with the
  oracle's solver.  The best placement has the largest flow value, then the
  smallest cost, then the smallest index; only instances solved with status
  OK take part.  The paper reports the gain (cost_now - cost_after) /
  cost_now; with a binding supply the value is fixed and the rule is the
  minimum cost.

parity: pinned by the paper's join example, by an independent network
construction with the candidates as extra nodes (networkx), by brute force on
tiny instances, and by invariants (zero-capacity candidates change nothing;
with a binding supply no placement raises the cost).
"""
from __future__ import annotations

import itertools
import math
from types import SimpleNamespace

import numpy as np

from . import solve


def placement_count(S: int, m: int) -> int:
    """Number of injective candidate-to-stage maps: S! / (S - m)!."""
    return math.perm(S, m)


def placements(S: int, m: int):
    """All placements as tuples (stage of candidate 0, ..., of candidate
    m-1), in lexicographic order (itertools.permutations emits them in
    that order)."""
    return list(itertools.permutations(range(S), m))


def _arr(a, shape):
    return np.zeros(shape, np.int64) if a is None else np.asarray(a, np.int64)


def expand_one(base, slot: int, cands, stages) -> dict:
    """The instance of placement ``stages`` (a tuple of the stage of each
    candidate) as int64 arrays of one instance."""
    S, n = int(base.S), int(base.n)
    m = len(stages)
    cap = np.asarray(base.node_cap, np.int64).reshape(S, n).copy()
    cost = np.asarray(base.node_cost, np.int64).reshape(S, n).copy()
    arc = (np.asarray(base.arc_cost, np.int64).reshape(S - 1, n, n).copy() if S > 1
           else np.zeros((0, n, n), np.int64))
    src = _arr(base.src_cost, (n,)).reshape(n).copy()
    snk = _arr(base.snk_cost, (n,)).reshape(n).copy()
    csrc = _arr(getattr(cands, "src", None), (m,))
    csnk = _arr(getattr(cands, "snk", None), (m,))
    at_stage = [-1] * S
    for c, k in enumerate(stages):
        at_stage[k] = c
    for k in range(S):
        c = at_stage[k]
        if c < 0:
            continue
        cap[k, slot] = cands.cap[c][k]
        cost[k, slot] = cands.cost[c][k]
        if k > 0:
            for i in range(n):
                arc[k - 1, i, slot] = cands.inn[c][k][i]
        if k < S - 1:
            for j in range(n):
                arc[k, slot, j] = cands.out[c][k][j]
        if k == 0:
            src[slot] = csrc[c]
        if k == S - 1:
            snk[slot] = csnk[c]
    for k in range(S - 1):
        if at_stage[k] >= 0 and at_stage[k + 1] >= 0:
            arc[k, slot, slot] = cands.link[at_stage[k]][at_stage[k + 1]]
    return {"node_cap": cap, "node_cost": cost, "arc_cost": arc, "src_cost": src,
            "snk_cost": snk, "supply": int(np.asarray(base.supply).reshape(-1)[0])}


def expand(base, slot: int, cands, first: int = 0, count: int | None = None):
    """Placements [first, first + count) as a batch (int32 arrays in the
    canonical layout) that ``oracle.solve`` accepts."""
    S, n = int(base.S), int(base.n)
    count = placement_count(S, int(cands.m)) - first if count is None else count
    chosen = itertools.islice(itertools.permutations(range(S), int(cands.m)), first, first + count)
    rows = [expand_one(base, slot, cands, stages) for stages in chosen]
    assert len(rows) == count, "placement range outside [0, S!/(S-m)!)"
    stack = lambda key, shape: np.ascontiguousarray(
        np.array([r[key] for r in rows], np.int64).reshape((count,) + shape).astype(np.int32))
    return SimpleNamespace(
        S=S, n=n, node_cap=stack("node_cap", (S, n)), node_cost=stack("node_cost", (S, n)),
        arc_cost=stack("arc_cost", (max(S - 1, 0), n, n)), src_cost=stack("src_cost", (n,)),
        snk_cost=stack("snk_cost", (n,)),
        supply=np.array([r["supply"] for r in rows], np.int32).reshape(count))


def best(F, cost, status):
    """(index, F, cost) of the best OK instance: largest F, then smallest
    cost, then smallest index; (-1, 0, 0) when no instance is OK."""
    bi, bF, bc = -1, 0, 0
    for i in range(len(F)):
        if int(status[i]) != 0:
            continue
        f, c = int(F[i]), int(cost[i])
        if bi < 0 or f > bF or (f == bF and c < bc):
            bi, bF, bc = i, f, c
    return bi, bF, bc


def whatif(base, slot: int, cands, nthreads: int | None = None) -> dict:
    """Solve every placement; returns the per-placement F, cost, status and
    the best placement with its stages."""
    batch = expand(base, slot, cands)
    r = solve(batch, nthreads=nthreads, flows=False, potentials=False)
    bi, bF, bc = best(r["F"], r["cost"], r["status"])
    allp = placements(int(base.S), int(cands.m))
    return {"F": r["F"], "cost": r["cost"], "status": r["status"], "best": (bi, bF, bc),
            "best_stages": allp[bi] if bi >= 0 else None, "count": len(allp)}
