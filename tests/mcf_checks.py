"""Independent checks for layered min-cost max-flow results.

None of these reuse the oracle's or the GPU library's arithmetic; each rests
on a separate mathematical fact:

* ``brute_force`` -- the original network is a DAG (stages are ordered), so
  every integral flow is a multiset of source-to-sink paths that visit one
  node per stage; enumerating all multisets that respect node capacities
  gives the maximum value and, at that value, the minimum cost of Eq. 2
  (paper Sec. V-A) directly from the definition.
* ``certify`` -- feasibility (capacity and conservation), the reported cost
  equals sum f * c, maximality (t unreachable from s0 in the residual graph,
  with the min-cut capacity equal to F, or F equal to the supply) and
  complementary slackness: no residual arc has negative reduced cost under
  the returned potentials, which proves minimum cost for the flow's value.
* ``closed_form_value`` -- with every inter-stage link present and of
  unbounded capacity, the maximum flow is min(supply, min over stages of the
  stage's total capacity) (the bottleneck stage of paper Sec. IV / V-B).
* ``assignment_cost`` -- with every capacity 1 and supply >= n each node
  carries exactly one unit, consecutive stages are joined by a permutation,
  and the optimum is the fixed node/source/sink cost plus one linear
  assignment per stage pair (scipy's linear_sum_assignment).
* ``single_stage_greedy`` -- with S = 1 each unit costs src + c + snk of its
  node, so filling the cheapest nodes first is optimal.
* ``transport_lp`` -- with S = 2 the problem is a transportation LP whose
  constraint matrix is totally unimodular; scipy's HiGHS solves it.
* ``networkx_mcmf`` -- networkx's max_flow_min_cost (network simplex).
"""
from __future__ import annotations

import numpy as np

NO_ARC = -1


def _inst(batch, b):
    S, n = batch.S, batch.n
    arc = batch.arc_cost[b] if S > 1 else np.zeros((0, n, n), np.int32)
    src = batch.src_cost[b] if batch.src_cost is not None else np.zeros(n, np.int32)
    snk = batch.snk_cost[b] if batch.snk_cost is not None else np.zeros(n, np.int32)
    return (batch.node_cap[b].astype(np.int64), batch.node_cost[b].astype(np.int64),
            arc.astype(np.int64), src.astype(np.int64), snk.astype(np.int64), int(batch.supply[b]))


def brute_force(batch, b, limit=3_000_000):
    """Exhaustive (F, cost) over all feasible path multisets of instance b."""
    S, n = batch.S, batch.n
    cap, ncost, arc, src, snk, supply = _inst(batch, b)
    paths, costs = [], []

    def rec(k, nodes, c):
        if k == S:
            paths.append(tuple(nodes))
            costs.append(c + snk[nodes[-1]])
            return
        for j in range(n):
            if cap[k, j] <= 0:
                continue
            if k == 0:
                rec(1, [j], src[j] + ncost[0, j])
            else:
                a = arc[k - 1, nodes[-1], j]
                if a == NO_ARC:
                    continue
                rec(k + 1, nodes + [j], c + a + ncost[k, j])

    rec(0, [], 0)
    order = np.argsort(costs, kind="stable")
    paths = [paths[i] for i in order]
    costs = [int(costs[i]) for i in order]
    best = {0: 0}
    used = np.zeros((S, n), np.int64)
    count = [0]

    def dfs(start, f, c):
        count[0] += 1
        if count[0] > limit:
            raise RuntimeError("brute force enumeration too large")
        if c < best.get(f, 1 << 62):
            best[f] = c
        if f == supply:
            return
        for p in range(start, len(paths)):
            nodes = paths[p]
            if all(used[k, nodes[k]] < cap[k, nodes[k]] for k in range(S)):
                for k in range(S):
                    used[k, nodes[k]] += 1
                dfs(p, f + 1, c + costs[p])
                for k in range(S):
                    used[k, nodes[k]] -= 1

    dfs(0, 0, 0)
    F = max(best)
    return F, best[F]


def closed_form_value(batch, b):
    """max flow = min(supply, min_k sum_i cap[k][i]) when all links exist."""
    cap = batch.node_cap[b].astype(np.int64)
    return int(min(int(batch.supply[b]), int(cap.sum(axis=1).min())))


def assignment_cost(batch, b):
    """Optimum for capacities all 1 and supply >= n (no missing links)."""
    from scipy.optimize import linear_sum_assignment

    S, n = batch.S, batch.n
    cap, ncost, arc, src, snk, supply = _inst(batch, b)
    assert (cap == 1).all() and supply >= n and (arc != NO_ARC).all()
    total = int(ncost.sum() + src.sum() + snk.sum())
    for k in range(S - 1):
        r, c = linear_sum_assignment(arc[k])
        total += int(arc[k][r, c].sum())
    return n, total


def single_stage_greedy(batch, b):
    """S = 1: fill the cheapest src + c + snk nodes first."""
    assert batch.S == 1
    cap, ncost, arc, src, snk, supply = _inst(batch, b)
    unit = src + ncost[0] + snk
    left, F, cost = supply, 0, 0
    for i in np.argsort(unit, kind="stable"):
        take = int(min(left, cap[0, i]))
        F += take
        cost += take * int(unit[i])
        left -= take
    return F, cost


def transport_lp(batch, b):
    """S = 2 transportation LP solved by HiGHS (integral by unimodularity)."""
    from scipy.optimize import linprog

    assert batch.S == 2
    n = batch.n
    cap, ncost, arc, src, snk, supply = _inst(batch, b)
    present = arc[0] != NO_ARC
    unit = (src + ncost[0])[:, None] + np.where(present, arc[0], 0) + (ncost[1] + snk)[None, :]
    idx = np.flatnonzero(present.ravel())
    m = idx.size
    if m == 0:
        return 0, 0
    rows, cols = np.divmod(idx, n)
    A = np.zeros((2 * n + 1, m))
    A[rows, np.arange(m)] = 1
    A[n + cols, np.arange(m)] = 1
    A[2 * n, :] = 1
    ub = np.concatenate([cap[0], cap[1], [supply]]).astype(float)
    r1 = linprog(-np.ones(m), A_ub=A, b_ub=ub, bounds=(0, None), method="highs")
    F = int(round(-r1.fun))
    r2 = linprog(unit.ravel()[idx].astype(float), A_ub=A, b_ub=ub, A_eq=np.ones((1, m)),
                 b_eq=[F], bounds=(0, None), method="highs")
    return F, int(round(r2.fun))


def networkx_mcmf(batch, b):
    """(F, cost) from networkx.max_flow_min_cost on the split-node network."""
    import networkx as nx

    S, n = batch.S, batch.n
    cap, ncost, arc, src, snk, supply = _inst(batch, b)
    G = nx.DiGraph()
    G.add_edge("s0", "s", capacity=supply, weight=0)
    for i in range(n):
        G.add_edge("s", ("in", 0, i), weight=int(src[i]))
        G.add_edge(("out", S - 1, i), "t", weight=int(snk[i]))
    for k in range(S):
        for i in range(n):
            G.add_edge(("in", k, i), ("out", k, i), capacity=int(cap[k, i]), weight=int(ncost[k, i]))
    for k in range(S - 1):
        for i in range(n):
            for j in range(n):
                if arc[k, i, j] != NO_ARC:
                    G.add_edge(("out", k, i), ("in", k + 1, j), weight=int(arc[k, i, j]))
    flow = nx.max_flow_min_cost(G, "s0", "t")
    F = sum(flow["s0"].values())
    return int(F), int(nx.cost_of_flow(G, flow))


def vertex_index(S, n):
    """Vertex numbering shared by the boundary's potential export."""
    k = np.arange(S)[:, None]
    i = np.arange(n)[None, :]
    return 3 + 2 * (k * n + i), 4 + 2 * (k * n + i)


def certify(batch, b, F, cost, node_flow, arc_flow, src_flow, snk_flow, potential):
    """Raise AssertionError unless the flow is feasible, maximum, of the
    reported cost and certified min-cost by the potentials."""
    S, n = batch.S, batch.n
    cap, ncost, arc, src, snk, supply = _inst(batch, b)
    nf = np.asarray(node_flow, np.int64)
    af = np.asarray(arc_flow, np.int64).reshape(max(S - 1, 0), n, n)
    sf = np.asarray(src_flow, np.int64)
    tf = np.asarray(snk_flow, np.int64)
    pi = np.asarray(potential, np.int64)
    present = arc != NO_ARC
    # feasibility
    assert (nf >= 0).all() and (nf <= cap).all(), "node flow outside [0, cap]"
    assert (af >= 0).all() and (af[~present] == 0).all(), "bad inter-stage flow"
    assert (sf >= 0).all() and (tf >= 0).all(), "negative source/sink flow"
    assert int(sf.sum()) == F == int(tf.sum()), "flow value mismatch"
    assert F <= supply, "flow above supply"
    assert (sf == nf[0]).all(), "conservation at stage-0 inputs"
    assert (tf == nf[S - 1]).all(), "conservation at last-stage outputs"
    for k in range(S - 1):
        assert (af[k].sum(axis=1) == nf[k]).all(), f"conservation at out of stage {k}"
        assert (af[k].sum(axis=0) == nf[k + 1]).all(), f"conservation at in of stage {k + 1}"
    c = int((src * sf).sum() + (ncost * nf).sum() + (np.where(present, arc, 0) * af).sum()
            + (snk * tf).sum())
    assert c == cost, f"cost {cost} != sum f*c {c}"
    # complementary slackness: reduced cost >= 0 on every residual arc
    vin, vout = vertex_index(S, n)
    p_s0, p_s, p_t = pi[0], pi[1], pi[2]
    p_in, p_out = pi[vin], pi[vout]

    def rc_ok(mask, rc, what):
        bad = mask & (rc < 0)
        assert not bad.any(), f"negative reduced cost on residual {what}"

    rc_ok(np.array(F < supply), np.array(p_s0 - p_s), "s0->s")
    rc_ok(np.array(F > 0), np.array(p_s - p_s0), "s->s0")
    rc_ok(np.ones(n, bool), src + p_s - p_in[0], "s->in0")
    rc_ok(sf > 0, -src + p_in[0] - p_s, "in0->s")
    rc_ok(nf < cap, ncost + p_in - p_out, "split")
    rc_ok(nf > 0, -ncost + p_out - p_in, "reverse split")
    rc_ok(np.ones(n, bool), snk + p_out[S - 1] - p_t, "out->t")
    rc_ok(tf > 0, -snk + p_t - p_out[S - 1], "t->out")
    for k in range(S - 1):
        red = arc[k] + p_out[k][:, None] - p_in[k + 1][None, :]
        rc_ok(present[k], red, f"inter-stage {k}")
        rc_ok(af[k] > 0, -red, f"reverse inter-stage {k}")
    # maximality: F == supply, or t unreachable in the residual graph with
    # the cut's capacity equal to F.
    if F < supply:
        reach_in = np.zeros((S, n), bool)
        reach_out = np.zeros((S, n), bool)
        reach_in[0] = True                       # s -> in0 has unbounded capacity
        reach_s = True
        changed = True
        while changed:
            changed = False
            new_out = reach_out | (reach_in & (nf < cap))
            new_in = reach_in | (reach_out & (nf > 0))
            for k in range(S - 1):
                new_in[k + 1] |= (new_out[k][:, None] & present[k]).any(axis=0)
                new_out[k] |= (new_in[k + 1][None, :] & (af[k] > 0)).any(axis=1)
            if (new_out != reach_out).any() or (new_in != reach_in).any():
                reach_out, reach_in, changed = new_out, new_in, True
        assert reach_s
        assert not reach_out[S - 1].any(), "augmenting path left (t reachable)"
        cut = int(cap[reach_in & ~reach_out].sum())
        assert cut == F, f"min cut {cut} != F {F}"
    return True


def networkx_with_candidates(base, slot, cands, stages):
    """(F, cost) of one what-if placement, built without slots: each stage
    holds the base nodes, except that a stage receiving candidate c holds c
    in place of the base node at ``slot``; links are looked up by the kind of
    their two ends (base-base, base-candidate, candidate-base,
    candidate-candidate).  networkx's max_flow_min_cost solves it."""
    import networkx as nx

    S, n = base.S, base.n
    cap, ncost, arc, src, snk, supply = _inst(base, 0)
    who = {k: c for c, k in enumerate(stages)}
    nodes = []
    for k in range(S):
        row = [("base", i) for i in range(n) if not (i == slot and k in who)]
        if k in who:
            row.append(("cand", who[k]))
        nodes.append(row)

    def node_cap(k, u):
        return int(cands.cap[u[1]][k]) if u[0] == "cand" else int(cap[k, u[1]])

    def node_cost(k, u):
        return int(cands.cost[u[1]][k]) if u[0] == "cand" else int(ncost[k, u[1]])

    def link(k, u, v):
        if u[0] == "base" and v[0] == "base":
            return int(arc[k, u[1], v[1]])
        if u[0] == "base":
            return int(cands.inn[v[1]][k + 1][u[1]])
        if v[0] == "base":
            return int(cands.out[u[1]][k][v[1]])
        return int(cands.link[u[1]][v[1]])

    G = nx.DiGraph()
    G.add_edge("s0", "s", capacity=supply, weight=0)
    for u in nodes[0]:
        G.add_edge("s", ("in", 0, u), weight=int(cands.src[u[1]]) if u[0] == "cand" else int(src[u[1]]))
    for u in nodes[S - 1]:
        G.add_edge(("out", S - 1, u), "t", weight=int(cands.snk[u[1]]) if u[0] == "cand" else int(snk[u[1]]))
    for k in range(S):
        for u in nodes[k]:
            G.add_edge(("in", k, u), ("out", k, u), capacity=node_cap(k, u), weight=node_cost(k, u))
    for k in range(S - 1):
        for u in nodes[k]:
            for v in nodes[k + 1]:
                d = link(k, u, v)
                if d != NO_ARC:
                    G.add_edge(("out", k, u), ("in", k + 1, v), weight=d)
    if "t" not in G:
        return 0, 0
    flow = nx.max_flow_min_cost(G, "s0", "t")
    return int(sum(flow["s0"].values())), int(nx.cost_of_flow(G, flow))


def networkx_located_hubs(lb, b):
    """(F, cost) of located instance b on a network with one hub vertex per
    stage boundary and location: exit (k, i) -> hub (k, location of i) at
    cost 0, hub (k, a) -> entry (k+1, j) at latency[a][location of j].  Every
    link is uncapacitated, so a path exit -> hub -> entry costs exactly the
    direct link and the optimum equals the direct network's."""
    import networkx as nx

    S, n = lb.S, lb.n
    cap, ncost = lb.node_cap[b].astype(int), lb.node_cost[b].astype(int)
    loc, lat = lb.location[b], lb.latency[b]
    G = nx.DiGraph()
    G.add_edge("s0", "s", capacity=int(lb.supply[b]), weight=0)
    for i in range(n):
        G.add_edge("s", ("in", 0, i), weight=int(lb.src_cost[b][i]))
        G.add_edge(("out", S - 1, i), "t", weight=int(lb.snk_cost[b][i]))
    for k in range(S):
        for i in range(n):
            G.add_edge(("in", k, i), ("out", k, i), capacity=int(cap[k, i]), weight=int(ncost[k, i]))
    for k in range(S - 1):
        for i in range(n):
            G.add_edge(("out", k, i), ("hub", k, int(loc[k, i])), weight=0)
        for a in set(int(x) for x in loc[k]):
            for j in range(n):
                G.add_edge(("hub", k, a), ("in", k + 1, j), weight=int(lat[a, loc[k + 1, j]]))
    flow = nx.max_flow_min_cost(G, "s0", "t")
    return int(sum(flow["s0"].values())), int(nx.cost_of_flow(G, flow))
