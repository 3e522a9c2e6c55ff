"""Pins for the what-if placement oracle (paper Sec. VI, handling joining
nodes): each check rests on something other than the oracle's own
expansion -- the paper's join example, a network built without slots and
solved by networkx, brute force over path multisets, and invariants."""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import oracle.whatif as OW
from paper_2509_21221_amd import workloads as W
import mcf_checks as C

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _single(batch, b=0):
    return batch.subset([b])


def _uniform_candidates(m, S, n, cap, cost):
    full = lambda shape, v: np.full(shape, v, np.int32)
    return W.Candidates(full((m, S), cap), full((m, S), cost), full((m, S, n), cost),
                        full((m, S, n), cost), full((m, m), cost), full(m, cost), full(m, cost))


def test_paper_join_example():
    d = json.load(open(os.path.join(GOLDEN, "whatif_paper_join.json")))
    S, n = d["S"], d["n"]
    base = W.Batch(S, n, np.asarray([d["node_cap"]], np.int32), np.asarray([d["node_cost"]], np.int32),
                   np.full((1, S - 1, n, n), d["arc_cost"], np.int32), np.full((1, n), d["src_cost"], np.int32),
                   np.full((1, n), d["snk_cost"], np.int32), np.asarray([d["supply"]], np.int32))
    cand = _uniform_candidates(1, S, n, d["candidate"]["cap"], d["candidate"]["cost"])
    for rnd in d["rounds"]:
        r = OW.whatif(base, rnd["slot"], cand)
        assert r["F"].tolist() == rnd["expect_F"]
        assert r["best"][0] == rnd["expect_best"]
        assert r["best_stages"] == (rnd["expect_best"],)
        nxt = OW.expand(base, rnd["slot"], cand, first=r["best"][0], count=1)
        base = W.Batch(S, n, nxt.node_cap, nxt.node_cost, nxt.arc_cost, nxt.src_cost, nxt.snk_cost,
                       nxt.supply)


@pytest.mark.parametrize("S,m", [(1, 0), (1, 1), (3, 0), (3, 1), (3, 3), (4, 2), (5, 5), (6, 3)])
def test_placement_enumeration(S, m):
    p = OW.placements(S, m)
    assert len(p) == OW.placement_count(S, m) == math.factorial(S) // math.factorial(S - m)
    assert len(set(p)) == len(p)
    assert all(len(set(t)) == m and all(0 <= k < S for k in t) for t in p)
    assert p == sorted(p)


@pytest.mark.parametrize("S,n,m,slot,occupied,holes", [
    (1, 2, 1, 1, False, 0.0), (2, 2, 1, 0, False, 0.0), (2, 3, 2, 2, True, 0.2),
    (3, 3, 2, 1, False, 0.0), (3, 3, 3, 0, True, 0.3), (3, 2, 1, 1, True, 0.0),
    (4, 2, 2, 1, False, 0.2),
])
def test_expansion_against_networkx(S, n, m, slot, occupied, holes):
    """Every placement's optimum equals that of a network built from the
    candidates directly (no slot arrays), solved by networkx."""
    for seed in range(3):
        base = W.random_small(1, S, n, seed=40 + seed, supply_hi=8, holes=holes)
        if not occupied:
            base.node_cap[0][:, slot] = 0
        cands = W.random_candidates(S, n, m, seed=seed, holes=holes)
        r = OW.whatif(base, slot, cands)
        for p, stages in enumerate(OW.placements(S, m)):
            assert r["status"][p] == 0
            assert (int(r["F"][p]), int(r["cost"][p])) == C.networkx_with_candidates(base, slot, cands, stages)


@pytest.mark.parametrize("S,n,m", [(2, 2, 2), (3, 2, 2), (2, 3, 1)])
def test_best_against_brute_force(S, n, m):
    """The best placement's (F, cost) from exhaustive path enumeration of
    every expanded instance."""
    for seed in range(3):
        base = W.random_small(1, S, n, seed=70 + seed, supply_hi=5)
        base.node_cap[0][:, n - 1] = 0
        cands = W.random_candidates(S, n, m, seed=seed + 5, cap_hi=2)
        r = OW.whatif(base, n - 1, cands)
        batch = OW.expand(base, n - 1, cands)
        brute = [C.brute_force(batch, p) for p in range(r["count"])]
        assert [tuple(map(int, x)) for x in zip(r["F"], r["cost"])] == brute
        key = min(range(len(brute)), key=lambda p: (-brute[p][0], brute[p][1], p))
        assert r["best"] == (key, *brute[key])


def test_zero_capacity_candidates_change_nothing():
    base = W.random_small(1, 3, 3, seed=3, supply_hi=8)
    base.node_cap[0][:, 2] = 0
    cands = W.random_candidates(3, 3, 3, seed=9)
    cands.cap[:] = 0
    r0 = oracle.solve(base, flows=False, potentials=False)
    r = OW.whatif(base, 2, cands)
    assert (r["F"] == r0["F"][0]).all() and (r["cost"] == r0["cost"][0]).all()


def test_binding_supply_never_raises_cost():
    """With the supply met before the join, any placement keeps F and can only
    lower the cost (the old flow stays feasible)."""
    base = W.random_small(1, 4, 4, seed=5, cap_hi=5, supply_hi=3)
    base.node_cap[0][:, 3] = 0
    r0 = oracle.solve(base, flows=False, potentials=False)
    assert r0["F"][0] == base.supply[0]
    cands = W.random_candidates(4, 4, 4, seed=2)
    r = OW.whatif(base, 3, cands)
    assert (r["F"] == r0["F"][0]).all() and (r["cost"] <= r0["cost"][0]).all()


def test_candidate_order_does_not_change_the_optimum():
    base = W.random_small(1, 4, 3, seed=8, supply_hi=8)
    base.node_cap[0][:, 0] = 0
    cands = W.random_candidates(4, 3, 3, seed=4)
    order = [2, 0, 1]
    r = OW.whatif(base, 0, cands)
    q = OW.whatif(base, 0, cands.permuted(order))
    assert r["best"][1:] == q["best"][1:]
    # placement of the permuted list: candidate j of it is candidate order[j]
    by_map = {tuple(s): (int(f), int(c)) for s, f, c in zip(OW.placements(4, 3), r["F"], r["cost"])}
    for s, f, c in zip(OW.placements(4, 3), q["F"], q["cost"]):
        orig = [0] * 3
        for j, k in enumerate(s):
            orig[order[j]] = k
        assert by_map[tuple(orig)] == (int(f), int(c))


def test_best_rule_against_lexsort():
    rng = np.random.default_rng(1)
    for trial in range(50):
        N = int(rng.integers(1, 40))
        F = rng.integers(0, 4, N)
        cost = rng.integers(0, 5, N)
        status = np.where(rng.random(N) < 0.2, rng.integers(1, 3, N), 0)
        ok = np.flatnonzero(status == 0)
        got = OW.best(F, cost, status)
        if len(ok) == 0:
            assert got == (-1, 0, 0)
            continue
        order = np.lexsort((ok, cost[ok], -F[ok]))
        i = int(ok[order[0]])
        assert got == (i, int(F[i]), int(cost[i]))


def test_node_addition_setting_shapes():
    for setting in (1, 2, 3, 4):
        base, slot, c = W.node_addition(setting)
        S = base.S
        assert base.n == 96 // S + 1 and slot == base.n - 1 and c.m == S
        assert (base.node_cap[0][:, slot] == 0).all()
        assert OW.placement_count(S, c.m) == math.factorial(S)
        base.check_layout()


# Each pin must be able to fail: plant one plausible mistake at a time in a
# private in-memory copy of the expansion oracle (never in the oracle itself)
# and check that the pins reject it.
WHATIF_MUTANTS = {
    "links_in_from_out": ("arc[k - 1, i, slot] = cands.inn[c][k][i]", "arc[k - 1, i, slot] = cands.out[c][k][i]"),
    "candidate_link_transposed": ("cands.link[at_stage[k]][at_stage[k + 1]]",
                                  "cands.link[at_stage[k + 1]][at_stage[k]]"),
    "no_candidate_link": ("arc[k, slot, slot] = cands.link", "arc[k, slot, slot] = 0 * cands.link"),
    "sink_delay_from_source": ("snk[slot] = csnk[c]", "snk[slot] = csrc[c]"),
    "source_delay_dropped": ("src[slot] = csrc[c]", "src[slot] = 0"),
    "stage_cost_index": ("cost[k, slot] = cands.cost[c][k]", "cost[k, slot] = cands.cost[c][0]"),
    "ties_to_last": ("(f == bF and c < bc)", "(f == bF and c <= bc)"),
    "cost_before_value": ("f > bF or (f == bF and c < bc)", "c < bc or (c == bc and f > bF)"),
}


def _variant(text, name):
    import types

    mod = types.ModuleType(f"oracle.{name}")
    mod.__package__ = "oracle"
    exec(compile(text, f"<whatif variant {name}>", "exec"), mod.__dict__)
    return mod


def _whatif_pins_pass(ow):
    try:
        for S, n, m, slot, holes, seed in [(3, 3, 2, 1, 0.0, 0), (3, 3, 3, 0, 0.3, 1), (2, 2, 1, 0, 0.0, 2),
                                           (4, 2, 2, 1, 0.2, 3)]:
            base = W.random_small(1, S, n, seed=40 + seed, supply_hi=8, holes=holes)
            base.node_cap[0][:, slot] = 0
            cands = W.random_candidates(S, n, m, seed=seed, holes=holes)
            r = ow.whatif(base, slot, cands)
            for p, stages in enumerate(ow.placements(S, m)):
                if (int(r["F"][p]), int(r["cost"][p])) != C.networkx_with_candidates(base, slot, cands, stages):
                    return False
        rng = np.random.default_rng(1)
        for _ in range(50):
            N = int(rng.integers(1, 40))
            F, cost = rng.integers(0, 4, N), rng.integers(0, 5, N)
            status = np.where(rng.random(N) < 0.2, 1, 0)
            ok = np.flatnonzero(status == 0)
            if len(ok) and ow.best(F, cost, status)[0] != int(ok[np.lexsort((ok, cost[ok], -F[ok]))[0]]):
                return False
    except AssertionError:
        return False
    return True


def test_unmutated_whatif_copy_passes():
    assert _whatif_pins_pass(_variant(open(OW.__file__).read(), "same"))


@pytest.mark.parametrize("name", sorted(WHATIF_MUTANTS))
def test_whatif_pins_reject_mutant(name):
    before, after = WHATIF_MUTANTS[name]
    text = open(OW.__file__).read()
    assert text.count(before) == 1, f"mutation anchor for {name} not unique"
    assert not _whatif_pins_pass(_variant(text.replace(before, after), name))
