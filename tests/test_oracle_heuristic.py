"""Pins of the decentralized-heuristic oracle (oracle/gwtf_heuristic.c).

The simulator has no closed form to compare against, so each part is pinned
by something outside it:

* the generator against numpy's independent Philox4x64-10;
* the paper's worked examples (Sec. V-C): the Request Change example (1 -> 2
  at 3 and 3 -> 4 at 8 become 1 -> 4 and 3 -> 2 at 6 each: taken under the
  max objective, 8 -> 6; under the sum objective 11 -> 12 it is taken exactly
  when the drawn U is below exp(-1 / 1.7)), and the Request Redirect example
  (1 -> 2 -> 3 at 11 moves to 1 -> 4 -> 3 at 9 in the first round in which
  node 4 proposes, which the shuffle's draws predict);
* the Request Flow rule (argmin of cost to the sink plus link cost) on a
  fixture where the nearest next hop is not the cheapest path;
* the annealing schedule (T = T0 * alpha^accepted moves, Sec. VI setup);
* invariants on random instances: the routed flow is feasible and conserved,
  its cost equals the sum over its links and nodes, F never exceeds the
  optimum and the cost never undercuts the exact minimum cost of the same
  flow value (the exact oracle run with supply = F);
* planted mistakes in a private copy of the C source, each rejected.
"""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from oracle import heuristic as H
from paper_2509_21221_amd import workloads as W

T0, ALPHA = 1.7, 0.95
MASK = 2**64 - 1


def numpy_philox(counter, key):
    """philox4x64-10(counter, key) from numpy's implementation, which
    increments the 256-bit counter before its first block."""
    c = sum(int(w) << (64 * q) for q, w in enumerate(counter))
    c = (c - 1) % (1 << 256)
    start = np.array([(c >> (64 * q)) & MASK for q in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.array([int(k) for k in key], dtype=np.uint64), counter=start)
    return [int(x) for x in bg.random_raw(4)]


def u_of(word):
    return (word >> 11) * 2.0**-53


def bounded(word, m):
    return ((word >> 32) * m) >> 32


def stage_perm(seed, instance, rnd, stage, n):
    perm = list(range(n))
    words, used, block = [], 4, 0
    for j in range(n - 1, 0, -1):
        if used == 4:
            words = numpy_philox([rnd, stage, 0, block], [seed, instance])
            block += 1
            used = 0
        r = bounded(words[used], j + 1)
        used += 1
        perm[j], perm[r] = perm[r], perm[j]
    return perm


def batch_of(S, n, cap, cost, arc, src, snk, supply):
    B = len(supply)
    i32 = lambda a, shape: np.ascontiguousarray(np.asarray(a, dtype=np.int32).reshape(shape))
    return W.Batch(S, n, i32(cap, (B, S, n)), i32(cost, (B, S, n)), i32(arc, (B, max(S - 1, 0), n, n)),
                   i32(src, (B, n)), i32(snk, (B, n)), i32(supply, (B,)))


def repeat(batch, B):
    return batch.subset([0] * B)


# ---------------------------------------------------------------- generator

@pytest.mark.parametrize("counter,key", [
    ([0, 0, 0, 0], [0, 0]),
    ([5, 7, 9, 11], [123, 456]),
    ([MASK, MASK, MASK, MASK], [MASK, MASK]),
    ([119, 9, 1, 3], [2509, 16383]),
    ([0, 3, 0, 0], [7, 1]),
])
def test_philox_matches_numpy(counter, key, lib=None):
    assert H.philox4x64_10(counter, key, lib=lib) == numpy_philox(counter, key)


# ---------------------------------------------------------------- paper examples

def change_example(B=1):
    """Sec. V-C Request Change: node 1 -> node 2 at 3, node 3 -> node 4 at 8;
    1 -> 4 and 3 -> 2 would cost 6 each.  Stage 0 = (node 1, node 3),
    stage 1 = (node 2, node 4); every capacity 1, so no redirect is possible."""
    arc = [[[3, 6], [6, 8]]]
    b = batch_of(2, 2, [[1, 1], [1, 1]], [[0, 0], [0, 0]], arc, [0, 0], [0, 0], [2])
    paths = np.array([[[0, 0], [1, 1]]], np.int32)  # 1 -> 2 and 3 -> 4
    return repeat(b, B), np.repeat(paths, B, axis=0)


def test_request_change_example_max_objective(lib=None):
    """Under the max objective the switch lowers the largest link from 8 to
    6, so it is always taken in the first round, and it cools the proposer."""
    b, paths = change_example(B=64)
    r = H.simulate(b, rounds=1, objective="max", paths=paths, seed=3, lib=lib)
    assert (r["status"] == 0).all()
    assert (r["arc_flow"][:, 0] == np.array([[0, 1], [1, 0]])).all()
    assert (r["cost"] == 12).all() and (r["F"] == 2).all()
    assert (r["accepted"][:, 0].sum(axis=1) == 1).all()
    assert np.allclose(np.sort(r["temperature"][:, 0], axis=1), [[T0 * ALPHA, T0]])


def test_request_change_example_sum_objective(lib=None):
    """Under the sum objective the switch raises 11 to 12: it is taken exactly
    when the pair's U draw is below exp(-1 / T0)."""
    b, paths = change_example(B=256)
    for seed in (0, 77):
        r = H.simulate(b, rounds=1, objective="sum", paths=paths, seed=seed, lib=lib)
        expect = np.array([u_of(numpy_philox([0, 0, 1, 0], [seed, inst])[3]) < math.exp(-1.0 / T0)
                           for inst in range(b.B)])
        taken = r["cost"] == 12
        assert (taken == expect).all()
        assert ((r["cost"] == 11) | taken).all()
        assert 0.45 < taken.mean() < 0.66  # exp(-1/1.7) = 0.555


def redirect_example():
    """Sec. V-C Request Redirect: 1 -> 2 -> 3 costs 11 (5 + 6), 1 -> 4 -> 3
    costs 9 (4 + 5).  Stage 0 = (node 1, empty), stage 1 = (node 2, node 4),
    stage 2 = (node 3, empty); node 4 is idle with capacity 1."""
    arc = [[[5, 4], [-1, -1]], [[6, -1], [5, -1]]]
    b = batch_of(3, 2, [[1, 0], [1, 1], [1, 0]], [[0, 0]] * 3, arc, [0, 0], [0, 0], [1])
    return b, np.array([[[0, 0, 0]]], np.int32)


def test_request_redirect_example(lib=None):
    b, paths = redirect_example()
    for seed in range(6):
        # node 4 (index 1 of stage 1) proposes in the first round whose
        # shuffle puts it first; before that nothing can move
        first = next(r for r in range(64) if stage_perm(seed, 0, r, 1, 2)[0] == 1)
        before = H.simulate(b, rounds=first, objective="sum", paths=paths, seed=seed, lib=lib)
        after = H.simulate(b, rounds=first + 1, objective="sum", paths=paths, seed=seed, lib=lib)
        assert before["cost"][0] == 11 and before["node_flow"][0, 1].tolist() == [1, 0]
        assert after["cost"][0] == 9 and after["node_flow"][0, 1].tolist() == [0, 1]
        assert after["accepted"][0, 1].tolist() == [0, 1]
        assert after["temperature"][0, 1, 1] == T0 * ALPHA
        assert after["used"][0, 1].tolist() == [0, 1]


def test_request_flow_argmin_of_cost_to_sink_plus_link(lib=None):
    """Relay a (stage 0) sees b at link 1 whose cost to the sink is 10 (its
    compute cost) and c at link 5 whose cost to the sink is 2: it must take
    c (7 < 11), not the nearest next hop."""
    arc = [[[1, 5], [-1, -1]]]
    b = batch_of(2, 2, [[1, 0], [1, 1]], [[3, 0], [10, 2]], arc, [4, 0], [0, 0], [2])
    r = H.simulate(b, rounds=3, lib=lib)
    assert r["F"][0] == 1
    assert r["arc_flow"][0, 0].tolist() == [[0, 1], [0, 0]]
    assert r["cost"][0] == 4 + 3 + 5 + 2 + 0
    assert r["used"][0, 1].tolist() == [1, 1]  # b keeps an unpaired outflow to the sink


# ---------------------------------------------------------------- invariants

def check_invariants(batch, r, exact=None):
    S, n = batch.S, batch.n
    ok = r["status"] == 0
    nf, af = r["node_flow"], r["arc_flow"]
    assert (nf <= batch.node_cap).all() and (nf >= 0).all()
    assert (r["used"] >= nf).all() and (r["used"] <= np.maximum(batch.node_cap, 0)).all()
    if S > 1:
        assert (af[batch.arc_cost < 0] == 0).all()
        assert (af.sum(axis=3) == nf[:, :-1]).all()       # out of stage k
        assert (af.sum(axis=2) == nf[:, 1:]).all()        # into stage k + 1
    assert (nf.sum(axis=2) == r["F"][:, None]).all()
    cost = (nf * batch.node_cost).sum(axis=(1, 2)) + (nf[:, 0] * batch.src_cost).sum(axis=1) \
        + (nf[:, -1] * batch.snk_cost).sum(axis=1)
    if S > 1:
        cost = cost + (af * np.maximum(batch.arc_cost, 0)).sum(axis=(1, 2, 3))
    assert (r["cost"][ok] == cost[ok]).all()
    assert (r["counters"][:, 0] == r["F"]).all()
    assert (r["counters"][:, 2] == r["accepted"].sum(axis=(1, 2))).all()
    assert (r["counters"][:, 3] == (r["used"] - nf).sum(axis=(1, 2))).all()
    # T0 cooled once per accepted move, by repeated multiplication
    acc = r["accepted"].copy()
    t = np.full(acc.shape, T0)
    for _ in range(int(acc.max(initial=0))):
        t = np.where(acc > 0, t * ALPHA, t)
        acc = acc - (acc > 0)
    assert (r["temperature"] == t).all()
    if exact is not None:
        assert (r["F"][ok] <= exact["F"][ok]).all()
        # the exact minimum cost of the heuristic's flow value
        sub = batch.subset(np.flatnonzero(ok))
        sub.supply[:] = r["F"][ok]
        best = oracle.solve(sub, flows=False, potentials=False)
        assert (best["F"] == r["F"][ok]).all()
        assert (r["cost"][ok] >= best["cost"]).all()


@pytest.mark.parametrize("setting", [1, 2, 3, 4])
def test_flow_test_settings_invariants(setting, lib=None):
    """Flow-test settings 1-4 of the paper's table: the heuristic reaches the
    optimal flow value within 120 rounds and never undercuts the optimum."""
    batch = W.paper_flow_test(setting, 64)
    exact = oracle.solve(batch, flows=False, potentials=False)
    for objective in ("sum", "max"):
        r = H.simulate(batch, rounds=120, objective=objective, seed=setting, lib=lib)
        assert (r["status"] == 0).all()
        check_invariants(batch, r, exact)
        assert (r["F"] == exact["F"]).all()
        assert (r["cost"] >= exact["cost"]).all()
        if objective == "sum":
            assert r["cost"].sum() < 1.4 * exact["cost"].sum()


@pytest.mark.parametrize("seed", range(6))
def test_random_instances_invariants(seed, lib=None):
    rng = np.random.default_rng(seed)
    S, n = int(rng.integers(1, 7)), int(rng.integers(1, 9))
    batch = W.random_small(40, S, n, seed=100 + seed, cap_hi=int(rng.integers(1, 5)),
                           cost_hi=int(rng.integers(0, 40)), supply_hi=int(rng.integers(0, 20)),
                           holes=float(rng.choice([0.0, 0.3])), zero_cap=float(rng.choice([0.0, 0.2])))
    exact = oracle.solve(batch, flows=False, potentials=False)
    for rounds in (0, 1, 7, 60):
        r = H.simulate(batch, rounds=rounds, objective=("sum", "max")[seed % 2], seed=seed, lib=lib)
        check_invariants(batch, r, exact)
        if rounds == 0:
            assert (r["F"] == 0).all() and (r["used"] == 0).all()


def test_deterministic_and_seeded(lib=None):
    batch = W.paper_flow_test(1, 32)
    a = H.simulate(batch, seed=5, lib=lib)
    b = H.simulate(batch, seed=5, nthreads=1, lib=lib)
    c = H.simulate(batch, seed=6, lib=lib)
    for key in ("F", "cost", "node_flow", "arc_flow", "used", "accepted", "temperature", "counters"):
        assert np.array_equal(a[key], b[key]), key
    assert not np.array_equal(a["accepted"], c["accepted"])


def test_status_and_initial_paths(lib=None):
    batch = W.paper_flow_test(1, 6)
    batch.node_cap[1, 2, 0] = -1               # bad capacity
    batch.arc_cost[2, 0, 0, 0] = -2            # bad link
    batch.node_cost[3, 0, 0] = 1 << 26         # overflow: (2S + 2) * max >= 2^30
    r = H.simulate(batch, max_slots=1024, lib=lib)
    assert r["status"].tolist()[:4] == [0, 1, 1, 2]
    assert (r["F"][1:4] == 0).all() and (r["cost"][1:4] == 0).all()
    small = H.simulate(batch.subset([0]), max_slots=int(batch.node_cap[0].sum()) - 1, lib=lib)
    assert small["status"][0] == 1              # total capacity above max_slots
    # initial paths: with zero rounds the result is the paths themselves
    b, paths = change_example()
    r = H.simulate(b, rounds=0, paths=paths, lib=lib)
    assert r["F"][0] == 2 and r["cost"][0] == 11
    bad = paths.copy()
    bad[0, 1] = [0, 1]                         # node 1 twice: over its capacity
    assert H.simulate(b, rounds=0, paths=bad, lib=lib)["status"][0] == 1
    unused = np.concatenate([paths, np.full((1, 1, 2), -1, np.int32)], axis=1)
    assert H.simulate(b, rounds=0, paths=unused, lib=lib)["F"][0] == 2


# ---------------------------------------------------------------- planted mistakes

MUTANTS = {
    "request_by_link_only": ("int64_t score = st->cs[u] + link(st, v, w);",
                             "int64_t score = link(st, v, w);"),
    "cost_to_sink_without_compute": ("st->cs[s] = st->cost[v] + (int64_t)edge",
                                     "st->cs[s] = 0 + (int64_t)edge"),
    "acceptance_sign_flipped": ("double delta = (double)(cur - nxt) * 0.5;",
                                "double delta = (double)(nxt - cur) * 0.5;"),
    "no_cooling": ("st->T[a] *= alpha;", "st->T[a] *= 1.0;"),
    "change_without_relink": ("if (oy != HS_DATA) st->in[oy] = x;", ";"),
    "redirect_keeps_old_slot": ("st->in[y] = HS_NONE;\n                    st->out[y] = HS_NONE;", ";"),
    "max_read_as_sum": ("cur = objective ? (c0 > c1 ? c0 : c1) : c0 + c1;\n                    nxt = objective ? (n0 > n1 ? n0 : n1) : n0 + n1;\n                    if (!accept_move(cur, nxt, st->T[a], w[3])) continue;\n                    st->out[x]",
                        "cur = c0 + c1;\n                    nxt = n0 + n1;\n                    if (!accept_move(cur, nxt, st->T[a], w[3])) continue;\n                    st->out[x]"),
    "u_from_low_bits": ("double U = (double)(w >> 11)", "double U = (double)(w & 0x1fffffffffffffULL)"),
    "shuffle_range_short": ("bounded(words[used_words++], (uint32_t)(j + 1))", "bounded(words[used_words++], (uint32_t)j)"),
}

PINS = [
    lambda lib: [test_philox_matches_numpy(c, k, lib=lib) for c, k in
                 [([0, 0, 0, 0], [0, 0]), ([5, 7, 9, 11], [123, 456])]],
    lambda lib: test_request_change_example_max_objective(lib=lib),
    lambda lib: test_request_change_example_sum_objective(lib=lib),
    lambda lib: test_request_redirect_example(lib=lib),
    lambda lib: test_request_flow_argmin_of_cost_to_sink_plus_link(lib=lib),
    lambda lib: [test_flow_test_settings_invariants(s, lib=lib) for s in (1, 3)],
    lambda lib: [test_random_instances_invariants(s, lib=lib) for s in (0, 1)],
]


@pytest.mark.slow
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(H.SRC).read()
    assert src.count(old) == 1, f"mutation site of {name} not found exactly once"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = H.bind(H.build(str(path), str(tmp_path / f"lib{name}.so")))
    caught = 0
    for pin in PINS:
        try:
            pin(lib)
        except AssertionError:
            caught += 1
    assert caught > 0, f"no pin rejects the planted mistake {name}"
