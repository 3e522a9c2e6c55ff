"""Pins for the CPU oracle: every check here is independent of the oracle's
own arithmetic (see mcf_checks for the fact each one rests on)."""
import glob
import json
import os

import numpy as np
import pytest

import oracle
from paper_2509_21221_amd import workloads as W
import mcf_checks as C

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def batch_from_json(path):
    d = json.load(open(path))
    S, n = d["S"], d["n"]
    arr = lambda key, shp: np.asarray(d[key], np.int32).reshape(shp)
    b = W.Batch(S, n, arr("node_cap", (1, S, n)), arr("node_cost", (1, S, n)),
                arr("arc_cost", (1, S - 1, n, n)), arr("src_cost", (1, n)),
                arr("snk_cost", (1, n)), np.asarray([d["supply"]], np.int32))
    b.check_layout()
    return b, d


def certify_all(batch, r):
    for b in range(batch.B):
        C.certify(batch, b, int(r["F"][b]), int(r["cost"][b]), r["node_flow"][b], r["arc_flow"][b],
                  r["src_flow"][b], r["snk_flow"][b], r["potential"][b])


@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(GOLDEN, "paper_*.json"))),
                         ids=lambda p: os.path.basename(p))
def test_paper_worked_examples(path):
    batch, d = batch_from_json(path)
    r = oracle.solve(batch)
    assert r["status"][0] == 0
    assert r["F"][0] == d["expect_F"]
    if "expect_cost" in d:
        assert r["cost"][0] == d["expect_cost"]
    certify_all(batch, r)


def test_request_change_is_sum_not_bottleneck():
    """Eq. 2 (sum) keeps 3 + 8 = 11; the max-objective swap would cost 12."""
    batch, _ = batch_from_json(os.path.join(GOLDEN, "paper_request_change.json"))
    r = oracle.solve(batch)
    assert (r["F"][0], r["cost"][0]) == (2, 11)
    # the optimal flow keeps links 1->2 and 3->4
    assert r["arc_flow"][0, 0].tolist() == [[1, 0], [0, 1]]


@pytest.mark.parametrize("S,n,holes,zero_cap", [
    (1, 1, 0.0, 0.0), (1, 3, 0.0, 0.2), (2, 2, 0.0, 0.0), (2, 3, 0.3, 0.1),
    (3, 2, 0.0, 0.0), (3, 3, 0.2, 0.1), (3, 3, 0.0, 0.0), (2, 1, 0.0, 0.0),
])
def test_brute_force_tiny(S, n, holes, zero_cap):
    batch = W.random_small(24, S, n, seed=11, cap_hi=3, cost_hi=20, supply_hi=6,
                           holes=holes, zero_cap=zero_cap)
    r = oracle.solve(batch)
    assert (r["status"] == 0).all()
    for b in range(batch.B):
        F, cost = C.brute_force(batch, b)
        assert (int(r["F"][b]), int(r["cost"][b])) == (F, cost), f"instance {b}"
    certify_all(batch, r)


def test_brute_force_asymmetric_links():
    """Transposing arc_cost (sender/receiver) must change these optima."""
    batch = W.random_small(40, 3, 3, seed=5, cap_hi=2, cost_hi=50, supply_hi=5)
    r = oracle.solve(batch)
    moved = 0
    for b in range(batch.B):
        F, cost = C.brute_force(batch, b)
        assert (int(r["F"][b]), int(r["cost"][b])) == (F, cost)
        t = batch.instance(b)
        t.arc_cost = np.ascontiguousarray(t.arc_cost.transpose(0, 1, 3, 2))
        moved += C.brute_force(t, 0) != (F, cost)
    assert moved > 0


@pytest.mark.parametrize("cfg,count", [(1, 256), (2, 128), (3, 128)])
def test_closed_form_value_and_certificate(cfg, count):
    batch = W.CONFIGS[cfg](count)
    r = oracle.solve(batch)
    assert (r["status"] == 0).all()
    for b in range(batch.B):
        assert r["F"][b] == C.closed_form_value(batch, b)
    certify_all(batch, r)


@pytest.mark.parametrize("cfg,count", [(1, 48), (2, 12), (3, 12)])
def test_networkx_cross_check(cfg, count):
    batch = W.CONFIGS[cfg](count)
    r = oracle.solve(batch, flows=False, potentials=False)
    for b in range(batch.B):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.networkx_mcmf(batch, b)


def test_networkx_with_missing_links():
    batch = W.random_small(20, 4, 4, seed=3, cap_hi=4, cost_hi=60, supply_hi=12,
                           holes=0.4, zero_cap=0.15)
    r = oracle.solve(batch)
    for b in range(batch.B):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.networkx_mcmf(batch, b)
    certify_all(batch, r)


def test_single_stage_greedy():
    batch = W.random_small(64, 1, 6, seed=9, cap_hi=4, cost_hi=30, supply_hi=20)
    r = oracle.solve(batch)
    for b in range(batch.B):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.single_stage_greedy(batch, b)


def test_two_stage_transport_lp():
    batch = W.random_small(24, 2, 7, seed=13, cap_hi=5, cost_hi=80, supply_hi=30, holes=0.2)
    r = oracle.solve(batch)
    for b in range(batch.B):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.transport_lp(batch, b)


def test_assignment_closed_form_c4_shape():
    """Capacities 1 on the 32 x 64 shape: one assignment per stage pair."""
    batch = W.config4(2)
    batch.node_cap[:] = 1
    r = oracle.solve(batch)
    for b in range(batch.B):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.assignment_cost(batch, b)
    certify_all(batch, r)


@pytest.mark.parametrize("setting", [1, 2, 3, 4])
def test_paper_flow_test_shapes(setting):
    batch = W.paper_flow_test(setting, B=6)
    r = oracle.solve(batch)
    for b in range(batch.B):
        assert r["F"][b] == C.closed_form_value(batch, b)
        assert (int(r["F"][b]), int(r["cost"][b])) == C.networkx_mcmf(batch, b)
    certify_all(batch, r)


def test_metamorphic():
    batch = W.config2(32)
    base = oracle.solve(batch, flows=False, potentials=False)
    # +k on every compute cost of one stage: each unit crosses it once
    t = batch.subset(range(batch.B))
    t.node_cost[:, 3] += 7
    r = oracle.solve(t, flows=False, potentials=False)
    assert (r["F"] == base["F"]).all() and (r["cost"] == base["cost"] + 7 * base["F"]).all()
    # +k on one stage pair's links
    t = batch.subset(range(batch.B))
    t.arc_cost[:, 5] += 3
    r = oracle.solve(t, flows=False, potentials=False)
    assert (r["cost"] == base["cost"] + 3 * base["F"]).all()
    # scale every cost by 3
    t = batch.subset(range(batch.B))
    t.node_cost *= 3
    t.arc_cost *= 3
    r = oracle.solve(t, flows=False, potentials=False)
    assert (r["cost"] == 3 * base["cost"]).all()
    # permute the nodes of stage 4 (and the links touching them)
    t = batch.subset(range(batch.B))
    p = np.random.default_rng(0).permutation(batch.n)
    t.node_cap[:, 4] = t.node_cap[:, 4][:, p]
    t.node_cost[:, 4] = t.node_cost[:, 4][:, p]
    t.arc_cost[:, 3] = t.arc_cost[:, 3][:, :, p]
    t.arc_cost[:, 4] = t.arc_cost[:, 4][:, p, :]
    r = oracle.solve(t, flows=False, potentials=False)
    assert (r["F"] == base["F"]).all() and (r["cost"] == base["cost"]).all()


def test_edge_cases():
    # zero supply, a whole stage deleted, S = 1, n = 1
    batch = W.config1(8)
    batch.supply[0] = 0
    batch.node_cap[1, 2] = 0
    r = oracle.solve(batch)
    assert r["F"][0] == 0 and r["cost"][0] == 0
    assert r["F"][1] == 0 and r["cost"][1] == 0
    certify_all(batch, r)
    one = W.random_small(5, 1, 1, seed=1, cap_hi=5, supply_hi=9)
    r = oracle.solve(one)
    for b in range(5):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.brute_force(one, b)


def test_bad_input_status():
    batch = W.config1(4)
    batch.node_cap[0, 0, 0] = -1
    batch.arc_cost[1, 0, 0, 0] = -2
    batch.supply[2] = -5
    r = oracle.solve(batch)
    assert r["status"].tolist() == [1, 1, 1, 0]
    assert r["F"][:3].tolist() == [0, 0, 0]


def test_thread_count_does_not_change_results():
    batch = W.config2(64)
    a = oracle.solve(batch, nthreads=1, flows=False, potentials=False)
    b = oracle.solve(batch, nthreads=4, flows=False, potentials=False)
    assert (a["F"] == b["F"]).all() and (a["cost"] == b["cost"]).all()
