"""GPU parity of location-factored instances (link delay = latency between
the two nodes' locations, the paper's Sec. VI testbed): gwtf_mcf_solve_located
through the C ABI against the located oracle, on every pass (the factored
grid pass for 64 < n <= 512, the expanded-delay passes below).

(F, cost, status) must match the oracle exactly; every returned flow is
certified (feasibility, maximality, complementary slackness) on the dense
instance the located one stands for.
"""
import hashlib
import json
import os
import sys

import numpy as np
import pytest

import oracle.located as OL
from paper_2509_21221_amd import mcf
from paper_2509_21221_amd import workloads as W
import mcf_checks as C

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gpu_solve_located(lb, flows=True, with_src=True):
    import torch

    dev = torch.device("cuda", 0)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    with mcf.Solver(lb.S, lb.n, lb.B) as s:
        F, cost, status = s.solve_located(t(lb.node_cap), t(lb.node_cost), t(lb.location), t(lb.latency),
                                          t(lb.supply), src_cost=t(lb.src_cost) if with_src else None,
                                          snk_cost=t(lb.snk_cost) if with_src else None)
        out = {"passes": s.passes().cpu().numpy(), "stats": s.stats().cpu().numpy()}
        if flows:
            out.update({k: v.cpu().numpy() for k, v in s.flows().items()})
        torch.cuda.synchronize()
        out.update(F=F.cpu().numpy(), cost=cost.cpu().numpy(), status=status.cpu().numpy())
    return out


def check(lb, g, ref, certify=None):
    assert (g["status"] == ref["status"]).all(), "status mismatch"
    bad = np.flatnonzero((g["F"] != ref["F"]) | (g["cost"] != ref["cost"]))
    assert bad.size == 0, (f"{bad.size} mismatches, first {bad[:5]}: gpu {g['F'][bad[:5]]}/"
                           f"{g['cost'][bad[:5]]} oracle {ref['F'][bad[:5]]}/{ref['cost'][bad[:5]]}")
    if "node_flow" not in g:
        return
    dense, _ = OL.to_dense(lb if certify is None else lb.subset(certify))
    idx = range(lb.B) if certify is None else range(len(certify))
    src = range(lb.B) if certify is None else certify
    for d, b in zip(idx, src):
        if g["status"][b] != 0:
            continue
        C.certify(dense, d, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                  g["src_flow"][b], g["snk_flow"][b], g["potential"][b])


@pytest.mark.parametrize("S,n,L,B,expect_pass", [
    (3, 6, 3, 24, mcf.GWTF_PASS_PACKED),
    (10, 6, 3, 8, mcf.GWTF_PASS_LDS),
    (4, 24, 5, 12, mcf.GWTF_PASS_REGISTER),
    (3, 80, 7, 4, mcf.GWTF_PASS_GRID),
    (2, 130, 32, 3, mcf.GWTF_PASS_GRID),
    (5, 200, 10, 2, mcf.GWTF_PASS_GRID),
    (1, 100, 4, 3, mcf.GWTF_PASS_GRID),
    (40, 48, 6, 3, mcf.GWTF_PASS_GRID),
    (2, 1, 1, 8, mcf.GWTF_PASS_PACKED),
])
def test_random_located(S, n, L, B, expect_pass):
    lb = W.random_located(B, S, n, L, seed=21, supply_hi=40)
    say("located", S, n, L, B)
    g = gpu_solve_located(lb)
    check(lb, g, OL.solve(lb))
    assert (g["passes"] == expect_pass).all()


def test_located_grid_batch_over_several_launches():
    """A located batch on the factored grid pass that needs several
    cooperative launches (40 workgroups per instance, six instances per
    launch on 256 CUs): every instance against the located oracle."""
    lb = W.random_located(14, 40, 70, 6, seed=29, supply_hi=60)
    say("located grid batch", 40, 70, 14)
    g = gpu_solve_located(lb, flows=False)
    check(lb, g, OL.solve(lb, flows=False, potentials=False))
    assert (g["passes"] == mcf.GWTF_PASS_GRID).all()


@pytest.mark.parametrize("S,n", [(3, 5), (3, 90)])
def test_invalid_locations_and_latencies(S, n):
    lb = W.random_located(5, S, n, 4, seed=8, supply_hi=20)
    lb.location[1][0, 0] = 4          # outside [0, L)
    lb.location[2][S - 1, n - 1] = -1  # outside, last stage
    lb.latency[3][0, 0] = -1           # negative latency (used or not)
    lb.latency[4][3, 3] = -5
    g = gpu_solve_located(lb, flows=False)
    ref = OL.solve(lb, flows=False, potentials=False)
    check(lb, g, ref)
    assert g["status"].tolist() == [0, 1, 1, 1, 1]


def test_without_data_node_delays():
    lb = W.random_located(6, 3, 70, 5, seed=4, supply_hi=30)
    g = gpu_solve_located(lb, with_src=False)
    lb.src_cost[:] = 0
    lb.snk_cost[:] = 0
    check(lb, g, OL.solve(lb))


def test_located_preset2_full():
    lb = W.located(2)
    g = gpu_solve_located(lb, flows=False)
    check(lb, g, OL.solve(lb, flows=False, potentials=False))


def _stored(preset, lb):
    """The stored optimum of the dense preset that the located batch
    expands to (checked by the input digest)."""
    rec = json.load(open(os.path.join(GOLDEN, f"c{preset}_oracle.json")))
    dense, bad = OL.to_dense(lb)
    assert not bad.any()
    h = hashlib.sha256()
    for key in ("node_cap", "node_cost", "arc_cost", "src_cost", "snk_cost", "supply"):
        h.update(np.ascontiguousarray(getattr(dense, key)).tobytes())
    assert h.hexdigest() == rec["input_sha256"]
    return dense, np.asarray(rec["F"]), np.asarray(rec["cost"])


def test_located_preset4_against_stored_optimum():
    lb = W.located(4)
    dense, F, cost = _stored(4, lb)
    g = gpu_solve_located(lb)
    assert (g["status"] == 0).all() and (g["F"] == F).all() and (g["cost"] == cost).all()
    assert (g["passes"] == mcf.GWTF_PASS_REGISTER).all()
    for b in range(0, lb.B, 37):
        C.certify(dense, b, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                  g["src_flow"][b], g["snk_flow"][b], g["potential"][b])


def test_located_preset5_factored_grid_pass():
    """The 64 x 512 instance on the factored grid pass: the stored optimum,
    the certificate, and fewer relaxation operations than the dense links
    stand for."""
    lb = W.located(5)
    dense, F, cost = _stored(5, lb)
    say("located c5 start")
    g = gpu_solve_located(lb)
    say("located c5 done", g["F"], g["cost"], g["stats"][0, :4])
    assert g["passes"][0] == mcf.GWTF_PASS_GRID
    assert g["status"][0] == 0 and g["F"][0] == F[0] and g["cost"][0] == cost[0]
    C.certify(dense, 0, int(g["F"][0]), int(g["cost"][0]), g["node_flow"][0], g["arc_flow"][0],
              g["src_flow"][0], g["snk_flow"][0], g["potential"][0])
