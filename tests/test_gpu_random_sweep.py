"""GPU parity on a seeded sweep of random shapes that crosses every pass.

Each case draws a pass-shaped random batch (packed: S <= 8, n <= 16;
pipelined: S <= 32, 16 < n <= 64 and wider pipelines; grid: 64 < n < 260;
LDS: n <= 16 with S > 8), with and without missing links, deleted nodes and
data-node delays, and checks (F, cost, status) against the oracle on every
instance and the certificate on the first instances of each case.  A second
sweep takes single instances over the grid pass's whole width (n <= 512) and
cost range, overflowing ones included.
"""
import sys

import numpy as np
import pytest

import mcf_checks as C
import oracle
from gpu_util import gpu_solve
from paper_2509_21221_amd import workloads as W

pytestmark = pytest.mark.gpu


def draw(rng):
    kind = int(rng.integers(0, 5))
    if kind == 0:  # packed pass
        S, n, B = int(rng.integers(1, 9)), int(rng.integers(1, 17)), int(rng.integers(1, 300))
        kw = dict(cap_hi=int(rng.integers(1, 9)), cost_hi=int(rng.integers(0, 300)), supply_hi=int(rng.integers(0, 80)))
    elif kind == 1:  # pipelined pass
        S, n, B = int(rng.integers(2, 33)), int(rng.integers(17, 65)), int(rng.integers(1, 40))
        kw = dict(cap_hi=int(rng.integers(1, 12)), cost_hi=int(rng.integers(1, 1100)), supply_hi=int(rng.integers(1, 300)))
    elif kind == 2:  # grid pass
        S, n, B = int(rng.integers(2, 12)), int(rng.integers(65, 260)), 1
        kw = dict(cap_hi=int(rng.integers(1, 6)), cost_hi=int(rng.integers(1, 400)), supply_hi=int(rng.integers(1, 60)))
    elif kind == 3:  # LDS pass
        S, n, B = int(rng.integers(9, 40)), int(rng.integers(1, 17)), int(rng.integers(1, 30))
        kw = dict(cap_hi=int(rng.integers(1, 6)), cost_hi=int(rng.integers(0, 200)), supply_hi=int(rng.integers(0, 40)))
    else:  # pipelines longer than the pipelined pass takes
        S, n, B = int(rng.integers(33, 48)), int(rng.integers(17, 65)), int(rng.integers(1, 8))
        kw = dict(cap_hi=int(rng.integers(1, 6)), cost_hi=int(rng.integers(1, 200)), supply_hi=int(rng.integers(1, 80)))
    holes = float(rng.choice([0.0, 0.0, 0.1, 0.4]))
    zero = float(rng.choice([0.0, 0.0, 0.2]))
    seed = int(rng.integers(0, 1 << 30))
    src_snk = bool(rng.integers(0, 2))
    return kind, W.random_small(B, S, n, seed, holes=holes, zero_cap=zero, src_snk=src_snk, **kw)


@pytest.mark.parametrize("block", range(4))
def test_random_sweep(block):
    rng = np.random.default_rng(np.random.SeedSequence(2509, spawn_key=(block,)))
    for case in range(75):
        kind, batch = draw(rng)
        print(f"block {block} case {case} kind {kind} S={batch.S} n={batch.n} B={batch.B}", flush=True)
        sys.stdout.flush()
        g = gpu_solve(batch)
        ref = oracle.solve(batch, flows=False, potentials=False)
        bad = np.flatnonzero((g["F"] != ref["F"]) | (g["cost"] != ref["cost"]) | (g["status"] != ref["status"]))
        assert bad.size == 0, (f"case {case}: instances {bad[:5]}: gpu {g['F'][bad[:3]]}/{g['cost'][bad[:3]]} "
                               f"oracle {ref['F'][bad[:3]]}/{ref['cost'][bad[:3]]}, passes {g['passes'][bad[:3]]}")
        for b in range(min(batch.B, 2)):
            if g["status"][b] == 0:
                C.certify(batch, b, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                          g["src_flow"][b], g["snk_flow"][b], g["potential"][b])


def max_cost(batch):
    arrays = [batch.node_cost, batch.arc_cost, batch.src_cost, batch.snk_cost]
    return max(int(np.max(a)) for a in arrays if a is not None and np.size(a))


@pytest.mark.parametrize("block", range(2))
def test_random_grid_sweep(block):
    """Single instances across the grid pass's whole range (64 < n <= 512,
    up to 19 stages, costs from a few values to tens of thousands, supply
    up to three times the stage width).  An instance whose label bound
    (2 S n + 3) * max cost reaches 2^29 must come back as an overflow with
    F = cost = 0 (the last two cases of each block are drawn long, wide and
    costly, so most of them do); every other one must match the oracle and
    pass the certificate."""
    rng = np.random.default_rng(np.random.SeedSequence(20261202, spawn_key=(block,)))
    for case in range(26):
        S, n = int(rng.integers(2, 20)), int(rng.integers(65, 513))
        holes = float(rng.choice([0.0, 0.0, 0.05, 0.3]))
        zero = float(rng.choice([0.0, 0.1, 0.3]))
        cost_hi = int(rng.choice([3, 50, 400, 3000, 60000]))
        if case >= 24:  # the last two: long, wide and costly
            S, n, cost_hi = int(rng.integers(12, 20)), int(rng.integers(300, 513)), 60000
        batch = W.random_small(1, S, n, int(rng.integers(0, 1 << 30)), cap_hi=int(rng.integers(1, 7)),
                               cost_hi=cost_hi, supply_hi=int(rng.integers(1, 3 * n)), holes=holes,
                               zero_cap=zero, src_snk=bool(rng.integers(0, 2)))
        overflow = (2 * S * n + 3) * max_cost(batch) >= 1 << 29
        print(f"grid block {block} case {case} S={S} n={n} cost_hi={cost_hi} overflow={overflow}", flush=True)
        g = gpu_solve(batch)
        if overflow:
            assert (g["status"] == 2).all() and (g["F"] == 0).all() and (g["cost"] == 0).all(), (case, g["status"])
            continue
        assert g["passes"][0] == 3, (case, g["passes"])
        ref = oracle.solve(batch, flows=False, potentials=False)
        assert g["F"][0] == ref["F"][0] and g["cost"][0] == ref["cost"][0] and g["status"][0] == ref["status"][0], (
            f"case {case}: gpu {g['F']}/{g['cost']}/{g['status']} oracle {ref['F']}/{ref['cost']}/{ref['status']}")
        if g["status"][0] == 0:
            C.certify(batch, 0, int(g["F"][0]), int(g["cost"][0]), g["node_flow"][0], g["arc_flow"][0],
                      g["src_flow"][0], g["snk_flow"][0], g["potential"][0])
