"""GPU parity on a seeded sweep of random shapes that crosses every pass.

Each case draws a pass-shaped random batch (packed: S <= 8, n <= 16;
pipelined: S <= 32, 16 < n <= 64 and wider pipelines; grid: 64 < n < 260;
LDS: n <= 16 with S > 8), with and without missing links, deleted nodes and
data-node delays, and checks (F, cost, status) against the oracle on every
instance and the certificate on the first instances of each case.
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
