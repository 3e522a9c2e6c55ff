"""Each pin must be able to fail: plant one plausible mistake at a time in
a private copy of the oracle's C source (never in the oracle itself),
compile it on the CPU, and check that the pin suite rejects it."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2509_21221_amd import workloads as W
import mcf_checks as C

SRC = os.path.join(os.path.dirname(oracle.__file__), "mcf_oracle.c")

MUTANTS = {
    "drop_node_cost": ("in->cap[k * n + i], in->ncost[k * n + i]);", "in->cap[k * n + i], 0);"),
    "reverse_cost_sign": ("g->cost[e + 1] = -c;", "g->cost[e + 1] = c;"),
    "transposed_links": ("int64_t q = ((int64_t)k * n + i) * n + j;",
                         "int64_t q = ((int64_t)k * n + j) * n + i;"),
    "drop_sink_cost": ("OR_INF_CAP, in->snk[i]);", "OR_INF_CAP, 0);"),
    "potential_not_clamped": ("pi[v] += (dist[v] < dt) ? dist[v] : dt;",
                              "pi[v] += (dist[v] < OR_INF_DIST) ? dist[v] : dt;"),
    "ignore_supply": ("add_arc(g, 0, 1, in->supply, 0);", "add_arc(g, 0, 1, OR_INF_CAP, 0);"),
    "unit_augment": ("r.F += delta;\n        r.cost += delta * (pi[2] - pi[0]);",
                     "r.F += 1;\n        r.cost += (pi[2] - pi[0]);"),
}


def _build_mutant(tmp_path, name):
    before, after = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(before) == 1, f"mutation anchor for {name} not unique"
    src = tmp_path / f"{name}.c"
    src.write_text(text.replace(before, after))
    so = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", "-pthread", str(src),
                           "-o", str(so)])
    return oracle.bind(str(so))


def _pins_pass(lib):
    """A small slice of the pin suite; True when every pin accepts ``lib``."""
    try:
        tiny = W.random_small(16, 3, 3, seed=21, cap_hi=3, cost_hi=20, supply_hi=6, holes=0.2)
        r = oracle.solve(tiny, lib=lib)
        for b in range(tiny.B):
            if r["status"][b] != 0 or (int(r["F"][b]), int(r["cost"][b])) != C.brute_force(tiny, b):
                return False
        geo = W.config2(8)
        r = oracle.solve(geo, lib=lib)
        for b in range(geo.B):
            if r["status"][b] != 0:
                return False
            C.certify(geo, b, int(r["F"][b]), int(r["cost"][b]), r["node_flow"][b], r["arc_flow"][b],
                      r["src_flow"][b], r["snk_flow"][b], r["potential"][b])
        ex = W.paper_flow_test(1, B=2)
        r = oracle.solve(ex, lib=lib)
        for b in range(ex.B):
            if (int(r["F"][b]), int(r["cost"][b])) != C.networkx_mcmf(ex, b):
                return False
    except AssertionError:
        return False
    return True


def test_unmutated_copy_passes(tmp_path):
    so = tmp_path / "libsame.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", "-pthread", SRC, "-o", str(so)])
    assert _pins_pass(oracle.bind(str(so)))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(tmp_path, name):
    assert not _pins_pass(_build_mutant(tmp_path, name))
