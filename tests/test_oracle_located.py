"""Pins for the located-instance oracle: each rests on something other than
its own dense expansion (a hub network solved by networkx, brute force, the
generator's dense presets and the stored optima of the dense presets)."""
import hashlib
import json
import os

import numpy as np
import pytest

import oracle
import oracle.located as OL
from paper_2509_21221_amd import workloads as W
import mcf_checks as C

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("S,n,L", [(1, 3, 2), (2, 3, 2), (3, 4, 3), (4, 5, 5), (3, 6, 10)])
def test_hub_network(S, n, L):
    lb = W.random_located(6, S, n, L, seed=3)
    r = OL.solve(lb, flows=False, potentials=False)
    for b in range(lb.B):
        assert r["status"][b] == 0
        assert (int(r["F"][b]), int(r["cost"][b])) == C.networkx_located_hubs(lb, b)


@pytest.mark.parametrize("S,n,L", [(2, 2, 2), (3, 2, 3), (2, 3, 2)])
def test_brute_force(S, n, L):
    lb = W.random_located(8, S, n, L, seed=5, cap_hi=2, supply_hi=5)
    r = OL.solve(lb, flows=False, potentials=False)
    dense, _ = OL.to_dense(lb)
    for b in range(lb.B):
        assert (int(r["F"][b]), int(r["cost"][b])) == C.brute_force(dense, b)


@pytest.mark.parametrize("preset", [2, 4])
def test_matches_generator_dense_presets(preset):
    lb = W.located(preset, B=3)
    d = W.CONFIGS[preset](3)
    dense, bad = OL.to_dense(lb)
    assert not bad.any()
    for key in ("node_cap", "node_cost", "arc_cost", "src_cost", "snk_cost", "supply"):
        assert (getattr(dense, key) == getattr(d, key)).all(), key


def test_c5_located_is_the_stored_instance():
    """The located 64 x 512 instance expands to exactly the dense instance
    whose optimum is stored (same input digest), so that optimum pins it."""
    g = json.load(open(os.path.join(GOLDEN, "c5_oracle.json")))
    dense, bad = OL.to_dense(W.located(5))
    assert not bad.any()
    h = hashlib.sha256()
    for key in ("node_cap", "node_cost", "arc_cost", "src_cost", "snk_cost", "supply"):
        h.update(np.ascontiguousarray(getattr(dense, key)).tobytes())
    assert h.hexdigest() == g["input_sha256"]


def test_invalid_location_or_latency():
    lb = W.random_located(4, 3, 3, 3, seed=1)
    lb.location[1][0, 0] = 3
    lb.latency[2][1, 2] = -1
    lb.location[3][2, 1] = -1
    r = OL.solve(lb, flows=False, potentials=False)
    assert r["status"].tolist() == [0, 1, 1, 1]
    assert r["F"][1:].tolist() == [0, 0, 0] and r["cost"][1:].tolist() == [0, 0, 0]


LOCATED_MUTANTS = {
    "latency_transposed": ("lat[loc[k, i], loc[k + 1, :]]", "lat[loc[k + 1, :], loc[k, i]]"),
    "same_stage_locations": ("lat[loc[k, i], loc[k + 1, :]]", "lat[loc[k, i], loc[k, :]]"),
    "negative_latency_accepted": ("or (lat < 0).any()", "or (lat < -1).any()"),
    "range_check_off_by_one": ("(loc >= L).any()", "(loc > L).any()"),
}


def _variant(text, name):
    import types

    mod = types.ModuleType(f"oracle.{name}")
    mod.__package__ = "oracle"
    exec(compile(text, f"<located variant {name}>", "exec"), mod.__dict__)
    return mod


def _located_pins_pass(ol):
    try:
        for S, n, L in [(3, 4, 3), (4, 5, 5)]:
            lb = W.random_located(4, S, n, L, seed=3)
            r = ol.solve(lb, flows=False, potentials=False)
            for b in range(lb.B):
                if (int(r["F"][b]), int(r["cost"][b])) != C.networkx_located_hubs(lb, b):
                    return False
        lb = W.random_located(3, 3, 3, 3, seed=1)
        lb.location[1][0, 0] = 3
        lb.latency[2][1, 2] = -1
        if ol.solve(lb, flows=False, potentials=False)["status"].tolist() != [0, 1, 1]:
            return False
    except (AssertionError, IndexError):
        return False
    return True


def test_unmutated_located_copy_passes():
    assert _located_pins_pass(_variant(open(OL.__file__).read(), "same"))


@pytest.mark.parametrize("name", sorted(LOCATED_MUTANTS))
def test_located_pins_reject_mutant(name):
    before, after = LOCATED_MUTANTS[name]
    text = open(OL.__file__).read()
    assert text.count(before) == 1, f"mutation anchor for {name} not unique"
    assert not _located_pins_pass(_variant(text.replace(before, after), name))


def test_single_stage_reads_no_location():
    lb = W.random_located(2, 1, 3, 2, seed=2)
    lb.location[0][0, 0] = 7
    lb.latency[1][0, 1] = -3
    r = OL.solve(lb, flows=False, potentials=False)
    assert r["status"].tolist() == [0, 0]
