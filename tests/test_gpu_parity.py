"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

(F, cost) must match the oracle bit for bit on every instance; flows may
differ where several are optimal, so every returned flow is checked for
feasibility, maximality and the complementary-slackness certificate with the
potentials the GPU returns.
"""
import hashlib
import json
import os
import sys

import numpy as np
import pytest

import oracle
from paper_2509_21221_amd import mcf
from paper_2509_21221_amd import workloads as W
import mcf_checks as C
from gpu_util import gpu_solve

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def compare(batch, g, ref, certify=None):
    assert (g["status"] == ref["status"]).all(), "status mismatch"
    bad = np.flatnonzero((g["F"] != ref["F"]) | (g["cost"] != ref["cost"]))
    assert bad.size == 0, (f"{bad.size} mismatches, first {bad[:5]}: gpu "
                           f"{g['F'][bad[:5]]}/{g['cost'][bad[:5]]} oracle "
                           f"{ref['F'][bad[:5]]}/{ref['cost'][bad[:5]]}")
    idx = range(batch.B) if certify is None else certify
    for b in idx:
        if g["status"][b] != 0:
            continue
        C.certify(batch, b, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                  g["src_flow"][b], g["snk_flow"][b], g["potential"][b])


def test_paper_examples():
    from test_oracle_pins import batch_from_json
    for name in sorted(os.listdir(GOLDEN)):
        if not (name.startswith("paper_") and name.endswith(".json")):
            continue
        batch, d = batch_from_json(os.path.join(GOLDEN, name))
        say("example", name)
        g = gpu_solve(batch)
        assert g["status"][0] == 0 and g["F"][0] == d["expect_F"]
        if "expect_cost" in d:
            assert g["cost"][0] == d["expect_cost"]
        compare(batch, g, oracle.solve(batch))


def test_config1_full():
    batch = W.config1()
    say("c1", batch.B)
    compare(batch, gpu_solve(batch), oracle.solve(batch, flows=False, potentials=False))


@pytest.mark.parametrize("cfg", [2, 3])
def test_config2_3_full(cfg):
    batch = W.CONFIGS[cfg]()
    say(f"c{cfg}", batch.B)
    g = gpu_solve(batch)
    ref = oracle.solve(batch, flows=False, potentials=False)
    compare(batch, g, ref, certify=range(0, batch.B, 16))


def _digest(batch):
    h = hashlib.sha256()
    for key in ("node_cap", "node_cost", "arc_cost", "src_cost", "snk_cost", "supply"):
        h.update(getattr(batch, key).tobytes())
    return h.hexdigest()


def test_config4_full_against_stored_oracle():
    gold = json.load(open(os.path.join(GOLDEN, "c4_oracle.json")))
    batch = W.config4()
    assert _digest(batch) == gold["input_sha256"], "generator no longer reproduces the stored inputs"
    say("c4", batch.B)
    g = gpu_solve(batch)
    assert (g["status"] == 0).all()
    assert (g["F"] == np.array(gold["F"])).all()
    assert (g["cost"] == np.array(gold["cost"])).all()
    for b in range(0, batch.B, 32):
        C.certify(batch, b, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                  g["src_flow"][b], g["snk_flow"][b], g["potential"][b])
        assert g["F"][b] == C.closed_form_value(batch, b)


def test_config4_sample_against_live_oracle():
    batch = W.config4(8)
    say("c4 sample", batch.B)
    compare(batch, gpu_solve(batch), oracle.solve(batch))


@pytest.mark.parametrize("S,n,holes,zero", [
    (1, 1, 0.0, 0.0), (1, 9, 0.0, 0.3), (2, 3, 0.3, 0.1), (3, 5, 0.2, 0.2), (4, 4, 0.5, 0.0),
    (6, 13, 0.1, 0.1), (9, 17, 0.0, 0.05), (5, 64, 0.05, 0.1), (12, 33, 0.2, 0.0), (40, 3, 0.0, 0.1),
])
def test_random_shapes(S, n, holes, zero):
    batch = W.random_small(48, S, n, seed=7, cap_hi=5, cost_hi=90, supply_hi=3 * n + 4,
                           holes=holes, zero_cap=zero)
    say("random", S, n)
    compare(batch, gpu_solve(batch), oracle.solve(batch))


@pytest.mark.parametrize("S,n", [(3, 65), (4, 100), (2, 130)])
def test_wide_stages(S, n):
    batch = W.random_small(6, S, n, seed=3, cap_hi=4, cost_hi=300, supply_hi=2 * n, holes=0.1,
                           zero_cap=0.1)
    say("wide", S, n)
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"] == mcf.GWTF_PASS_GRID).all()


@pytest.mark.parametrize("S,n,holes,zero", [
    (1, 200, 0.0, 0.1), (2, 512, 0.1, 0.0), (5, 128, 0.2, 0.1), (4, 129, 0.0, 0.0),
    (3, 300, 0.3, 0.2), (16, 256, 0.05, 0.05), (40, 97, 0.1, 0.1),
])
def test_grid_pass_shapes(S, n, holes, zero):
    """Shapes served by the grid-cooperative pass (64 < n <= 512): one
    ragged or full column block per workgroup, one to many stages."""
    batch = W.random_small(3, S, n, seed=23, cap_hi=6, cost_hi=400, supply_hi=3 * n,
                           holes=holes, zero_cap=zero)
    say("grid pass", S, n)
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"] == mcf.GWTF_PASS_GRID).all()


@pytest.mark.parametrize("S,n,B", [(6, 90, 40), (4, 130, 70), (33, 100, 9), (1, 300, 300)])
def test_grid_pass_batches(S, n, B):
    """Batches on the grid pass: as many instances per cooperative launch as
    can be resident together (each with its own labels, ring, predecessors,
    path and control block), the batch split over several launches when it
    holds more, every instance against the oracle."""
    batch = W.random_small(B, S, n, seed=47, cap_hi=5, cost_hi=300, supply_hi=2 * n, holes=0.1, zero_cap=0.1)
    say("grid batch", S, n, B)
    g = gpu_solve(batch, stats=True)
    compare(batch, g, oracle.solve(batch), certify=[0, B // 2, B - 1])
    assert (g["passes"] == mcf.GWTF_PASS_GRID).all()
    # Each instance's searches converge as they do when it is solved alone:
    # the label iterations per instance (stats column 1) vary a little with
    # timing (about 10 % for a single stage), but a convergence count that
    # mixed instances would multiply them.
    for b in (0, B - 1):
        one = gpu_solve(batch.subset([b]), flows=False, stats=True)
        assert one["F"][0] == g["F"][b] and one["cost"][0] == g["cost"][b]
        r_batch, r_one = int(g["stats"][b, 1]), int(one["stats"][0, 1])
        assert r_batch <= 2 * r_one + 16 and r_one <= 2 * r_batch + 16, (b, r_batch, r_one)


@pytest.mark.parametrize("S,n,B,expect", [(40, 64, 5, mcf.GWTF_PASS_GRID), (33, 17, 2, mcf.GWTF_PASS_GRID),
                                         (64, 40, 32, mcf.GWTF_PASS_GRID), (36, 32, 200, mcf.GWTF_PASS_LDS)])
def test_long_narrow_pipelines(S, n, B, expect):
    """More stages than the register pass holds, 16 < n <= 64: a batch that
    needs at most eight grid launches runs on the grid pass (one workgroup
    per stage), a larger one on the LDS pass (one workgroup per instance)."""
    batch = W.random_small(B, S, n, seed=53, cap_hi=5, cost_hi=300, supply_hi=2 * n, holes=0.1, zero_cap=0.1)
    say("long narrow", S, n, B)
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch), certify=[0, B - 1])
    assert (g["passes"] == expect).all(), np.bincount(g["passes"])


@pytest.mark.parametrize("S,n,cost_hi", [(3, 200, 0), (6, 130, 1), (12, 300, 2), (4, 512, 3)])
def test_grid_pass_tied_exits(S, n, cost_hi):
    """Costs drawn from a handful of values make many exits of the last
    stage reach the sink at the same label: the grid pass augments them along
    their tree paths without a new search while their bottleneck is positive,
    and skips those whose path the previous one saturated."""
    batch = W.random_small(2, S, n, seed=31, cap_hi=3, cost_hi=cost_hi, supply_hi=80)
    for a in (batch.node_cost, batch.arc_cost, batch.src_cost, batch.snk_cost):
        a += 1  # every cost in [1, cost_hi + 1]: no free path, many equal ones
    say("grid pass ties", S, n, cost_hi)
    g = gpu_solve(batch, stats=True)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"] == mcf.GWTF_PASS_GRID).all()


def test_grid_pass_wide_labels():
    """Every cost between 55,000 and 65,000 on a 48-stage chain: shortest
    path labels pass 2^22 - 2^16, where the grid pass's packed 32-bit keys
    (label << 9 | row) stop, so its link sweep takes the exact 64-bit keys."""
    batch = W.random_small(2, 48, 80, seed=41, cap_hi=3, cost_hi=10000, supply_hi=40)
    for a in (batch.node_cost, batch.arc_cost, batch.src_cost, batch.snk_cost):
        a[a >= 0] += 55000
    say("grid pass wide labels")
    g = gpu_solve(batch)
    ref = oracle.solve(batch)
    compare(batch, g, ref)
    assert (g["passes"] == mcf.GWTF_PASS_GRID).all()
    assert (ref["F"] > 0).all() and (ref["cost"] // ref["F"] > (1 << 22)).all()


def test_grid_pass_routing_and_status():
    """At n = 512 a workgroup's LDS holds about 1400 flow-list slots: an
    instance with capacities of 64 reserves 128 * 64 and moves to the global
    pass, as does one with a link cost above 16 bits; bad input and label
    overflow are reported by the grid pass itself."""
    batch = W.random_small(6, 3, 512, seed=29, cap_hi=8, cost_hi=900, supply_hi=600, holes=0.05,
                           zero_cap=0.05)
    batch.node_cap[1] = 64
    batch.supply[1] = 600
    batch.arc_cost[2, 1, 7, 9] = 70000
    batch.node_cap[3, 2, 5] = -1
    batch.node_cost[4, 0, 3] = 2 ** 28
    say("grid routing")
    g = gpu_solve(batch)
    assert g["status"].tolist() == [0, 0, 0, 1, 2, 0]
    assert g["passes"].tolist() == [3, 4, 4, 3, 3, 3]
    assert (g["F"][3:5] == 0).all() and (g["cost"][3:5] == 0).all()
    keep = [0, 1, 2, 5]
    ref = oracle.solve(batch.subset(keep))
    assert (g["F"][keep] == ref["F"]).all() and (g["cost"][keep] == ref["cost"]).all()
    for b in keep:
        C.certify(batch, b, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                  g["src_flow"][b], g["snk_flow"][b], g["potential"][b])


@pytest.mark.parametrize("S,n,B,holes,zero", [
    (1, 1, 5, 0.0, 0.0), (2, 16, 7, 0.2, 0.1), (8, 16, 33, 0.1, 0.1), (8, 13, 64, 0.0, 0.0),
    (5, 9, 10, 0.3, 0.2), (3, 4, 1, 0.0, 0.0), (7, 11, 6, 0.0, 0.3),
    (8, 8, 37, 0.2, 0.1), (6, 7, 9, 0.0, 0.2), (4, 2, 13, 0.3, 0.0), (8, 5, 70, 0.1, 0.1),
])
def test_packed_pass_shapes(S, n, B, holes, zero):
    """Shapes served by the packed pass (S <= 8, n <= 16) in small batches
    (one instance per wave), missing links, deleted nodes."""
    batch = W.random_small(B, S, n, seed=31, cap_hi=9, cost_hi=400, supply_hi=4 * n + 8,
                           holes=holes, zero_cap=zero)
    say("packed", S, n, B)
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"] == mcf.GWTF_PASS_PACKED).all()


@pytest.mark.parametrize("S,n,B", [
    (4, 6, 512), (4, 6, 513), (4, 6, 1024), (4, 6, 1025), (4, 6, 2040), (4, 6, 2041), (3, 12, 1100),
])
def test_packed_pass_instances_per_wave(S, n, B):
    """Every launch shape of the packed pass at its batch-size boundaries:
    one instance per wave up to 512 instances, two up to 1,024, four above
    (n > 8, or up to 2,040 instances), eight per wave from 2,041 (n <= 8),
    with the last wave partly empty."""
    batch = W.random_small(B, S, n, seed=43, cap_hi=9, cost_hi=400, supply_hi=4 * n + 8, holes=0.1, zero_cap=0.1)
    say("packed per wave", S, n, B)
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch), certify=[0, 1, B // 2, B - 2, B - 1])
    assert (g["passes"] == mcf.GWTF_PASS_PACKED).all()


def test_packed_pass_routing_and_status():
    """Instances outside the packed bounds (supply above 255, a cost above
    2047) move to the global pass; bad input and label overflow are reported
    by the packed pass itself."""
    batch = W.random_small(9, 4, 8, seed=37, cap_hi=9, cost_hi=400, supply_hi=40)
    batch.supply[1] = 256
    batch.arc_cost[2, 1, 3, 4] = 2048
    batch.node_cost[3, 2, 2] = 5000
    batch.src_cost[4, 0] = 3000
    batch.node_cap[5, 1, 1] = -3
    batch.node_cost[6, 0, 0] = 2 ** 27    # (2Sn+3) * max cost >= 2^29
    say("packed routing")
    g = gpu_solve(batch)
    assert g["status"].tolist() == [0, 0, 0, 0, 0, 1, 2, 0, 0]
    assert g["passes"].tolist() == [5, 4, 4, 4, 4, 5, 5, 5, 5]
    keep = [0, 1, 2, 3, 4, 7, 8]
    ref = oracle.solve(batch.subset(keep))
    assert (g["F"][keep] == ref["F"]).all() and (g["cost"][keep] == ref["cost"]).all()
    for b in keep:
        C.certify(batch, b, int(g["F"][b]), int(g["cost"][b]), g["node_flow"][b], g["arc_flow"][b],
                  g["src_flow"][b], g["snk_flow"][b], g["potential"][b])


def test_packed_pass_bounds():
    """Supply 255 and a cost of 2047 are the largest the packed pass keeps
    (flows in 8 bits, costs shifted by 5 in 16 bits); parity at the bounds."""
    batch = W.random_small(12, 6, 10, seed=41, cap_hi=60, cost_hi=2047, supply_hi=255)
    batch.supply[:] = 255
    batch.node_cost[:, 0, 0] = 2047
    batch.arc_cost[:, 2, 3, 4] = 2047
    batch.src_cost[:, 1] = 2047
    say("packed bounds")
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"] == mcf.GWTF_PASS_PACKED).all()


def test_lists_outgrow_lds_use_fallback():
    """Capacities of 64 make every exit vertex reserve 64 flow-list slots,
    more than LDS holds at this shape, so the global-memory pass runs."""
    batch = W.config4(3)
    batch.node_cap[:] = 64
    batch.supply[:] = 150
    say("fallback c4-shape")
    g = gpu_solve(batch, stats=True)
    compare(batch, g, oracle.solve(batch))


def test_paper_flow_test_shapes():
    for setting in (1, 2, 3, 4):
        batch = W.paper_flow_test(setting, B=32)
        say("paper setting", setting)
        compare(batch, gpu_solve(batch), oracle.solve(batch))


def test_edge_cases():
    batch = W.config1(8)
    batch.supply[0] = 0
    batch.node_cap[1, 2] = 0              # stage 2 deleted -> F = 0
    batch.node_cap[2] = 0                 # everything deleted
    batch.supply[3] = 1
    batch.supply[4] = 2_000_000_000       # huge supply: stage capacity binds
    batch.node_cost[5] = 0
    batch.arc_cost[5] = 0                 # all-zero costs: ties everywhere
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert g["F"][0] == 0 and g["F"][1] == 0 and g["F"][2] == 0


def test_bad_input_and_overflow_status():
    batch = W.config1(6)
    batch.node_cap[0, 0, 0] = -1
    batch.arc_cost[1, 0, 0, 0] = -2
    batch.supply[2] = -5
    batch.src_cost[3, 0] = -1
    batch.node_cost[4, 1, 1] = 2 ** 28    # (2Sn+3) * max cost >= 2^29
    g = gpu_solve(batch)
    assert g["status"].tolist() == [1, 1, 1, 1, 2, 0]
    assert (g["F"][:5] == 0).all() and (g["cost"][:5] == 0).all()
    ref = oracle.solve(batch.subset([5]))
    assert g["F"][5] == ref["F"][0] and g["cost"][5] == ref["cost"][0]


def test_deterministic_flows():
    batch = W.config2(512)
    a = gpu_solve(batch)
    b = gpu_solve(batch)
    for key in ("F", "cost", "node_flow", "arc_flow", "potential"):
        assert (a[key] == b[key]).all(), key


def test_api_errors():
    import torch
    from paper_2509_21221_amd import mcf

    s = mcf.Solver(4, 4, 8)
    with pytest.raises(mcf.GwtfError) as e:
        s.flows(0, 1)
    assert e.value.code == mcf.GWTF_ERR_NOT_SOLVED
    batch = W.config1(4)
    gpu_solve(batch, flows=False, solver=s)
    with pytest.raises(mcf.GwtfError) as e:
        s.flows(2, 3)
    assert e.value.code == mcf.GWTF_ERR_RANGE
    dev = torch.device("cuda", 0)
    z = lambda *shape: torch.zeros(shape, dtype=torch.int32, device=dev)
    out = [torch.zeros(9, dtype=torch.int64, device=dev)] * 2 + [z(9)]
    with pytest.raises(mcf.GwtfError) as e:
        mcf.gwtf_mcf_solve_batch(s.handle, 9, z(9, 4, 4).data_ptr(), z(9, 4, 4).data_ptr(),
                                 z(9, 3, 4, 4).data_ptr(), 0, 0, z(9).data_ptr(), out[0].data_ptr(),
                                 out[1].data_ptr(), out[2].data_ptr())
    assert e.value.code == mcf.GWTF_ERR_INVALID_ARG
    with pytest.raises(mcf.GwtfError) as e:
        mcf.gwtf_mcf_solve_batch(s.handle, 2, z(2, 4, 4).data_ptr(), z(2, 4, 4).data_ptr(), 0, 0, 0,
                                 z(2).data_ptr(), out[0].data_ptr(), out[1].data_ptr(),
                                 out[2].data_ptr())
    assert e.value.code == mcf.GWTF_ERR_INVALID_ARG
    s.close()


@pytest.mark.parametrize("S,n,holes,zero", [
    (1, 40, 0.0, 0.1), (2, 20, 0.2, 0.0), (31, 50, 0.1, 0.05), (32, 64, 0.0, 0.0), (7, 64, 0.3, 0.2),
])
def test_register_pass_shapes(S, n, holes, zero):
    """Shapes served by the register-resident pass (S <= 32, 16 < n <= 64)."""
    batch = W.random_small(12, S, n, seed=19, cap_hi=6, cost_hi=250, supply_hi=4 * n,
                           holes=holes, zero_cap=zero)
    say("register pass", S, n)
    compare(batch, gpu_solve(batch), oracle.solve(batch))


def test_register_pass_routes_wide_costs():
    """Link costs above 16 bits send an instance to the fallback pass; the
    others in the same batch stay on the register pass."""
    batch = W.config4(4)
    batch.arc_cost[1, 3, 5, 7] = 70000
    batch.arc_cost[2, 0, 0, :] = 65535
    say("register pass routing")
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))


@pytest.mark.parametrize("S,n,holes", [(3, 40, 0.0), (32, 64, 0.0), (9, 64, 0.2)])
def test_register_pass_unscaled_costs(S, n, holes):
    """Costs above 1023 do not fit the keyed relaxation (labels times 64 plus
    the row in 32 bits, costs times 64 in 16): the unscaled variant of the
    register pass solves these instances."""
    batch = W.random_small(8, S, n, seed=43, cap_hi=6, cost_hi=6000, supply_hi=4 * n, holes=holes)
    say("register pass unscaled", S, n)
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"] == mcf.GWTF_PASS_REGISTER).all()


def test_register_pass_keyed_and_unscaled_in_one_batch():
    """One batch split over both variants of the register pass and the
    fallback: the keyed variant keeps instances whose costs are at most 1023
    (a link, a compute and a data-node cost at exactly 1023 included)."""
    batch = W.config4(8)
    batch.arc_cost[1, 3, 5, 7] = 1023
    batch.node_cost[1, 4, 9] = 1023
    batch.snk_cost[1, 2] = 1023
    batch.arc_cost[2, 0, 0, 1] = 1024   # link cost over the keyed limit
    batch.node_cost[4, 31, 63] = 4000   # compute cost over it
    batch.src_cost[5, 0] = 1500         # data-node cost over it
    batch.arc_cost[6, 7, 2, 2] = 70000  # over 16 bits: the fallback pass
    say("register pass keyed / unscaled / fallback")
    g = gpu_solve(batch)
    compare(batch, g, oracle.solve(batch))
    assert (g["passes"][[0, 1, 2, 3, 4, 5, 7]] == mcf.GWTF_PASS_REGISTER).all()
    assert g["passes"][6] != mcf.GWTF_PASS_REGISTER


def test_config5_full_against_stored_oracle():
    """The single 64 x 512 instance: (F, cost) equal to the stored oracle
    optimum, the closed-form flow value, and the returned flow certified."""
    gold = json.load(open(os.path.join(GOLDEN, "c5_oracle.json")))
    batch = W.config5()
    assert _digest(batch) == gold["input_sha256"], "generator no longer reproduces the stored inputs"
    say("c5 (about a minute)")
    g = gpu_solve(batch)
    assert g["status"][0] == 0 and g["passes"][0] == mcf.GWTF_PASS_GRID
    assert int(g["F"][0]) == gold["F"][0] == C.closed_form_value(batch, 0)
    assert int(g["cost"][0]) == gold["cost"][0]
    C.certify(batch, 0, int(g["F"][0]), int(g["cost"][0]), g["node_flow"][0], g["arc_flow"][0],
              g["src_flow"][0], g["snk_flow"][0], g["potential"][0])
