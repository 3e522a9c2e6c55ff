"""GPU test of gwtf_mcf_solve_batch_noalloc, the solve whose workspace lives in
the library's fixed per-device array instead of allocated memory.

Each case solves a batch with the ordinary handle entry point
(gwtf_mcf_solve_batch) and with the no-allocation one on the same device
inputs, twice in a row with the second batch smaller, and requires identical
(F, cost, status) on every instance; the ordinary results are in turn checked
against the CPU oracle.  The shapes cover the packed pass (with instances it
hands to the fallback pass), the pipelined register pass and the grid pass.
A batch whose workspace exceeds the array is refused with nothing enqueued.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2509_21221_amd import mcf
from paper_2509_21221_amd import workloads as W

pytestmark = pytest.mark.gpu


def _dev(batch):
    import torch

    dev = torch.device("cuda", 0)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    return {"node_cap": t(batch.node_cap), "node_cost": t(batch.node_cost),
            "arc_cost": t(batch.arc_cost) if batch.S > 1 else None, "src_cost": t(batch.src_cost),
            "snk_cost": t(batch.snk_cost), "supply": t(batch.supply)}


def _noalloc(batch, d, max_batch):
    import torch

    dev = torch.device("cuda", 0)
    B = batch.B
    F = torch.full((B,), -7, dtype=torch.int64, device=dev)
    cost = torch.full((B,), -7, dtype=torch.int64, device=dev)
    status = torch.full((B,), -7, dtype=torch.int32, device=dev)
    ptr = lambda x: x.data_ptr() if x is not None else 0
    mcf.gwtf_mcf_solve_batch_noalloc(batch.S, batch.n, max_batch, 0, torch.cuda.current_stream().cuda_stream, B,
                                     ptr(d["node_cap"]), ptr(d["node_cost"]), ptr(d["arc_cost"]),
                                     ptr(d["src_cost"]), ptr(d["snk_cost"]), ptr(d["supply"]),
                                     F.data_ptr(), cost.data_ptr(), status.data_ptr())
    return F, cost, status


def _handle(batch, d):
    from paper_2509_21221_amd.mcf import Solver

    with Solver(batch.S, batch.n, batch.B) as s:
        out = s.solve(d["node_cap"], d["node_cost"], d["arc_cost"], d["supply"], d["src_cost"], d["snk_cost"])
        s.torch.cuda.synchronize()
        return [x.cpu().numpy() for x in out]


def _check_pair(name, first, second, max_batch):
    import torch

    for step, batch in (("first", first), ("second", second)):
        print(f"no-alloc {name} {step}: S={batch.S} n={batch.n} B={batch.B}", flush=True)
        sys.stdout.flush()
        d = _dev(batch)
        F, cost, status = [x.cpu().numpy() for x in _noalloc(batch, d, max_batch)]
        torch.cuda.synchronize()
        hF, hcost, hstatus = _handle(batch, d)
        assert np.array_equal(F, hF) and np.array_equal(cost, hcost) and np.array_equal(status, hstatus), \
            f"{name} {step}: no-alloc results differ from gwtf_mcf_solve_batch"
        ref = oracle.solve(batch, flows=False, potentials=False)
        assert np.array_equal(hF, ref["F"]) and np.array_equal(hcost, ref["cost"]) \
            and np.array_equal(hstatus, ref["status"]), f"{name} {step}: differs from the oracle"


def test_noalloc_packed_and_fallback():
    """8 x 8 batches on the packed pass, with instances whose link costs
    exceed the packed bounds (solved by the fallback pass)."""
    first = W.concat([W.config2(1800), W.random_small(200, 8, 8, seed=31, cost_hi=2600, supply_hi=40)])
    second = W.concat([W.config2(500, first=4000), W.random_small(40, 8, 8, seed=32, cost_hi=2600, supply_hi=40)])
    _check_pair("packed", first, second, max_batch=2000)


def test_noalloc_pipelined():
    """32 x 64 instances on the stage-pipelined register pass."""
    _check_pair("pipelined", W.config4(6), W.config4(3, first=40), max_batch=6)


def test_noalloc_grid():
    """Instances wider than 64 nodes on the grid-cooperative pass."""
    first = W.random_small(2, 6, 96, seed=33, cap_hi=4, cost_hi=300, supply_hi=40)
    # second call: one smaller instance, the first's second instance with half
    # of a middle stage deleted and half the supply
    second = first.instance(1)
    second.node_cap[0, 3, ::2] = 0
    second.supply[0] = max(1, int(second.supply[0]) // 2)
    _check_pair("grid", first, second, max_batch=2)


def test_noalloc_refuses_batches_beyond_the_array():
    import torch

    batch = W.config2(7000)
    d = _dev(batch)
    print("no-alloc oversize 8x8 B=7000", flush=True)
    with pytest.raises(mcf.GwtfError) as err:
        _noalloc(batch, d, max_batch=7000)
    assert err.value.code == mcf.GWTF_ERR_INVALID_ARG
    assert "scratch" in str(err.value)
    torch.cuda.synchronize()
    # nothing was enqueued and the array still serves a batch that fits
    small = batch.subset(range(64))
    F, cost, status = [x.cpu().numpy() for x in _noalloc(small, _dev(small), max_batch=64)]
    ref = oracle.solve(small, flows=False, potentials=False)
    assert np.array_equal(F, ref["F"]) and np.array_equal(cost, ref["cost"]) and (status == 0).all()
