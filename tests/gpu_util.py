"""Helpers for the GPU tests: run a workloads.Batch through the C ABI."""
import numpy as np


def have_gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def gpu_solve(batch, flows=True, stats=False, solver=None):
    import torch
    from paper_2509_21221_amd.mcf import Solver

    dev = torch.device("cuda", 0)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    own = solver is None
    if own:
        solver = Solver(batch.S, batch.n, batch.B)
    F, cost, status = solver.solve(t(batch.node_cap), t(batch.node_cost),
                                   t(batch.arc_cost) if batch.S > 1 else None, t(batch.supply),
                                   t(batch.src_cost), t(batch.snk_cost))
    out = {}
    if flows:
        out.update({k: v.cpu().numpy() for k, v in solver.flows().items()})
    if stats:
        out["stats"] = solver.stats().cpu().numpy()
    out["passes"] = solver.passes().cpu().numpy()
    torch.cuda.synchronize()
    out.update(F=F.cpu().numpy(), cost=cost.cpu().numpy(), status=status.cpu().numpy())
    if own:
        solver.close()
    return out
