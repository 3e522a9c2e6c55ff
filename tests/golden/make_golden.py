"""Write the oracle's (F, cost) for the large presets into tests/golden/.

Calls only the CPU oracle and the seeded workload generator.  Usage:

    python tests/golden/make_golden.py 4        # 256 instances, ~1 min
    python tests/golden/make_golden.py 5        # one 64 x 512 instance, long

The stored input digest lets a test detect a generator that no longer
reproduces the same instances.
"""
import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2509_21221_amd import workloads as W  # noqa: E402


def digest(batch):
    h = hashlib.sha256()
    for key in ("node_cap", "node_cost", "arc_cost", "src_cost", "snk_cost", "supply"):
        h.update(getattr(batch, key).tobytes())
    return h.hexdigest()


def main(cfg):
    batch = W.CONFIGS[cfg]()
    t0 = time.time()
    r = oracle.solve(batch, flows=False, potentials=False)
    dt = time.time() - t0
    assert (r["status"] == 0).all()
    out = {
        "citation": "Optimum of Eq. 2 (Sec. V-A) computed by the CPU oracle on the seeded preset; "
                    "no paper value exists for these synthetic instances.",
        "preset": cfg, "B": batch.B, "S": batch.S, "n": batch.n,
        "input_sha256": digest(batch),
        "F": r["F"].tolist(), "cost": r["cost"].tolist(),
        "augmentations": r["augmentations"].tolist(),
        "oracle_seconds": round(dt, 2), "oracle_threads": r["threads"],
    }
    with open(os.path.join(HERE, f"c{cfg}_oracle.json"), "w") as f:
        json.dump(out, f)
    print(f"c{cfg}: {batch.B} instances in {dt:.1f}s on {r['threads']} threads")


if __name__ == "__main__":
    for a in sys.argv[1:]:
        main(int(a))
