"""Write tests/golden/oracle_digests.json: CPU-oracle outputs of workloads too
large to re-run inside a GPU test (the 100000-request single instance).

Only the oracle and the seeded generator are called.  Run from the repo root:
    python tests/golden/make_oracle_digests.py
"""
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2508_14544_amd import workloads as W  # noqa: E402


def digest(name, algos):
    batch = W.generate(name, 0)
    inst = batch.instance(0)
    out = {}
    for a in algos:
        t0 = time.time()
        r = O.simulate(inst, O.ALGOS[a], batch.M)
        out[a] = {
            "status": r["status"], "tel": r["tel"], "makespan": r["makespan"],
            "request_steps": r["request_steps"], "total_evictions": r["total_evictions"],
            "completion_sha256": hashlib.sha256(r["completion"].astype("<i4").tobytes()).hexdigest(),
            "evictions_sha256": hashlib.sha256(r["evictions"].astype("<i4").tobytes()).hexdigest(),
            "oracle_seconds": round(time.time() - t0, 1),
        }
        print(name, a, out[a], flush=True)
    return out


if __name__ == "__main__":
    res = {"_note": "written by tests/golden/make_oracle_digests.py from the CPU oracle (seed 0)",
           "single_n100000_m1048576": digest("single_n100000_m1048576", ["amin", "amax"])}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_digests.json")
    with open(path, "w") as f:
        json.dump(res, f, indent=1)
    print("wrote", path)
