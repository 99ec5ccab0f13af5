"""Write tests/golden/oracle_digests.json: CPU-oracle outputs of every instance
of the named workloads, as block digests (format: tests/digests.py).

Only the oracle and the seeded generator are called.  Run from the repo root:
    python tests/golden/make_oracle_digests.py [workload[:algo,...] ...] [--threads T]
With no arguments every (workload, policy) pair below is (re)computed; the
file is rewritten after each pair, so an interrupted run keeps what finished.
The whole set takes about 9 hours of CPU time (the 65536-instance sweep
under A_min is most of it).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

from oracle import oracle as O  # noqa: E402
from paper_2508_14544_amd import workloads as W  # noqa: E402
import digests as D  # noqa: E402

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_digests.json")

# (workload, policies, whether A_max's upper bounds are passed)
PLAN = [
    ("single_n200_m512", ["amin", "amax", "hsf"], True),
    ("batch4096_n1000_m16384", ["amin", "amax", "hsf", "aell", "adaptive"], True),
    ("single_n100000_m1048576", ["amin", "amax", "hsf"], True),
    ("online1024_n10000_m65536", ["amin", "amax", "hsf", "aell"], True),
    # A_min is given only the lower bounds here (H-SF reads neither bound)
    ("sweep65536_n2000_m32768", ["amin", "hsf"], False),
    # the two-point workload of Section 5.1 (A_l and the adaptive switch)
    ("twopoint4096_n1000_m16384", ["aell", "adaptive", "amin", "hsf"], True),
]
CHUNK = 2048  # instances generated and simulated at once (a multiple of the digest block)


def oracle_source_hash() -> str:
    h = hashlib.sha256()
    for p in ("oracle/sched_oracle.c", "oracle/sched_oracle.h"):
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


def run(name, algo, with_upper, threads):
    w = W.WORKLOADS[name]
    blocks, parts = [], []
    t0 = time.time()
    inputs = hashlib.sha256()
    for c0 in range(0, w.num_instances, CHUNK):
        ids = range(c0, min(w.num_instances, c0 + CHUNK))
        batch = W.generate(name, 0, instance_ids=ids, with_upper=with_upper)
        inputs.update(D.inputs_digest(batch).encode())
        out = O.simulate_batch(batch, O.ALGOS[algo], threads=threads)
        blocks += D.block_digests(batch.offsets, out, first=c0)
        parts.append({f: out[f] for f in D.FIELDS})
        print(f"  {name} {algo}: {ids.stop}/{w.num_instances} instances, {time.time() - t0:.0f} s", flush=True)
    import numpy as np
    merged = {f: np.concatenate([p[f] for p in parts]) for f in D.FIELDS}
    return {
        "inputs_sha": inputs.hexdigest()[:32],
        "totals": D.totals(merged),
        "blocks": blocks,
        "oracle_seconds": round(time.time() - t0, 1),
        "oracle_threads": threads,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("only", nargs="*", help="workload or workload:algo1,algo2")
    ap.add_argument("--threads", type=int, default=len(os.sched_getaffinity(0)))
    args = ap.parse_args()
    want = {}
    for spec in args.only:
        nm, _, al = spec.partition(":")
        want[nm] = al.split(",") if al else None
    data = json.load(open(PATH)) if os.path.exists(PATH) else {}
    if data.get("format") != 2:
        data = {}
    data.update({
        "_note": "written by tests/golden/make_oracle_digests.py from the CPU oracle (seed 0); "
                 "block digests as defined in tests/digests.py",
        "format": 2,
        "block": D.BLOCK,
        "oracle_source_sha16": oracle_source_hash(),
    })
    data.setdefault("workloads", {})
    for name, algos, with_upper in PLAN:
        if want and name not in want:
            continue
        for algo in algos:
            if want and want[name] and algo not in want[name]:
                continue
            print(f"{name} {algo} ...", flush=True)
            entry = data["workloads"].setdefault(name, {"with_upper": with_upper, "algos": {}})
            entry["algos"][algo] = run(name, algo, with_upper, args.threads)
            print(f"{name} {algo}: {entry['algos'][algo]['totals']}", flush=True)
            tmp = PATH + ".tmp"
            with open(tmp, "w") as f:
                json.dump(data, f, indent=1)
            os.replace(tmp, PATH)
    print("wrote", PATH)


if __name__ == "__main__":
    main()
