"""Write tests/golden/opt_pool_tiny8.json: the oracle's hindsight optimum
(exhaustive search over start steps, equations (1) and (3)) of a few
eight-request instances of the tiny competitive-ratio workload (seed 0, 65536
instances, s ~ U{0..3}, o ~ U{1..6}, M = 12, random intervals), chosen among
those whose GPU branch and bound needs more nodes than a one-wave search is
given at first, so that their optimum comes from the device-wide second
search.  The last one is the workload's hardest (about 3.4e7 nodes).

Only the oracle and the seeded generator are called.  Run from the repo root:
    python tests/golden/make_opt_pool.py [--threads T]
It takes a few minutes on eight threads (one to three minutes per instance).
"""
import argparse
import json
import os
import sys
from concurrent.futures import ProcessPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2508_14544_amd import workloads as W  # noqa: E402

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "opt_pool_tiny8.json")
SEED, K, N, M, O_MAX = 0, 65536, 8, 12, 6
INDICES = [2967, 17800, 18140, 24577, 26321, 28200, 37071, 41124, 49227, 52507, 52969, 55289, 58671]


def _one(k):
    d = W.tiny(SEED, K, N, M=M, o_max=O_MAX, alpha=None).instance(k)
    n = len(d["output"])
    inst = {f: [int(x) for x in (d[f] if d[f] is not None else [0] * n)] for f in ("arrival", "prompt", "output")}
    return k, inst, O.opt_tel(inst, M)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=min(8, len(os.sched_getaffinity(0))))
    a = ap.parse_args()
    with ProcessPoolExecutor(a.threads) as ex:
        rows = list(ex.map(_one, INDICES))
    out = {"workload": f"tiny seed {SEED}: {K} instances x {N} requests, s ~ U{{0..3}}, o ~ U{{1..{O_MAX}}}, "
                       f"random intervals, M = {M}",
           "M": M,
           "instances": [{"index": k, **inst, "opt_tel": int(v)} for k, inst, v in rows]}
    json.dump(out, open(PATH, "w"), indent=1)
    print("wrote", PATH, [(k, v) for k, _, v in rows])


if __name__ == "__main__":
    main()
