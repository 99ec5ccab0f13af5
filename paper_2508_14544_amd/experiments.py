"""Analogue of the paper's numerical experiments (Section 6), in unit time steps.

For every prediction setting (Experiment 1: intervals [1, 1000]; Experiment 2:
buckets of 100; Experiment 3: [(1-x) o, (1+x) o] for x in 0.10, 0.95, 0.99)
and instance size n in 200, 400, ..., 2000, it simulates `replicates`
instances with A_max, A_min, H-SF, A_l and the adaptive A_min/A_l switch on
the GPU and reports the average end-to-end latency (total latency / n) in
steps, averaged over the replicates.  Inputs come from
``workloads.experiment``; the paper's batch-time model (Section 6: a linear
regression predictor of batch time for LLaMA2-70B on two linked A100 GPUs)
and its data set are not used: every step costs one unit.

    python -m paper_2508_14544_amd.experiments [--replicates 64] [--json out.json]

The GPU results of these cells are checked against the CPU oracle by
``tests/test_gpu_experiments.py``.
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import binding as B
from . import workloads as W

POLICIES = ("amax", "amin", "hsf", "aell", "adaptive")
SIZES = tuple(range(200, 2001, 200))


def run(replicates: int = 64, sizes=SIZES, settings=W.EXP_SETTINGS, policies=POLICIES, seed: int = 0,
        log=None):
    import torch
    B.load_library()
    rows = []
    gpu_ms = 0.0
    request_steps = 0
    for setting in settings:
        for n in sizes:
            batch = W.experiment(setting, n, replicates, seed)
            db = B.to_device(batch)
            for pol in policies:
                out = B.alloc_results(db)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                B.simulate_into(db, B.ALGOS[pol], out)
                e1.record()
                torch.cuda.synchronize()
                gpu_ms += e0.elapsed_time(e1)
                g = {k: v.cpu().numpy() for k, v in out.items() if v is not None}
                if not (g["status"] == 0).all():
                    raise RuntimeError(f"{setting} n={n} {pol}: status {np.unique(g['status'])}")
                request_steps += int(g["request_steps"].sum())
                lat = g["tel"] / n
                row = {"setting": setting, "n": n, "policy": pol, "avg_latency": float(lat.mean()),
                       "std_over_replicates": float(lat.std()), "replicates": replicates}
                if pol == "adaptive":
                    row["a_l_instances"] = int((g["algo_used"] == B.AELL).sum())
                rows.append(row)
                if log:
                    log(f"{setting} n={n} {pol}: {row['avg_latency']:.1f}")
    hs = {(r["setting"], r["n"]): r["avg_latency"] for r in rows if r["policy"] == "hsf"}
    for r in rows:
        r["ratio_to_hsf"] = r["avg_latency"] / hs[(r["setting"], r["n"])] if (r["setting"], r["n"]) in hs else None
    summary = {"gpu_ms": gpu_ms, "request_steps": request_steps,
               "request_steps_per_s": request_steps / (gpu_ms / 1e3) if gpu_ms else None}
    return rows, summary


def cr_study(num_instances: int = 1 << 18, sizes=(4, 6, 8), seed: int = 0, M: int = 12, o_max: int = 6,
             alphas=(None, 1, 2), log=None):
    """Empirical competitive ratios against the hindsight optimum on many tiny
    instances (all requests at step 0): for each size and interval recipe, the
    optimum comes from ``sched_optimum`` and each policy's total latency from
    ``sched_simulate``; reports the largest and the mean ratio per policy."""
    import torch
    from fractions import Fraction
    B.load_library()
    rows = []
    gpu_ms_opt = 0.0
    for n in sizes:
        for al in alphas:
            alpha = None if al is None else Fraction(al)
            batch = W.tiny(seed, num_instances, n, M=M, o_max=o_max, alpha=alpha)
            db = B.to_device(batch)
            hsf = B.simulate(db, B.HSF)   # an achievable total: prunes the search
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            opt = B.optimum(db, upper_bound=hsf["tel"])
            e1.record()
            torch.cuda.synchronize()
            gpu_ms_opt += e0.elapsed_time(e1)
            ot = opt["tel"].cpu().numpy().astype(np.float64)
            ok = opt["status"].cpu().numpy() == 0
            for pol in ("amax", "amin", "hsf", "aell", "adaptive"):
                out = B.simulate(db, B.ALGOS[pol])
                torch.cuda.synchronize()
                tel = out["tel"].cpu().numpy().astype(np.float64)
                good = ok & (out["status"].cpu().numpy() == 0)
                ratio = tel[good] / ot[good]
                rows.append({"n": n, "intervals": "random" if al is None else f"geometric alpha={al}",
                             "policy": pol, "instances": int(good.sum()), "max_ratio": float(ratio.max()),
                             "mean_ratio": float(ratio.mean()),
                             "opt_nodes_mean": float(opt["nodes"].cpu().numpy()[ok].mean())})
                if log:
                    log(f"n={n} alpha={al} {pol}: max {ratio.max():.4f} mean {ratio.mean():.4f}")
    return rows, {"opt_gpu_ms": gpu_ms_opt, "opt_instances": num_instances * len(sizes) * len(alphas)}


def markdown(rows, policies=POLICIES) -> str:
    out = []
    for setting in W.EXP_SETTINGS:
        sel = [r for r in rows if r["setting"] == setting]
        if not sel:
            continue
        out.append(f"\n{setting}: average latency (steps), ratio to H-SF in parentheses\n")
        out.append("| n | " + " | ".join(policies) + " |")
        out.append("|---|" + "---|" * len(policies))
        for n in sorted({r["n"] for r in sel}):
            cells = []
            for p in policies:
                r = [x for x in sel if x["n"] == n and x["policy"] == p]
                cells.append("" if not r else f"{r[0]['avg_latency']:.0f} ({r[0]['ratio_to_hsf']:.2f})")
            out.append(f"| {n} | " + " | ".join(cells) + " |")
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--replicates", type=int, default=64)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--sizes", default=",".join(map(str, SIZES)))
    ap.add_argument("--json", default="")
    ap.add_argument("--cr", action="store_true", help="run the competitive-ratio study on tiny instances instead")
    ap.add_argument("--cr-instances", type=int, default=1 << 18)
    a = ap.parse_args(argv)
    if a.cr:
        rows, summary = cr_study(a.cr_instances, seed=a.seed, log=lambda m: print(m, file=sys.stderr, flush=True))
        print("| n | intervals | policy | instances | max TEL/OPT | mean TEL/OPT |")
        print("|---|---|---|---|---|---|")
        for r in rows:
            print(f"| {r['n']} | {r['intervals']} | {r['policy']} | {r['instances']} | {r['max_ratio']:.4f} | "
                  f"{r['mean_ratio']:.4f} |")
        print(json.dumps(summary))
        if a.json:
            json.dump({"rows": rows, "summary": summary}, open(a.json, "w"), indent=1)
        return
    sizes = tuple(int(x) for x in a.sizes.split(","))
    t0 = time.perf_counter()
    rows, summary = run(a.replicates, sizes=sizes, seed=a.seed,
                        log=lambda m: print(m, file=sys.stderr, flush=True))
    summary["wall_s"] = time.perf_counter() - t0
    print(markdown(rows))
    print(json.dumps(summary))
    if a.json:
        json.dump({"rows": rows, "summary": summary}, open(a.json, "w"), indent=1)


if __name__ == "__main__":
    main()
