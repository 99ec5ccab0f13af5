"""GPU parity on every instance of the named workloads (the five configurations
of the benchmark set and their policies), in the launch configuration the
benchmark uses (one sched_simulate call over the whole batch).

The expected outputs are the CPU oracle's, stored as block digests by
tests/golden/make_oracle_digests.py (format: tests/digests.py): every
per-request completion step and cancellation count and every per-instance
total is compared bit for bit through its block's digest.  A mismatch names
the first differing instance, found by re-running the oracle on its block.
"""
import json
import os

import numpy as np
import pytest

import digests as D
from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, gpu_run, _say  # noqa: F401 (B is a fixture)

pytestmark = pytest.mark.gpu

PATH = os.path.join(os.path.dirname(__file__), "golden", "oracle_digests.json")
DIG = json.load(open(PATH)) if os.path.exists(PATH) else {"workloads": {}}
CASES = [(w, a) for w, e in DIG["workloads"].items() for a in e["algos"]]
CHUNK = 2048  # the chunking of the stored input digests

_batches = {}


def _batch(name, with_upper):
    """The whole workload, generated in chunks (bounded host memory) and kept
    for the module's other policies."""
    key = (name, with_upper)
    if key not in _batches:
        _batches.clear()
        w = W.WORKLOADS[name]
        parts = [W.generate(name, 0, instance_ids=range(c0, min(w.num_instances, c0 + CHUNK)), with_upper=with_upper)
                 for c0 in range(0, w.num_instances, CHUNK)]
        cat = lambda f: (None if getattr(parts[0], f) is None
                         else np.concatenate([getattr(p, f) for p in parts]).astype(np.int32))
        offsets = np.arange(w.num_instances + 1, dtype=np.int64) * w.n
        whole = W.Instances(name, w.M, offsets, cat("arrival"), cat("prompt"), cat("output"), cat("lower"),
                            cat("upper"), np.arange(w.num_instances, dtype=np.int64), {"seed": 0})
        import hashlib
        h = hashlib.sha256()
        for p in parts:
            h.update(D.inputs_digest(p).encode())
        _batches[key] = (whole, h.hexdigest()[:32])
    return _batches[key]


def _first_difference(batch, g, algo, block):
    """Re-run the oracle on one block and describe the first differing instance."""
    k0, k1 = block * D.BLOCK, min(batch.num_instances, (block + 1) * D.BLOCK)
    ref = O.simulate_batch(batch, O.ALGOS[algo], instances=range(k0, k1))
    pos = 0
    for j, k in enumerate(range(k0, k1)):
        n = int(batch.offsets[k + 1] - batch.offsets[k])
        for f in D.FIELDS:
            if int(g[f][k]) != int(ref[f][j]):
                return f"instance {k}: {f} gpu {int(g[f][k])} oracle {int(ref[f][j])}"
        lo = int(batch.offsets[k])
        for f in ("completion", "evictions"):
            a, r = g[f][lo:lo + n], ref[f][pos:pos + n]
            if not np.array_equal(a, r):
                i = int(np.flatnonzero(a != r)[0])
                return f"instance {k} request {i}: {f} gpu {int(a[i])} oracle {int(r[i])}"
        pos += n
    return f"block {block}: digests differ but the oracle re-run agrees (stale digest file?)"


@pytest.mark.timeout(900)
@pytest.mark.parametrize("workload,algo", CASES, ids=[f"{w}-{a}" for w, a in CASES])
def test_every_instance_matches_oracle(B, workload, algo):
    entry = DIG["workloads"][workload]
    d = entry["algos"][algo]
    batch, inputs_sha = _batch(workload, entry["with_upper"])
    assert inputs_sha == d["inputs_sha"], "the generator no longer produces the inputs the oracle saw"
    g = gpu_run(B, batch, O.ALGOS[algo], pass_upper=entry["with_upper"])
    # every instance completes (the stored oracle run says so too)
    assert d["totals"]["status_counts"] == {"0": batch.num_instances}
    assert (g["status"] == 0).all(), f"statuses {dict(zip(*np.unique(g['status'], return_counts=True)))}"
    assert D.totals(g) == d["totals"]
    got = D.block_digests(batch.offsets, g)
    bad = [i for i, (x, y) in enumerate(zip(got, d["blocks"])) if x != y]
    assert len(got) == len(d["blocks"])
    if bad:
        pytest.fail(f"{len(bad)} of {len(got)} blocks differ; first: {_first_difference(batch, g, algo, bad[0])}")
    _say(f"[digest] {workload} {algo}: {batch.num_instances} instances bit-exact")


# the large single instance simulated by a workgroup of 2 or 4 waves from the
# start (the running set split over the waves): the same bits as one wave's
WG_CASES = [(w, a, ww) for (w, a) in CASES if w == "single_n100000_m1048576" and a in ("amax", "amin", "hsf")
            for ww in (2, 4)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("workload,algo,ww", WG_CASES, ids=[f"{w}-{a}-w{ww}" for w, a, ww in WG_CASES])
def test_workgroup_matches_oracle(B, workload, algo, ww):
    entry = DIG["workloads"][workload]
    d = entry["algos"][algo]
    batch, inputs_sha = _batch(workload, entry["with_upper"])
    assert inputs_sha == d["inputs_sha"]
    g = gpu_run(B, batch, O.ALGOS[algo], pass_upper=entry["with_upper"], workgroup_waves=ww)
    assert (g["status"] == 0).all()
    assert D.totals(g) == d["totals"]
    assert D.block_digests(batch.offsets, g) == d["blocks"]
    _say(f"[digest] {workload} {algo} workgroup of {ww}: bit-exact")
