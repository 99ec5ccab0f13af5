"""Launch shapes.  A_min batches with more instances than the device holds at
once take their instances in a launch order (the widest gaps between the
lower bounds and the outputs first), batches of at most four instances per CU
run the 256-VGPR bodies, and A_min batches in between may set issue
priorities by class.  The outputs must not depend on any of it: every
instance equals the oracle (Algorithm 2 with equation (2)), invalid and
empty instances keep their statuses, the batch reversed gives the same
outputs per instance, the no-allocation entry point gives the same bits, and
the same instances alone or inside a larger batch give the same outputs under
every policy."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run  # noqa: F401

pytestmark = pytest.mark.gpu

FIELDS = ("status", "tel", "makespan", "request_steps", "total_evictions")


def _many(K=5000):
    # more instances than 16 waves on each of 256 CUs, with a few invalid and
    # empty ones among them
    base = W.random_small(21, K, 14, s_max=4, o_max=10, M=40, arrivals=True)
    insts = [{f: base.instance(k)[f] for f in ("arrival", "prompt", "output", "lower", "upper")} for k in range(K)]
    good = insts[0]
    bad = [dict(good, lower=[x + 100 for x in good["lower"]]),             # l > o
           {"arrival": [], "prompt": [], "output": [], "lower": [], "upper": []},
           {"arrival": [1, 0], "prompt": [1, 1], "output": [2, 2], "lower": [1, 1], "upper": [3, 3]}]  # unsorted
    for j, b in enumerate(bad):
        insts[1000 * (j + 1) + 7] = b
    return W.from_lists(40, insts, name="amin_many_instances")


def test_launch_order_many_instances(B):
    import torch
    batch = _many()
    ref = oracle_run(batch, O.AMIN)
    assert (ref["status"] != 0).sum() >= 2
    g = gpu_run(B, batch, O.AMIN)
    assert_parity(batch, g, ref)
    # the same instances in reverse: the same outputs per instance
    K = batch.num_instances
    rev = batch.subset(list(range(K - 1, -1, -1)))
    gr = gpu_run(B, rev, O.AMIN)
    for f in FIELDS:
        assert np.array_equal(gr[f][::-1], g[f]), f
    # the no-allocation entry point: the same bits, twice, the second batch smaller
    for b in (batch, batch.subset(list(range(4200, 4900)))):
        db = B.to_device(b)
        out = B.alloc_results(db)
        ref_t = B.simulate(db, B.AMIN)
        B.simulate_into(db, B.AMIN, out, no_alloc=True)
        torch.cuda.synchronize()
        for f in ("status", "tel", "makespan", "request_steps", "total_evictions", "completion", "evictions"):
            assert torch.equal(out[f], ref_t[f]), f


@pytest.mark.parametrize("algo", ["amin", "amax", "hsf", "aell", "adaptive", "arandom"])
def test_same_instances_in_every_launch_shape(B, algo):
    # 300 instances of the benchmark batch alone (a batch of at most 4 per CU:
    # the 256-VGPR bodies) and inside the whole 4096-instance batch (the
    # 128-VGPR bodies; A_min with issue-priority classes): the same outputs
    a = O.ALGOS[algo]
    full = W.generate("batch4096_n1000_m16384", 0)
    if algo == "arandom":
        full = W.with_random_order(full, seed=1)   # A_random's per-request order
    ks = list(range(2800, 3100))
    g = gpu_run(B, full, a)
    s = gpu_run(B, full.subset(ks), a)
    for f in FIELDS:
        assert np.array_equal(s[f], g[f][ks]), (algo, f)
    sel = np.concatenate([np.arange(full.offsets[k], full.offsets[k + 1]) for k in ks])
    for f in ("completion", "evictions"):
        assert np.array_equal(s[f], g[f][sel]), (algo, f)
