"""The no-allocation entry point (sched_simulate_noalloc) through the C ABI:
bit-identical outputs to sched_simulate_opts on two calls in a row, the
second with a smaller input (the scratch array keeps the first call's
contents), and the size limit of its scratch array."""
import numpy as np
import pytest

from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, _growth_sweep  # noqa: F401 (B is a fixture)

pytestmark = pytest.mark.gpu
FIELDS = ("completion", "evictions", "tel", "makespan", "request_steps", "total_evictions", "status", "algo_used")


def _run(B, db, algo, no_alloc, **kw):
    import torch
    out = B.alloc_results(db)
    for v in out.values():
        v.fill_(-77)  # stale values the call must overwrite
    B.simulate_into(db, algo, out, no_alloc=no_alloc, **kw)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _same(a, b):
    for f in FIELDS:
        assert np.array_equal(a[f], b[f]), f


@pytest.mark.parametrize("name", ["amin", "amax", "hsf", "aell", "adaptive"])
def test_noalloc_equals_opts_twice_second_smaller(B, name):
    algo = B.ALGOS[name]
    big = W.generate("batch4096_n1000_m16384", 0, instance_ids=range(2600, 3400))
    small = W.generate("batch4096_n1000_m16384", 0, instance_ids=range(2980, 3000))
    for batch in (big, small):
        db = B.to_device(batch)
        ref = _run(B, db, algo, False)
        assert (ref["status"] == 0).all()
        _same(_run(B, db, algo, True), ref)


@pytest.mark.parametrize("name", ["amin", "aell"])
def test_noalloc_retries_tie_keys_and_global_set(B, name):
    # retry launches, tie keys and a global-memory cancelled set, all inside the scratch array
    algo = B.ALGOS[name]
    big = W.with_tie_keys(_growth_sweep(1, K=48), 2)
    small = W.with_tie_keys(_growth_sweep(0, K=12), 5)
    for batch in (big, small):
        db = B.to_device(batch)
        for kw in ({}, {"evicted_capacity": 4, "evicted_lds_limit": 8}):
            ref = _run(B, db, algo, False, **kw)
            _same(_run(B, db, algo, True, **kw), ref)


def test_noalloc_rejects_workspace_beyond_scratch(B):
    import torch
    # 50 instances of 110000 requests: 5.5 million requests need about 110 MB
    K, n = 50, 110000
    dev = torch.device("cuda")
    z = torch.ones(K * n, dtype=torch.int32, device=dev)
    db = B.DeviceBatch(1 << 20, n, torch.arange(K + 1, dtype=torch.int64, device=dev) * n,
                       None, z, z, z, z)
    out = B.alloc_results(db)
    with pytest.raises(B.SchedError) as e:
        B.simulate_into(db, B.AMIN, out, no_alloc=True)
    assert e.value.code == B.E_SCRATCH
