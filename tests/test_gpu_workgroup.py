"""GPU parity of the workgroup kernels: several waves simulate one instance,
each holding part of the running set, and agree on every decision through
LDS.  Their outputs must equal the oracle's bit for bit, whether the workgroup
runs from the start (workgroup_waves) or takes over an instance whose running
set outgrows one wave (more than 1024 runs).  The policies are Algorithms 1-5
with equation (2); the closed-form case pins a schedule in which every request
fits at once (every start at its arrival)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run, _growth_sweep, _say  # noqa: F401

pytestmark = pytest.mark.gpu

FIELDS = ("status", "tel", "makespan", "request_steps", "total_evictions", "completion", "evictions")


@pytest.mark.parametrize("ww", [2, 4])
@pytest.mark.parametrize("algo", ["amax", "amin", "hsf"])
@pytest.mark.parametrize("seed,arrivals", [(0, True), (1, False)])
def test_workgroup_random_small(B, ww, algo, seed, arrivals):
    a = O.ALGOS[algo]
    batch = W.random_small(seed, 64, 60, s_max=6, o_max=12, M=40, arrivals=arrivals)
    ref = oracle_run(batch, a)
    assert_parity(batch, gpu_run(B, batch, a, workgroup_waves=ww), ref)


@pytest.mark.parametrize("ww", [2, 4])
@pytest.mark.parametrize("algo", ["amax", "amin", "hsf"])
def test_workgroup_growth_sweep(B, ww, algo):
    # running sets of up to ~800 runs, cancellations and arrivals in bursts;
    # also with random tie keys (equal planning lengths in random order)
    a = O.ALGOS[algo]
    batch = _growth_sweep(0, K=40)
    ref = oracle_run(batch, a)
    assert (ref["status"] == 0).all()
    g = gpu_run(B, batch, a, workgroup_waves=ww)
    assert_parity(batch, g, ref)
    g1 = gpu_run(B, batch, a)
    for f in FIELDS:
        assert np.array_equal(g[f], g1[f]), f
    tb = W.with_tie_keys(batch, seed=3)
    assert_parity(tb, gpu_run(B, tb, a, workgroup_waves=ww), oracle_run(tb, a))


def test_workgroup_global_cancelled_sets_fewer_workgroups_than_instances(B):
    # LDS cancelled sets capped at one slot: A_min's sets live in global memory,
    # n_max entries per wave; with a 70000-request instance in the batch the
    # launch has fewer workgroups than instances, each simulating several
    batch0 = _growth_sweep(1, K=39)
    insts = [{f: batch0.instance(k)[f] for f in ("arrival", "prompt", "output", "lower", "upper")}
             for k in range(39)]
    rng = np.random.default_rng(11)
    n = 70000
    o = rng.integers(1, 4, n)
    insts.append({"arrival": np.sort(rng.integers(0, 30000, n)), "prompt": np.ones(n, int), "output": o,
                  "lower": np.ones(n, int), "upper": o + 1})
    batch = W.from_lists(1400, insts, name="many_with_one_large")
    ref = oracle_run(batch, O.AMIN)
    assert (ref["status"] == 0).all()
    g = gpu_run(B, batch, O.AMIN, workgroup_waves=4, evicted_lds_limit=1)
    assert_parity(batch, g, ref)


def _wide_instances():
    # more than 1024 concurrent runs: all 3000 requests at step 0 with
    # footprints of one to seven tokens under M = 2000 (A_min admits 2000 and
    # cancels ~1400 times; A_l promotes every request), and a stream of 3000
    # requests over 21 steps under M = 12000 (about 1090 runs at once under
    # every policy)
    rng = np.random.default_rng(5)
    n = 3000
    o = rng.integers(2, 7, n)
    burst = {"arrival": np.zeros(n, int), "prompt": np.zeros(n, int), "output": o, "lower": np.ones(n, int),
             "upper": o + 1, "priority": rng.permutation(n)}
    rng = np.random.default_rng(0)
    o = rng.integers(3, 13, n)
    s = rng.integers(0, 3, n)
    a = np.sort(rng.integers(0, 21, n))
    lo = np.maximum(1, (o * rng.uniform(0.5, 1.0, n)).astype(int))
    stream = {"arrival": a, "prompt": s, "output": o, "lower": lo, "upper": o + rng.integers(0, 4, n),
              "priority": rng.permutation(n)}
    return W.from_lists(2000, [burst], name="burst3000"), W.from_lists(12000, [stream], name="stream3000")


@pytest.mark.parametrize("algo", ["amin", "amax", "hsf", "aell", "adaptive", "arandom"])
def test_more_than_1024_runs(B, algo):
    a = O.ALGOS[algo]
    for batch in _wide_instances():
        ref = oracle_run(batch, a, stats=True)
        assert (ref["status"] == 0).all()
        peak = ref["stats"][0]["max_running"]
        g = gpu_run(B, batch, a)
        _say(f"[wide] {batch.name} {algo}: peak {peak} runs, gpu status {g['status'].tolist()}")
        assert_parity(batch, g, ref)


@pytest.mark.parametrize("algo", ["amin", "hsf"])
def test_more_than_1024_runs_inside_a_batch(B, algo):
    # the wide instance between two small batches' worth of instances: the
    # others finish in the first launch, the wide one in a workgroup launch
    a = O.ALGOS[algo]
    burst = _wide_instances()[0]
    small = _growth_sweep(0, K=20)
    pick = lambda b, k: {f: b.instance(k)[f] for f in ("arrival", "prompt", "output", "lower", "upper", "priority")}
    insts = [pick(small, k) for k in range(10)] + [pick(burst, 0)] + [pick(small, k) for k in range(10, 20)]
    batch = W.from_lists(2000, insts, name="wide_in_batch")
    ref = oracle_run(batch, a)
    assert (ref["status"] == 0).all()
    assert_parity(batch, gpu_run(B, batch, a), ref)


@pytest.mark.parametrize("algo", ["amax", "amin", "hsf", "aell", "adaptive", "arandom"])
def test_more_than_4096_runs_closed_form(B, algo):
    # every request fits at once: all start at step 0 and complete at their
    # output length (intervals [o, o + 1], so A_l never promotes), TEL = sum o,
    # request-steps = sum o; 5000 runs at once go to the eight-wave workgroup.
    # The closed form is first checked against the oracle on a small copy.
    a = O.ALGOS[algo]
    rng = np.random.default_rng(9)

    def inst(n):
        o = rng.integers(1, 6, n)
        s = rng.integers(0, 3, n)
        return {"arrival": np.zeros(n, int), "prompt": s, "output": o, "lower": o, "upper": o + 1,
                "priority": rng.permutation(n)}, int((s + o + 1).sum())

    d, M = inst(40)
    ref = oracle_run(W.from_lists(M, [d], name="fits40"), a)
    assert ref["completion"].tolist() == d["output"].tolist() and int(ref["tel"][0]) == int(d["output"].sum())
    assert int(ref["request_steps"][0]) == int(d["output"].sum()) and int(ref["total_evictions"][0]) == 0
    d, M = inst(5000)
    g = gpu_run(B, W.from_lists(M, [d], name="fits5000"), a)
    o = d["output"]
    assert g["status"].tolist() == [0]
    assert g["completion"].tolist() == o.tolist()
    assert int(g["tel"][0]) == int(o.sum()) and int(g["makespan"][0]) == int(o.max())
    assert int(g["request_steps"][0]) == int(o.sum()) and int(g["total_evictions"][0]) == 0
    assert (g["evictions"] == 0).all()


def test_workgroup_option_checks(B):
    batch = W.random_small(0, 4, 10)
    db = B.to_device(batch)
    for ww, algo in [(3, O.AMIN), (8, O.AMAX), (-1, O.HSF), (2, O.AELL), (4, O.ADAPTIVE), (2, O.ARANDOM)]:
        with pytest.raises(B.SchedError) as e:
            B.simulate(db, algo, workgroup_waves=ww)
        assert e.value.code == B.E_INVAL
    with pytest.raises(B.SchedError):
        B.simulate(db, O.AMIN, workgroup_waves=2, running_capacity=128)
    # 0 and 1 are the default
    for ww in (0, 1):
        g = gpu_run(B, batch, O.AMIN, workgroup_waves=ww)
        assert_parity(batch, g, oracle_run(batch, O.AMIN))


@pytest.mark.parametrize("ww", [2, 4])
@pytest.mark.parametrize("cap", [3, 17])
def test_workgroup_step_cap(B, ww, cap):
    # a step cap ends every wave of the workgroup at the same step, with the
    # oracle's partial outputs
    batch = _growth_sweep(1, K=12)
    for algo in (O.AMIN, O.AMAX, O.HSF):
        ref = oracle_run(batch, algo, step_cap=cap)
        assert (ref["status"] == O.E_STEP_CAP).any()
        assert_parity(batch, gpu_run(B, batch, algo, step_cap=cap, workgroup_waves=ww), ref)


def test_workgroup_launches_without_allocation(B):
    # the no-allocation entry point with workgroups: from the start (global
    # cancelled sets) and as the tier above 1024 runs; twice, the second batch
    # smaller, against the allocating entry point
    import torch
    burst = _wide_instances()[0]
    small = _growth_sweep(2, K=6)
    pick = lambda b, k: {f: b.instance(k)[f] for f in ("arrival", "prompt", "output", "lower", "upper", "priority")}
    big = W.from_lists(2000, [pick(small, k) for k in range(6)] + [pick(burst, 0)], name="noalloc_wide")
    for batch in (big, W.from_lists(2000, [pick(small, k) for k in range(3)], name="noalloc_small")):
        db = B.to_device(batch)
        for kw in ({}, {"workgroup_waves": 4, "evicted_lds_limit": 1}):
            ref = B.simulate(db, B.AMIN, **kw)
            out = B.alloc_results(db)
            B.simulate_into(db, B.AMIN, out, no_alloc=True, **kw)
            torch.cuda.synchronize()
            for f in ("status", "tel", "makespan", "request_steps", "total_evictions", "completion", "evictions"):
                assert torch.equal(out[f], ref[f]), (batch.name, kw, f)
            assert (out["status"] == 0).all()


@pytest.mark.parametrize("ww", [2, 4])
def test_workgroup_statuses_and_empty_instances(B, ww):
    # invalid and empty instances next to valid ones: the same statuses and
    # outputs as one wave per instance
    good = {"arrival": [0, 1, 1], "prompt": [1, 2, 1], "output": [3, 2, 4], "lower": [1, 2, 2], "upper": [4, 2, 6]}
    insts = [good, dict(good, lower=[4, 2, 2]), dict(good, output=[0, 2, 4]), dict(good, prompt=[1, 2, 9]),
             dict(good, arrival=[1, 0, 1]), {"arrival": [], "prompt": [], "output": [], "lower": [], "upper": []},
             dict(good, upper=[2, 2, 6]), good]
    batch = W.from_lists(10, insts, name="wg_statuses")
    for algo in (O.AMAX, O.AMIN, O.HSF):
        g1 = gpu_run(B, batch, algo)
        g = gpu_run(B, batch, algo, workgroup_waves=ww)
        for f in FIELDS:
            assert np.array_equal(g[f], g1[f]), (algo, f)
        ok = [k for k in range(batch.num_instances) if g["status"][k] == 0]
        assert_parity(batch, g, oracle_run(batch, algo, instances=ok), instances=ok)
