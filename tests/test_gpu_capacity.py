"""GPU parity where an instance outgrows the room of a launch: its cancelled set
(A_min's cancelled requests, A_l's promoted queue) or its running set.  The
library then simulates it again with more room, down to a cancelled set in
global memory; whether an instance completes, and its outputs, never depend on
the other instances of its batch or on the capacities chosen (Algorithm 2's
cancellation step; Algorithm 5's queue)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run, _growth_sweep, _say  # noqa: F401

pytestmark = pytest.mark.gpu


def _many_cancelled():
    # 3000 requests with l = 1 and outputs of 20..40 at M = 1500: up to 750
    # run at once and up to 2808 cancelled requests wait at once (oracle)
    rng = np.random.default_rng(0)
    n = 3000
    o = rng.integers(20, 41, n)
    return {"arrival": np.zeros(n, int), "prompt": np.ones(n, int), "output": o, "lower": np.ones(n, int),
            "upper": o}


def test_more_than_1024_waiting_cancellations_alone_and_in_a_batch(B):
    big = _many_cancelled()
    st = O.simulate(big, O.AMIN, 1500, stats=True)["stats"]
    assert st["max_evicted_waiting"] > 1024 and 640 < st["max_running"] <= 1024
    alone = W.from_lists(1500, [big], name="many_cancelled")
    ref1 = oracle_run(alone, O.AMIN)
    assert (ref1["status"] == 0).all()
    assert_parity(alone, gpu_run(B, alone, O.AMIN), ref1)
    # the same instance as the 65th of a batch (whose first launch gives each
    # instance fewer cancelled-set slots than it needs)
    others = W.random_small(7, 64, 60, s_max=8, o_max=40, M=1500)
    insts = [{f: others.instance(k)[f] for f in ("arrival", "prompt", "output", "lower", "upper")}
             for k in range(64)] + [big]
    batch = W.from_lists(1500, insts, name="batch65")
    ref = oracle_run(batch, O.AMIN)
    assert (ref["status"] == 0).all()
    g = gpu_run(B, batch, O.AMIN)
    assert_parity(batch, g, ref)
    lo = int(batch.offsets[64])
    assert np.array_equal(g["completion"][lo:], ref1["completion"])


@pytest.mark.parametrize("algo", ["amin", "aell", "adaptive"])
@pytest.mark.parametrize("cap,lds_limit", [(4, 0), (16, 0), (4, 8), (2, 2)])
def test_small_cancelled_sets_retry(B, algo, cap, lds_limit):
    # tiny first-launch capacities: instances that outgrow them are simulated
    # again with the LDS maximum (lds_limit 0) or a global-memory set
    a = O.ALGOS[algo]
    batch = _growth_sweep(0, K=48)
    ref = oracle_run(batch, a, stats=True)
    assert (ref["status"] == 0).all()
    assert max(st["max_evicted_waiting"] for st in ref["stats"]) > max(cap, lds_limit)
    g = gpu_run(B, batch, a, evicted_capacity=cap, evicted_lds_limit=lds_limit)
    assert_parity(batch, g, ref)


def test_global_cancelled_set_large_instance(B):
    # the 3000-request instance with at most 512 LDS slots: its cancelled set
    # lives in global memory in the last launch
    batch = W.from_lists(1500, [_many_cancelled()], name="many_cancelled_global")
    ref = oracle_run(batch, O.AMIN)
    g = gpu_run(B, batch, O.AMIN, evicted_lds_limit=512)
    assert_parity(batch, g, ref)


@pytest.mark.parametrize("algo", ["amin", "aell"])
def test_forced_running_capacity_with_cancelled_set_retry(B, algo):
    # a caller's running capacity holds in the retry launches too
    a = O.ALGOS[algo]
    batch = _growth_sweep(1, K=40)
    ref = oracle_run(batch, a)
    g = gpu_run(B, batch, a, running_capacity=1024, evicted_capacity=4)
    assert_parity(batch, g, ref)
    g = gpu_run(B, batch, a, running_capacity=384, evicted_capacity=4, evicted_lds_limit=8)
    peak = np.array([O.simulate(batch.instance(k), a, batch.M, stats=True)["stats"]["max_running"]
                     for k in range(batch.num_instances)])
    fits = peak <= 384
    assert fits.any() and (~fits).any()
    assert (g["status"][~fits] == -6).all()
    ks = list(np.flatnonzero(fits))
    assert_parity(batch, g, oracle_run(batch, a, instances=ks), instances=ks)


def test_validate_matches_simulate_statuses(B):
    good = {"arrival": [0, 1, 1], "prompt": [1, 2, 1], "output": [3, 2, 4], "lower": [1, 2, 2], "upper": [4, 2, 6]}
    insts = [good, dict(good, lower=[4, 2, 2]), dict(good, output=[0, 2, 4]), dict(good, prompt=[1, 2, 9]),
             dict(good, arrival=[1, 0, 1]), dict(good, upper=[2, 2, 6]), dict(good, upper=[4, 2, 10]),
             {"arrival": [], "prompt": [], "output": [], "lower": [], "upper": []}]
    batch = W.from_lists(10, insts, name="validate")
    db = B.to_device(batch)
    import torch
    for algo in (O.AMAX, O.AMIN, O.HSF, O.AELL, O.ADAPTIVE):
        v = B.validate(db, algo)
        g = gpu_run(B, batch, algo)
        torch.cuda.synchronize()
        assert v.cpu().numpy().tolist() == g["status"].tolist(), algo
