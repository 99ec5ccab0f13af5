"""GPU parity of the auxiliary random-order policy A_random (Appendix, proof of
Theorem 3.1) through the C ABI: the random order is an input (per-request
priorities drawn by the generator); outputs are bit-exact with the oracle."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run  # noqa: F401 (B is a fixture)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed,arrivals", [(0, True), (1, False), (2, True)])
def test_random_small(B, seed, arrivals):
    batch = W.with_random_order(W.random_small(seed, 300, 12, s_max=6, o_max=10, M=30, arrivals=arrivals), seed)
    g = gpu_run(B, batch, O.ARANDOM)
    assert_parity(batch, g, oracle_run(batch, O.ARANDOM))


@pytest.mark.parametrize("cap", [150, 384, 1024])
def test_ragged_and_rows(B, cap):
    rng = np.random.default_rng(17)
    insts = []
    for k in range(150):
        n = int(rng.integers(0, 151)) if k % 13 else 0
        o = rng.integers(1, 40, n)
        insts.append({"arrival": np.sort(rng.integers(0, 40, n)) if k % 2 else np.zeros(n, int),
                      "prompt": rng.integers(0, 10, n), "output": o, "lower": np.ones(n, int), "upper": o + 3,
                      "priority": rng.permutation(n)})
    batch = W.from_lists(300, insts, name="ragged_random_order")
    g = gpu_run(B, batch, O.ARANDOM, running_capacity=cap)
    assert_parity(batch, g, oracle_run(batch, O.ARANDOM))


def test_hsf_order_is_hsf_and_priority_range(B):
    b = W.random_small(8, 50, 12, s_max=6, o_max=10, M=30)
    insts = []
    for k in range(b.num_instances):
        d = dict(b.instance(k))
        o = np.asarray(d["output"])
        rank = np.empty(len(o), np.int64)
        rank[np.lexsort((np.arange(len(o)), o))] = np.arange(len(o))
        d["priority"] = rank
        insts.append(d)
    batch = W.from_lists(b.M, insts, name="hsf_order")
    g = gpu_run(B, batch, O.ARANDOM)
    h = gpu_run(B, batch, O.HSF)
    for f in ("status", "tel", "makespan", "request_steps", "completion"):
        assert np.array_equal(g[f], h[f]), f
    bad = W.from_lists(30, [dict(insts[0], priority=[1 << 15] + [0] * (len(insts[0]["output"]) - 1))], name="prio")
    assert int(gpu_run(B, bad, O.ARANDOM)["status"][0]) == B.E_UNSUPPORTED


def test_batch4096_random_order_sampled(B):
    batch = W.with_random_order(W.generate("batch4096_n1000_m16384", 0))
    g = gpu_run(B, batch, O.ARANDOM)
    assert (g["status"] == 0).all()
    ks = list(range(0, 4096, 64)) + [1364, 1365, 2730, 4095]
    assert_parity(batch, g, oracle_run(batch, O.ARANDOM, instances=ks), instances=ks)


def test_growth_mid_simulation_random_order(B):
    # the running set outgrows the first register rows in the middle of the
    # simulation (as in test_gpu_parity's growth test), under a random order
    from test_gpu_parity import _growth_instances
    batch = W.with_random_order(_growth_instances(), 5)
    ref = oracle_run(batch, O.ARANDOM)
    assert (ref["status"] == 0).all()
    g = gpu_run(B, batch, O.ARANDOM)
    assert_parity(batch, g, ref)
    g1 = gpu_run(B, batch, O.ARANDOM, running_capacity=1024)
    for f in ("status", "tel", "makespan", "request_steps", "completion"):
        assert np.array_equal(g[f], g1[f]), f
