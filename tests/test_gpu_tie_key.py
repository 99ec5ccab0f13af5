"""GPU parity with caller-given tie keys: requests whose planning keys are equal
are ordered by (tie key, index) in admission and cancellation (the paper breaks
these ties uniformly at random; Algorithms 1, 2 and 4), A_l's fresh queue by
(arrival, tie key, index).  Bit-exact against the CPU oracle."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run, _growth_sweep  # noqa: F401

pytestmark = pytest.mark.gpu
NAMES = ["amax", "amin", "hsf", "aell", "adaptive", "arandom"]


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("seed,arrivals", [(0, False), (1, True)])
def test_random_small_with_tie_keys(B, name, seed, arrivals):
    batch = W.with_tie_keys(W.with_random_order(
        W.random_small(seed + 70, 300, 12, s_max=6, o_max=10, M=30, arrivals=arrivals, alpha=1.0), seed), seed)
    a = O.ALGOS[name]
    ref = oracle_run(batch, a)
    assert_parity(batch, gpu_run(B, batch, a), ref)


@pytest.mark.parametrize("name", ["amin", "amax", "aell"])
def test_repeated_and_negative_tie_keys(B, name):
    # tie keys with repeats (then the index decides) and negative values
    base = W.random_small(80, 200, 14, s_max=5, o_max=9, M=28, arrivals=True, alpha=1.0)
    rng = np.random.default_rng(1)
    import dataclasses
    batch = dataclasses.replace(base, tie_key=rng.integers(-3, 3, base.total_requests).astype(np.int32))
    a = O.ALGOS[name]
    assert_parity(batch, gpu_run(B, batch, a), oracle_run(batch, a))


@pytest.mark.parametrize("name", ["amin", "aell", "hsf"])
def test_growth_with_tie_keys(B, name):
    # instances that outgrow the first register rows and are simulated again
    batch = W.with_tie_keys(_growth_sweep(2, K=48), 3)
    a = O.ALGOS[name]
    ref = oracle_run(batch, a)
    assert (ref["status"] == 0).all()
    assert_parity(batch, gpu_run(B, batch, a), ref)
    assert_parity(batch, gpu_run(B, batch, a, evicted_capacity=4, evicted_lds_limit=8), ref)


@pytest.mark.parametrize("name", ["amin", "amax", "hsf"])
def test_batch4096_subset_with_tie_keys(B, name):
    # the benchmark's instances with random tie keys (A_min cancels far less
    # when ties among equal lower bounds are random rather than by index)
    batch = W.with_tie_keys(W.generate("batch4096_n1000_m16384", 0, instance_ids=range(2900, 3100)), 0)
    a = O.ALGOS[name]
    ref = oracle_run(batch, a)
    assert (ref["status"] == 0).all()
    assert_parity(batch, gpu_run(B, batch, a), ref)
