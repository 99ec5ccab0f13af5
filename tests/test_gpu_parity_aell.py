"""GPU parity of the promote-l policy A_l and the adaptive A_min/A_l switch
(Section 5.1) through the C ABI, against the CPU oracle, bit-exact on every
integer output, plus the policy each instance ran under the adaptive switch."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run, _say  # noqa: F401 (B is a fixture)

pytestmark = pytest.mark.gpu

POLICIES = {"aell": O.AELL, "adaptive": O.ADAPTIVE}


def choices(batch, ks=None):
    ks = range(batch.num_instances) if ks is None else ks
    return [O.adaptive_choice(batch.instance(k)) for k in ks]


def check_algo_used(batch, g, algo, ks=None):
    ks = list(range(batch.num_instances)) if ks is None else list(ks)
    ok = g["status"][ks] != O.E_INVAL
    want = np.array(choices(batch, ks)) if algo == O.ADAPTIVE else np.full(len(ks), algo)
    assert np.array_equal(g["algo_used"][ks][ok], want[ok])


@pytest.mark.parametrize("algo", ["aell", "adaptive"])
@pytest.mark.parametrize("seed,arrivals,alpha", [(0, True, 1.0), (1, False, 1.0), (2, True, 2.0), (3, False, 0.5)])
def test_random_small(B, algo, seed, arrivals, alpha):
    batch = W.random_small(seed, 300, 12, s_max=6, o_max=10, M=30, arrivals=arrivals, alpha=alpha)
    g = gpu_run(B, batch, POLICIES[algo])
    ref = oracle_run(batch, POLICIES[algo])
    assert_parity(batch, g, ref)
    check_algo_used(batch, g, POLICIES[algo])
    if algo == "aell":
        assert ref["total_evictions"].sum() > 0  # promotions happen


@pytest.mark.parametrize("algo", ["aell", "adaptive"])
def test_ragged(B, algo):
    # instances of 0..150 requests (empty ones included), several rows of 64 lanes
    rng = np.random.default_rng(7)
    insts = []
    for k in range(200):
        n = int(rng.integers(0, 151)) if k % 17 else 0
        lo = int(rng.integers(1, 12))
        hi = lo + int(rng.integers(0, 40))
        o = np.where(rng.random(n) < 0.5, lo, rng.integers(lo, hi + 1, n))
        s = rng.integers(0, 20, n)
        a = np.sort(rng.integers(0, 60, n)) if k % 2 else np.zeros(n, int)
        insts.append({"arrival": a, "prompt": s, "output": o, "lower": np.full(n, lo), "upper": np.full(n, hi)})
    batch = W.from_lists(400, insts, name="ragged_two_point")
    g = gpu_run(B, batch, POLICIES[algo])
    assert_parity(batch, g, oracle_run(batch, POLICIES[algo]))
    check_algo_used(batch, g, POLICIES[algo])


@pytest.mark.parametrize("cap", [150, 384, 512, 1024])
def test_row_variants(B, cap):
    rng = np.random.default_rng(13)
    insts = []
    for k in range(100):
        n = int(rng.integers(1, 151))
        o = rng.integers(1, 30, n)
        insts.append({"arrival": np.zeros(n, int), "prompt": rng.integers(0, 4, n), "output": o,
                      "lower": np.maximum(1, o // 3), "upper": o + 8})
    batch = W.from_lists(600, insts, name="rows_aell")
    for algo in (O.AELL, O.ADAPTIVE):
        g = gpu_run(B, batch, algo, running_capacity=cap)
        assert_parity(batch, g, oracle_run(batch, algo))


def test_statuses(B):
    good = {"arrival": [0, 1, 1], "prompt": [1, 2, 1], "output": [3, 2, 4], "lower": [1, 2, 2], "upper": [4, 2, 6]}
    insts = [
        good,
        dict(good, upper=[2, 2, 6]),     # u < o
        dict(good, lower=[4, 2, 2]),     # l > o
        dict(good, upper=[4, 2, 10]),    # s + u > M
        dict(good, arrival=[1, 0, 1]),   # unsorted arrivals
        {"arrival": [], "prompt": [], "output": [], "lower": [], "upper": []},
    ]
    batch = W.from_lists(10, insts, name="errors_aell")
    g = gpu_run(B, batch, O.AELL)
    assert g["status"].tolist() == [0, O.E_INTERVAL, O.E_INTERVAL, O.E_TOO_BIG, O.E_ARRIVAL, 0]
    assert_parity(batch, g, oracle_run(batch, O.AELL))
    # the adaptive switch validates with the policy it picks: with (sum l)/(sum u)
    # = 4/7 it picks A_min, which does not read u, so u < o is accepted
    hi = {"arrival": [0, 0], "prompt": [1, 1], "output": [4, 3], "lower": [2, 2], "upper": [3, 4]}
    lo = {"arrival": [0, 0], "prompt": [1, 1], "output": [4, 3], "lower": [1, 1], "upper": [9, 9]}
    b2 = W.from_lists(10, [hi, lo, dict(lo, upper=[3, 9])], name="adaptive_validation")
    g = gpu_run(B, b2, O.ADAPTIVE)
    assert g["algo_used"].tolist() == [O.AMIN, O.AELL, O.AELL]
    assert g["status"].tolist() == [0, 0, O.E_INTERVAL]
    assert_parity(b2, g, oracle_run(b2, O.ADAPTIVE))


@pytest.mark.parametrize("cap", [1, 7, 30])
def test_step_cap(B, cap):
    batch = W.random_small(5, 100, 10, s_max=6, o_max=10, M=30, alpha=1.0)
    for algo in (O.AELL, O.ADAPTIVE):
        g = gpu_run(B, batch, algo, step_cap=cap)
        assert_parity(batch, g, oracle_run(batch, algo, step_cap=cap))


@pytest.mark.parametrize("algo", ["aell", "adaptive", "amin"])
def test_twopoint4096_sampled(B, algo):
    # the two-point workload at full size, in the benchmark's launch configuration
    batch = W.generate("twopoint4096_n1000_m16384", 0)
    a = {"aell": O.AELL, "adaptive": O.ADAPTIVE, "amin": O.AMIN}[algo]
    g = gpu_run(B, batch, a)
    assert (g["status"] == 0).all()
    ks = list(range(0, 4096, 16)) + [681, 682, 1363, 1364, 2045, 2046, 2727, 2728, 3409, 3410, 4095]
    _say(f"[oracle] twopoint4096 {algo} on {len(ks)} instances")
    assert_parity(batch, g, oracle_run(batch, a, instances=ks), instances=ks)
    check_algo_used(batch, g, a)  # every instance's choice
