"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Integer outputs must match bit-exactly: per-request completion steps and
cancellation counts, per-instance total latency, makespan, request-steps,
total cancellations and status.
"""
import json
import os
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W

pytestmark = pytest.mark.gpu

ALGOS = {"amax": O.AMAX, "amin": O.AMIN, "hsf": O.HSF, "aell": O.AELL, "adaptive": O.ADAPTIVE}


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def B():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_14544_amd import binding
    binding.load_library()
    return binding


def gpu_run(B, batch, algo, *, pass_upper=True, **opts):
    import torch
    _say(f"[gpu] {batch.name} K={batch.num_instances} N={batch.total_requests} algo={algo} opts={opts}")
    db = B.to_device(batch)
    out = B.simulate(db, algo, pass_upper=pass_upper, **opts)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}


def oracle_run(batch, algo, instances=None, step_cap=0, stats=False):
    return O.simulate_batch(batch, algo, instances=instances, step_cap=step_cap, stats=stats)


def assert_parity(batch, g, ref, instances=None):
    ks = list(range(batch.num_instances)) if instances is None else list(instances)
    assert g["status"][ks].tolist() == ref["status"].tolist()
    assert g["tel"][ks].tolist() == ref["tel"].tolist()
    assert g["makespan"][ks].tolist() == ref["makespan"].tolist()
    assert g["request_steps"][ks].tolist() == ref["request_steps"].tolist()
    assert g["total_evictions"][ks].tolist() == ref["total_evictions"].tolist()
    sel = np.concatenate([np.arange(batch.offsets[k], batch.offsets[k + 1]) for k in ks]) if ks else np.zeros(0, int)
    sel = sel.astype(np.int64)
    assert np.array_equal(g["completion"][sel], ref["completion"])
    assert np.array_equal(g["evictions"][sel], ref["evictions"])


def _golden():
    here = os.path.join(os.path.dirname(__file__), "golden")
    files = [os.path.join(here, f) for f in sorted(os.listdir(here)) if f.endswith(".json")]
    return [f for f in files if "instance" in json.load(open(f))]


@pytest.mark.parametrize("path", _golden(), ids=os.path.basename)
def test_paper_examples(B, path):
    g = json.load(open(path))
    batch = W.from_lists(g["M"], [g["instance"]], name=os.path.basename(path))
    for name, exp in g["expected"].items():
        if name not in ALGOS:
            continue
        out = gpu_run(B, batch, ALGOS[name])
        assert int(out["status"][0]) == 0
        assert out["completion"].tolist() == exp["completion"]
        assert int(out["tel"][0]) == exp["tel"]
        for f in ("evictions",):
            if f in exp:
                assert out[f].tolist() == exp[f]
        for f in ("makespan", "request_steps"):
            if f in exp:
                assert int(out[f][0]) == exp[f]


@pytest.mark.parametrize("algo", ["amax", "amin", "hsf"])
@pytest.mark.parametrize("seed,arrivals", [(0, True), (1, False), (2, True)])
def test_random_small(B, algo, seed, arrivals):
    batch = W.random_small(seed, 300, 12, s_max=6, o_max=10, M=30, arrivals=arrivals)
    g = gpu_run(B, batch, ALGOS[algo])
    assert_parity(batch, g, oracle_run(batch, ALGOS[algo]))


@pytest.mark.parametrize("algo", ["amax", "amin", "hsf"])
def test_random_medium_ragged(B, algo):
    # instances of 0..150 requests (empty ones included), several rows of 64 lanes
    rng = np.random.default_rng(5)
    insts = []
    for k in range(200):
        n = int(rng.integers(0, 151)) if k % 17 else 0
        o = rng.integers(1, 40, n)
        l = np.maximum(1, (o * rng.uniform(0.3, 1.0, n)).astype(int))
        u = o + rng.integers(0, 30, n)
        s = rng.integers(0, 20, n)
        a = np.sort(rng.integers(0, 60, n)) if k % 2 else np.zeros(n, int)
        insts.append({"arrival": a, "prompt": s, "output": o, "lower": l, "upper": u})
    batch = W.from_lists(400, insts, name="ragged")
    g = gpu_run(B, batch, ALGOS[algo])
    assert_parity(batch, g, oracle_run(batch, ALGOS[algo]))


@pytest.mark.parametrize("algo", ["amax", "amin", "hsf"])
def test_single_n200(B, algo):
    batch = W.generate("single_n200_m512", 0)
    g = gpu_run(B, batch, ALGOS[algo])
    assert_parity(batch, g, oracle_run(batch, ALGOS[algo]))


@pytest.mark.parametrize("cap", [384, 512, 1024])
def test_launch_shape_independence(B, cap):
    # 6, 8 and 16 register rows give the same bits as the default launches (a
    # 6-row kernel that re-runs outgrown instances with 8 rows, then 16)
    batch = W.generate("batch4096_n1000_m16384", 0, instance_ids=range(0, 4096, 97))
    ref = gpu_run(B, batch, O.AMIN)
    g = gpu_run(B, batch, O.AMIN, running_capacity=cap)
    for f in ("status", "tel", "makespan", "request_steps", "total_evictions", "completion", "evictions"):
        assert np.array_equal(ref[f], g[f]), f


@pytest.mark.parametrize("cap", [150, 192, 512, 1024])
def test_row_variants_against_oracle(B, cap):
    # 3 -> 4, 4, 8 and 16 register rows on instances of up to 150 requests
    rng = np.random.default_rng(11)
    insts = []
    for k in range(120):
        n = int(rng.integers(1, 151))
        o = rng.integers(1, 30, n)
        insts.append({"arrival": np.zeros(n, int), "prompt": rng.integers(0, 4, n), "output": o,
                      "lower": np.maximum(1, o // 2), "upper": o + 5})
    batch = W.from_lists(600, insts, name="rows")
    for algo in (O.AMAX, O.AMIN, O.HSF):
        g = gpu_run(B, batch, algo, running_capacity=cap)
        assert_parity(batch, g, oracle_run(batch, algo))


def test_errors_and_statuses(B):
    good = {"arrival": [0, 1, 1], "prompt": [1, 2, 1], "output": [3, 2, 4], "lower": [1, 2, 2], "upper": [4, 2, 6]}
    insts = [
        good,
        dict(good, lower=[4, 2, 2]),          # l > o
        dict(good, lower=[0, 2, 2]),          # l < 1
        dict(good, output=[0, 2, 4]),         # o < 1
        dict(good, prompt=[-1, 2, 1]),        # s < 0
        dict(good, prompt=[1, 2, 9]),         # s + o > M
        dict(good, arrival=[1, 0, 1]),        # unsorted
        dict(good, arrival=[-2, 0, 1]),       # negative
        {"arrival": [], "prompt": [], "output": [], "lower": [], "upper": []},
        good,
    ]
    batch = W.from_lists(10, insts, name="errors")
    for algo in (O.AMAX, O.AMIN, O.HSF):
        g = gpu_run(B, batch, algo)
        assert_parity(batch, g, oracle_run(batch, algo))
    # A_max-specific: u < o and s + u > M
    insts2 = [good, dict(good, upper=[2, 2, 6]), dict(good, upper=[4, 2, 10])]
    b2 = W.from_lists(10, insts2, name="errors_amax")
    g = gpu_run(B, b2, O.AMAX)
    assert g["status"].tolist() == [0, O.E_INTERVAL, O.E_TOO_BIG]
    assert_parity(b2, g, oracle_run(b2, O.AMAX))


@pytest.mark.parametrize("cap", [1, 5, 15, 60])
def test_step_cap(B, cap):
    batch = W.random_small(3, 100, 10, s_max=6, o_max=10, M=30)
    for algo in (O.AMAX, O.AMIN, O.HSF):
        g = gpu_run(B, batch, algo, step_cap=cap)
        ref = oracle_run(batch, algo, step_cap=cap)
        if cap <= 5:
            assert (ref["status"] == O.E_STEP_CAP).any()
        assert_parity(batch, g, ref)


def test_capacity_overflow_reported(B):
    # 200 requests that all fit at once need more than 64 running slots
    n = 200
    batch = W.from_lists(10 ** 6, [{"prompt": [1] * n, "output": [5] * n, "lower": [5] * n, "upper": [5] * n}])
    g = gpu_run(B, batch, O.HSF, running_capacity=64)
    assert int(g["status"][0]) == -6 and (g["completion"] == -1).all()
    g = gpu_run(B, batch, O.HSF, running_capacity=256)
    assert int(g["status"][0]) == 0 and (g["completion"] == 5).all()


@pytest.mark.parametrize("algo", ["amin", "hsf", "amax", "aell", "adaptive"])
def test_default_passes_after_cancellations(B, algo):
    # 140 long requests are cancelled (A_min, A_l) from step 1 on; a burst of
    # tiny requests at step 3000 then lifts the running set past 320 and 384
    # (the wave continues with more rows), past 512 (a second launch with 640
    # slots simulates the instance again) or past 640 (a third with 1024).
    # The outputs, cancellation counts included, must be those of a run that
    # never outgrew its rows.
    rng = np.random.default_rng(3)
    insts = []
    for burst in (300, 450, 600, 0, 450, 600, 900):
        g1 = 140
        o1 = rng.integers(10, 30, g1)
        o = np.r_[o1, np.ones(burst, int)]
        insts.append({"arrival": np.r_[np.zeros(g1, int), np.full(burst, 3000)],
                      "prompt": np.r_[np.full(g1, 4), np.zeros(burst, int)], "output": o,
                      "lower": np.ones(g1 + burst, int), "upper": o + 2})
    batch = W.from_lists(1000, insts, name="bursts")
    g = gpu_run(B, batch, ALGOS[algo])
    ref = oracle_run(batch, ALGOS[algo])
    assert (ref["status"] == 0).all()
    if algo in ("amin", "aell"):
        assert (ref["total_evictions"] > 0).all()
    assert_parity(batch, g, ref)


def _growth_instances():
    # a first group of long runs is cancelled (A_min) from the first steps; a
    # burst of tiny requests then lifts the running set past 320 while
    # cancelled requests still wait, so the wave continues with more rows in
    # the middle of the churn (and, for some, past 512)
    insts = []
    for seed, (n1, n2, t2, o1max) in [(1, (250, 500, 8, 20)), (1, (300, 600, 12, 30)), (0, (350, 500, 10, 25)),
                                      (2, (250, 500, 8, 20)), (0, (200, 400, 6, 20))]:
        rng = np.random.default_rng(seed)
        o = np.r_[rng.integers(5, o1max + 1, n1), rng.integers(1, 4, n2)]
        insts.append({"arrival": np.r_[np.zeros(n1, int), np.sort(rng.integers(t2, t2 + 4, n2))],
                      "prompt": np.r_[np.ones(n1, int), np.zeros(n2, int)], "output": o,
                      "lower": np.ones(n1 + n2, int), "upper": o + 2})
    return W.from_lists(1600, insts, name="growth")


@pytest.mark.parametrize("algo", ["amin", "hsf", "amax", "aell", "adaptive"])
def test_growth_mid_simulation(B, algo):
    batch = _growth_instances()
    ref = oracle_run(batch, ALGOS[algo])
    assert (ref["status"] == 0).all()
    g = gpu_run(B, batch, ALGOS[algo])
    assert_parity(batch, g, ref)
    # the same bits from one launch that never runs out of rows
    g1 = gpu_run(B, batch, ALGOS[algo], running_capacity=1024)
    for f in ("status", "tel", "makespan", "request_steps", "total_evictions", "completion", "evictions"):
        assert np.array_equal(g[f], g1[f]), f


@pytest.mark.parametrize("cap", [18, 30])
def test_growth_then_step_cap(B, cap):
    # the step cap ends the simulation after the running set has outgrown the
    # first rows (crossings at steps 0, 14, 15, 22): partial outputs as the oracle's
    batch = _growth_instances()
    for algo in (O.AMIN, O.HSF):
        ref = oracle_run(batch, algo, step_cap=cap)
        assert (ref["status"] == O.E_STEP_CAP).any()
        assert_parity(batch, gpu_run(B, batch, algo, step_cap=cap), ref)


def _growth_sweep(seed, K=96):
    # random instances whose running sets peak on both sides of 320, 384 and
    # 512 runs: a first group that fills the memory (cancellations under
    # A_min, promotions under A_l) and a burst of short requests a few steps
    # later; every policy's priority input is a random order
    rng = np.random.default_rng(seed)
    insts = []
    for _ in range(K):
        n1, n2 = int(rng.integers(100, 350)), int(rng.integers(150, 550))
        o = np.r_[rng.integers(3, int(rng.integers(8, 40)), n1), rng.integers(1, int(rng.integers(2, 6)), n2)]
        t2 = int(rng.integers(0, 20))
        a = np.r_[np.sort(rng.integers(0, 3, n1)), np.sort(rng.integers(t2, t2 + int(rng.integers(1, 6)), n2))]
        order = np.argsort(a, kind="stable")
        s = np.r_[rng.integers(0, 3, n1), rng.integers(0, 2, n2)]
        l = np.maximum(1, (o * rng.uniform(0.2, 1.0, n1 + n2)).astype(int))
        u = o + rng.integers(0, 4, n1 + n2)
        insts.append({"arrival": a[order], "prompt": s[order], "output": o[order], "lower": l[order],
                      "upper": u[order], "priority": rng.permutation(n1 + n2)})
    return W.from_lists(1400, insts, name=f"growth_sweep{seed}")


@pytest.mark.parametrize("seed", [0, 1])
@pytest.mark.parametrize("name", ["amin", "amax", "hsf", "aell", "adaptive", "arandom"])
def test_growth_random_sweep(B, seed, name):
    algo = O.ALGOS[name]
    batch = _growth_sweep(seed)
    ref = oracle_run(batch, algo)
    assert (ref["status"] == 0).all()
    g = gpu_run(B, batch, algo)
    assert_parity(batch, g, ref)
    g1 = gpu_run(B, batch, algo, running_capacity=1024)
    for f in ("status", "tel", "makespan", "request_steps", "total_evictions", "completion", "evictions"):
        assert np.array_equal(g[f], g1[f]), f


def _arrival_word_sweep(seed, K=128):
    # fresh requests keep arriving while earlier ones wait: arrivals land in
    # the bitmap word of the current smallest waiting rank (often below it:
    # short outputs arriving late), words empty as their requests start and
    # refill later; memory is tight so the waiting set stays long
    rng = np.random.default_rng(1000 + seed)
    M = int(rng.integers(80, 400))
    insts = []
    for _ in range(K):
        n = int(rng.integers(60, 400))
        o = rng.integers(1, int(rng.integers(4, 60)), n)
        a = np.sort(rng.integers(0, int(rng.integers(1, 200)), n))
        s = rng.integers(0, 6, n)
        l = np.maximum(1, (o * rng.uniform(0.1, 1.0, n)).astype(int))
        u = o + rng.integers(0, 10, n)
        insts.append({"arrival": a, "prompt": s, "output": o, "lower": l, "upper": u,
                      "priority": rng.permutation(n)})
    return W.from_lists(M, insts, name=f"arrival_word_sweep{seed}")


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", ["amin", "amax", "hsf", "aell", "adaptive", "arandom"])
def test_arrivals_into_waiting_words(B, seed, name):
    algo = O.ALGOS[name]
    batch = _arrival_word_sweep(seed)
    ref = oracle_run(batch, algo)
    assert (ref["status"] == 0).all()
    assert_parity(batch, gpu_run(B, batch, algo), ref)


def test_determinism_and_chunking(B):
    batch = W.generate("batch4096_n1000_m16384", 0, instance_ids=range(1000, 1300))
    a = gpu_run(B, batch, O.AMIN)
    b = gpu_run(B, batch, O.AMIN)
    for f in a:
        if a[f] is not None:
            assert np.array_equal(a[f], b[f]), f
    h1 = gpu_run(B, batch.subset(range(0, 150)), O.AMIN)
    h2 = gpu_run(B, batch.subset(range(150, 300)), O.AMIN)
    assert np.array_equal(np.concatenate([h1["tel"], h2["tel"]]), a["tel"])
    assert np.array_equal(np.concatenate([h1["completion"], h2["completion"]]), a["completion"])
