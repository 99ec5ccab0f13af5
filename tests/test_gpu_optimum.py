"""The hindsight optimum of tiny instances on the GPU (sched_optimum) against
the oracle's exhaustive search, and the paper's printed OPT values."""
import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B  # noqa: F401 (fixture)

pytestmark = pytest.mark.gpu


def gpu_opt(B, batch, **kw):
    import torch
    db = B.to_device(batch)
    out = B.optimum(db, **kw)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def test_paper_examples_opt(B):
    here = os.path.join(os.path.dirname(__file__), "golden")
    n_checked = 0
    for f in sorted(x for x in os.listdir(here) if x.endswith(".json")):
        g = json.load(open(os.path.join(here, f)))
        if "instance" in g and "opt_tel" in g:
            batch = W.from_lists(g["M"], [g["instance"]], name=f)
            r = gpu_opt(B, batch)
            assert int(r["status"][0]) == 0 and int(r["tel"][0]) == g["opt_tel"], f
            n_checked += 1
    assert n_checked >= 2


@pytest.mark.parametrize("seed,arrivals", [(0, False), (1, True), (2, False)])
def test_random_tiny_against_oracle(B, seed, arrivals):
    b = W.random_small(seed + 40, 30, 6, s_max=3, o_max=5, M=12, arrivals=arrivals)
    r = gpu_opt(B, b)
    assert (r["status"] == 0).all()
    ref = [O.opt_tel(b.instance(k), b.M) for k in range(b.num_instances)]
    assert r["tel"].tolist() == ref
    # OPT is a lower bound of every policy (per instance); a policy's total as
    # the starting bound gives the same optimum
    import torch
    for algo in (O.AMAX, O.AMIN, O.HSF):
        tel = O.simulate_batch(b, algo)["tel"]
        assert (r["tel"] <= tel).all()
        rb = gpu_opt(B, b, upper_bound=torch.from_numpy(tel).cuda())
        assert rb["tel"].tolist() == ref


def test_closed_forms(B):
    from test_oracle_pins import spt_single_machine_tel
    rng = np.random.default_rng(11)
    excl, roomy = [], []
    for _ in range(200):
        n = int(rng.integers(1, 9))
        o = rng.integers(1, 8, n).tolist()
        # runs that never overlap leave the search only its weak bound (sum of
        # o): every order is explored, so keep these to n <= 6
        excl.append({"prompt": rng.integers(11, 14, min(n, 6)).tolist(), "output": o[:6]})
        roomy.append({"prompt": rng.integers(0, 3, n).tolist(), "output": o})
    r = gpu_opt(B, W.from_lists(20, excl, name="opt_exclusive"), node_cap=1 << 26)
    assert (r["status"] == 0).all()
    assert r["tel"].tolist() == [spt_single_machine_tel(i["output"]) for i in excl]
    r = gpu_opt(B, W.from_lists(16 + 7 * 8, roomy, name="opt_roomy"))
    assert (r["status"] == 0).all()
    assert r["tel"].tolist() == [sum(i["output"]) for i in roomy]


def test_statuses_and_node_cap(B):
    good = {"arrival": [0, 0, 1], "prompt": [1, 2, 1], "output": [3, 2, 4]}
    # the last one: a search horizon (max a + sum(o + 1) + 1) of 2^27 is not searched
    insts = [good, dict(good, arrival=[1, 0, 1]), dict(good, output=[0, 2, 4]), dict(good, prompt=[1, 2, 9]),
             {"arrival": [], "prompt": [], "output": []}, dict(good, arrival=[(1 << 27) - 10] * 3)]
    r = gpu_opt(B, W.from_lists(10, insts, name="opt_status"))
    assert r["status"].tolist() == [0, O.E_ARRIVAL, O.E_INTERVAL, O.E_TOO_BIG, 0, B.E_UNSUPPORTED]
    assert r["tel"][0] == O.opt_tel(good, 10) and r["tel"][4] == 0
    b = W.random_small(3, 20, 8, s_max=2, o_max=8, M=14, arrivals=False)
    capped = gpu_opt(B, b, node_cap=5)
    full = gpu_opt(B, b)
    hit = capped["status"] == O.E_STEP_CAP
    assert hit.any()
    assert (capped["tel"][hit] >= full["tel"][hit]).all()   # an upper bound when the search was cut


def _pool_golden():
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "opt_pool_tiny8.json")))
    insts = [{f: i[f] for f in ("arrival", "prompt", "output")} for i in g["instances"]]
    return g, insts


def test_device_wide_second_search(B):
    # eight-request instances whose search outlasts the first launch's budget
    # (2^17 start steps per wave): their optimum comes from the second launch,
    # in which every workgroup claims pieces of any unfinished instance.  The
    # oracle's values are stored (tests/golden/make_opt_pool.py); alone, among
    # easy instances, and with a policy's total as the starting bound.
    import torch
    g, insts = _pool_golden()
    ref = [i["opt_tel"] for i in g["instances"]]
    r = gpu_opt(B, W.from_lists(g["M"], insts, name="opt_pool"))
    assert (r["status"] == 0).all()
    assert (r["nodes"] > (1 << 17)).all()
    assert r["tel"].tolist() == ref
    easy = W.random_small(7, 300, 6, s_max=3, o_max=5, M=g["M"], arrivals=False)
    mixed = [{f: easy.instance(k)[f] for f in ("arrival", "prompt", "output")} for k in range(300)]
    pos = list(range(0, 300, 300 // len(insts)))[:len(insts)]
    for p, inst in zip(reversed(pos), reversed(insts)):
        mixed.insert(p, inst)
    b = W.from_lists(g["M"], mixed, name="opt_pool_mixed")
    r = gpu_opt(B, b)
    at = [p + i for i, p in enumerate(pos)]
    assert (r["status"] == 0).all()
    assert r["tel"][at].tolist() == ref
    rest = [k for k in range(b.num_instances) if k not in at]
    assert r["tel"][rest[:40]].tolist() == [O.opt_tel(b.instance(k), b.M) for k in rest[:40]]
    hsf = O.simulate_batch(b, O.HSF)["tel"]
    rb = gpu_opt(B, b, upper_bound=torch.from_numpy(hsf).cuda())
    assert rb["tel"].tolist() == r["tel"].tolist()
    assert (r["tel"] <= hsf).all()


def test_device_wide_second_search_node_cap(B):
    # a budget just above the first launch's: the second search may run out on
    # some piece; an instance it gives up on reports SCHED_E_STEP_CAP with a
    # schedule at least as long as the optimum, the others the optimum
    g, insts = _pool_golden()
    ref = np.array([i["opt_tel"] for i in g["instances"]])
    r = gpu_opt(B, W.from_lists(g["M"], insts, name="opt_pool_cap"), node_cap=(1 << 17) + 64)
    ok = r["status"] == 0
    assert ((r["status"] == 0) | (r["status"] == O.E_STEP_CAP)).all()
    assert (r["tel"][ok] == ref[ok]).all()
    assert (r["tel"][~ok] >= ref[~ok]).all()
