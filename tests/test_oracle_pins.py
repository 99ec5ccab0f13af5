"""Pins of the CPU oracle to things other than itself (no GPU needed).

* worked examples the paper prints (Example 1, Example 2) and two examples
  derived by hand from Algorithms 2/4 (tests/golden/*.json);
* a closed form the paper states: H-SF's total latency on the instance built in
  the proof of Theorem 3.2;
* a closed form of the memory model: identical requests with s >= 1 run in
  batches that restart one step after completion (a completing run still
  holds s+o at its completion step);
* a second, independently written step loop that evaluates equation (2)
  densely at every step (``literal_simulate``), fuzzed against the C oracle;
* brute-force hindsight optimum on tiny instances (OPT <= every algorithm);
* an event-log auditor (memory <= M before and after evictions at every step,
  completion = start + o, equation (3), evictions only on overflow);
* reductions: exact predictions make A_min = A_max = H-SF; l = o makes
  A_min = H-SF; a huge M makes every completion a + o.
"""
import glob
import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W

FIELDS_I = ("status", "tel", "makespan", "request_steps", "total_evictions")
FIELDS_A = ("completion", "evictions")


def same(r1, r2):
    return all(r1[f] == r2[f] for f in FIELDS_I) and all(np.array_equal(r1[f], r2[f]) for f in FIELDS_A)


def _golden_files():
    here = os.path.join(os.path.dirname(__file__), "golden")
    files = sorted(glob.glob(os.path.join(here, "*.json")))
    return [f for f in files if "instance" in json.load(open(f))]


@pytest.mark.parametrize("path", _golden_files(), ids=lambda p: os.path.basename(p))
def test_golden_examples(path):
    g = json.load(open(path))
    inst, M = g["instance"], g["M"]
    for name, exp in g["expected"].items():
        algo = O.ALGOS[name]
        r = O.simulate(inst, algo, M, events=True)
        assert r["status"] == O.OK
        for k, v in exp.items():
            if k == "starts":
                starts = {}
                for (t, kind, i) in r["events"]:
                    if kind == O.EV_START:
                        starts[i] = t
                assert [starts[i] for i in range(len(v))] == v
            elif k in FIELDS_A:
                assert r[k].tolist() == v, (name, k)
            else:
                assert r[k] == v, (name, k)
        O.audit(inst, algo, M, r)
        assert same(r, O.literal_simulate(inst, algo, M))
    if "opt_tel" in g:
        assert O.opt_tel(inst, M) == g["opt_tel"]


@pytest.mark.parametrize("l,u,a,b,seed", [(2, 8, 10, 20, 0), (3, 12, 15, 30, 2), (4, 9, 12, 18, 3), (1, 4, 5, 10, 4)])
def test_hsf_closed_form_theorem32_instance(l, u, a, b, seed):
    # Proof of Theorem 3.2: s=0, M=l*u, a*u jobs of length l and b*l of length u.
    # H-SF runs the short jobs in a batches of u and then the long ones in b
    # batches of l:  TEL = u*l*(1+..+a) + b*l*a*l + u*l*(1+..+b).
    rng = np.random.default_rng(seed)
    o = np.array([l] * (a * u) + [u] * (b * l))
    rng.shuffle(o)
    n = len(o)
    inst = {"prompt": np.zeros(n, int), "output": o, "lower": np.full(n, l), "upper": np.full(n, u)}
    r = O.simulate(inst, O.HSF, l * u)
    assert r["tel"] == u * l * a * (a + 1) // 2 + b * l * a * l + u * l * b * (b + 1) // 2


@pytest.mark.parametrize("s,k,m,B", [(1, 3, 4, 5), (2, 5, 3, 7), (4, 1, 6, 4)])
def test_identical_requests_batches(s, k, m, B):
    # n = m*B identical requests (prompt s>=1, output k, exact prediction), M = m*(s+k).
    # A batch of m fills M exactly at its completion step k, so the next batch
    # can only start one step later: batch j completes at j*(k+1) + k.
    n = m * B
    inst = {"prompt": [s] * n, "output": [k] * n, "lower": [k] * n, "upper": [k] * n}
    expect = np.repeat(np.arange(B) * (k + 1) + k, m)
    for algo in (O.AMAX, O.AMIN, O.HSF):
        r = O.simulate(inst, algo, m * (s + k))
        assert r["completion"].tolist() == expect.tolist()
        assert r["tel"] == int(expect.sum())
        assert r["request_steps"] == n * k


@pytest.mark.parametrize("seed", range(4))
def test_c_oracle_equals_literal_dense_eq2(seed):
    b = W.random_small(seed, 120, 7, s_max=5, o_max=8, M=20, arrivals=(seed % 2 == 0))
    n_ev = 0
    for k in range(b.num_instances):
        inst = b.instance(k)
        for algo in (O.AMAX, O.AMIN, O.HSF):
            r = O.simulate(inst, algo, b.M)
            assert same(r, O.literal_simulate(inst, algo, b.M)), (k, algo)
            n_ev += r["total_evictions"]
    assert n_ev > 0  # the eviction path was exercised


@pytest.mark.parametrize("seed", range(3))
def test_audit_invariants(seed):
    b = W.random_small(10 + seed, 150, 10, s_max=6, o_max=10, M=30, arrivals=(seed != 1))
    for k in range(b.num_instances):
        inst = b.instance(k)
        for algo in (O.AMAX, O.AMIN, O.HSF):
            O.audit(inst, algo, b.M, O.simulate(inst, algo, b.M, events=True))


def test_audit_on_generated_workloads():
    for name, ids in (("single_n200_m512", [0]), ("batch4096_n1000_m16384", [2731])):
        b = W.generate(name, 0, instance_ids=ids)
        inst = b.instance(0)
        for algo in (O.AMAX, O.AMIN, O.HSF):
            O.audit(inst, algo, b.M, O.simulate(inst, algo, b.M, events=True))


def test_audit_rejects_planted_overflow():
    # The auditor must notice a schedule that breaks equation (1).
    inst = {"prompt": [1, 1], "output": [3, 3], "lower": [1, 1], "upper": [3, 3]}
    r = O.simulate(inst, O.HSF, 4, events=True)
    bad = dict(r)
    bad["events"] = [(0, O.EV_START, 0), (0, O.EV_START, 1), (3, O.EV_COMPLETE, 0), (3, O.EV_COMPLETE, 1)]
    bad["completion"] = np.array([3, 3], np.int32)
    bad["tel"], bad["makespan"], bad["request_steps"] = 6, 3, 6
    with pytest.raises(AssertionError):
        O.audit(inst, O.HSF, 4, bad)


@pytest.mark.parametrize("seed", range(2))
def test_opt_is_a_lower_bound(seed):
    b = W.random_small(100 + seed, 40, 5, s_max=3, o_max=4, M=10, arrivals=(seed == 0))
    for k in range(b.num_instances):
        inst = b.instance(k)
        opt = O.opt_tel(inst, b.M)
        for algo in (O.AMAX, O.AMIN, O.HSF):
            assert opt <= O.simulate(inst, algo, b.M)["tel"]


def spt_single_machine_tel(o):
    """Sum of completion times when runs cannot overlap: a run of output o
    occupies o + 1 steps and shortest-first sequencing is optimal (Smith's
    rule); the j-th run in ascending o completes at sum_{k<=j}(o_k + 1) - 1."""
    t, total = 0, 0
    for x in sorted(int(v) for v in o):
        total += t + x
        t += x + 1
    return total


@pytest.mark.parametrize("seed", range(3))
def test_opt_closed_forms(seed):
    rng = np.random.default_rng(seed)
    for _ in range(15):
        n = int(rng.integers(1, 6))
        o = rng.integers(1, 8, n)
        # two prompts together exceed M: no two runs ever overlap
        M = 20
        inst = {"prompt": rng.integers(11, 14, n), "output": o}
        assert O.opt_tel(inst, M) == spt_single_machine_tel(o)
        # room for every run at once: each completes at o
        inst = {"prompt": rng.integers(0, 5, n), "output": o}
        assert O.opt_tel(inst, int(sum(inst["prompt"]) + sum(o))) == int(sum(o))


def test_reduction_exact_predictions_all_equal():
    from fractions import Fraction
    b = W.random_small(7, 100, 10, s_max=6, o_max=10, M=30, alpha=Fraction(0))
    for k in range(b.num_instances):
        inst = b.instance(k)
        rs = [O.simulate(inst, a, b.M) for a in (O.AMAX, O.AMIN, O.HSF)]
        assert same(rs[0], rs[2]) and same(rs[1], rs[2])
    # a generated batch instance with alpha = 0
    g = W.generate("sweep65536_n2000_m32768", 0, instance_ids=[3], with_upper=True)
    inst = g.instance(0)
    assert np.array_equal(inst["lower"], inst["output"])
    rs = [O.simulate(inst, a, g.M) for a in (O.AMAX, O.AMIN, O.HSF)]
    assert same(rs[0], rs[2]) and same(rs[1], rs[2])


def test_reduction_lower_equals_output_amin_is_hsf():
    b = W.random_small(8, 100, 10, s_max=6, o_max=10, M=30)
    for k in range(b.num_instances):
        inst = dict(b.instance(k))
        inst["lower"] = inst["output"]
        assert same(O.simulate(inst, O.AMIN, b.M), O.simulate(inst, O.HSF, b.M))


def test_reduction_huge_memory_and_single_request():
    b = W.random_small(9, 50, 10, s_max=6, o_max=10, M=30)
    for k in range(b.num_instances):
        inst = b.instance(k)
        for algo in (O.AMAX, O.AMIN, O.HSF):
            r = O.simulate(inst, algo, 10 ** 6)
            assert r["completion"].tolist() == (inst["arrival"] + inst["output"]).tolist()
            one = {f: (None if v is None else v[:1]) for f, v in inst.items()}
            r1 = O.simulate(one, algo, b.M)
            assert r1["completion"].tolist() == [int(inst["arrival"][0] + inst["output"][0])]


def test_step_cap_and_error_codes():
    inst = {"prompt": [1, 1], "output": [3, 3], "lower": [1, 1], "upper": [3, 3]}
    r = O.simulate(inst, O.AMIN, 4, step_cap=5)
    assert r["status"] == O.E_STEP_CAP and r["completion"].tolist() == [-1, 3]
    assert same(r, O.literal_simulate(inst, O.AMIN, 4, step_cap=5))
    assert O.simulate(inst, O.AMIN, 4, step_cap=7)["status"] == O.OK
    base = {"arrival": [0, 1], "prompt": [1, 1], "output": [3, 3], "lower": [1, 1], "upper": [3, 3]}
    cases = [
        (dict(base, lower=[4, 1]), O.AMIN, O.E_INTERVAL),   # l > o
        (dict(base, lower=[0, 1]), O.AMIN, O.E_INTERVAL),   # l < 1
        (dict(base, upper=[2, 3]), O.AMAX, O.E_INTERVAL),   # u < o
        (dict(base, output=[0, 3]), O.HSF, O.E_INTERVAL),   # o < 1
        (dict(base, prompt=[-1, 1]), O.HSF, O.E_INTERVAL),  # s < 0
        (dict(base, prompt=[2, 1]), O.HSF, O.E_TOO_BIG),    # s + o > M
        (dict(base, upper=[3, 4]), O.AMAX, O.E_TOO_BIG),    # s + u > M
        (dict(base, arrival=[1, 0]), O.HSF, O.E_ARRIVAL),   # not sorted
        (dict(base, arrival=[-1, 0]), O.HSF, O.E_ARRIVAL),  # negative
        (dict(base, arrival=[1, 0], lower=[4, 1]), O.AMIN, O.E_ARRIVAL),  # priority
        (dict(base, prompt=[2, 1], lower=[4, 1]), O.AMIN, O.E_INTERVAL),  # priority
    ]
    for inst_, algo, code in cases:
        r = O.simulate(inst_, algo, 4)
        assert r["status"] == code, (inst_, algo)
        assert r["completion"].tolist() == [-1, -1] and r["tel"] == 0 and r["request_steps"] == 0
    e = O.simulate({"prompt": [], "output": [], "lower": [], "upper": []}, O.AMIN, 4)
    assert e["status"] == O.OK and e["tel"] == 0 and e["makespan"] == 0


@pytest.mark.parametrize("l,u", [(2, 8), (3, 6), (5, 10)])
def test_theorem31_upper_bound_soft(l, u):
    # Theorem 3.1: CR(A_max) <= alpha^-1 (1 + alpha^-1) / 2 + O(1/M), alpha = l/u,
    # with one interval [l, u] shared by all jobs.  Checked on random outputs.
    rng = np.random.default_rng(l * 100 + u)
    alpha = l / u
    bound = (1 / alpha) * (1 + 1 / alpha) / 2
    for trial in range(5):
        n = 300
        o = rng.integers(l, u + 1, n)
        inst = {"prompt": np.ones(n, int), "output": o, "lower": np.full(n, l), "upper": np.full(n, u)}
        M = 40 * (1 + u)
        ratio = O.simulate(inst, O.AMAX, M)["tel"] / O.simulate(inst, O.HSF, M)["tel"]
        assert ratio <= bound


def test_work_counter_definition():
    """The reported algorithmic work count W_alg: per step |S_t| (twice for A_min,
    whose projection reads the running set again), per feasibility test |Q|
    including the candidate, per eviction event |S_t| ceil(log2 |S_t|).  A single
    request (s=1, o=3, ample M) is tested once with |Q| = 1 and runs in steps
    0, 1, 2 (it completes at step 3), so W = 1 + 3 = 4, and 1 + 2*3 = 7 for A_min."""
    inst = {"arrival": np.zeros(1, np.int32), "prompt": np.array([1], np.int32),
            "output": np.array([3], np.int32), "lower": np.array([1], np.int32),
            "upper": np.array([3], np.int32)}
    for algo, want in ((O.AMAX, 4), (O.HSF, 4), (O.AMIN, 7)):
        r = O.simulate(inst, algo, 100, stats=True)
        assert r["stats"]["work"] == want
        assert r["request_steps"] == 3
    # two requests that cannot run together (M = 4, s + o = 4 each), H-SF: the
    # second is refused at steps 0, 1, 2 (|Q| = 2 with the running one) and at
    # step 3, where the run completing at 3 still holds s + o = 4 (|Q| = 2); it is
    # admitted at step 4 (|Q| = 1) and completes at 7.  Tests: 1 + 2+2+2+2 + 1 = 10;
    # request-steps: 1 at steps 0..2, 0 at step 3, 1 at steps 4..6.
    inst2 = {"arrival": np.zeros(2, np.int32), "prompt": np.array([1, 1], np.int32),
             "output": np.array([3, 3], np.int32), "lower": np.array([3, 3], np.int32),
             "upper": np.array([3, 3], np.int32)}
    r = O.simulate(inst2, O.HSF, 4, stats=True)
    assert r["completion"].tolist() == [3, 7]
    assert r["stats"]["tests"] == 6
    assert r["request_steps"] == 6
    assert r["stats"]["work"] == 10 + 6


def _two_point(l, u, a, b, seed, s=0):
    rng = np.random.default_rng(seed)
    o = np.array([l] * (a * u) + [u] * (b * l))
    rng.shuffle(o)
    n = len(o)
    return {"prompt": np.full(n, s), "output": o, "lower": np.full(n, l), "upper": np.full(n, u)}, o


@pytest.mark.parametrize("l,u,a,b,seed", [(2, 8, 3, 5, 0), (3, 12, 4, 6, 1), (4, 9, 10, 10, 2), (5, 20, 6, 4, 3)])
def test_aell_closed_form_theorem52_instance(l, u, a, b, seed):
    # The construction of Theorem 5.2's proof: two-point outputs {l, u}, s = 0,
    # M = l*u, a*u short and b*l long requests in random index order.  A_l plans
    # every fresh request with l: batch j takes requests [j*u, (j+1)*u) at step
    # j*l (they hold l each at their planned end); shorts complete at (j+1)*l,
    # longs are promoted then.  After the B1 = n/u fresh batches the longs run in
    # promotion order, l at a time (u each at the end): batch m completes at
    # B1*l + (m+1)*u.  Runs never overlap a refused step because s = 0.
    inst, o = _two_point(l, u, a, b, seed)
    n = len(o)
    r = O.simulate(inst, O.AELL, l * u)
    b1 = n // u
    tel = sum((i // u + 1) * l for i in range(n) if o[i] == l)
    tel += sum(b1 * l + (q // l + 1) * u for q in range(b * l))
    assert r["tel"] == tel
    assert r["total_evictions"] == b * l
    assert r["request_steps"] == n * l + b * l * u


def test_aell_ratio_approaches_theorem52():
    # Theorem 5.2 (proof, eq. (3)): TEL(A_l)/TEL(H-SF) = 1 + (a^2 t + 2 a^2)/(a^2 t^2
    # + 2 a^2 t + 1) + O(1/M) with a = l/u and t = (#short)/(#long).  The exact
    # H-SF total on the construction is Theorem 3.2's (u*l*(1+..+A) + B*l*A*l +
    # u*l*(1+..+B)); the discrete ratio approaches the limit from below.
    l, u, a, b = 10, 40, 20, 20
    inst, o = _two_point(l, u, a, b, 4)
    M = l * u
    ra = O.simulate(inst, O.AELL, M)["tel"]
    rh = O.simulate(inst, O.HSF, M)["tel"]
    assert rh == u * l * a * (a + 1) // 2 + b * l * a * l + u * l * b * (b + 1) // 2
    al, t = l / u, (a * u) / (b * l)
    limit = 1 + (al ** 2 * t + 2 * al ** 2) / (al ** 2 * t ** 2 + 2 * al ** 2 * t + 1)
    assert limit - 0.01 <= ra / rh <= limit


def test_amin_two_point_theorem51_soft():
    # Theorem 5.1: under two-point outputs CR(A_min) <= (3 - alpha)/2 + O(1/M).
    # Checked (soft, in the limit sense) at M = 4000 on 4000 shuffled requests.
    l, u = 10, 40
    rng = np.random.default_rng(0)
    o = np.array([l] * 2000 + [u] * 2000)
    rng.shuffle(o)
    n = len(o)
    inst = {"prompt": np.ones(n, int), "output": o, "lower": np.full(n, l), "upper": np.full(n, u)}
    ratio = O.simulate(inst, O.AMIN, 4000)["tel"] / O.simulate(inst, O.HSF, 4000)["tel"]
    assert ratio <= (3 - l / u) / 2


def test_aell_reduction_exact_lower_bounds_sorted():
    # With l = o (the lower bound is exact) nothing is ever promoted; if o is
    # non-decreasing in the index, A_l's queue order is H-SF's (o, index) order,
    # so the two schedules coincide.
    b = W.random_small(11, 40, 9, s_max=5, o_max=9, M=25)
    for k in range(b.num_instances):
        inst = dict(b.instance(k))
        order = np.argsort(inst["output"], kind="stable")
        inst = {f: (None if v is None else np.asarray(v)[order]) for f, v in inst.items()}
        inst["arrival"] = np.zeros(len(order), np.int32)
        inst["lower"] = inst["output"].copy()
        inst["upper"] = np.maximum(inst["upper"], inst["output"])
        ra = O.simulate(inst, O.AELL, b.M)
        rh = O.simulate(inst, O.HSF, b.M)
        assert ra["total_evictions"] == 0
        assert same(ra, rh)


@pytest.mark.parametrize("l,u,want", [(1, 3, "aell"), (2, 5, "amin"), (19, 50, "aell"), (191, 500, "amin"),
                                      (1, 1, "amin"), (38, 100, "aell"), (382, 1000, "amin")])
def test_adaptive_switch_threshold(l, u, want):
    # Section 5.1: A_l when alpha = l/u < alpha* = (3 - sqrt 5)/2 = 0.381966...,
    # A_min otherwise; 0.38 < alpha* < 0.382.  ADAPTIVE reproduces the choice.
    rng = np.random.default_rng(l + u)
    n = 30
    o = rng.choice([l, u], n)
    inst = {"prompt": np.ones(n, int), "output": o, "lower": np.full(n, l), "upper": np.full(n, u)}
    assert O.adaptive_choice(inst) == O.ALGOS[want]
    M = 4 * (1 + u)
    assert same(O.simulate(inst, O.ADAPTIVE, M), O.simulate(inst, O.ALGOS[want], M))


@pytest.mark.parametrize("seed", range(3))
def test_aell_c_oracle_equals_literal_and_audit(seed):
    # the C loop against the pure-Python loop with dense equation (2), and the
    # event-log audit (memory before/after each step, promotions at exactly l
    # tokens and only for o > l, once per request)
    b = W.random_small(seed + 20, 60, 8, s_max=5, o_max=9, M=24, arrivals=(seed % 2 == 1), alpha=1.0)
    n_prom = 0
    for k in range(b.num_instances):
        inst = b.instance(k)
        for algo in (O.AELL, O.ADAPTIVE):
            r = O.simulate(inst, algo, b.M, events=True)
            assert same(r, O.literal_simulate(inst, algo, b.M))
            O.audit(inst, algo, b.M, r)
            n_prom += r["total_evictions"]
    assert n_prom > 0


def test_arandom_reductions():
    # A_random plans with the true o (like H-SF) and walks a given random order;
    # with the order of H-SF's key (o, index) it is H-SF bit-exactly
    b = W.random_small(21, 40, 9, s_max=5, o_max=9, M=25)
    for k in range(b.num_instances):
        inst = dict(b.instance(k))
        o = np.asarray(inst["output"])
        rank = np.empty(len(o), np.int32)
        rank[np.lexsort((np.arange(len(o)), o))] = np.arange(len(o))
        inst["priority"] = rank
        assert same(O.simulate(inst, O.ARANDOM, b.M), O.simulate(inst, O.HSF, b.M))


def test_arandom_theorem31_random_order_bound_soft():
    # Appendix (proof of Theorem 3.1): CR(A_random) <= (1 + 1/alpha)/2 + O(1/M),
    # in expectation over the random order; checked on the mean over 12 random
    # orders of two-point instances (the worst case of that theorem), M large.
    l, u = 5, 20
    rng = np.random.default_rng(3)
    n = 600
    o = rng.choice([l, u], n)
    base = {"prompt": np.ones(n, int), "output": o, "lower": np.full(n, l), "upper": np.full(n, u)}
    M = 40 * (1 + u)
    hsf = O.simulate(base, O.HSF, M)["tel"]
    tels = []
    for rep in range(12):
        inst = dict(base, priority=rng.permutation(n).astype(np.int32))
        r = O.simulate(inst, O.ARANDOM, M, events=True)
        O.audit(inst, O.ARANDOM, M, r)
        tels.append(r["tel"])
    assert np.mean(tels) / hsf <= (1 + u / l) / 2


@pytest.mark.parametrize("seed", range(2))
def test_arandom_c_oracle_equals_literal(seed):
    b = W.with_random_order(W.random_small(seed + 30, 60, 8, s_max=5, o_max=9, M=24, arrivals=(seed == 1)), seed)
    for k in range(b.num_instances):
        inst = b.instance(k)
        r = O.simulate(inst, O.ARANDOM, b.M, events=True)
        assert same(r, O.literal_simulate(inst, O.ARANDOM, b.M))
        O.audit(inst, O.ARANDOM, b.M, r)


# ---------------------------------------------------------------------------
# Tie keys: the paper breaks ties among equal planning lengths uniformly at
# random (Algorithm 1's random sample; Algorithm 2's eviction and admission
# sorts); a caller-given tie key is that order, index order without one.
# ---------------------------------------------------------------------------

def _relabel(inst, perm):
    """Instance j of the result is request perm[j] of `inst`."""
    out = {}
    for f, v in inst.items():
        out[f] = None if v is None else np.asarray(v)[perm]
    return out


@pytest.mark.parametrize("seed", range(3))
def test_tie_key_relabelling(seed):
    # Renumber the requests (inside each group of equal arrivals, so arrivals
    # stay sorted) and give each its old index as tie key: every policy must
    # produce the old outputs, renumbered.  A tie decided by the new index
    # anywhere (admission, cancellation, A_l's queue) breaks this.
    rng = np.random.default_rng(40 + seed)
    b = W.random_small(seed + 40, 40, 10, s_max=4, o_max=8, M=22, arrivals=(seed == 2), alpha=1.0)
    b = W.with_random_order(b, seed)
    n_ev = 0
    for k in range(b.num_instances):
        inst = dict(b.instance(k))
        inst.pop("tie_key", None)
        a = np.asarray(inst["arrival"])
        perm = np.concatenate([rng.permutation(np.flatnonzero(a == v)) for v in np.unique(a)]).astype(np.int64)
        new = _relabel(inst, perm)
        new["tie_key"] = perm.astype(np.int32)
        for algo in (O.AMAX, O.AMIN, O.HSF, O.AELL, O.ADAPTIVE, O.ARANDOM):
            r0 = O.simulate(inst, algo, b.M)
            r1 = O.simulate(new, algo, b.M)
            assert all(r0[f] == r1[f] for f in FIELDS_I), (k, algo)
            assert np.array_equal(r0["completion"][perm], r1["completion"]), (k, algo)
            assert np.array_equal(r0["evictions"][perm], r1["evictions"]), (k, algo)
            n_ev += r0["total_evictions"]
    assert n_ev > 0


def test_tie_key_neutral_forms():
    # the identity and a constant tie key both leave index order
    b = W.random_small(50, 40, 9, s_max=4, o_max=8, M=22, alpha=1.0)
    for k in range(b.num_instances):
        inst = dict(b.instance(k))
        n = len(inst["output"])
        for algo in (O.AMAX, O.AMIN, O.HSF, O.AELL):
            r = O.simulate(inst, algo, b.M)
            assert same(r, O.simulate(dict(inst, tie_key=np.arange(n, dtype=np.int32)), algo, b.M))
            assert same(r, O.simulate(dict(inst, tie_key=np.full(n, 7, np.int32)), algo, b.M))


@pytest.mark.parametrize("seed", range(2))
def test_tie_key_c_oracle_equals_literal_and_audit(seed):
    # random tie keys with repeats (ties among tie keys fall back to the index)
    b = W.random_small(seed + 60, 60, 8, s_max=5, o_max=9, M=24, arrivals=(seed == 1), alpha=1.0)
    rng = np.random.default_rng(seed)
    for k in range(b.num_instances):
        inst = dict(b.instance(k))
        inst["tie_key"] = rng.integers(0, 4, len(inst["output"])).astype(np.int32)
        for algo in (O.AMAX, O.AMIN, O.HSF, O.AELL):
            r = O.simulate(inst, algo, b.M, events=True)
            assert same(r, O.literal_simulate(inst, algo, b.M)), (k, algo)
            O.audit(inst, algo, b.M, r)
