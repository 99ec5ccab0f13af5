"""The seeded input generator: determinism, per-instance independence, ranges, bins."""
from fractions import Fraction

import numpy as np
import pytest

from paper_2508_14544_amd import workloads as W


def test_bins_match_exact_ceil_and_known_tables():
    # bins start at 1; u = ceil(l * (1 + alpha)) exactly; the next bin starts at u + 1
    known = {
        Fraction(1, 2): [(1, 2), (3, 5), (6, 9), (10, 15), (16, 24), (25, 38), (39, 59), (60, 90)],
        Fraction(1, 1): [(1, 2), (3, 6), (7, 14), (15, 30), (31, 62), (63, 126), (127, 254), (255, 510)],
        Fraction(1, 10): [(1, 2), (3, 4), (5, 6), (7, 8), (9, 10), (11, 13), (14, 16), (17, 19)],
        Fraction(2, 1): [(1, 3), (4, 12), (13, 39), (40, 120), (121, 363), (364, 1092)],
        Fraction(1, 4): [(1, 2), (3, 4), (5, 7), (8, 10), (11, 14), (15, 19), (20, 25), (26, 33)],
    }
    for alpha, bins in known.items():
        tab = W.geometric_bins(alpha, 2000)
        for lo, hi in bins:
            assert tab[0][lo] == lo and tab[1][lo] == hi and tab[0][min(hi, 2000)] == lo
    for alpha in [Fraction(k, 20) for k in range(0, 41)]:
        tab = W.geometric_bins(alpha, 5000)
        for o in range(1, 5001):
            l, u = int(tab[0][o]), int(tab[1][o])
            assert l <= o <= u
            assert Fraction(u) >= l * (1 + alpha) > u - 1  # u = ceil(l (1 + alpha))
    # the exact rule differs from a float ceil(l * 1.1) on some bin starts
    import math
    tab = W.geometric_bins(Fraction(1, 10), 5000)
    starts = sorted(set(int(x) for x in tab[0][1:]))
    assert any(math.ceil(l * 1.1) != int(tab[1][l]) for l in starts)


def test_deterministic_and_subset_independent():
    a = W.generate("batch4096_n1000_m16384", 0, instance_ids=[5, 1400, 4095])
    b = W.generate("batch4096_n1000_m16384", 0, instance_ids=[4095])
    assert np.array_equal(a.instance(2)["output"], b.instance(0)["output"])
    c = W.generate("batch4096_n1000_m16384", 0, instance_ids=[5, 1400, 4095])
    for f in ("arrival", "prompt", "output", "lower", "upper"):
        assert np.array_equal(getattr(a, f), getattr(c, f))
    d = W.generate("batch4096_n1000_m16384", 1, instance_ids=[5])
    assert not np.array_equal(a.instance(0)["output"], d.instance(0)["output"])


@pytest.mark.parametrize("name,ids", [
    ("single_n200_m512", [0]),
    ("batch4096_n1000_m16384", [0, 1365, 4095]),
    ("online1024_n10000_m65536", [0, 1023]),
    ("single_n100000_m1048576", [0]),
    ("sweep65536_n2000_m32768", [0, 7281, 65535]),
])
def test_ranges(name, ids):
    w = W.WORKLOADS[name]
    b = W.generate(name, 0, instance_ids=ids, with_upper=True)
    assert b.M == w.M and b.max_requests == w.n and b.num_instances == len(ids)
    assert np.all(b.lower >= 1) and np.all(b.lower <= b.output) and np.all(b.output <= b.upper)
    assert np.all(b.prompt + b.upper <= b.M)
    for k in range(b.num_instances):
        a = b.instance(k)["arrival"]
        assert np.all(a >= 0) and np.all(np.diff(a) >= 0)
    ranges = {
        "single_n200_m512": ((1, 16), (1, 64)),
        "batch4096_n1000_m16384": ((1, 64), (1, 512)),
        "online1024_n10000_m65536": ((8, 256), (1, 2048)),
        "single_n100000_m1048576": ((16, 2048), (1, 4096)),
        "sweep65536_n2000_m32768": ((1, 128), (1, 1024)),
    }[name]
    assert ranges[0][0] <= b.prompt.min() and b.prompt.max() <= ranges[0][1]
    assert ranges[1][0] <= b.output.min() and b.output.max() <= ranges[1][1]


def test_distribution_shapes():
    b = W.generate("online1024_n10000_m65536", 0, instance_ids=[3])
    a = b.arrival
    rate = len(a) / (a[-1] + 1)
    assert 3.8 < rate < 4.2                          # Poisson arrivals, 4 per step
    assert 120 < np.median(b.output) < 180           # lognormal(5, 1): median e^5 ~ 148
    s = W.generate("sweep65536_n2000_m32768", 0, instance_ids=[9000])
    short = np.mean(s.output <= 64)
    assert 0.67 < short < 0.73                       # 70 % short outputs
    assert np.all((s.output <= 64) | (s.output >= 512))
    g = W.generate("single_n100000_m1048576", 0)
    assert g.arrival.max() <= 19999 and abs(g.prompt.mean() - 1032) < 10


def test_alpha_blocks():
    idx = W._alpha_blocks(4096, [0, 1, 2])
    assert np.bincount(idx).tolist() == [1365, 1365, 1366]
    idx = W._alpha_blocks(65536, list(range(9)))
    assert np.bincount(idx).tolist() == [7281] * 8 + [7288]


def test_twopoint_recipe():
    b = W.generate("twopoint4096_n1000_m16384", 0, instance_ids=[0, 681, 682, 2045, 2046, 4095])
    alphas = [Fraction(1, 10), Fraction(1, 10), Fraction(1, 5), Fraction(3, 10), Fraction(2, 5), Fraction(3, 5)]
    for j in range(b.num_instances):
        inst = b.instance(j)
        lk, uk = int(inst["lower"][0]), int(inst["upper"][0])
        assert (inst["lower"] == lk).all() and (inst["upper"] == uk).all()
        assert 2 <= lk <= 64
        a = alphas[j]
        assert uk == -((-lk * a.denominator) // a.numerator)  # ceil(l / alpha)
        assert set(np.unique(inst["output"])) <= {lk, uk}
        assert 0.4 < (inst["output"] == uk).mean() < 0.6
        assert (inst["arrival"] == 0).all()
        assert str(a) == b.meta["alpha"][j]


def test_experiment_recipe():
    # Section 6's statistics (prompts mean 41, median 11; outputs mean 85, median 43)
    # approximately, nested sizes, and the three interval settings
    b = W.experiment("exp1", 2000, 16)
    s, o = b.prompt, b.output
    assert 1 <= s.min() and s.max() <= 468 and 1 <= o.min() and o.max() <= 883
    assert 36 < s.mean() < 45 and np.median(s) in (10, 11, 12)
    assert 72 < o.mean() < 88 and 40 <= np.median(o) <= 48
    assert (b.lower == 1).all() and (b.upper == 1000).all() and (b.arrival == 0).all()
    small = W.experiment("exp1", 200, 16)
    for k in range(16):
        assert (small.instance(k)["output"] == b.instance(k)["output"][:200]).all()
    e2 = W.experiment("exp2", 2000, 4)
    assert ((e2.lower - 1) % 100 == 0).all() and (e2.upper - e2.lower == 99).all()
    assert ((e2.lower <= e2.output) & (e2.output <= e2.upper)).all()
    e3 = W.experiment("exp3_x95", 2000, 4)
    oo = e3.output.astype(np.int64)
    assert (e3.lower == np.maximum(1, 5 * oo // 100)).all()
    assert (e3.upper == -((-195 * oo) // 100)).all()


def test_chunked_generation_equals_drawing_at_once(monkeypatch):
    # large batches are drawn in chunks of instances; every instance has its
    # own random streams, so the result is the same batch
    import paper_2508_14544_amd.workloads as WW
    a = W.generate("batch4096_n1000_m16384", 0, instance_ids=range(100, 400))
    monkeypatch.setattr(WW, "_CHUNK_REQUESTS", 1 << 15)
    b = W.generate("batch4096_n1000_m16384", 0, instance_ids=range(100, 400))
    for f in ("offsets", "arrival", "prompt", "output", "lower", "upper", "instance_ids"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    assert a.meta["alpha"] == b.meta["alpha"]
    assert W.generate("sweep65536_n2000_m32768", 0, instance_ids=range(3)).upper is None
