"""The step-cap bisection that locates the first divergent (instance, step)
of two simulations (tests/divergence.py), checked on the CPU with a mistake
planted on one side: one request's output made one token longer.  The policy
plans with l or u, not o, so both sides decide alike until that request's
original completion step, where one side completes it and the other does not
(a run holds s + o at its last step on both sides): the bisection must name
exactly that step."""
import dataclasses

import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from divergence import _one, first_divergence


def _oracle(algo):
    return lambda b, T: O.simulate_batch(b, algo, step_cap=T)


@pytest.mark.parametrize("algo", [O.AMAX, O.AMIN])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_bisection_finds_the_planted_step(algo, seed):
    batch = W.random_small(seed, 6, 40, s_max=4, o_max=10, M=30)
    ref = O.simulate_batch(batch, algo)
    assert (ref["status"] == 0).all()
    rng = np.random.default_rng(seed)
    k = int(rng.integers(0, batch.num_instances))
    lo, hi = int(batch.offsets[k]), int(batch.offsets[k + 1])
    cand = [i for i in range(lo, hi) if batch.output[i] < batch.upper[i]]
    i = cand[int(rng.integers(0, len(cand)))]
    out = batch.output.copy()
    out[i] += 1
    planted = dataclasses.replace(batch, output=out)
    one_a, one_b = _one(batch, k), _one(planted, k)
    found = first_divergence(one_a, _oracle(algo), lambda b, T: _oracle(algo)(one_b, T))
    assert found == [(0, int(ref["completion"][i]))]
    # over the whole batch, only instance k differs
    run_b = lambda b, T: _oracle(algo)(one_b if b.name.endswith(f"[{k}]") else b, T)
    assert first_divergence(batch, _oracle(algo), run_b) == [(k, int(ref["completion"][i]))]


def test_identical_sides_agree():
    batch = W.random_small(3, 4, 30, s_max=4, o_max=10, M=30)
    assert first_divergence(batch, _oracle(O.HSF), _oracle(O.HSF)) == []
