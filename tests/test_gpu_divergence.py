"""The step-cap bisection (tests/divergence.py) with the GPU path on one side:
no divergence from the oracle, and with one request's output made a token
longer on the oracle's side (a planted mistake), exactly that request's
completion step under policies that plan with l or u."""
import dataclasses

import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from divergence import _one, first_divergence
from test_gpu_parity import B, gpu_run  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("algo", [O.AMAX, O.AMIN, O.AELL])
def test_gpu_against_oracle_and_planted(B, algo):
    batch = W.random_small(4, 4, 40, s_max=4, o_max=10, M=30)
    gpu = lambda b, T: gpu_run(B, b, algo, step_cap=T)
    ora = lambda b, T: O.simulate_batch(b, algo, step_cap=T)
    assert first_divergence(batch, gpu, ora) == []
    if algo == O.AELL:
        return
    ref = O.simulate_batch(batch, algo)
    k = 1
    lo, hi = int(batch.offsets[k]), int(batch.offsets[k + 1])
    i = next(j for j in range(lo, hi) if batch.output[j] < batch.upper[j])
    out = batch.output.copy()
    out[i] += 1
    one_b = _one(dataclasses.replace(batch, output=out), k)
    found = first_divergence(_one(batch, k), gpu, lambda b, T: ora(one_b, T))
    assert found == [(0, int(ref["completion"][i]))]
