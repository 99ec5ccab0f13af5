"""The Section 6 analogue on the GPU: every policy's outputs on sampled
replicates equal the CPU oracle's, for every prediction setting."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2508_14544_amd import workloads as W
from test_gpu_parity import B, assert_parity, gpu_run, oracle_run  # noqa: F401 (B is a fixture)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("setting", W.EXP_SETTINGS)
def test_experiment_cells_against_oracle(B, setting):
    for n in (200, 2000):
        batch = W.experiment(setting, n, 8)
        ks = [0, 7] if n == 2000 else list(range(8))
        for algo in (O.AMAX, O.AMIN, O.HSF, O.AELL, O.ADAPTIVE):
            g = gpu_run(B, batch, algo)
            assert (g["status"] == 0).all()
            assert_parity(batch, g, oracle_run(batch, algo, instances=ks), instances=ks)
