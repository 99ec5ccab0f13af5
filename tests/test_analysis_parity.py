"""The competitive-ratio numerics of the package (numpy / LAPACK) against the
exact-rational oracle, at sizes the oracle finishes in seconds, and against
properties and printed values at full size (u up to 1000, Figure 1's range)."""
import random
from fractions import Fraction as F

import numpy as np
import pytest

from oracle import analysis_oracle as AO
from paper_2508_14544_amd import analysis as AN


@pytest.mark.parametrize("seed", range(4))
def test_lemma_cr_against_oracle(seed):
    rng = random.Random(seed)
    for _ in range(6):
        l = rng.randint(1, 4)
        u = l + rng.randint(0, 25)
        s = rng.randint(0, 5)
        x = [F(rng.randint(0, 12), 11) for _ in range(u - l + 1)]
        if not any(x):
            x[-1] = F(1)
        want = float(AO.lemma_cr({l + j: v for j, v in enumerate(x)}, s, l, u))
        got = AN.lemma_cr([float(v) for v in x], s, l)
        assert abs(got - want) <= 1e-12 * want


def test_matrices_and_rayleigh_against_oracle():
    A, B = AN.matrices(15)
    Ae, Be = AO.matrices_exact(15)
    assert np.allclose(A, np.array(Ae, dtype=float), rtol=1e-14, atol=0)
    assert np.array_equal(B, np.array(Be, dtype=float))
    x = [F(k % 5 + 1, 3) for k in range(12)]
    assert abs(AN.rayleigh([float(v) for v in x]) - float(AO.rayleigh(x, 12))) < 1e-13


@pytest.mark.parametrize("u", range(1, 11))
def test_lambda_max_against_oracle(u):
    lam, vec = AN.lambda_max(u)
    want = AO.lambda_max_exact(u, F(1, 10 ** 13))
    assert abs(lam - float(want)) < 1e-11
    assert (vec > 0).all() and abs(vec.sum() - 1) < 1e-12
    # the eigenvector attains the maximum of the Rayleigh quotient
    assert abs(AN.rayleigh(vec) - lam) < 1e-11


@pytest.mark.parametrize("u", [1, 2, 5, 12])
def test_b_inverse_against_oracle(u):
    _, Be = AO.matrices_exact(u)
    assert np.allclose(AN.b_inverse(u), np.array(AO.inverse_exact(Be), dtype=float), rtol=0, atol=1e-15)


@pytest.mark.parametrize("u", [50, 300, 1000])
def test_full_size_properties(u):
    # B_u^-1 B_u = I; tr(B_u^-1 A_u) = H_u; 1 <= lambda_max <= H_u; a positive
    # top eigenvector (so the maximum over distributions is the eigenvalue)
    A, B = AN.matrices(u)
    assert np.allclose(AN.b_inverse(u) @ B, np.eye(u), atol=1e-9)
    h = float(sum(1.0 / i for i in range(1, u + 1)))
    assert abs(AN.trace_c(u) - h) < 1e-10 * h
    lam, vec = AN.lambda_max(u)
    assert 1 <= lam <= h and (vec > 0).all()


@pytest.mark.parametrize("u", [100, 300, 1000])
def test_figure1_fitted_curve(u):
    # Figure 1 prints 0.2555 ln(u + 0.2793) + 1.1587 as a fit with R^2 > 0.9999
    lam, _ = AN.lambda_max(u)
    a, b, c = AN.FIG1_FIT
    assert abs(lam - (a * np.log(u + b) + c)) < 0.005


def test_closed_forms_against_oracle():
    for alpha in (F(1, 10), F(3, 8), F(1, 2), F(9, 10)):
        for t in (F(0), F(1, 2), F(3), F(40)):
            assert abs(AN.two_point_cr(float(alpha), float(t)) - float(AO.two_point_closed_form(alpha, t))) < 1e-15
            assert abs(AN.aell_two_point_cr(float(alpha), float(t)) - float(AO.aell_two_point(alpha, t))) < 1e-15
    for q in (F(0), F(1, 3), F(7, 8), F(1)):
        assert abs(AN.lg_cr_closed(float(q)) - float(AO.lg_closed_form(q))) < 1e-15


def test_figure2_curves():
    # Figure 2: geometric outputs stay below 1.7; linearly weighted geometric
    # outputs approach Theorem 5.3's closed form (at most 14/9)
    qs = np.linspace(0.0, 0.99, 100)
    assert max(AN.geometric_cr(q, 400) for q in qs) <= 1.7
    for q in (0.2, 0.6, 0.9):
        assert abs(AN.lg_cr(q, 600) - AN.lg_cr_closed(q)) < 1e-9
    assert max(AN.lg_cr(q, 600) for q in qs) <= 14 / 9 + 1e-12
