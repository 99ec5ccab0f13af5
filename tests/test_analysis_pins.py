"""Pins of the oracle of the competitive-ratio analysis (Sections 4.1 and 5):
each check ties a literal, exact-arithmetic evaluation to something other
than itself -- a second form the paper prints, a value derived by hand, an
independent exact computation, or a limit the paper proves."""
import random
from fractions import Fraction as F

import pytest

from oracle import analysis_oracle as AO


def a_closed(i, j):
    # the Corollary's simplified entry: min^2/(ij) * ((i+j)^2/2 - min^2)
    m = min(i, j)
    return F(m * m, i * j) * (F((i + j) ** 2, 2) - m * m)


def test_a_entries_sum_form_equals_closed_form():
    # the proof's sum and the Corollary's statement are two printed forms of a_ij
    for i in range(1, 31):
        for j in range(1, 31):
            assert AO.a_entry_sum(i, j) == a_closed(i, j)


@pytest.mark.parametrize("seed", range(3))
def test_rayleigh_quotient_equals_lemma(seed):
    # Corollary: at s = 0, l = 1 the Lemma's ratio is x'Ax / x'Bx for every x
    rng = random.Random(seed)
    for u in (1, 2, 3, 5, 8):
        x = [F(rng.randint(0, 9), 7) for _ in range(u)]
        if not any(x):
            x[0] = F(1)
        assert AO.rayleigh(x, u) == AO.lemma_cr({k + 1: x[k] for k in range(u)}, 0, 1, u)


def test_lemma_two_point_equals_theorem51_closed_form():
    # proof of Theorem 5.1: with outputs in {l, u} and s = 0 the Lemma reduces
    # to 1 + alpha(1 - alpha^2) t / (alpha^2 t^2 + 2 alpha^2 t + 1), t = x_l / x_u,
    # which never exceeds (3 - alpha) / 2
    for l, u in ((1, 2), (2, 8), (3, 7), (5, 20)):
        for t in (F(0), F(1, 3), F(1), F(5, 2), F(9)):
            x = {l: t / (1 + t), u: 1 / (1 + t)}
            cr = AO.lemma_cr(x, 0, l, u)
            alpha = F(l, u)
            assert cr == AO.two_point_closed_form(alpha, t)
            assert cr <= (3 - alpha) / 2


def test_lemma_point_mass_is_one():
    # all mass at l: A_min plans every request with its true length and never
    # cancels, so its ratio to the hindsight schedule is 1
    for s in (0, 3):
        for l, u in ((1, 5), (4, 9)):
            assert AO.lemma_cr({l: F(1)}, s, l, u) == 1


def test_lambda_max_small_cases():
    # u = 1: a_11 = b_11 = 1.  u = 2: A = [[1, 7/4], [7/4, 4]], B = [[1, 1], [1, 4]],
    # det(A - lam B) = 4(1 - lam)^2 - (7/4 - lam)^2, roots 1/4 and 5/4 (by hand)
    tol = F(1, 10 ** 12)
    assert abs(AO.lambda_max_exact(1, tol) - 1) <= tol
    assert abs(AO.lambda_max_exact(2, tol) - F(5, 4)) <= tol
    assert a_closed(1, 2) == F(7, 4) and a_closed(2, 2) == 4


@pytest.mark.parametrize("u", [3, 5, 8])
def test_lambda_max_bounds(u):
    # the maximum of the Rayleigh quotient is at least its value at any x and
    # at most tr(B^-1 A) = H_u (all eigenvalues are positive; Section 4.1)
    tol = F(1, 10 ** 12)
    lam = AO.lambda_max_exact(u, tol)
    rng = random.Random(u)
    for _ in range(20):
        x = [F(rng.randint(1, 20)) for _ in range(u)]
        assert AO.rayleigh(x, u) <= lam + tol
    assert lam <= AO.harmonic(u)


@pytest.mark.parametrize("u", [1, 2, 3, 6, 12])
def test_b_inverse_tridiagonal_and_trace(u):
    # Section 4.1: B_u^-1 is tridiagonal with 4i/(4i^2-1) (i < u), 1/(2u-1) at
    # (u, u) and -1/(2 min(i,j)+1) beside the diagonal; tr(B_u^-1 A_u) = H_u
    A, B = AO.matrices_exact(u)
    inv = AO.inverse_exact(B)
    for i in range(1, u + 1):
        for j in range(1, u + 1):
            if i == j:
                want = F(4 * i, 4 * i * i - 1) if i < u else F(1, 2 * u - 1)
            elif abs(i - j) == 1:
                want = F(-1, 2 * min(i, j) + 1)
            else:
                want = F(0)
            assert inv[i - 1][j - 1] == want
    tr = sum(inv[i][k] * A[k][i] for i in range(u) for k in range(u))
    assert tr == AO.harmonic(u)


def test_lg_closed_form_limits():
    # Theorem 5.3: the ratio is 1 at q = 0 and its supremum 14/9 at q -> 1
    assert AO.lg_closed_form(F(0)) == 1
    assert AO.lg_closed_form(F(1)) == F(14, 9)
    for q in (F(1, 10), F(1, 2), F(9, 10), F(99, 100)):
        assert 1 <= AO.lg_closed_form(q) <= F(14, 9)


def test_lemma_lg_distribution_tends_to_theorem53():
    # the Lemma with P(o = k) = k p^2 q^(k-1) on [1, u] (renormalised) at s = 0,
    # l = 1 approaches Theorem 5.3's closed form as u grows (tail mass ~ u q^u)
    for q in (F(1, 4), F(1, 2)):
        p = 1 - q
        u = 60
        w = {k: k * p * p * q ** (k - 1) for k in range(1, u + 1)}
        z = sum(w.values())
        x = {k: v / z for k, v in w.items()}
        assert abs(float(AO.lemma_cr(x, 0, 1, u)) - float(AO.lg_closed_form(q))) < 1e-9


def test_aell_two_point_theorem52_shape():
    # Theorem 5.2's expression is 1 + 2 alpha^2 at t = 0 (only long requests)
    # and tends to 1 as t grows (only short requests)
    for alpha in (F(1, 10), F(1, 2), F(9, 10)):
        assert AO.aell_two_point(alpha, F(0)) == 1 + 2 * alpha * alpha
        assert AO.aell_two_point(alpha, F(10 ** 6)) - 1 < F(1, 10 ** 5)
