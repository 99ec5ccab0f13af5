"""Plain oracle of the competitive-ratio analysis of A_min (arXiv 2508.14544,
Sections 4.1 and 5).

TEST INFRASTRUCTURE ONLY: tests compare the analysis module of the package
against these slow, literal evaluations.  Nothing in the product imports this
file.  Every function works in exact rational arithmetic (fractions.Fraction)
unless it says otherwise, and follows the paper's formulas term by term:

* ``lemma_cr``: the Lemma of Section 4.1 (the fluid competitive ratio of A_min
  for an output distribution x on [l, u] and prompt size s), its double sums
  written out as loops.
* ``a_entry_sum`` / ``b_entry``: the entries of A_u and B_u of the Corollary of
  Section 4.1 (s = 0, l = 1), A_u taken from the sum in the Corollary's proof
  (Appendix) before it is simplified.
* ``lambda_max_exact``: the largest generalised eigenvalue of (A_u, B_u) (the
  maximum of the Rayleigh quotient, B_u being positive definite), by bisection
  on the number of eigenvalues above a point, counted exactly from the signs
  of the pivots of A_u - lam B_u (Sylvester's law of inertia).
* ``inverse_exact``: B_u^{-1} by exact Gauss-Jordan elimination.
* ``two_point_closed_form``: the closed form in the proof of Theorem 5.1.
* ``aell_two_point``: Theorem 5.2's expression for A_l.
* ``lg_closed_form``: Theorem 5.3 (linearly weighted geometric outputs).
"""
from fractions import Fraction
from typing import Dict, List, Sequence


def delta(s: int, l: int, k: int) -> Fraction:
    """delta_{s,l}(k) of the Lemma: s + l at k = l, else 1."""
    return Fraction(s + l) if k == l else Fraction(1)


def lemma_cr(x: Dict[int, Fraction], s: int, l: int, u: int) -> Fraction:
    """The Lemma of Section 4.1 without its O(1/M) term; x maps each length
    k in [l, u] to its probability (missing keys are 0)."""
    X = lambda i: Fraction(x.get(i, 0))
    num = Fraction(0)
    for k in range(l, u + 1):
        d = delta(s, l, k)
        first = sum((i * X(i) for i in range(k, u + 1)), Fraction(0))
        second = sum((d / (s + i) * X(i) for i in range(k, u + 1)), Fraction(0))
        third = sum((Fraction(i - k, s + i) * X(i) for i in range(k + 1, u + 1)), Fraction(0))
        num += d * first * (second + 2 * third)
    den = Fraction(0)
    for k in range(l, u + 1):
        tail = sum((X(i) for i in range(k + 1, u + 1)), Fraction(0))
        den += k * (s + k) * X(k) * (X(k) + 2 * tail)
    return num / den


def a_entry_sum(i: int, j: int) -> Fraction:
    """a_ij from the sum in the proof of the Corollary: half of
    (1/ij) sum_{k=1}^{min(i,j)} (i^2 (1 + 2j - 2k) + j^2 (1 + 2i - 2k))."""
    m = min(i, j)
    tot = sum(i * i * (1 + 2 * j - 2 * k) + j * j * (1 + 2 * i - 2 * k) for k in range(1, m + 1))
    return Fraction(tot, 2 * i * j)


def b_entry(i: int, j: int) -> Fraction:
    return Fraction(min(i, j) ** 2)


def matrices_exact(u: int):
    A = [[a_entry_sum(i, j) for j in range(1, u + 1)] for i in range(1, u + 1)]
    B = [[b_entry(i, j) for j in range(1, u + 1)] for i in range(1, u + 1)]
    return A, B


def inverse_exact(M: List[List[Fraction]]) -> List[List[Fraction]]:
    """Inverse by Gauss-Jordan elimination over the rationals."""
    n = len(M)
    aug = [row[:] + [Fraction(int(i == j)) for j in range(n)] for i, row in enumerate(M)]
    for c in range(n):
        p = next(r for r in range(c, n) if aug[r][c] != 0)
        aug[c], aug[p] = aug[p], aug[c]
        piv = aug[c][c]
        aug[c] = [v / piv for v in aug[c]]
        for r in range(n):
            if r != c and aug[r][c] != 0:
                f = aug[r][c]
                aug[r] = [a - f * b for a, b in zip(aug[r], aug[c])]
    return [row[n:] for row in aug]


def rayleigh(x: Sequence[Fraction], u: int) -> Fraction:
    A, B = matrices_exact(u)
    num = sum(x[i] * A[i][j] * x[j] for i in range(u) for j in range(u))
    den = sum(x[i] * B[i][j] * x[j] for i in range(u) for j in range(u))
    return num / den


def count_above(A, B, lam: Fraction) -> int:
    """Number of generalised eigenvalues of (A, B) above lam: by Sylvester's law
    of inertia (B positive definite), the number of positive pivots of the
    symmetric elimination of A - lam B, run without row exchanges.  Returns -1
    when a pivot is exactly zero (lam hits a root of a leading minor)."""
    u = len(A)
    S = [[A[i][j] - lam * B[i][j] for j in range(u)] for i in range(u)]
    pos = 0
    for c in range(u):
        piv = S[c][c]
        if piv == 0:
            return -1
        pos += piv > 0
        for r in range(c + 1, u):
            f = S[r][c] / piv
            if f:
                for q in range(c + 1, u):
                    S[r][q] -= f * S[c][q]
    return pos


def lambda_max_exact(u: int, tol: Fraction = Fraction(1, 10 ** 15)) -> Fraction:
    """The largest generalised eigenvalue of (A_u, B_u), the maximum of the
    Rayleigh quotient, to within tol: bisection on count_above >= 1 between 0
    (A_u is positive definite, so every eigenvalue is above 0) and a doubled
    upper end with nothing above it."""
    A, B = matrices_exact(u)

    def above(lam):
        c = count_above(A, B, lam)
        while c < 0:  # a zero pivot: move off the root of that minor
            lam += tol / 7
            c = count_above(A, B, lam)
        return c

    lo, hi = Fraction(0), Fraction(1)
    while above(hi) > 0:
        lo, hi = hi, hi * 2
    while hi - lo > tol:
        mid = (lo + hi) / 2
        if above(mid) > 0:
            lo = mid
        else:
            hi = mid
    return (lo + hi) / 2


def harmonic(u: int) -> Fraction:
    return sum((Fraction(1, i) for i in range(1, u + 1)), Fraction(0))


def two_point_closed_form(alpha: Fraction, t: Fraction) -> Fraction:
    """Proof of Theorem 5.1 (s = 0): 1 + alpha (1 - alpha^2) t / (alpha^2 t^2 + 2 alpha^2 t + 1),
    with t = x_l / x_u."""
    return 1 + alpha * (1 - alpha * alpha) * t / (alpha * alpha * t * t + 2 * alpha * alpha * t + 1)


def aell_two_point(alpha: Fraction, t: Fraction) -> Fraction:
    """Theorem 5.2: the competitive ratio of A_l on two-point outputs,
    1 + (alpha^2 t + 2 alpha^2) / (alpha^2 t^2 + 2 alpha^2 t + 1)."""
    a2 = alpha * alpha
    return 1 + (a2 * t + 2 * a2) / (a2 * t * t + 2 * a2 * t + 1)


def lg_closed_form(q: Fraction) -> Fraction:
    """Theorem 5.3: (1+q)^2 (1 + 3q + 6q^2 + 3q^3 + q^4) / (1 + 2q + 11q^2 + 8q^3 + 11q^4 + 2q^5 + q^6)."""
    num = (1 + q) ** 2 * (1 + 3 * q + 6 * q ** 2 + 3 * q ** 3 + q ** 4)
    den = 1 + 2 * q + 11 * q ** 2 + 8 * q ** 3 + 11 * q ** 4 + 2 * q ** 5 + q ** 6
    return num / den
