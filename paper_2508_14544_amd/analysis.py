"""Competitive-ratio numerics of A_min (arXiv 2508.14544, Sections 4.1 and 5):
small dense problems solved on the host with LAPACK (numpy / scipy).

* ``lemma_cr``: the Lemma of Section 4.1, the fluid (M -> infinity)
  competitive ratio of A_min for an output distribution x on [l, u] and
  prompt size s, in O(u) with suffix sums.
* ``matrices``: A_u and B_u of the Corollary of Section 4.1 (s = 0, l = 1),
  whose Rayleigh quotient x'A_u x / x'B_u x is that ratio.
* ``lambda_max``: the largest generalised eigenvalue of (A_u, B_u) and its
  eigenvector (LAPACK's symmetric-definite solver).  When the eigenvector is
  positive, rescaled it is the worst output distribution on [1, u] and the
  eigenvalue is A_min's competitive ratio at alpha = 1/u (Figure 1's curve).
* ``b_inverse`` and ``trace_c``: the tridiagonal inverse of B_u stated in
  Section 4.1 and tr(B_u^-1 A_u), which the paper shows equals H_u.
* ``two_point_cr``, ``aell_two_point_cr``, ``lg_cr_closed``: Theorems 5.1,
  5.2 and 5.3; ``geometric_cr`` and ``lg_cr``: the Lemma on geometric and
  linearly weighted geometric outputs (Figure 2).
* ``fit_log``: least-squares fit of a*ln(u + b) + c, the form of Figure 1.

``python -m paper_2508_14544_amd.analysis`` prints Figure 1's curve against
the paper's fitted function, the refitted parameters, and Figure 2's maxima.
"""
from __future__ import annotations

import argparse
import json
import time
from typing import Dict, Optional, Sequence

import numpy as np

# Figure 1's fitted curve, as printed: 0.2555 ln(u + 0.2793) + 1.1587 (s = 0, l = 1)
FIG1_FIT = (0.2555, 0.2793, 1.1587)


def lemma_cr(x: Sequence[float], s: int, l: int) -> float:
    """The Lemma of Section 4.1 (without its O(1/M) term).  x[j] is the mass
    of output length l + j, for lengths l .. u = l + len(x) - 1."""
    x = np.asarray(x, dtype=np.float64)
    u = l + len(x) - 1
    k = np.arange(l, u + 1, dtype=np.float64)
    delta = np.ones_like(k)
    delta[0] = s + l
    suffix = lambda v: np.cumsum(v[::-1])[::-1]   # sum over i >= k
    after = lambda v: np.concatenate([suffix(v)[1:], [0.0]])  # sum over i > k
    s1 = suffix(k * x)                 # sum_{i>=k} i x_i
    s2 = suffix(x / (s + k))           # sum_{i>=k} x_i / (s + i)
    s3 = after(k * x / (s + k)) - k * after(x / (s + k))   # sum_{i>k} (i - k) x_i / (s + i)
    num = np.sum(delta * s1 * (delta * s2 + 2.0 * s3))
    den = np.sum(k * (s + k) * x * (x + 2.0 * after(x)))
    return float(num / den)


def matrices(u: int):
    """A_u and B_u of the Corollary: a_ij = m^2/(ij) ((i+j)^2/2 - m^2),
    b_ij = m^2, m = min(i, j)."""
    i = np.arange(1, u + 1, dtype=np.float64)
    I, J = np.meshgrid(i, i, indexing="ij")
    m = np.minimum(I, J)
    A = m * m / (I * J) * (0.5 * (I + J) ** 2 - m * m)
    B = m * m
    return A, B


def rayleigh(x: Sequence[float]) -> float:
    x = np.asarray(x, dtype=np.float64)
    A, B = matrices(len(x))
    return float(x @ A @ x / (x @ B @ x))


def lambda_max(u: int):
    """(largest generalised eigenvalue of (A_u, B_u), its eigenvector rescaled
    to sum 1 with a positive first entry)."""
    from scipy.linalg import eigh
    A, B = matrices(u)
    w, v = eigh(A, B, subset_by_index=[u - 1, u - 1])
    vec = v[:, 0]
    vec = vec / vec.sum()
    return float(w[0]), vec


def b_inverse(u: int) -> np.ndarray:
    """Section 4.1's tridiagonal inverse of B_u: 4i/(4i^2-1) on the diagonal
    for i < u, 1/(2u-1) at (u, u), -1/(2 min(i,j)+1) beside the diagonal."""
    i = np.arange(1, u + 1, dtype=np.float64)
    inv = np.diag(4 * i / (4 * i * i - 1))
    inv[u - 1, u - 1] = 1.0 / (2 * u - 1)
    off = -1.0 / (2 * i[:-1] + 1)
    inv[np.arange(u - 1), np.arange(1, u)] = off
    inv[np.arange(1, u), np.arange(u - 1)] = off
    return inv


def trace_c(u: int) -> float:
    """tr(B_u^-1 A_u) from the diagonal and first off-diagonals (B_u^-1 is
    tridiagonal and A_u symmetric), in O(u)."""
    i = np.arange(1, u + 1, dtype=np.float64)
    a_diag = i * i                                             # a_ii = (2i)^2/2 - i^2
    d = 4 * i / (4 * i * i - 1)
    d[-1] = 1.0 / (2 * u - 1)
    j = i[:-1]
    a_off = j / (j + 1) * (0.5 * (2 * j + 1) ** 2 - j * j)     # a_{i,i+1}
    return float(np.sum(d * a_diag) + 2 * np.sum(-1.0 / (2 * j + 1) * a_off))


def two_point_cr(alpha, t):
    """Theorem 5.1's closed form (s = 0): 1 + alpha(1-alpha^2) t / (alpha^2 t^2 + 2 alpha^2 t + 1)."""
    alpha, t = np.asarray(alpha, np.float64), np.asarray(t, np.float64)
    a2 = alpha * alpha
    return 1 + alpha * (1 - a2) * t / (a2 * t * t + 2 * a2 * t + 1)


def aell_two_point_cr(alpha, t):
    """Theorem 5.2: 1 + (alpha^2 t + 2 alpha^2) / (alpha^2 t^2 + 2 alpha^2 t + 1)."""
    alpha, t = np.asarray(alpha, np.float64), np.asarray(t, np.float64)
    a2 = alpha * alpha
    return 1 + (a2 * t + 2 * a2) / (a2 * t * t + 2 * a2 * t + 1)


def lg_cr_closed(q):
    """Theorem 5.3 (u, M -> infinity, s = 0, l = 1)."""
    q = np.asarray(q, np.float64)
    num = (1 + q) ** 2 * (1 + 3 * q + 6 * q ** 2 + 3 * q ** 3 + q ** 4)
    den = 1 + 2 * q + 11 * q ** 2 + 8 * q ** 3 + 11 * q ** 4 + 2 * q ** 5 + q ** 6
    return num / den


def geometric_cr(q: float, u: int) -> float:
    """The Lemma (s = 0, l = 1) for P(o = k) proportional to q^(k-1) on [1, u]."""
    k = np.arange(1, u + 1, dtype=np.float64)
    return lemma_cr(q ** (k - 1), 0, 1)


def lg_cr(q: float, u: int) -> float:
    """The Lemma (s = 0, l = 1) for P(o = k) proportional to k q^(k-1) on [1, u]."""
    k = np.arange(1, u + 1, dtype=np.float64)
    return lemma_cr(k * q ** (k - 1), 0, 1)


def fit_log(us: np.ndarray, ys: np.ndarray):
    """Least-squares a*ln(u + b) + c through (us, ys); returns (a, b, c), R^2."""
    from scipy.optimize import curve_fit
    f = lambda u, a, b, c: a * np.log(u + b) + c
    (a, b, c), _ = curve_fit(f, us, ys, p0=FIG1_FIT, bounds=([0, -0.99, -10], [10, 100, 10]))
    res = ys - f(us, a, b, c)
    r2 = 1 - np.sum(res ** 2) / np.sum((ys - ys.mean()) ** 2)
    return (float(a), float(b), float(c)), float(r2)


def fig1_curve(u_max: int = 1000, us: Optional[Sequence[int]] = None) -> Dict[str, object]:
    us = np.arange(1, u_max + 1) if us is None else np.asarray(us)
    t0 = time.perf_counter()
    lam = np.empty(len(us))
    positive = True
    for n, u in enumerate(us):
        lam[n], vec = lambda_max(int(u))
        positive &= bool((vec > 0).all())
    secs = time.perf_counter() - t0
    return {"u": us, "lambda_max": lam, "eigvec_positive": positive, "seconds": secs}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--u-max", type=int, default=1000)
    ap.add_argument("--json", default="")
    a = ap.parse_args(argv)
    fig = fig1_curve(a.u_max)
    us, lam = fig["u"].astype(np.float64), fig["lambda_max"]
    paper = FIG1_FIT[0] * np.log(us + FIG1_FIT[1]) + FIG1_FIT[2]
    sel = [u for u in (1, 2, 5, 10, 20, 50, 100, 200, 500, 1000, 2000) if u <= a.u_max]
    print("Figure 1: competitive ratio of A_min (s = 0, l = 1) against u = 1/alpha")
    print("| u | lambda_max(A_u, B_u) | paper's fit | H_u (trace bound) |")
    print("|---|---|---|---|")
    for u in sel:
        print(f"| {u} | {lam[u - 1]:.4f} | {paper[u - 1]:.4f} | {trace_c(u):.4f} |")
    mask = us >= 10
    (fa, fb, fc), r2 = fit_log(us[mask], lam[mask])
    gap = np.abs(lam - paper)
    print(f"refit on u in [10, {a.u_max}]: {fa:.4f} ln(u + {fb:.4f}) + {fc:.4f}, R^2 = {r2:.6f}")
    print(f"max |lambda_max - paper's fit| for u >= 100: {gap[us >= 100].max():.4f}; "
          f"top eigenvectors all positive: {fig['eigvec_positive']}; {len(us)} eigenproblems in {fig['seconds']:.2f} s")
    qs = np.linspace(0.0, 0.999, 1000)
    g = np.array([geometric_cr(q, 400) for q in qs])
    lg = np.array([lg_cr(q, 400) for q in qs])
    print(f"Figure 2 (u = 400): max over q of geometric CR = {g.max():.4f} at q = {qs[g.argmax()]:.3f}; "
          f"LG CR = {lg.max():.4f} at q = {qs[lg.argmax()]:.3f}; Theorem 5.3 limit 14/9 = {14 / 9:.4f}")
    if a.json:
        json.dump({"u": us.tolist(), "lambda_max": lam.tolist(), "fit": [fa, fb, fc], "r2": r2,
                   "geometric_max": float(g.max()), "lg_max": float(lg.max())}, open(a.json, "w"))


if __name__ == "__main__":
    main()
