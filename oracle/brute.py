"""Oracle: exhaustive enumeration on tiny inputs.

Test infrastructure only (see the package header).  Used to pin the exact
solvers of the other modules.

* ``nnls_enumerate``: every support A of the cone problem (Sec. 3.3.1,
  Eq. (proj) over the cone), w_A = K_AA^-1 s_A, keep the feasible candidate
  with the smallest objective 1/2 w^T K w - s^T w.
* ``topk_enumerate``: every k-subset, maximise the exact (rational) sum of
  scores; among maximisers take the lexicographically smallest sorted index
  tuple, which is the lowest-index tie break.
* ``subset_projection``: the exact Global Subset Update of Sec. 3.3.2,
  argmin over |S| = k of ||g_S - g_star_hat||^2 with g_S the subset mean.
"""

import itertools
from fractions import Fraction

import numpy as np


def nnls_enumerate(K, s):
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    best, best_f = np.zeros(n), 0.0
    for r in range(1, n + 1):
        for A in itertools.combinations(range(n), r):
            A = list(A)
            try:
                wA = np.linalg.solve(K[np.ix_(A, A)], s[A])
            except np.linalg.LinAlgError:
                continue
            if np.any(wA < 0):
                continue
            w = np.zeros(n)
            w[A] = wA
            f = 0.5 * w @ (K @ w) - s @ w
            if f < best_f:
                best, best_f = w, f
    return best


def topk_enumerate(s, k):
    s = [Fraction(float(v)) for v in np.asarray(s, dtype=np.float64)]
    n = len(s)
    best, best_sum = None, None
    for S in itertools.combinations(range(n), k):
        tot = sum((s[i] for i in S), Fraction(0))
        if best_sum is None or tot > best_sum:
            best, best_sum = S, tot
    return np.array(best if best is not None else (), dtype=np.int64)


def subset_projection(G, gbar, k):
    G = np.asarray(G, dtype=np.float64)
    gbar = np.asarray(gbar, dtype=np.float64)
    best, best_v = None, None
    for S in itertools.combinations(range(G.shape[0]), k):
        gS = G[list(S)].mean(axis=0)
        v = float(np.sum((gS - gbar) ** 2))
        if best_v is None or v < best_v - 1e-12 * max(1.0, abs(best_v)):
            best, best_v = S, v
    return np.array(best, dtype=np.int64), best_v
