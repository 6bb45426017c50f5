"""Oracle: the other subset rules of Sec. 3.3.2 (thresholding, greedy).

Test infrastructure only (see the package header).

With a subset S the update is the subset average g_S = (1/|S|) sum_{i in S} g_i,
and the projection objective of Eq. (proj) over subsets reduces, after
dropping the term that does not depend on S, to
    f(S) = ||g_S||^2 - 2 <g_S, g_star_hat>
         = (1/|S|^2) sum_{i,i' in S} K_ii'  -  (2/|S|) sum_{i in S} s_i
(alignment versus redundancy, Sec. 3.3.2).  Top-k drops the redundancy
term; the two rules here are:

* Thresholding: keep every example whose score exceeds a fixed threshold
  (a subset of variable size).  Negative score filtering (the rule of the
  RL experiments of Sec. 5, whose data-regularization settings the
  experimental appendix gives) is the case that keeps the non-negative
  scores.
  Readings: "exceeds" is strict (s_i > tau); negative filtering keeps
  s_i >= 0, so the rule takes an `inclusive` switch; w_i = 1/|S| on S (the
  subset average), all zero when nothing is kept; a NaN score is an error.
* Greedy construction: start from the empty set and add, k times, the
  example whose addition gives the smallest f (the full objective, so the
  redundancy term is accounted for at every step).  Readings: exactly k
  additions (the same k as top-k); ties go to the lowest index; a NaN in K
  or s is an error.  The set is returned in ascending index order.

Parity: pinned by tests (hand fixtures; greedy equals top-k when K is a
multiple of the identity; k = 1 closed form; every greedy step is the best
single addition by brute force; thresholding against direct comparisons).
"""

import numpy as np


def threshold_ref(s, tau, inclusive=False):
    """Kept indices (ascending) and weights 1/|S| on them."""
    s = np.asarray(s, dtype=np.float64)
    if np.isnan(s).any():
        raise ValueError("NaN score")
    keep = [i for i in range(s.shape[0]) if (s[i] >= tau if inclusive else s[i] > tau)]
    w = np.zeros(s.shape[0])
    if keep:
        w[keep] = 1.0 / len(keep)
    return np.array(keep, dtype=np.int64), w


def subset_objective(K, s, S):
    """f(S) = (1/|S|^2) 1^T K_SS 1 - (2/|S|) 1^T s_S (the S-dependent part of
    ||g_S - g_star_hat||^2)."""
    S = list(S)
    t = len(S)
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    return K[np.ix_(S, S)].sum() / t ** 2 - 2.0 * s[S].sum() / t


def greedy_ref(K, s, k):
    """Greedy subset of size k (ascending indices) and the order of addition.

    Each step evaluates, for every candidate c outside S,
        f(S + c) = (A + 2 r_c + K_cc) / t^2 - 2 (B + s_c) / t,   t = |S| + 1
    with A = sum_{i,i' in S} K_ii', B = sum_{i in S} s_i, r_c = sum_{i in S} K_ic,
    and keeps the smallest (lowest index on ties).
    """
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    if not 0 <= k <= n:
        raise ValueError("k must satisfy 0 <= k <= n")
    if np.isnan(K).any() or np.isnan(s).any():
        raise ValueError("NaN input")
    chosen = []
    in_set = np.zeros(n, dtype=bool)
    diag = np.diag(K).copy()
    A = 0.0
    B = 0.0
    r = np.zeros(n)
    for step in range(k):
        t = float(step + 1)
        # f(S + c) for every candidate at once (the same operations, in the
        # same order, as the formula above applied to each c)
        f = (A + 2.0 * r + diag) / (t * t) - 2.0 * (B + s) / t
        f[in_set] = np.inf
        best = int(np.argmin(f))          # first minimum: lowest index on ties
        A = A + 2.0 * r[best] + K[best, best]
        B = B + s[best]
        r = r + K[best]
        in_set[best] = True
        chosen.append(best)
    return np.array(sorted(chosen), dtype=np.int64), np.array(chosen, dtype=np.int64)
