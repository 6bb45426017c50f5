"""Oracle: target mean, Gram matrix and scores per parameter group.

Test infrastructure only (see the package header).

Definitions followed
--------------------
* Mean target gradient g_star_hat = (1/m) sum_j g*_j (Sec. 3.2, batch
  gradients); in sketch space the mean of the m target sketches.
* Alignment scores s_i = <g_i, g_star_hat> and the redundancy term
  (1/k^2) sum_{i,i' in S} <g_i, g_i'> (Sec. 3.3.2, Global Subset Update).
  The Gram matrix K = G G^T collects every <g_i, g_i'>.
* Group-wise decomposition (Sec. 3.3.3): for a partition of the coordinates
  into groups p, every quantity above is formed on the group's sub-vectors.
  Groups are column ranges [goff[p], goff[p+1]) of the sketch matrix.
* t2_p = ||g_star_hat^(p)||^2, the constant term of ||u - g_star_hat||^2.

Parity: pinned by tests (brute-force double loops, symmetry / PSD / diagonal
invariants, linearity of the scores in the target rows, redundancy identity).
"""

import numpy as np


def gram_ref(G, Gt, goff=None):
    """Per-group Gram matrix, scores and squared target norm.

    G  [n, kappa] general-data sketches; Gt [m, kappa] target sketches.
    goff: group column offsets, length P+1 (None: one group, all columns).
    Returns (K [P, n, n], s [P, n], t2 [P]) in float64.
    """
    G = np.asarray(G, dtype=np.float64)
    Gt = np.asarray(Gt, dtype=np.float64)
    n, kappa = G.shape
    if goff is None:
        goff = [0, kappa]
    P = len(goff) - 1
    m = Gt.shape[0]
    K = np.zeros((P, n, n))
    s = np.zeros((P, n))
    t2 = np.zeros(P)
    for p in range(P):
        a, b = int(goff[p]), int(goff[p + 1])
        Gp = G[:, a:b]
        gbar = Gt[:, a:b].sum(axis=0) / m if m > 0 else np.zeros(b - a)
        K[p] = Gp @ Gp.T
        s[p] = Gp @ gbar
        t2[p] = gbar @ gbar
    return K, s, t2
