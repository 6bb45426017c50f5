"""Oracle: the exact per-sample scorers of Sec. 4.3 and the compressed one.

Test infrastructure only (see the package header).

For one linear layer with retained pairs (a, dL/de) the alignment score of a
general example i against the mean target gradient is
    s_i = < g_star_hat , g_i >          (Sec. 3.3.2, alignment term)
Sec. 4.3 gives three exact ways to evaluate it, differing only in the order
of the contractions:
* Direct: materialise g_i and the mean target gradient, take the inner
  product.
* Ghost Inner Product (GIP): (1/m) sum_j < D_i D*_j^T , X_i X*_j^T >, two
  T x T cross-correlations per (train, target) pair.
* Per-Token Inner Product (PIP): sum_tau dL/de_{i,tau}^T  G_star_hat  a_{i,tau}.
Compressed scoring replaces the two gradients by their sketches and takes
the inner product in sketch space (Sec. 4.3.3).

Rows are token-major here ([T, d]); the paper stores tokens as columns, which
only transposes the T x T products.  Padding rows (tau >= len) are dropped.

Parity: the three exact scorers pin each other (they must agree to float64
rounding) and pin sketch_ref with identity projectors.
"""

import numpy as np

from .sketch import per_example_gradient


def _valid(a, length):
    return np.asarray(a, dtype=np.float64)[: int(length)]


def _mean_target_gradient(xs, dys, lens):
    m = len(xs)
    G = None
    for x, dy, L in zip(xs, dys, lens):
        g = per_example_gradient(x, dy, L)
        G = g if G is None else G + g
    return G / m


def score_direct(x, dy, lens, xt, dyt, lens_t):
    """Direct scorer: s_i = <mean_j G*_j, G_i> with explicit gradients.

    x [n, T, d_in], dy [n, T, d_out], lens [n]; xt, dyt, lens_t for the m
    target examples.  Returns float64 [n].
    """
    Gs = _mean_target_gradient(xt, dyt, lens_t)
    return np.array([np.sum(Gs * per_example_gradient(x[i], dy[i], lens[i]))
                     for i in range(len(x))])


def score_gip(x, dy, lens, xt, dyt, lens_t):
    """Ghost Inner Product: (1/m) sum_j sum_{tau,tau'} (D_i D*_j^T)(X_i X*_j^T)."""
    m = len(xt)
    out = np.zeros(len(x))
    for i in range(len(x)):
        Xi, Di = _valid(x[i], lens[i]), _valid(dy[i], lens[i])
        acc = 0.0
        for j in range(m):
            Xj, Dj = _valid(xt[j], lens_t[j]), _valid(dyt[j], lens_t[j])
            acc += np.sum((Di @ Dj.T) * (Xi @ Xj.T))
        out[i] = acc / m
    return out


def score_pip(x, dy, lens, xt, dyt, lens_t):
    """Per-Token Inner Product: sum_tau dy_tau^T  G*  x_tau with G* the mean target gradient."""
    Gs = _mean_target_gradient(xt, dyt, lens_t)
    out = np.zeros(len(x))
    for i in range(len(x)):
        Xi, Di = _valid(x[i], lens[i]), _valid(dy[i], lens[i])
        out[i] = sum(float(Di[t] @ (Gs @ Xi[t])) for t in range(Xi.shape[0]))
    return out


def score_compressed(S_train, S_target):
    """Compressed scoring: s_i = <mean_j S*_j, S_i> in sketch space."""
    S_train = np.asarray(S_train, dtype=np.float64)
    gbar = np.asarray(S_target, dtype=np.float64).mean(axis=0)
    return S_train @ gbar
