"""Oracle: projection of the mean target gradient onto the convex cone of the
general-data gradients (non-negative least squares).

Test infrastructure only (see the package header).

Definitions followed
--------------------
* Eq. (proj), Sec. 3.3.1, with U = { G^T w : w >= 0 }: the conic member of
  the feasible-set family (a reading -- the paper's discussion names the
  simplex of soft weights, whose conic hull this is).  Expanding
  ||G^T w - g_star_hat||^2 gives the equivalent quadratic program
      minimise 1/2 w^T K w - s^T w  subject to  w >= 0,
  with K = G G^T and s = G g_star_hat.
* Exact solution: the Lawson-Hanson active-set method on that quadratic
  program (textbook NNLS; grow a passive set by the most violated dual
  coordinate, solve the unconstrained sub-problem on it, step back to
  feasibility when a coordinate would turn negative).
* Optimality (KKT): w >= 0, grad = K w - s >= 0 and w_i grad_i = 0.
  ``cone_kkt_residual`` measures this on the Jacobi-scaled problem
  (K~ = D^-1/2 K D^-1/2, s~ = D^-1/2 s, w~ = D^1/2 w, D = diag K) as
      rho = max_i |min(w~_i, grad~_i)| / max(max_i |s~_i|, tiny).
* ``cone_pg_replay`` is the iterative solver of the design reading (projected
  gradient on the Jacobi-scaled problem with the Gershgorin step); it is kept
  to check that a fixed iteration budget reaches the exact optimum on the
  workloads, not as the parity reference.

Parity: pinned by tests (scipy.optimize.nnls on the primal least-squares
form, enumeration of every support for n <= 10, KKT, target-in-cone,
all-negative scores, n = 0, hand-solved 2x2 fixture).
"""

import numpy as np


def _objective(K, s, w):
    return 0.5 * w @ (K @ w) - s @ w


def nnls_active_set(K, s, max_outer=None):
    """Exact minimiser of 1/2 w^T K w - s^T w over w >= 0 (K symmetric PSD).

    Returns float64 [n].
    """
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    w = np.zeros(n)
    if n == 0:
        return w
    scale = max(np.abs(K).max(), np.abs(s).max(), 1e-300)
    tol = 64.0 * n * np.finfo(np.float64).eps * scale
    passive = np.zeros(n, dtype=bool)
    max_outer = 3 * n + 10 if max_outer is None else max_outer
    for _ in range(max_outer):
        dual = s - K @ w                     # minus the gradient
        cand = np.where(~passive, dual, -np.inf)
        j = int(np.argmax(cand))
        if passive.all() or cand[j] <= tol:
            break
        passive[j] = True
        while True:
            idx = np.flatnonzero(passive)
            z = np.zeros(n)
            z[idx] = np.linalg.lstsq(K[np.ix_(idx, idx)], s[idx], rcond=None)[0]
            if np.all(z[idx] > 0.0):
                w = z
                break
            bad = idx[z[idx] <= 0.0]
            alpha = np.min(w[bad] / (w[bad] - z[bad]))
            w = w + alpha * (z - w)
            passive &= w > tol / scale * np.maximum(1.0, np.abs(w).max())
            w[~passive] = 0.0
            if not passive.any():
                break
    return w


def cone_kkt_residual(K, s, w):
    """Scaled natural KKT residual rho of a candidate w (see header)."""
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n = s.shape[0]
    if n == 0:
        return 0.0
    d = np.diag(K)
    r = np.where(d > 0, 1.0 / np.sqrt(np.where(d > 0, d, 1.0)), 0.0)
    wt = w / np.where(r > 0, r, 1.0) * (r > 0)
    gt = r * (K @ w - s)
    st = r * s
    den = max(np.abs(st).max(), np.finfo(np.float64).tiny)
    return float(np.abs(np.minimum(wt, gt)).max() / den)


def cone_ref(K, s, t2=None):
    """Exact cone projection of one group.

    Returns (w [n], resid2) where resid2 = ||g_star_hat - G^T w||^2 if t2 is
    given (else None).
    """
    w = nnls_active_set(K, s)
    resid2 = None
    if t2 is not None:
        K = np.asarray(K, dtype=np.float64)
        s = np.asarray(s, dtype=np.float64)
        resid2 = float(t2 - 2.0 * (s @ w) + w @ (K @ w))
    return w, resid2


def cone_pg_replay(K, s, max_iter, kkt_tol=0.0):
    """Projected gradient on the Jacobi-scaled problem (design reading).

    w~ <- max(0, w~ - (K~ w~ - s~) / Lhat), Lhat = max_i sum_j |K~_ij|,
    starting from w~ = 0.  With kkt_tol > 0 the loop stops as soon as the
    scaled KKT residual of the current iterate is <= kkt_tol.
    Returns (w [n], iters, rho).
    """
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    if n == 0:
        return np.zeros(0), 0, 0.0
    d = np.diag(K)
    r = np.where(d > 0, 1.0 / np.sqrt(np.where(d > 0, d, 1.0)), 0.0)
    Kt = K * r[:, None] * r[None, :]
    st = s * r
    Lhat = np.abs(Kt).sum(axis=1).max()
    den = max(np.abs(st).max(), np.finfo(np.float64).tiny)
    wt = np.zeros(n)
    it = 0
    while True:
        g = Kt @ wt - st
        rho = np.abs(np.minimum(wt, g)).max() / den
        if (kkt_tol > 0 and rho <= kkt_tol) or it >= max_iter or Lhat == 0:
            break
        wt = np.maximum(0.0, wt - g / Lhat)
        it += 1
    return wt * r, it, float(rho)
