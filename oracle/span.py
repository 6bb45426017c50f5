"""Oracle: projection of the mean target gradient onto the span of the
general-data gradients (ridge least squares).

Test infrastructure only (see the package header).

Definitions followed
--------------------
* Eq. (proj), Sec. 3.3.1: u = argmin_{u in U} ||u - g_star_hat||^2, with the
  feasible set U = { G^T w : w in R^n } built from the training batch alone
  (Sec. 3.2: U depends only on the training gradients).  The paper names the
  template and several feasible sets but not this one; the span is the
  linear-subspace member of the family (reading, listed in the design notes).
* Ridge (Tikhonov) form: w = argmin ||G^T w - g_star_hat||^2 + lam_eff ||w||^2,
  whose normal equations are (K + lam_eff I) w = s with K = G G^T and
  s = G g_star_hat.  lam_eff -> 0 recovers Eq. (proj) exactly.
* lam_eff is either the given lambda (absolute) or lambda * tr(K) / n
  (relative to the mean squared gradient norm).  Reading: the relative form
  is the default because an absolute ridge of 1e-2 is below the float32 ulp
  of the diagonal at the workloads' gradient scales.
* Empty feasible set (n = 0, or K = 0 under the relative ridge): span{} =
  {0}, so w = 0 and u = 0.
* A matrix K + lam_eff I that is not positive definite is reported
  LAPACK-style through ``info`` = the 1-based index of the first
  non-positive pivot; w is then undefined (zeros).

The factorisation is LAPACK's Cholesky (a library primitive) followed by two
triangular solves; the plain column loop below is used only to report the
failing pivot's index.

Parity: pinned by tests (normal-equation identity G r = lam_eff w, exact
orthogonality at lam = 0, target-in-span, least squares on the stacked
primal system, empty cases, hand-solved 2x2 fixture).
"""

import numpy as np
from scipy.linalg import solve_triangular

RIDGE_ABS = 0
RIDGE_REL_TRACE = 1


def ridge_lambda(K, lam, mode):
    """Effective ridge for one group."""
    K = np.asarray(K, dtype=np.float64)
    n = K.shape[0]
    if mode == RIDGE_ABS:
        return float(lam)
    if mode == RIDGE_REL_TRACE:
        return float(lam) * float(np.trace(K)) / n if n > 0 else 0.0
    raise ValueError("unknown ridge mode")


def _first_bad_pivot(A):
    """Plain Cholesky column loop; returns the 1-based index of the first
    pivot that is not positive, or 0 if A is positive definite."""
    n = A.shape[0]
    L = np.zeros_like(A)
    for j in range(n):
        d = A[j, j] - L[j, :j] @ L[j, :j]
        if not d > 0.0:
            return j + 1
        L[j, j] = np.sqrt(d)
        L[j + 1:, j] = (A[j + 1:, j] - L[j + 1:, :j] @ L[j, :j]) / L[j, j]
    return 0


def span_ref(K, s, lam, mode=RIDGE_REL_TRACE, lam_eff=None):
    """Solve (K + lam_eff I) w = s for one group.

    Returns (w float64 [n], lam_eff, info).  If ``lam_eff`` is given it is
    used as is (to replay exactly the ridge another implementation chose).
    """
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    if n == 0:
        return np.zeros(0), 0.0, 0
    if lam_eff is None:
        lam_eff = ridge_lambda(K, lam, mode)
    if mode == RIDGE_REL_TRACE and np.trace(K) == 0.0:
        return np.zeros(n), float(lam_eff), 0
    A = K + lam_eff * np.eye(n)
    try:
        L = np.linalg.cholesky(A)
    except np.linalg.LinAlgError:
        return np.zeros(n), float(lam_eff), _first_bad_pivot(A) or 1
    y = solve_triangular(L, s, lower=True)
    w = solve_triangular(L.T, y, lower=False)
    return w, float(lam_eff), 0


def span_residual2(K, s, t2, w):
    """||g_star_hat - G^T w||^2 from the Gram quantities alone:
    t2 - 2 s^T w + w^T K w."""
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    return float(t2 - 2.0 * (s @ w) + w @ (K @ w))


def combine_ref(G, w, goff=None):
    """Update direction in sketch space: u^(p) = G^(p)^T w_p per group.

    G [n, kappa]; w [P, n] (or [n] for one group).  Returns u [kappa].
    """
    G = np.asarray(G, dtype=np.float64)
    w = np.atleast_2d(np.asarray(w, dtype=np.float64))
    n, kappa = G.shape
    if goff is None:
        goff = [0, kappa]
    u = np.zeros(kappa)
    for p in range(len(goff) - 1):
        a, b = int(goff[p]), int(goff[p + 1])
        u[a:b] = G[:, a:b].T @ w[p]
    return u
