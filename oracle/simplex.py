"""Oracle: soft weighting over the probability simplex, and back-projection.

Test infrastructure only (see the package header).

Definitions followed
--------------------
* Soft weighting (the first new feasible set of Sec. 6, "Designing New
  Feasible Sets"): U_soft = { sum_i w_i g_i : w in the simplex }.  With
  K = G G^T and s = G g_star_hat, Eq. (proj) over U_soft is the quadratic
  program
      minimise  f(w) = w^T K w - 2 s^T w   subject to  w >= 0, sum_i w_i = 1
  (||G^T w - g_star_hat||^2 = f(w) + ||g_star_hat||^2).  ``simplex_ref`` solves
  it exactly with a primal active-set method: keep a support P, solve the
  equality-constrained problem on P from its KKT system
      [2 K_PP  1; 1^T 0] [w_P; mu] = [2 s_P; 1],
  step back to feasibility when a coordinate would turn negative, and add
  the coordinate with the most negative multiplier grad_i + mu outside P
  until none is negative.
  Optimality: w on the simplex, grad = 2 (K w - s), grad_i + mu = 0 on the
  support and >= 0 off it.  ``simplex_residual`` measures it as the
  fixed-point residual of a projected-gradient step,
      rho = max_i |w_i - proj(w - grad / L)_i|,  L = 2 max_i sum_j |K_ij|,
  zero exactly at the optimum.
* Back-projection (App. C.3, "Backward projection"): for a sketch-space
  vector x~ and a layer with first-stage projectors P_in, P_out (second
  stage the identity), Pi^T x~ reshaped to d_out x d_in is
      P_out^T X' P_in,   X' = x~ reshaped to [k_out][k_in] (row-major, the
  layout of the sketches).  Applied to u~ = G~^T w it maps a sketch-space
  update to parameter space (the MeSO variant of the layer-wise update).

Parity: pinned by tests (enumeration of every support for small n; the
scaled-identity case equals the textbook sort-based simplex projection of
s / c; KKT; vertex and interior solutions; the adjoint identity
<Pi vec(G), x~> = <vec(G), Pi^T x~> with the explicit Kronecker matrix).
"""

import numpy as np


def project_simplex_threshold(v):
    """theta with sum_i max(v_i - theta, 0) = 1 (Michelot's iteration)."""
    v = np.asarray(v, dtype=np.float64)
    S = np.ones(v.shape[0], dtype=bool)
    while True:
        theta = (v[S].sum() - 1.0) / S.sum()
        S2 = v > theta
        if (S2 == S).all():
            return theta
        S = S2


def simplex_objective(K, s, w):
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    return w @ (K @ w) - 2.0 * s @ w


def simplex_residual(K, s, w):
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    L = 2.0 * max(np.abs(K).sum(axis=1).max(), 1e-300)
    v = w - 2.0 * (K @ w - s) / L
    theta = project_simplex_threshold(v)
    return float(np.abs(w - np.maximum(v - theta, 0.0)).max())


def _solve_on_support(K, s, P):
    """KKT system of the equality-constrained problem on the support P.  The
    constraint row and column are scaled by c = max |2 K_PP| (the system
    [2K_PP c1; c1^T 0][w; mu/c] = [2 s_P; c] has the same solution), so that
    the least-squares solve treats both blocks on the same scale."""
    idx = np.flatnonzero(P)
    k = idx.size
    KP = 2.0 * K[np.ix_(idx, idx)]
    c = max(np.abs(KP).max(), 1e-300)
    A = np.zeros((k + 1, k + 1))
    A[:k, :k] = KP
    A[:k, k] = c
    A[k, :k] = c
    b = np.concatenate([2.0 * s[idx], [c]])
    sol = np.linalg.lstsq(A, b, rcond=None)[0]
    z = np.zeros(K.shape[0])
    z[idx] = sol[:k]
    return z, sol[k] * c


def simplex_ref(K, s, max_outer=None):
    """Exact minimiser of w^T K w - 2 s^T w over the probability simplex."""
    K = np.asarray(K, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    if n == 0:
        return np.zeros(0)
    scale = max(np.abs(K).max(), np.abs(s).max(), 1e-300)
    tol = 64.0 * n * np.finfo(np.float64).eps * scale
    i0 = int(np.argmin(np.diag(K) - 2.0 * s))
    w = np.zeros(n)
    w[i0] = 1.0
    P = np.zeros(n, dtype=bool)
    P[i0] = True
    max_outer = 3 * n + 10 if max_outer is None else max_outer
    for _ in range(max_outer):
        # inner loop: restore feasibility of the sub-problem solution
        while True:
            z, mu = _solve_on_support(K, s, P)
            neg = P & (z <= 0.0)
            if not neg.any():
                w = z
                break
            alpha = np.min(w[neg] / (w[neg] - z[neg]))
            w = w + alpha * (z - w)
            P &= w > 0.0
            w[~P] = 0.0
            w = w / w.sum()
        grad = 2.0 * (K @ w - s)
        mu = -np.mean(grad[P])
        lam = np.where(P, np.inf, grad + mu)
        j = int(np.argmin(lam))
        if P.all() or lam[j] >= -tol:
            break
        P[j] = True
    return w


def backproject_ref(u, layers):
    """Per-layer P_out^T X' P_in (float64 [d_out, d_in]) of a sketch-space vector.

    layers: dicts with p_in [k_in, d_in], p_out [k_out, d_out], col_offset.
    """
    u = np.asarray(u, dtype=np.float64)
    out = []
    for L in layers:
        p_in = np.asarray(L["p_in"], dtype=np.float64)
        p_out = np.asarray(L["p_out"], dtype=np.float64)
        k_in, k_out = p_in.shape[0], p_out.shape[0]
        o = int(L["col_offset"])
        X = u[o:o + k_out * k_in].reshape(k_out, k_in)
        out.append(p_out.T @ X @ p_in)
    return out
