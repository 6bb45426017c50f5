"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests re-type an oracle formula: each checks the oracle
against an independent route (autograd, an explicit Kronecker matrix, a
different contraction order, a library solver on the primal problem,
exhaustive enumeration, a hand-derived fixture or an invariant).
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.optimize
import torch

import oracle
from oracle import brute
from oracle.span import RIDGE_ABS, RIDGE_REL_TRACE

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def _num(v):
    return float(v) if not isinstance(v, str) else float(v)


# --------------------------------------------------------------------------
# Sketch oracle
# --------------------------------------------------------------------------

def _linear_layer_batch(seed, N=5, T=7, d_in=6, d_out=4):
    """Per-example loss through one linear layer with a non-linear head.

    Returns x, W, per-example output gradients dL/de (from autograd) and
    the per-example weight gradients from torch.func (vmap of grad).
    """
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(N, T, d_in, generator=g, dtype=torch.float64)
    W = torch.randn(d_out, d_in, generator=g, dtype=torch.float64)
    c = torch.randn(N, T, d_out, generator=g, dtype=torch.float64)
    lens = torch.randint(0, T + 1, (N,), generator=g)
    mask = (torch.arange(T)[None, :] < lens[:, None]).to(torch.float64)

    def loss_one(Wm, xi, ci, mi):
        e = xi @ Wm.T                        # [T, d_out] pre-activations
        return (mi[:, None] * (torch.tanh(e) - ci) ** 2).sum()

    per_ex = torch.func.vmap(torch.func.grad(loss_one), in_dims=(None, 0, 0, 0))(W, x, c, mask)
    e = (x @ W.T).requires_grad_(True)
    loss = (mask[..., None] * (torch.tanh(e) - c) ** 2).sum()
    (dy,) = torch.autograd.grad(loss, e)
    Wg = W.clone().requires_grad_(True)
    loss_w = (mask[..., None] * (torch.tanh(x @ Wg.T) - c) ** 2).sum()
    loss_w.backward()
    return x.numpy(), dy.numpy(), lens.numpy(), per_ex.numpy(), Wg.grad.numpy()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_sketch_identity_projectors_equal_per_example_autograd(seed):
    x, dy, lens, per_ex, _ = _linear_layer_batch(seed)
    N, T, d_in = x.shape
    d_out = dy.shape[2]
    # padding positions hold NaN: they must be excluded, not multiplied by 0
    x = x.copy(); dy = dy.copy()
    for i in range(N):
        x[i, lens[i]:] = np.nan
        dy[i, lens[i]:] = np.nan
    layer = dict(x=x, dy=dy, p_in=np.eye(d_in), p_out=np.eye(d_out))
    S = oracle.sketch_ref([layer], lens)
    np.testing.assert_allclose(S, per_ex.reshape(N, -1), rtol=1e-12, atol=1e-12)


def test_sum_of_per_example_gradients_is_the_batch_weight_gradient():
    x, dy, lens, _, wgrad = _linear_layer_batch(7)
    G = sum(oracle.per_example_gradient(x[i], dy[i], lens[i]) for i in range(x.shape[0]))
    np.testing.assert_allclose(G, wgrad, rtol=1e-12, atol=1e-12)


def test_factorised_sketch_equals_explicit_kronecker_projector():
    """Pi = P_in kron P_out acting on vec(G) (App. C.3) equals P_out G P_in^T
    stored [k_out][k_in]: with row-major vec, kron(P_out, P_in) vec(G)."""
    rng = np.random.default_rng(3)
    d_in, d_out, k_in, k_out, T = 9, 7, 3, 4, 5
    x = rng.standard_normal((1, T, d_in))
    dy = rng.standard_normal((1, T, d_out))
    p_in = rng.standard_normal((k_in, d_in))
    p_out = rng.standard_normal((k_out, d_out))
    S = oracle.sketch_ref([dict(x=x, dy=dy, p_in=p_in, p_out=p_out)])[0]
    # explicit gradient via a per-token loop of outer products, then the full matrix
    G = np.zeros((d_out, d_in))
    for t in range(T):
        G += np.outer(dy[0, t], x[0, t])
    Pi = np.kron(p_out, p_in)                 # [k_out*k_in, d_out*d_in]
    np.testing.assert_allclose(S, Pi @ G.reshape(-1), rtol=1e-12, atol=1e-12)
    # per-token factorised form: sum_t (P_out dy_t)(P_in x_t)^T
    Sf = sum(np.outer(p_out @ dy[0, t], p_in @ x[0, t]) for t in range(T))
    np.testing.assert_allclose(S, Sf.reshape(-1), rtol=1e-12, atol=1e-12)


def test_sketch_hand_fixture(golden_dir):
    fx = _load(golden_dir, "sketch_hand.json")
    x = np.array([[_num(v) for v in r] for r in fx["x"]])[None]
    dy = np.array([[_num(v) for v in r] for r in fx["dy"]])[None]
    G = oracle.per_example_gradient(x[0], dy[0], fx["length"])
    np.testing.assert_array_equal(G, np.array(fx["G"], dtype=float))
    for c in fx["cases"]:
        layer = dict(x=x, dy=dy, p_in=np.array(c["p_in"], float), p_out=np.array(c["p_out"], float))
        S = oracle.sketch_ref([layer], [fx["length"]])[0]
        np.testing.assert_array_equal(S, np.array(c["S"], dtype=float))


def test_sketch_empty_and_rank_one_and_linearity():
    rng = np.random.default_rng(5)
    N, T, d_in, d_out, k_in, k_out = 3, 6, 8, 5, 4, 2
    x = rng.standard_normal((N, T, d_in))
    dy = rng.standard_normal((N, T, d_out))
    p_in = rng.standard_normal((k_in, d_in))
    p_out = rng.standard_normal((k_out, d_out))
    L = dict(x=x, dy=dy, p_in=p_in, p_out=p_out)
    S = oracle.sketch_ref([L], [0, 1, T])
    assert np.all(S[0] == 0.0)
    np.testing.assert_allclose(S[1], np.outer(p_out @ dy[1, 0], p_in @ x[1, 0]).reshape(-1), rtol=1e-12)
    S2 = oracle.sketch_ref([dict(L, dy=2.5 * dy)], [0, 1, T])
    np.testing.assert_allclose(S2, 2.5 * S, rtol=1e-12, atol=1e-12)
    S3 = oracle.sketch_ref([dict(L, x=x + x[::-1])], [0, 1, T])
    S4 = oracle.sketch_ref([dict(L, x=x[::-1])], [0, 1, T])
    np.testing.assert_allclose(S3, S + S4, rtol=1e-10, atol=1e-10)


def test_multi_layer_column_offsets():
    rng = np.random.default_rng(11)
    N, T = 2, 4
    Ls = []
    for (d_in, d_out, k_in, k_out) in [(5, 3, 2, 2), (4, 6, 3, 1)]:
        Ls.append(dict(x=rng.standard_normal((N, T, d_in)), dy=rng.standard_normal((N, T, d_out)),
                       p_in=rng.standard_normal((k_in, d_in)), p_out=rng.standard_normal((k_out, d_out))))
    S = oracle.sketch_ref(Ls)
    assert S.shape == (N, 4 + 3)
    for l, off in zip(Ls, [0, 4]):
        Sl = oracle.sketch_ref([l])
        np.testing.assert_allclose(S[:, off:off + Sl.shape[1]], Sl)


def test_exact_scorers_agree_and_match_identity_sketch():
    """Direct, GIP and PIP (Sec. 4.3) are the same inner product in three
    contraction orders; compressed scoring with identity projectors is Direct."""
    rng = np.random.default_rng(8)
    n, m, T, d_in, d_out = 5, 3, 6, 7, 4
    x = rng.standard_normal((n, T, d_in)); dy = rng.standard_normal((n, T, d_out))
    xt = rng.standard_normal((m, T, d_in)); dyt = rng.standard_normal((m, T, d_out))
    lens = rng.integers(1, T + 1, n); lens_t = rng.integers(1, T + 1, m)
    sd = oracle.score_direct(x, dy, lens, xt, dyt, lens_t)
    sg = oracle.score_gip(x, dy, lens, xt, dyt, lens_t)
    sp = oracle.score_pip(x, dy, lens, xt, dyt, lens_t)
    np.testing.assert_allclose(sg, sd, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(sp, sd, rtol=1e-11, atol=1e-11)
    I_in, I_out = np.eye(d_in), np.eye(d_out)
    S = oracle.sketch_ref([dict(x=x, dy=dy, p_in=I_in, p_out=I_out)], lens)
    St = oracle.sketch_ref([dict(x=xt, dy=dyt, p_in=I_in, p_out=I_out)], lens_t)
    np.testing.assert_allclose(oracle.score_compressed(S, St), sd, rtol=1e-11, atol=1e-11)
    _, s_g, _ = oracle.gram_ref(S, St)
    np.testing.assert_allclose(s_g[0], sd, rtol=1e-11, atol=1e-11)


def test_gaussian_sketch_preserves_inner_products_in_expectation():
    """With P entries ~ N(0, 1/k), E <Pi g, Pi h> = <g, h> (statistical pin of
    the projector scale reading)."""
    rng = np.random.default_rng(21)
    d_in, d_out, k, T = 12, 10, 6, 3
    x = rng.standard_normal((2, T, d_in)); dy = rng.standard_normal((2, T, d_out))
    g = oracle.per_example_gradient(x[0], dy[0], T)
    h = oracle.per_example_gradient(x[1], dy[1], T)
    exact = float(np.sum(g * h))
    est = []
    for _ in range(400):
        p_in = rng.standard_normal((k, d_in)) / math.sqrt(k)
        p_out = rng.standard_normal((k, d_out)) / math.sqrt(k)
        est.append(float(np.sum(oracle.sketch_block(g, p_in, p_out) * oracle.sketch_block(h, p_in, p_out))))
    est = np.array(est)
    se = est.std() / math.sqrt(len(est))
    assert abs(est.mean() - exact) < 5 * se


# --------------------------------------------------------------------------
# Gram oracle
# --------------------------------------------------------------------------

def test_gram_against_python_loops_and_invariants():
    rng = np.random.default_rng(1)
    n, m, kappa = 6, 3, 10
    G = rng.standard_normal((n, kappa)); Gt = rng.standard_normal((m, kappa))
    goff = [0, 4, 10]
    K, s, t2 = oracle.gram_ref(G, Gt, goff)
    for p in range(2):
        a, b = goff[p], goff[p + 1]
        gbar = [sum(Gt[j][c] for j in range(m)) / m for c in range(a, b)]
        for i in range(n):
            assert math.isclose(s[p, i], sum(G[i][c] * gbar[c - a] for c in range(a, b)), rel_tol=1e-12, abs_tol=1e-12)
            for j in range(n):
                assert math.isclose(K[p, i, j], sum(G[i][c] * G[j][c] for c in range(a, b)), rel_tol=1e-12, abs_tol=1e-12)
        assert math.isclose(t2[p], sum(v * v for v in gbar), rel_tol=1e-12)
        np.testing.assert_array_equal(K[p], K[p].T)
        assert np.linalg.eigvalsh(K[p]).min() > -1e-10
    # groups partition the coordinates: per-group quantities add up
    K1, s1, t21 = oracle.gram_ref(G, Gt)
    np.testing.assert_allclose(K.sum(0), K1[0], rtol=1e-12)
    np.testing.assert_allclose(s.sum(0), s1[0], rtol=1e-12)
    # scores are the mean of the per-target scores (linearity in g_star)
    per_target = np.stack([oracle.gram_ref(G, Gt[j:j + 1])[1][0] for j in range(m)])
    np.testing.assert_allclose(per_target.mean(0), s1[0], rtol=1e-12)


def test_redundancy_term_identity():
    """(1/k^2) sum_{i,i' in S} <g_i, g_i'> = ||g_S||^2 (Sec. 3.3.2)."""
    rng = np.random.default_rng(2)
    G = rng.standard_normal((7, 9))
    K, _, _ = oracle.gram_ref(G, G[:1])
    S = [1, 4, 5]
    gS = G[S].mean(0)
    assert math.isclose(K[0][np.ix_(S, S)].sum() / 9.0, float(gS @ gS), rel_tol=1e-12)


# --------------------------------------------------------------------------
# Span oracle
# --------------------------------------------------------------------------

def test_span_hand_fixture(golden_dir):
    fx = _load(golden_dir, "span_2x2.json")
    for c in fx["cases"]:
        w, lam_eff, info = oracle.span_ref(fx["K"], fx["s"], c["lam"], c["mode"])
        assert info == 0 and math.isclose(lam_eff, c["lam_eff"])
        np.testing.assert_allclose(w, c["w"], rtol=1e-14, atol=1e-14)
        assert math.isclose(oracle.span_residual2(fx["K"], fx["s"], fx["t2"], w), c["resid2"], rel_tol=1e-13)


@pytest.mark.parametrize("lam,mode", [(0.0, RIDGE_ABS), (1e-3, RIDGE_REL_TRACE), (0.3, RIDGE_ABS)])
def test_span_normal_equations_and_primal_least_squares(lam, mode):
    rng = np.random.default_rng(4)
    n, kappa = 6, 20
    G = rng.standard_normal((n, kappa)); gbar = rng.standard_normal(kappa)
    K, s, t2 = oracle.gram_ref(G, gbar[None])
    w, lam_eff, info = oracle.span_ref(K[0], s[0], lam, mode)
    assert info == 0
    u = oracle.combine_ref(G, w)
    r = gbar - u
    # normal equations: G r = lam_eff w  (exact orthogonality when lam = 0)
    np.testing.assert_allclose(G @ r, lam_eff * w, atol=1e-10 * np.abs(G).max() * np.abs(r).max() * kappa)
    # stacked primal least squares [G^T; sqrt(lam) I] w = [gbar; 0]
    A = np.vstack([G.T, math.sqrt(lam_eff) * np.eye(n)])
    b = np.concatenate([gbar, np.zeros(n)])
    w_ls = np.linalg.lstsq(A, b, rcond=None)[0]
    np.testing.assert_allclose(w, w_ls, rtol=1e-9, atol=1e-12)
    assert math.isclose(oracle.span_residual2(K[0], s[0], t2[0], w), float(r @ r), rel_tol=1e-9, abs_tol=1e-12)


def test_span_target_in_span_and_empty_sets():
    rng = np.random.default_rng(6)
    n, kappa = 4, 12
    G = rng.standard_normal((n, kappa))
    c = rng.standard_normal(n)
    gbar = G.T @ c
    K, s, t2 = oracle.gram_ref(G, gbar[None])
    w, _, info = oracle.span_ref(K[0], s[0], 0.0, RIDGE_ABS)
    np.testing.assert_allclose(w, c, rtol=1e-9)
    np.testing.assert_allclose(oracle.combine_ref(G, w), gbar, rtol=1e-9, atol=1e-12)
    assert abs(oracle.span_residual2(K[0], s[0], t2[0], w)) < 1e-9 * t2[0]
    # n = 0: empty feasible set
    w0, _, info0 = oracle.span_ref(np.zeros((0, 0)), np.zeros(0), 1e-2, RIDGE_REL_TRACE)
    assert w0.shape == (0,) and info0 == 0
    # K = 0 (all general gradients zero): span{} = {0}
    wz, lz, iz = oracle.span_ref(np.zeros((3, 3)), np.zeros(3), 1e-2, RIDGE_REL_TRACE)
    assert iz == 0 and lz == 0.0 and np.all(wz == 0)


def test_span_reports_first_non_positive_pivot():
    K = np.diag([1.0, -1.0, 1.0])
    _, _, info = oracle.span_ref(K, np.ones(3), 0.0, RIDGE_ABS)
    assert info == 2
    K = np.array([[1.0, 2.0], [2.0, 1.0]])            # indefinite
    _, _, info = oracle.span_ref(K, np.ones(2), 0.0, RIDGE_ABS)
    assert info == 2


def test_span_relative_ridge_definition():
    rng = np.random.default_rng(9)
    G = rng.standard_normal((5, 8))
    K, s, _ = oracle.gram_ref(G, G[:1])
    _, lam_eff, _ = oracle.span_ref(K[0], s[0], 0.01, RIDGE_REL_TRACE)
    assert math.isclose(lam_eff, 0.01 * np.mean(np.sum(G * G, axis=1)), rel_tol=1e-12)


# --------------------------------------------------------------------------
# Cone oracle
# --------------------------------------------------------------------------

def test_cone_hand_fixture(golden_dir):
    fx = _load(golden_dir, "cone_2x2.json")
    for c in fx["cases"]:
        w, _ = oracle.cone_ref(fx["K"], c["s"])
        np.testing.assert_allclose(w, c["w"], rtol=1e-14, atol=1e-14)


def test_cone_kkt_residual_hand_fixture_away_from_the_optimum(golden_dir):
    """rho at non-optimal points, hand-computed: a wrong power of D in the
    scaling, a flipped gradient sign or a dropped scaling all change it."""
    fx = _load(golden_dir, "cone_kkt_hand.json")
    for c in fx["cases"]:
        rho = oracle.cone_kkt_residual(c["K"], c["s"], c["w"])
        assert math.isclose(rho, c["rho"], rel_tol=1e-14), (c, rho)


@pytest.mark.parametrize("seed", range(6))
def test_cone_matches_scipy_nnls_and_enumeration(seed):
    rng = np.random.default_rng(100 + seed)
    n, kappa = 8, 14
    G = rng.standard_normal((n, kappa))
    gbar = rng.standard_normal(kappa)
    K, s, t2 = oracle.gram_ref(G, gbar[None])
    w, resid2 = oracle.cone_ref(K[0], s[0], t2[0])
    w_sp, rnorm = scipy.optimize.nnls(G.T, gbar)
    np.testing.assert_allclose(w, w_sp, rtol=1e-8, atol=1e-10)
    assert math.isclose(resid2, rnorm ** 2, rel_tol=1e-8)
    np.testing.assert_allclose(w, brute.nnls_enumerate(K[0], s[0]), rtol=1e-9, atol=1e-12)
    assert oracle.cone_kkt_residual(K[0], s[0], w) < 1e-10
    # KKT in the primal form: <g_i, r> <= 0 for every i, = 0 on the support
    r = gbar - G.T @ w
    gr = G @ r
    assert np.all(gr <= 1e-9)
    assert np.all(np.abs(gr[w > 0]) < 1e-9)


def test_cone_special_cases():
    rng = np.random.default_rng(12)
    n, kappa = 5, 9
    G = rng.standard_normal((n, kappa))
    c = np.abs(rng.standard_normal(n)) + 0.1
    K, s, _ = oracle.gram_ref(G, (G.T @ c)[None])
    np.testing.assert_allclose(oracle.cone_ref(K[0], s[0])[0], c, rtol=1e-9)   # target inside the cone
    Q, _ = np.linalg.qr(rng.standard_normal((kappa, n)))
    Go = Q.T                                                                    # orthonormal rows
    K, s, _ = oracle.gram_ref(Go, (-Go[0])[None])                                # s <= 0 everywhere
    assert np.all(s[0] <= 1e-12)
    assert np.all(oracle.cone_ref(K[0], s[0])[0] == 0.0)
    assert oracle.cone_ref(np.zeros((0, 0)), np.zeros(0))[0].shape == (0,)


def test_projected_gradient_reaches_exact_cone_optimum_on_near_orthogonal_gradients():
    """Workload-like K: rows nearly orthogonal (independent examples); 200
    Jacobi-scaled projected-gradient steps reach the exact optimum."""
    rng = np.random.default_rng(13)
    n, kappa = 64, 4096
    G = rng.standard_normal((n, kappa)) * rng.uniform(0.5, 2.0, (n, 1))
    gbar = rng.standard_normal(kappa) * 0.1 + G[:3].sum(0) * 0.05
    K, s, _ = oracle.gram_ref(G, gbar[None])
    w_ex = oracle.nnls_active_set(K[0], s[0])
    w_pg, it, rho = oracle.cone_pg_replay(K[0], s[0], 200)
    assert it == 200
    np.testing.assert_allclose(w_pg, w_ex, rtol=1e-9, atol=1e-12 * np.abs(w_ex).max())
    w_pg2, it2, rho2 = oracle.cone_pg_replay(K[0], s[0], 10000, kkt_tol=1e-6)
    assert rho2 <= 1e-6 and it2 < 200


# --------------------------------------------------------------------------
# Top-k oracle
# --------------------------------------------------------------------------

def test_topk_hand_fixture(golden_dir):
    fx = _load(golden_dir, "topk_ties.json")
    for c in fx["cases"]:
        s = [_num(v) for v in c["s"]]
        assert list(oracle.topk_ref(s, c["k"])) == c["idx"], c


@pytest.mark.parametrize("seed", range(5))
def test_topk_matches_enumeration(seed):
    rng = np.random.default_rng(200 + seed)
    n = 10
    s = rng.integers(-3, 4, n).astype(float)        # many exact ties
    for k in range(0, n + 1):
        np.testing.assert_array_equal(oracle.topk_ref(s, k), brute.topk_enumerate(s, k))
    s = rng.standard_normal(n)
    for k in (1, 3, 7):
        np.testing.assert_array_equal(oracle.topk_ref(s, k), brute.topk_enumerate(s, k))


def test_topk_errors_and_full_training_case():
    with pytest.raises(ValueError):
        oracle.topk_ref([1.0, float("nan")], 1)
    with pytest.raises(ValueError):
        oracle.topk_ref([1.0], 2)
    rng = np.random.default_rng(3)
    G = rng.standard_normal((6, 5))
    idx = oracle.topk_ref(rng.standard_normal(6), 6)
    np.testing.assert_array_equal(idx, np.arange(6))
    np.testing.assert_allclose(G[idx].mean(0), G.mean(0))      # k = n is the full-training update


@pytest.mark.parametrize("seed", range(4))
def test_topk_is_exact_subset_projection_when_gram_is_scaled_identity(seed):
    """With K = cI the redundancy term is constant, so top-k solves the
    Global Subset projection exactly (Sec. 3.3.2)."""
    rng = np.random.default_rng(300 + seed)
    n, kappa, k = 8, 12, 3
    Q, _ = np.linalg.qr(rng.standard_normal((kappa, n)))
    G = 2.0 * Q.T
    gbar = rng.standard_normal(kappa)
    K, s, _ = oracle.gram_ref(G, gbar[None])
    np.testing.assert_allclose(K[0], 4.0 * np.eye(n), atol=1e-12)
    S_exact, _ = brute.subset_projection(G, gbar, k)
    np.testing.assert_array_equal(oracle.topk_ref(s[0], k), S_exact)


# --------------------------------------------------------------------------
# Update assembly oracle
# --------------------------------------------------------------------------

def test_update_hand_fixture(golden_dir):
    fx = _load(golden_dir, "update_hand.json")
    x = np.array([[[_num(v) for v in r] for r in ex] for ex in fx["x"]])
    dy = np.array([[[_num(v) for v in r] for r in ex] for ex in fx["dy"]])
    for c in fx["cases"]:
        (U,) = oracle.update_ref([dict(x=x, dy=dy)], c["w"], fx["lengths"])
        np.testing.assert_array_equal(U, np.array(c["U"], dtype=float))


@pytest.mark.parametrize("seed", [0, 3])
def test_update_one_hot_and_unit_weights_match_autograd(seed):
    x, dy, lens, per_ex, wgrad = _linear_layer_batch(seed)
    N = x.shape[0]
    x = x.copy(); dy = dy.copy()
    for i in range(N):
        x[i, lens[i]:] = np.nan
        dy[i, lens[i]:] = np.nan
    layer = dict(x=x, dy=dy)
    for i in range(N):
        (U,) = oracle.update_ref([layer], np.eye(N)[i], lens)
        np.testing.assert_allclose(U, per_ex[i], rtol=1e-12, atol=1e-12)
    (U,) = oracle.update_ref([layer], np.ones(N), lens)
    np.testing.assert_allclose(U, wgrad, rtol=1e-12, atol=1e-12)


def test_update_subset_mean_is_the_gradient_of_the_subset_mean_loss():
    """u = g_S (Sec. 3.3.2): with w = 1/k on S the assembled update equals
    autograd's weight gradient of (1/k) sum_{i in S} loss_i."""
    g = torch.Generator().manual_seed(21)
    N, T, d_in, d_out = 6, 5, 4, 3
    x = torch.randn(N, T, d_in, generator=g, dtype=torch.float64)
    W = torch.randn(d_out, d_in, generator=g, dtype=torch.float64)
    c = torch.randn(N, T, d_out, generator=g, dtype=torch.float64)
    lens = torch.tensor([5, 2, 0, 4, 1, 3])
    mask = (torch.arange(T)[None, :] < lens[:, None]).to(torch.float64)
    e = (x @ W.T).requires_grad_(True)
    per_example_loss = (mask[..., None] * torch.sin(e - c) ** 2).sum(dim=(1, 2))
    (dy,) = torch.autograd.grad(per_example_loss.sum(), e)
    S = [0, 3, 4]
    Wg = W.clone().requires_grad_(True)
    loss_S = (mask[..., None] * torch.sin(x @ Wg.T - c) ** 2).sum(dim=(1, 2))[S].mean()
    loss_S.backward()
    w = np.zeros(N)
    w[S] = 1.0 / len(S)
    (U,) = oracle.update_ref([dict(x=x.numpy(), dy=dy.numpy())], w, lens.numpy())
    np.testing.assert_allclose(U, Wg.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_update_sketch_equals_weighted_sum_of_sketches_per_group():
    """P_out U_l P_in^T = sum_i w_{g(l),i} S_i^(l): sketching is linear, so
    the sketch of the assembled update is the same weighted sum of the
    (separately pinned) per-example sketches.  Two layers in two groups,
    NaN padding, a NaN row with weight 0 and NaN target rows after n."""
    rng = np.random.default_rng(8)
    n, m, T = 5, 2, 6
    N = n + m
    lens = np.array([6, 3, 0, 1, 5, 6, 6])
    dims = [(7, 5, 3, 2), (4, 6, 2, 3)]
    layers = []
    for d_in, d_out, k_in, k_out in dims:
        x = rng.standard_normal((N, T, d_in))
        dy = rng.standard_normal((N, T, d_out))
        for i in range(N):
            x[i, lens[i]:] = np.nan
            dy[i, lens[i]:] = np.nan
        x[1] = np.nan
        dy[1] = np.nan
        x[n:] = np.nan
        layers.append(dict(x=x, dy=dy, p_in=rng.standard_normal((k_in, d_in)),
                           p_out=rng.standard_normal((k_out, d_out))))
    w = rng.standard_normal((2, n))
    w[:, 1] = 0.0
    w[1, 3] = 0.0
    U = oracle.update_ref(layers, w, lens, group_of_layer=[1, 0])
    for li, (L, g) in enumerate(zip(layers, [1, 0])):
        assert np.all(np.isfinite(U[li]))
        rows = [i for i in range(n) if w[g, i] != 0.0]
        S = oracle.sketch_ref([L], lens, rows=rows)
        want = sum(w[g, i] * S[i] for i in rows)
        got = (L["p_out"] @ U[li] @ L["p_in"].T).reshape(-1)
        np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-11)


# --------------------------------------------------------------------------
# Thresholding and greedy selection oracles
# --------------------------------------------------------------------------

def test_selection_hand_fixture(golden_dir):
    fx = _load(golden_dir, "select_hand.json")
    s = np.array(fx["s"], dtype=float)
    K = np.array(fx["K"], dtype=float)
    for c in fx["threshold"]:
        idx, w = oracle.threshold_ref(s, c["tau"], c["inclusive"])
        assert idx.tolist() == c["idx"]
        np.testing.assert_array_equal(w[idx], np.full(len(idx), 1.0 / max(1, len(idx))))
    idx, order = oracle.greedy_ref(K, s, fx["greedy"]["k"])
    assert order.tolist() == fx["greedy"]["order"]
    assert oracle.topk_ref(s, fx["greedy"]["k"]).tolist() == fx["greedy"]["topk"]
    for S, f in fx["objective"]:
        assert oracle.subset_objective(K, s, S) == pytest.approx(f, rel=1e-15, abs=1e-15)


def test_threshold_against_comparisons_and_errors():
    rng = np.random.default_rng(4)
    s = np.round(rng.standard_normal(40), 1)          # many exact ties and zeros
    s[3] = 0.0
    s[7] = -0.0
    for tau, inc in [(0.0, True), (0.0, False), (0.3, False), (-0.5, True), (9.0, False)]:
        idx, w = oracle.threshold_ref(s, tau, inc)
        want = np.flatnonzero(s >= tau) if inc else np.flatnonzero(s > tau)
        assert idx.tolist() == want.tolist()
        assert w.sum() == pytest.approx(1.0 if len(want) else 0.0)
    assert 3 in oracle.threshold_ref(s, 0.0, True)[0] and 7 in oracle.threshold_ref(s, 0.0, True)[0]
    with pytest.raises(ValueError):
        oracle.threshold_ref(np.array([1.0, np.nan]), 0.0)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_greedy_matches_topk_for_orthogonal_equal_norm_gradients(seed):
    """K = cI: f(S) = c/|S| - (2/|S|) sum s, so every greedy step adds the
    largest remaining score -- the top-k set, ties to the lowest index."""
    rng = np.random.default_rng(seed)
    n, k = 12, 5
    s = np.round(rng.standard_normal(n), 1)
    idx, _ = oracle.greedy_ref(2.5 * np.eye(n), s, k)
    assert idx.tolist() == oracle.topk_ref(s, k).tolist()


@pytest.mark.parametrize("seed", [3, 4])
def test_greedy_steps_are_best_single_additions_by_brute_force(seed):
    rng = np.random.default_rng(seed)
    n, k = 9, 5
    Gm = rng.standard_normal((n, 6))
    gstar = rng.standard_normal(6)
    K, s = Gm @ Gm.T, Gm @ gstar
    _, order = oracle.greedy_ref(K, s, k)
    S = []
    for c in order:
        cands = [j for j in range(n) if j not in S]
        vals = [oracle.subset_objective(K, s, S + [j]) for j in cands]
        assert c == cands[int(np.argmin(vals))]
        # the objective is the S-dependent part of the projection distance
        g_S = Gm[S + [c]].mean(axis=0)
        assert np.sum((g_S - gstar) ** 2) - gstar @ gstar == pytest.approx(min(vals), rel=1e-10, abs=1e-10)
        S.append(c)
    # k = 1 closed form: argmin K_cc - 2 s_c
    assert oracle.greedy_ref(K, s, 1)[0].tolist() == [int(np.argmin(np.diag(K) - 2 * s))]
    with pytest.raises(ValueError):
        oracle.greedy_ref(K, np.where(np.arange(n) == 2, np.nan, s), 2)


# --------------------------------------------------------------------------
# Simplex soft weighting and back-projection oracles
# --------------------------------------------------------------------------

def _simplex_by_enumeration(K, s):
    """Best KKT point over every support (the QP restricted to a support is an
    equality-constrained least-squares problem)."""
    n = s.shape[0]
    best, best_f = None, np.inf
    for mask in range(1, 1 << n):
        idx = [i for i in range(n) if mask >> i & 1]
        k = len(idx)
        A = np.zeros((k + 1, k + 1))
        A[:k, :k] = 2 * K[np.ix_(idx, idx)]
        A[:k, k] = 1
        A[k, :k] = 1
        try:
            sol = np.linalg.solve(A, np.concatenate([2 * s[idx], [1.0]]))
        except np.linalg.LinAlgError:
            continue
        if (sol[:k] < -1e-12).any():
            continue
        w = np.zeros(n)
        w[idx] = np.maximum(sol[:k], 0)
        w /= w.sum()
        f = w @ K @ w - 2 * s @ w
        if f < best_f - 1e-14:
            best, best_f = w, f
    return best


def _sort_projection(v):
    """Textbook Euclidean projection onto the simplex (sort, find the pivot)."""
    u = np.sort(v)[::-1]
    css = np.cumsum(u)
    rho = max(j for j in range(len(v)) if u[j] - (css[j] - 1) / (j + 1) > 0)
    theta = (css[rho] - 1) / (rho + 1)
    return np.maximum(v - theta, 0)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_simplex_matches_support_enumeration(seed):
    rng = np.random.default_rng(seed)
    n = 7
    Gm = rng.standard_normal((n, 5 + seed))            # rank-deficient for seeds 0, 1
    gs = rng.standard_normal(5 + seed) * (0.3 + seed)
    K, s = Gm @ Gm.T + 1e-3 * np.eye(n), Gm @ gs
    w = oracle.simplex_ref(K, s)
    we = _simplex_by_enumeration(K, s)
    assert w.min() >= 0 and w.sum() == pytest.approx(1.0, abs=1e-12)
    assert oracle.simplex_objective(K, s, w) == pytest.approx(oracle.simplex_objective(K, s, we), abs=1e-10)
    np.testing.assert_allclose(w, we, atol=1e-7)
    assert oracle.simplex_residual(K, s, w) < 1e-10


@pytest.mark.parametrize("seed", [4, 5])
def test_simplex_scaled_identity_is_the_projection_of_the_scores(seed):
    """K = cI: f = c||w||^2 - 2 s^T w = c ||w - s/c||^2 + const, so the
    optimum is the Euclidean projection of s / c onto the simplex."""
    rng = np.random.default_rng(seed)
    s = rng.standard_normal(30)
    w = oracle.simplex_ref(3.0 * np.eye(30), s)
    np.testing.assert_allclose(w, _sort_projection(s / 3.0), atol=1e-12)


@pytest.mark.parametrize("c", [1e-6, 1e4, 1e8, 1e12])
def test_simplex_is_invariant_to_scaling_the_objective(c):
    """argmin of c (w^T K w - 2 s^T w) over the simplex does not depend on c > 0
    (sketch Gram matrices have entries of order 1e6 and more)."""
    rng = np.random.default_rng(12)
    Gm = rng.standard_normal((40, 300))
    K, s = Gm @ Gm.T, Gm @ (0.05 * rng.standard_normal(300))
    w1 = oracle.simplex_ref(K, s)
    wc = oracle.simplex_ref(c * K, c * s)
    assert wc.sum() == pytest.approx(1.0, abs=1e-12) and wc.min() >= 0
    np.testing.assert_allclose(wc, w1, atol=1e-9)
    assert oracle.simplex_residual(c * K, c * s, wc) < 1e-10


def test_simplex_special_cases():
    # one example: the only point of the simplex
    np.testing.assert_allclose(oracle.simplex_ref(np.array([[2.0]]), np.array([-5.0])), [1.0], atol=1e-14)
    # target inside the convex hull: zero residual distance
    Gm = np.array([[1.0, 0.0], [0.0, 1.0], [-1.0, -1.0]])
    gstar = np.array([0.2, 0.3])                        # = 0.5 g0 + 0.6 g1 ... inside the hull
    K, s = Gm @ Gm.T, Gm @ gstar
    w = oracle.simplex_ref(K, s)
    assert np.sum((Gm.T @ w - gstar) ** 2) == pytest.approx(0.0, abs=1e-12)
    # a dominant example: the vertex
    s2 = np.array([10.0, 0.0, 0.0])
    w2 = oracle.simplex_ref(np.eye(3), s2)
    np.testing.assert_allclose(w2, [1.0, 0.0, 0.0], atol=1e-14)


def test_backprojection_is_the_adjoint_of_the_factorised_sketch():
    rng = np.random.default_rng(6)
    layers = []
    off = 0
    for d_in, d_out, k_in, k_out in [(7, 5, 3, 2), (4, 6, 2, 3)]:
        layers.append(dict(p_in=rng.standard_normal((k_in, d_in)), p_out=rng.standard_normal((k_out, d_out)),
                           col_offset=off, d_in=d_in, d_out=d_out))
        off += k_in * k_out
    u = rng.standard_normal(off)
    Us = oracle.backproject_ref(u, layers)
    for L, U in zip(layers, Us):
        G = rng.standard_normal((L["d_out"], L["d_in"]))
        Pi = np.kron(L["p_out"], L["p_in"])            # row-major vec, sketch layout [k_out][k_in]
        x = u[L["col_offset"]:L["col_offset"] + Pi.shape[0]]
        assert np.sum(G * U) == pytest.approx((Pi @ G.reshape(-1)) @ x, rel=1e-12)
        np.testing.assert_allclose(U.reshape(-1), Pi.T @ x, rtol=1e-12, atol=1e-12)
