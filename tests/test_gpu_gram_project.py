"""GPU parity of dr_gram, dr_project_span, dr_project_cone, dr_select_topk and
dr_combine against the oracle, on identical inputs, plus the invariants the
paper's problem statement fixes."""

import itertools

import numpy as np
import pytest
import torch

import oracle
from oracle.span import RIDGE_ABS, RIDGE_REL_TRACE
from paper_2605_07063_amd import api, workloads
from gpu_helpers import TOL_GRAM, TOL_SOLVE, host64, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def rand(shape, seed, dtype=torch.float32, scale=1.0):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * scale).to(dtype)


# --------------------------------------------------------------------------- Gram

@pytest.mark.parametrize("n,kappa,goff,dtype", [
    (65, 4096, None, torch.float32),                    # ragged row tile
    (16, 256, None, torch.float32),
    (130, 2048 + 512, [0, 512, 512, 2560], torch.float32),   # three groups, one empty
    (200, 3000 // 8 * 8, None, torch.bfloat16),
    (1, 64, None, torch.float32),
    (64, 2048 + 512 + 68, [0, 512, 512, 2628], torch.float32),   # one-pass small path: groups, one empty, ragged chunk
    (127, 8192, None, torch.float32),                 # largest n of the one-pass path
    (150, 1068, [0, 604, 1068], torch.float32),       # LDS-staged tiles: ragged 32-column steps in both groups
    (128, 2048, None, torch.float32),                 # LDS-staged tiles: two full row tiles
    (178, 1568, [0, 768, 1568], torch.float32),       # LDS-staged tiles: 50 rows in the third row tile
    (130, 2400, [8 * i for i in range(301)], torch.float32),   # 300 groups: two launches (256 + 44 groups)
    # 300 groups of one chunk each (tiles written without the reduction), two of them empty
    (130, 2400, [0] + list(itertools.accumulate([0 if g in (5, 100) else (16 if g in (6, 101) else 8)
                                                 for g in range(300)])), torch.float32),
])
def test_gram_matches_oracle(n, kappa, goff, dtype):
    G = rand((n, kappa), 10 + n, dtype)
    Gt = rand((5, kappa), 20 + n, dtype)
    K, s, t2 = api.gram(G, Gt, goff)
    torch.cuda.synchronize()
    Kr, sr, t2r = oracle.gram_ref(host64(G), host64(Gt), goff)
    Kg, sg, t2g = host64(K), host64(s), host64(t2)
    for p in range(Kr.shape[0]):
        assert np.array_equal(Kg[p], Kg[p].T), "K must be exactly symmetric"
        assert rel(Kg[p], Kr[p]) <= TOL_GRAM
        assert rel(sg[p], sr[p]) <= TOL_GRAM
        assert rel(t2g[p], t2r[p]) <= TOL_GRAM


def test_gram_no_general_rows_and_determinism():
    Gt = rand((3, 512), 5)
    G = torch.empty(0, 512, device=DEV)
    K, s, t2 = api.gram(G, Gt)
    torch.cuda.synchronize()
    _, _, t2r = oracle.gram_ref(np.zeros((0, 512)), host64(Gt))
    assert rel(host64(t2), t2r) <= TOL_GRAM
    G = rand((70, 4096), 6)
    a = api.gram(G, Gt[:, :1].expand(3, 4096).contiguous())
    b = api.gram(G, Gt[:, :1].expand(3, 4096).contiguous())
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    # the LDS-staged tile path (n + 1 > 128), with the scores formed in the
    # diagonal tiles: bit-identical on a repeat
    G = rand((200, 6144), 7)
    Gt2 = rand((5, 6144), 8)
    a = api.gram(G, Gt2, [0, 1024, 6144])
    b = api.gram(G, Gt2, [0, 1024, 6144])
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_gram_dominated_full_size_sampled():
    """16384 + 32 bf16 rows of dim 8192 (rank-32 spike): K rows sampled."""
    cfg = workloads.CONFIGS["gram"]
    rows = workloads.gram_rows(cfg, DEV)
    G, Gt = rows[:cfg["n"]], rows[cfg["n"]:]
    K, s, t2 = api.gram(G, Gt)
    torch.cuda.synchronize()
    pick = [0, 1, 4095, 8192, 16383]
    Gh = host64(G)
    gbar = host64(Gt).mean(0)
    Kref = Gh[pick] @ Gh.T
    Kg = host64(K[0, pick])
    assert rel(Kg, Kref) <= TOL_GRAM
    assert rel(host64(s[0]), Gh @ gbar) <= TOL_GRAM
    assert rel(host64(t2), [gbar @ gbar]) <= TOL_GRAM
    # exact symmetry on a sampled block
    assert torch.equal(K[0, :64, 8000:8064], K[0, 8000:8064, :64].T)


@pytest.mark.parametrize("n", [8200, 8195])
def test_gram_large_tiles_ragged_groups(n):
    """The 256x256-tile path: ragged n (8200 rows; 8195, whose K rows are not
    16-byte aligned), a ragged group width (1000 columns), an empty group and
    a full-width one; sampled rows of each K_p against the oracle, every K_p
    exactly symmetric."""
    goff = [0, 1000, 1000, 2600]
    G = rand((n, 2600), 77, torch.bfloat16)
    Gt = rand((3, 2600), 78, torch.bfloat16)
    K, s, t2 = api.gram(G, Gt, goff)
    torch.cuda.synchronize()
    pick = [0, 255, 256, 4100, 8191, n - 1]
    Gh, Gth = host64(G), host64(Gt)
    for p in range(3):
        c0, c1 = goff[p], goff[p + 1]
        Kref = Gh[pick, c0:c1] @ Gh[:, c0:c1].T
        if c1 == c0:
            assert torch.all(K[p] == 0)
        else:
            assert rel(host64(K[p, pick]), Kref) <= TOL_GRAM
        gbar = Gth[:, c0:c1].mean(0)
        if c1 > c0:
            assert rel(host64(s[p]), Gh[:, c0:c1] @ gbar) <= TOL_GRAM
        assert torch.equal(K[p], K[p].T)


# --------------------------------------------------------------------------- span

def spd_problem(n, kappa, seed, target_in_span=False):
    G = rand((n, kappa), seed)
    gbar = rand((kappa,), seed + 1)
    if target_in_span:
        gbar = (rand((n,), seed + 2) @ G)
    K, s, t2 = api.gram(G, gbar[None, :].contiguous())
    return G, gbar, K, s, t2


@pytest.mark.parametrize("n,kappa,lam,mode", [
    (16, 256, 1e-3, RIDGE_REL_TRACE),       # the tiny workload's shape
    (1, 64, 0.0, RIDGE_ABS),
    (64, 4096, 0.0, RIDGE_ABS),
    (200, 8192, 1e-2, RIDGE_REL_TRACE),
    (256, 16384, 0.0, RIDGE_ABS),           # the Llama-shaped n
    (37, 512, 0.5, RIDGE_ABS),
    (17, 256, 1e-3, RIDGE_REL_TRACE),       # every small-n kernel: 17..32 and 33..64, padded and full
    (32, 1024, 0.0, RIDGE_ABS),
    (48, 2048, 1e-2, RIDGE_REL_TRACE),
    (63, 4096, 0.0, RIDGE_ABS),
    (65, 4096, 0.0, RIDGE_ABS),             # 16x16-tile path: one row in the last tile
    (129, 8192, 1e-2, RIDGE_REL_TRACE),
    (255, 16384, 0.0, RIDGE_ABS),
])
def test_span_matches_oracle_and_normal_equations(n, kappa, lam, mode):
    G, gbar, K, s, t2 = spd_problem(n, kappa, 100 + n)
    w, lam_eff, resid2, info = api.project_span(K, s, t2, lam, mode)
    u = api.combine(G, w)
    torch.cuda.synchronize()
    assert int(info[0]) == 0
    Kh, sh, t2h = host64(K[0]), host64(s[0]), float(host64(t2)[0])
    le = float(host64(lam_eff)[0])
    if mode == RIDGE_REL_TRACE:
        assert abs(le - lam * np.trace(Kh) / n) <= 1e-6 * le
    w_ref, _, info_ref = oracle.span_ref(Kh, sh, lam, mode, lam_eff=le)
    assert info_ref == 0
    assert rel(host64(w[0]), w_ref) <= TOL_SOLVE
    u_ref = oracle.combine_ref(host64(G), w_ref)
    assert rel(host64(u), u_ref) <= TOL_SOLVE
    r2_ref = oracle.span_residual2(Kh, sh, t2h, w_ref)
    assert abs(float(host64(resid2)[0]) - r2_ref) <= 1e-5 * t2h
    # normal equations on the GPU output: G r = lam_eff w (orthogonality at lam = 0)
    r = host64(gbar) - host64(u)
    Gr = host64(G) @ r
    scale = np.linalg.norm(host64(G), axis=1).max() * np.linalg.norm(host64(gbar))
    assert np.abs(Gr - le * host64(w[0])).max() <= 1e-4 * scale


def test_span_special_cases():
    # target inside the span, lam = 0: u = gbar, residual ~ 0
    G, gbar, K, s, t2 = spd_problem(8, 512, 7, target_in_span=True)
    w, _, resid2, info = api.project_span(K, s, t2, 0.0, RIDGE_ABS)
    u = api.combine(G, w)
    torch.cuda.synchronize()
    assert int(info[0]) == 0
    assert rel(host64(u), host64(gbar)) <= 1e-5
    assert abs(float(resid2[0])) <= 1e-5 * float(t2[0])
    # not positive definite: first bad pivot reported, w = 0
    K = torch.diag(torch.tensor([1.0, -1.0, 1.0], device=DEV))[None].contiguous()
    s = torch.ones(1, 3, device=DEV)
    t2 = torch.ones(1, device=DEV)
    w, _, _, info = api.project_span(K, s, t2, 0.0, RIDGE_ABS)
    torch.cuda.synchronize()
    assert int(info[0]) == 2 and torch.all(w == 0)
    # relative ridge with K = 0: empty span, w = 0
    w, le, resid2, info = api.project_span(torch.zeros(1, 4, 4, device=DEV), torch.zeros(1, 4, device=DEV),
                                           torch.full((1,), 3.0, device=DEV), 1e-2, RIDGE_REL_TRACE)
    torch.cuda.synchronize()
    assert int(info[0]) == 0 and torch.all(w == 0) and float(resid2[0]) == 3.0
    # non-finite input
    Kn = torch.eye(3, device=DEV)[None].contiguous()
    Kn[0, 1, 1] = float("nan")
    w, _, _, info = api.project_span(Kn, torch.ones(1, 3, device=DEV), torch.ones(1, device=DEV), 0.0, RIDGE_ABS)
    torch.cuda.synchronize()
    assert int(info[0]) == -3
    # n = 0 with P = 2 groups
    w, le, resid2, info = api.project_span(torch.zeros(2, 0, 0, device=DEV), torch.zeros(2, 0, device=DEV),
                                           torch.tensor([1.0, 2.0], device=DEV), 1e-2, RIDGE_REL_TRACE)
    torch.cuda.synchronize()
    assert torch.all(info == 0) and torch.equal(resid2.cpu(), torch.tensor([1.0, 2.0]))


@pytest.mark.parametrize("n", [12, 20, 32, 40, 64, 100, 150, 256])
def test_span_bad_pivot_and_batched_groups(n):
    # group 0: K = diag(1, ..., -1 at j = n - 3, ..., 1) -> info = n - 2 (1-based), w = 0, resid2 = t2;
    # groups 1, 2: random SPD problems of the same n, each against the oracle
    j = n - 3
    d = torch.ones(n, device=DEV)
    d[j] = -1.0
    Ks, ss, t2s = [torch.diag(d)], [torch.ones(n, device=DEV)], [torch.full((), 2.0, device=DEV)]
    for g in (1, 2):
        _, _, K, s, t2 = spd_problem(n, 2048, 700 + 10 * n + g)
        Ks.append(K[0]), ss.append(s[0]), t2s.append(t2[0])
    K, s, t2 = torch.stack(Ks).contiguous(), torch.stack(ss).contiguous(), torch.stack(t2s).contiguous()
    w, lam_eff, resid2, info = api.project_span(K, s, t2, 1e-3, RIDGE_ABS)
    torch.cuda.synchronize()
    assert int(info[0]) == j + 1 and torch.all(w[0] == 0) and float(resid2[0]) == 2.0
    for g in (1, 2):
        assert int(info[g]) == 0
        w_ref, _, info_ref = oracle.span_ref(host64(K[g]), host64(s[g]), 1e-3, RIDGE_ABS)
        assert info_ref == 0
        assert rel(host64(w[g]), w_ref) <= TOL_SOLVE
        r2_ref = oracle.span_residual2(host64(K[g]), host64(s[g]), float(t2[g]), w_ref)
        assert abs(float(resid2[g]) - r2_ref) <= 1e-5 * float(t2[g])


def test_span_tiles_first_pivot_and_upper_nan():
    # 64 < n <= 256 (16x16 LDS tiles): a non-positive pivot in the first tile
    # (factored before the look-ahead starts) and one at the last column
    for n, j in ((150, 5), (150, 149), (200, 16)):
        d = torch.ones(n, device=DEV)
        d[j] = 0.0
        w, _, resid2, info = api.project_span(torch.diag(d)[None].contiguous(), torch.ones(1, n, device=DEV),
                                              torch.full((1,), 2.0, device=DEV), 0.0, RIDGE_ABS)
        torch.cuda.synchronize()
        assert int(info[0]) == j + 1 and torch.all(w == 0) and float(resid2[0]) == 2.0
    # a NaN strictly above the diagonal (never factored) is still reported
    _, _, K, s, t2 = spd_problem(200, 2048, 901)
    K[0, 3, 170] = float("nan")
    w, _, _, info = api.project_span(K, s, t2, 0.0, RIDGE_ABS)
    torch.cuda.synchronize()
    assert int(info[0]) == -3 and torch.all(w == 0)


# ------------------------------------------------------------ span, n > 256 (blocked)

@pytest.mark.parametrize("n,kappa,lam,mode", [
    (257, 4096, 1e-3, RIDGE_REL_TRACE),     # one full panel + a 1-row panel
    (300, 256, 1e-2, RIDGE_REL_TRACE),      # rank-deficient G: the ridge carries it
    (1000, 4096, 0.0, RIDGE_ABS),           # no ridge, full rank
    (2085, 8192, 0.5, RIDGE_ABS),           # ragged last panel, several trailing tiles
    (6144, 8192, 1e-3, RIDGE_REL_TRACE),    # the first panel pairs' bulk updates on split bf16 planes
    (7000, 8192, 0.0, RIDGE_ABS),           # ... with a partial last 256-row tile, no ridge
    (6998, 8192, 1e-3, RIDGE_ABS),          # ... with n not a multiple of 4: partial float4 column tails
])
def test_span_blocked_matches_oracle(n, kappa, lam, mode):
    G, gbar, K, s, t2 = spd_problem(n, kappa, 900 + n)
    w, lam_eff, resid2, info = api.project_span(K, s, t2, lam, mode)
    torch.cuda.synchronize()
    assert int(info[0]) == 0
    Kh, sh, t2h = host64(K[0]), host64(s[0]), float(host64(t2)[0])
    le = float(host64(lam_eff)[0])
    if mode == RIDGE_REL_TRACE:
        assert abs(le - lam * np.trace(Kh) / n) <= 1e-6 * le
    w_ref, _, info_ref = oracle.span_ref(Kh, sh, lam, mode, lam_eff=le)
    assert info_ref == 0
    assert rel(host64(w[0]), w_ref) <= TOL_SOLVE, rel(host64(w[0]), w_ref)
    r2_ref = oracle.span_residual2(Kh, sh, t2h, w_ref)
    assert abs(float(host64(resid2)[0]) - r2_ref) <= 1e-5 * t2h


def test_span_blocked_special_cases():
    n = 400
    # non-positive pivots: in the first diagonal tile of the first block, at
    # the end of the first tile of the second block, inside a later tile of
    # it (factored one step ahead), and in the last row (a 16-row block)
    for j in (5, 143, 200, n - 1):
        d = torch.ones(n, device=DEV)
        d[j] = -1.0
        w, _, r2, info = api.project_span(torch.diag(d)[None].contiguous(), torch.ones(1, n, device=DEV),
                                          torch.full((1,), 5.0, device=DEV), 0.0, RIDGE_ABS)
        torch.cuda.synchronize()
        assert int(info[0]) == j + 1 and torch.all(w == 0) and float(r2[0]) == 5.0
    # a NaN in the upper triangle (the factorisation never reads it; the residual does)
    G, gbar, K, s, t2 = spd_problem(n, 1024, 31)
    Kn = K.clone()
    Kn[0, 3, 300] = float("nan")
    w, le, r2, info = api.project_span(Kn, s, t2, 1e-3, RIDGE_REL_TRACE)
    torch.cuda.synchronize()
    assert int(info[0]) == -3 and torch.all(w == 0) and float(le[0]) == 0.0
    # a non-finite entry outranks a non-positive pivot, wherever each lies
    # (the first panels are factored while the rest of K is still scanned):
    # a pivot failure in the first block with a NaN in a late column, below
    # and above the diagonal
    for (i, j) in ((390, 350), (300, 399)):
        d = torch.ones(n, device=DEV)
        d[2] = -1.0
        Kb = torch.diag(d)[None].contiguous()
        Kb[0, i, j] = float("nan")
        w, le, r2, info = api.project_span(Kb, torch.ones(1, n, device=DEV), torch.full((1,), 5.0, device=DEV), 0.0,
                                           RIDGE_ABS)
        torch.cuda.synchronize()
        assert int(info[0]) == -3 and torch.all(w == 0) and float(le[0]) == 0.0 and float(r2[0]) == 5.0
    # relative ridge with K = 0: empty span
    w, le, r2, info = api.project_span(torch.zeros(1, n, n, device=DEV), torch.zeros(1, n, device=DEV),
                                       torch.full((1,), 3.0, device=DEV), 1e-2, RIDGE_REL_TRACE)
    torch.cuda.synchronize()
    assert int(info[0]) == 0 and torch.all(w == 0) and float(r2[0]) == 3.0
    # two groups in one call share the workspace one after another; the
    # target inside the span is reproduced at lam = 0
    G1, g1, K1, s1, t21 = spd_problem(n, 2048, 41, target_in_span=True)
    G2, g2, K2, s2, t22 = spd_problem(n, 2048, 42)
    K = torch.cat([K1, K2]).contiguous()
    s = torch.cat([s1, s2]).contiguous()
    t2 = torch.cat([t21, t22]).contiguous()
    w, le, r2, info = api.project_span(K, s, t2, 0.0, RIDGE_ABS)
    u1 = api.combine(G1, w[:1].contiguous())
    torch.cuda.synchronize()
    assert torch.all(info == 0)
    assert rel(host64(u1), host64(g1)) <= 1e-4
    w_ref, _, _ = oracle.span_ref(host64(K2[0]), host64(s2[0]), 0.0, RIDGE_ABS)
    assert rel(host64(w[1]), w_ref) <= TOL_SOLVE


@pytest.mark.parametrize("n", [128, 320])
def test_span_refinement_flag_tracks_accuracy_over_a_conditioning_sweep(n):
    """n = 128 (one-workgroup tiles) and n = 320 (blocked): K = Q diag(l) Q^T
    with l from 1 down to 1 / cond, cond = 1e2 .. 1e7, rounded to fp32.  A
    result reported converged (info = 0) must be within 1e-5 of the fp64
    solution of the same fp32 system; the ill-conditioned end of the sweep
    must be reported (DR_INFO_NOT_CONVERGED, or a non-positive pivot), not
    returned silently."""
    rng = np.random.default_rng(31 + n)
    Q, _ = np.linalg.qr(rng.standard_normal((n, n)))
    out = []
    for cond in (1e2, 1e3, 1e4, 1e5, 1e6, 1e7):
        lam = np.geomspace(1.0, 1.0 / cond, n)
        K32 = ((Q * lam) @ Q.T).astype(np.float32)
        K32 = ((K32 + K32.T) / 2).astype(np.float32)
        s32 = (K32.astype(np.float64) @ rng.standard_normal(n)).astype(np.float32)
        K = torch.from_numpy(K32)[None].to(DEV)
        s = torch.from_numpy(s32)[None].to(DEV)
        t2 = torch.ones(1, device=DEV)
        w, le, r2, info = api.project_span(K, s, t2, 0.0, RIDGE_ABS)
        torch.cuda.synchronize()
        w_ref = np.linalg.solve(K32.astype(np.float64), s32.astype(np.float64))
        err = rel(host64(w[0]), w_ref)
        inf = int(info[0])
        out.append((cond, inf, err))
        print(f"n={n} cond {cond:.0e}: info {inf}, rel err {err:.2e}", flush=True)
        if inf == 0:
            assert err <= TOL_SOLVE, (cond, err)
        else:
            assert inf == -2 or inf > 0, (cond, inf)
    assert out[0][1] == 0 and out[1][1] == 0
    assert out[-1][1] != 0


def test_span_gram_dominated_full_size():
    """n = 16384 from the 16384 x 8192 bf16 rows with a rank-32 spike, relative ridge 1e-2:
    parity with the fp64 LAPACK oracle and the ridge normal equations G (gbar - G^T w) = lam w."""
    cfg = workloads.CONFIGS["gram"]
    rows = workloads.gram_rows(cfg, DEV)
    G, Gt = rows[:cfg["n"]], rows[cfg["n"]:]
    K, s, t2 = api.gram(G, Gt)
    w, lam_eff, resid2, info = api.project_span(K, s, t2, cfg["lam"], RIDGE_REL_TRACE)
    torch.cuda.synchronize()
    assert int(info[0]) == 0
    le = float(lam_eff[0])
    Kh, sh = host64(K[0]), host64(s[0])
    w_ref, _, info_ref = oracle.span_ref(Kh, sh, cfg["lam"], RIDGE_REL_TRACE, lam_eff=le)
    assert info_ref == 0
    wg = host64(w[0])
    assert rel(wg, w_ref) <= TOL_SOLVE, rel(wg, w_ref)
    r2_ref = oracle.span_residual2(Kh, sh, float(t2[0]), w_ref)
    assert abs(float(resid2[0]) - r2_ref) <= 1e-5 * float(t2[0])
    # ridge normal equations in the sketch space: K w + lam w = s
    res = Kh @ wg + le * wg - sh
    assert np.linalg.norm(res) <= 1e-5 * np.linalg.norm(sh)


def test_span_batched_groups_and_hand_fixture(golden_dir):
    import json, os
    fx = json.load(open(os.path.join(golden_dir, "span_2x2.json")))
    P = len(fx["cases"])
    K = torch.tensor([fx["K"]] * P, dtype=torch.float32, device=DEV)
    s = torch.tensor([fx["s"]] * P, dtype=torch.float32, device=DEV)
    t2 = torch.full((P,), float(fx["t2"]), device=DEV)
    for p, c in enumerate(fx["cases"]):
        w, le, r2, info = api.project_span(K[p:p + 1].contiguous(), s[p:p + 1].contiguous(), t2[p:p + 1].contiguous(),
                                           c["lam"], c["mode"])
        torch.cuda.synchronize()
        assert int(info[0]) == 0
        np.testing.assert_allclose(host64(w[0]), c["w"], rtol=1e-6, atol=1e-7)
        assert abs(float(le[0]) - c["lam_eff"]) <= 1e-7
        assert abs(float(r2[0]) - c["resid2"]) <= 1e-5


# --------------------------------------------------------------------------- cone

@pytest.mark.parametrize("n,kappa,iters,tol", [
    (64, 8192, 200, 0.0),       # the small-block workload: 200 projected-gradient steps
    (32, 16384, 100000, 1e-6),  # the long-context workload: run to KKT residual 1e-6
    (16, 1024, 3000, 1e-6),
    (24, 4096, 400, 0.0),       # padded 17..32 path at a fixed step count
    (45, 4096, 5000, 1e-6),     # padded 33..64 path to tolerance
    (200, 32768, 20000, 1e-6),  # n > 128: K read from memory each step
    (1, 64, 10, 0.0),
])
def test_cone_matches_exact_nnls(n, kappa, iters, tol):
    G = rand((n, kappa), 300 + n) * (0.5 + rand((n, 1), 301 + n).abs())
    gbar = rand((kappa,), 302 + n) * 0.3 + 0.05 * G[: max(1, n // 8)].sum(0)
    K, s, t2 = api.gram(G.contiguous(), gbar[None, :].contiguous())
    w, resid2, it, kkt, info = api.project_cone(K, s, t2, iters, tol)
    u = api.combine(G.contiguous(), w)
    torch.cuda.synchronize()
    Kh, sh, t2h = host64(K[0]), host64(s[0]), float(host64(t2)[0])
    w_ref = oracle.nnls_active_set(Kh, sh)
    assert int(info[0]) == 0
    if tol > 0:
        assert float(kkt[0]) <= tol and int(it[0]) < iters
    else:
        assert int(it[0]) == iters
    wg = host64(w[0])
    assert np.all(wg >= 0)
    assert rel(wg, w_ref) <= TOL_SOLVE, rel(wg, w_ref)
    assert rel(host64(u), oracle.combine_ref(host64(G), w_ref)) <= TOL_SOLVE
    _, r2_ref = oracle.cone_ref(Kh, sh, t2h)
    assert abs(float(resid2[0]) - r2_ref) <= 1e-5 * t2h
    # KKT of the GPU output, in primal form: <g_i, r> <= 0, = 0 on the support
    rho = oracle.cone_kkt_residual(Kh, sh, wg)
    assert rho <= 1e-5
    if tol > 0:
        assert abs(rho - float(kkt[0])) <= 1e-6


def test_cone_special_cases(golden_dir):
    import json, os
    fx = json.load(open(os.path.join(golden_dir, "cone_2x2.json")))
    P = len(fx["cases"])
    K = torch.tensor([fx["K"]] * P, dtype=torch.float32, device=DEV)
    s = torch.tensor([c["s"] for c in fx["cases"]], dtype=torch.float32, device=DEV)
    t2 = torch.ones(P, device=DEV) * 100.0
    w, _, it, kkt, info = api.project_cone(K, s, t2, 10000, 1e-7)
    torch.cuda.synchronize()
    for p, c in enumerate(fx["cases"]):
        np.testing.assert_allclose(host64(w[p]), c["w"], rtol=1e-6, atol=1e-7)
        assert int(info[p]) == 0
    # target inside the cone: w = c
    G = rand((6, 512), 9)
    c = rand((6,), 10).abs() + 0.2
    gbar = c @ G
    K, s, t2 = api.gram(G, gbar[None, :].contiguous())
    w, resid2, it, kkt, info = api.project_cone(K, s, t2, 100000, 1e-7)
    torch.cuda.synchronize()
    assert rel(host64(w[0]), host64(c)) <= 1e-4
    # not converged within the budget
    w, resid2, it, kkt, info = api.project_cone(K, s, t2, 2, 1e-12)
    torch.cuda.synchronize()
    assert int(info[0]) == -2 and int(it[0]) == 2
    # n = 0
    w, resid2, it, kkt, info = api.project_cone(torch.zeros(1, 0, 0, device=DEV), torch.zeros(1, 0, device=DEV),
                                                torch.ones(1, device=DEV), 10, 0.0)
    torch.cuda.synchronize()
    assert int(info[0]) == 0 and float(resid2[0]) == 1.0


# --------------------------------------------------------------------------- top-k

def check_topk(s, k):
    idx, w, info = api.select_topk(s, k)
    torch.cuda.synchronize()
    sh = s.cpu().numpy()
    for p in range(s.shape[0]):
        ref = oracle.topk_ref(sh[p].astype(np.float64), k)
        got = idx[p].cpu().numpy()
        assert np.array_equal(got, ref), (p, got[:10], ref[:10])
        wp = w[p].cpu().numpy()
        assert np.all(wp[ref] == np.float32(1.0 / k)) if k > 0 else True
        mask = np.ones(s.shape[1], bool)
        mask[ref] = False
        assert np.all(wp[mask] == 0.0)
        assert int(info[p]) == 0


@pytest.mark.parametrize("n,k,P", [(256, 64, 1), (16384, 1024, 1), (64, 32, 3), (1000, 1, 2), (1000, 1000, 1),
                                   (70000, 5000, 1), (5, 0, 1)])
def test_topk_exact_on_random_scores(n, k, P):
    check_topk(rand((P, n), 400 + n), k)


def test_topk_ties_signed_zero_infinities_and_nan(golden_dir):
    import json, os
    fx = json.load(open(os.path.join(golden_dir, "topk_ties.json")))
    for c in fx["cases"]:
        s = torch.tensor([[float(v) for v in c["s"]]], dtype=torch.float32, device=DEV)
        idx, w, info = api.select_topk(s, c["k"])
        torch.cuda.synchronize()
        assert idx[0].cpu().tolist() == c["idx"], c
    # heavy ties: integers in [-3, 3]
    s = torch.randint(-3, 4, (2, 5000), device=DEV).float()
    for k in (1, 7, 2500, 4999):
        check_topk(s, k)
    s = torch.zeros(1, 10, device=DEV)
    s[0, 3] = float("nan")
    idx, w, info = api.select_topk(s, 4)
    torch.cuda.synchronize()
    assert int(info[0]) == -3 and torch.all(idx == -1) and torch.all(w == 0)


# --------------------------------------------------------------------------- combine

@pytest.mark.parametrize("dtype,n", [(torch.float32, 300), (torch.bfloat16, 300), (torch.float32, 64),
                                     (torch.bfloat16, 64), (torch.float32, 1), (torch.float32, 13)])
def test_combine_groups(dtype, n):
    kappa = 4096
    G = rand((n, kappa), 500, dtype)
    goff = [0, 1024, 1024, 4096]
    w = rand((3, n), 501)
    u = api.combine(G, w, goff)
    torch.cuda.synchronize()
    ref = oracle.combine_ref(host64(G), host64(w), goff)
    assert rel(host64(u), ref) <= 1e-6
