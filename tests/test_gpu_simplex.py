"""GPU parity of the soft-weighting (simplex) projection and of the
back-projection against the oracle.

Simplex: the GPU iterates accelerated projected gradient to a step residual
of 1e-9; the exact optimum is the oracle's active-set solution.  With K
positive definite the optimum is unique: weights must agree to 1e-5 and the
residual distance resid2 to a relative 1e-5 (the fp32 1e-5 bar of the
solves).  Back-projection: fp32 sums of at most 64 products per stage, rel
1e-5 per layer block.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2605_07063_amd import api, workloads
from gpu_helpers import host64, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def gram_problem(P, n, dim, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    G = torch.randn(P, n, dim, generator=g, dtype=torch.float64)
    gs = torch.randn(P, dim, generator=g, dtype=torch.float64) * scale
    K = (G @ G.transpose(1, 2)).to(torch.float32)
    s = torch.einsum("pnd,pd->pn", G, gs).to(torch.float32)
    t2 = (gs * gs).sum(dim=1).to(torch.float32)
    return K, s, t2


def check(K, s, t2, max_iter=20000, tol=1e-9):
    w, r2, it, res, info = api.project_simplex(K.to(DEV), s.to(DEV), t2.to(DEV), max_iter, tol)
    torch.cuda.synchronize()
    for p in range(K.shape[0]):
        Kh, sh = host64(K[p]), host64(s[p])
        wref = oracle.simplex_ref(Kh, sh)
        wg = host64(w[p])
        assert int(info[p]) == 0, f"group {p}: info {int(info[p])} after {int(it[p])} steps, res {float(res[p])}"
        assert wg.min() >= 0.0 and abs(wg.sum() - 1.0) < 1e-6
        np.testing.assert_allclose(wg, wref, atol=1e-5)
        r2ref = float(t2[p]) + oracle.simplex_objective(Kh, sh, wref)
        assert abs(float(r2[p]) - r2ref) <= 1e-5 * max(abs(r2ref), float(t2[p])), (float(r2[p]), r2ref)
        assert oracle.simplex_residual(Kh, sh, wg) <= 1e-5
    return w, it


@pytest.mark.parametrize("n,dim,scale", [(7, 9, 1.0), (40, 60, 0.3), (64, 96, 3.0), (200, 240, 1.0)])
def test_simplex_matches_the_exact_optimum(n, dim, scale):
    K, s, t2 = gram_problem(3, n, dim, seed=n, scale=scale)
    _, it = check(K, s, t2)
    print(f"n={n}: steps {it.tolist()}")


def test_simplex_special_cases():
    # K = cI: the projection of s / c onto the simplex (sort-based, textbook)
    s = torch.randn(1, 50, generator=torch.Generator().manual_seed(3))
    c = 2.0
    v = (s[0] / c).double().numpy()
    u = np.sort(v)[::-1]
    css = np.cumsum(u)
    rho = max(j for j in range(50) if u[j] - (css[j] - 1) / (j + 1) > 0)
    want = np.maximum(v - (css[rho] - 1) / (rho + 1), 0)
    w, _, _, _, info = api.project_simplex((c * torch.eye(50)).unsqueeze(0).to(DEV), s.to(DEV),
                                           torch.ones(1, device=DEV), 20000, 1e-10)
    torch.cuda.synchronize()
    assert int(info[0]) == 0
    np.testing.assert_allclose(host64(w[0]), want, atol=1e-6)
    # one example; non-finite input; no examples
    w, r2, _, _, info = api.project_simplex(torch.full((1, 1, 1), 3.0, device=DEV), torch.tensor([[1.0]], device=DEV),
                                            torch.tensor([2.0], device=DEV), 10, 0.0)
    torch.cuda.synchronize()
    assert float(w[0, 0]) == 1.0 and abs(float(r2[0]) - (2.0 + 3.0 - 2.0)) < 1e-6
    K, s2, t2 = gram_problem(1, 10, 12, seed=4)
    s2[0, 3] = float("nan")
    _, _, _, _, info = api.project_simplex(K.to(DEV), s2.to(DEV), t2.to(DEV), 100, 1e-6)
    torch.cuda.synchronize()
    assert int(info[0]) == -3
    w0 = torch.empty(1, 0, device=DEV)
    r20 = torch.empty(1, device=DEV)
    it0 = torch.empty(1, dtype=torch.int32, device=DEV)
    rs0 = torch.empty(1, device=DEV)
    in0 = torch.empty(1, dtype=torch.int32, device=DEV)
    api.dr_project_simplex(torch.empty(1, 0, 0, device=DEV), torch.empty(1, 0, device=DEV),
                           torch.tensor([4.0], device=DEV), 10, 0.0, w0, r20, it0, rs0, in0)
    torch.cuda.synchronize()
    assert float(r20[0]) == 4.0 and int(in0[0]) == 0


def test_simplex_on_the_small_block_gram():
    """The small-block workload's own K and s (64 general examples over 32768
    sketch columns), one group and one group per layer."""
    cfg = workloads.CONFIGS["small"]
    layers, lens, ktot = workloads.sketch_inputs(cfg, DEV)
    S = api.sketch(layers, lens)
    n = cfg["n"]
    for goff in ([0, ktot], [int(L["col_offset"]) for L in layers] + [ktot]):
        K, s, t2 = api.gram(S[:n], S[n:], goff)
        check(K, s, t2, max_iter=50000, tol=1e-9)


@pytest.mark.parametrize("dtype,tol,specs", [
    (torch.float32, 1e-5, [(200, 136, 64, 64), (128, 264, 16, 32), (72, 64, 32, 16)]),
    # bf16, every dimension a multiple of 8: the bf16-MFMA path (T as three bf16 planes)
    (torch.bfloat16, 1e-5, [(200, 136, 64, 64), (128, 264, 16, 32), (72, 64, 32, 16)]),
    # bf16 with d_in = 100 (not a multiple of 8): the fp32 path for the whole launch
    (torch.bfloat16, 1e-5, [(100, 60, 8, 12), (136, 40, 64, 33)]),
])
def test_back_projection_matches_oracle(dtype, tol, specs):
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    layers, off = [], 0
    for d_in, d_out, k_in, k_out in specs:
        layers.append(dict(p_in=(torch.randn(k_in, d_in, generator=g, device=DEV) / k_in ** 0.5).to(dtype),
                           p_out=(torch.randn(k_out, d_out, generator=g, device=DEV) / k_out ** 0.5).to(dtype),
                           col_offset=off))
        off += k_in * k_out
    u = torch.randn(off + 5, generator=g, device=DEV)
    U = api.back_project(layers, u)
    torch.cuda.synchronize()
    hl = [dict(p_in=host64(L["p_in"]), p_out=host64(L["p_out"]), col_offset=L["col_offset"]) for L in layers]
    for got, ref in zip(U, oracle.backproject_ref(host64(u), hl)):
        assert rel(host64(got), ref) <= tol


def test_back_projection_of_the_small_block_update():
    """Sketch-space top-k update of the small-block workload (dr_combine) back
    to parameter space: 8 layers of 2048 x 2048 from 64 x 64 sketches."""
    cfg = workloads.CONFIGS["small"]
    layers, lens, ktot = workloads.sketch_inputs(cfg, DEV)
    n = cfg["n"]
    S = api.sketch(layers, lens)
    K, s, t2 = api.gram(S[:n], S[n:])
    _, w, _ = api.select_topk(s, n // 2)
    u = api.combine(S[:n], w)
    U = api.back_project(layers, u)
    torch.cuda.synchronize()
    hl = [dict(p_in=host64(L["p_in"]), p_out=host64(L["p_out"]), col_offset=L["col_offset"]) for L in layers]
    for got, ref in zip(U, oracle.backproject_ref(host64(u), hl)):
        assert rel(host64(got), ref) <= 1e-5
