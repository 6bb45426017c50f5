"""End-to-end hot path on the GPU (sketch -> Gram -> projection -> combine),
each stage checked against the oracle on the stage's exact inputs, and the
end-to-end result checked against the oracle run from the raw inputs."""

import numpy as np
import pytest
import torch

import oracle
from oracle.span import RIDGE_REL_TRACE
from paper_2605_07063_amd import api, workloads
from gpu_helpers import TOL_GRAM, TOL_SKETCH_F32, TOL_SOLVE, host64, layers_to_host, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_tiny_workload_end_to_end():
    cfg = workloads.CONFIGS["tiny"]
    n, m = cfg["n"], cfg["m"]
    layers, lens, kt = workloads.sketch_inputs(cfg, DEV)
    S = api.sketch(layers, lens)
    K, s, t2 = api.gram(S[:n], S[n:])
    w, lam_eff, resid2, info = api.project_span(K, s, t2, cfg["lam"], RIDGE_REL_TRACE)
    u = api.combine(S[:n], w)
    torch.cuda.synchronize()
    assert int(info[0]) == 0
    # oracle from the raw inputs: explicit gradients -> sketches -> Gram -> ridge solve
    S_ref = oracle.sketch_ref(layers_to_host(layers), lens.cpu().numpy())
    assert rel(host64(S), S_ref) <= TOL_SKETCH_F32
    K_ref, s_ref, t2_ref = oracle.gram_ref(S_ref[:n], S_ref[n:])
    assert rel(host64(K[0]), K_ref[0]) <= TOL_GRAM
    assert rel(host64(s[0]), s_ref[0]) <= TOL_GRAM
    w_ref, le_ref, _ = oracle.span_ref(K_ref[0], s_ref[0], cfg["lam"], RIDGE_REL_TRACE)
    assert abs(float(lam_eff[0]) - le_ref) <= 1e-6 * le_ref
    # stage-wise: same (K, s, lam_eff) as the GPU used
    w_stage, _, _ = oracle.span_ref(host64(K[0]), host64(s[0]), cfg["lam"], RIDGE_REL_TRACE,
                                    lam_eff=float(lam_eff[0]))
    assert rel(host64(w[0]), w_stage) <= TOL_SOLVE
    # end to end (bounded by cond(K + lam I) times the sketch error)
    e2e = rel(host64(u), oracle.combine_ref(S_ref[:n], w_ref))
    print(f"tiny end-to-end rel err of u: {e2e:.2e}")
    assert e2e <= 1e-4


def test_small_block_workload_end_to_end_with_all_projections():
    """The benchmark's step at full size: 8 layers, 72 examples, cone 200
    iterations, span and top-k on the same Gram; stages after the sketch are
    checked in full against the oracle on the GPU's own sketches."""
    cfg = workloads.CONFIGS["small"]
    n, m = cfg["n"], cfg["m"]
    layers, lens, kt = workloads.sketch_inputs(cfg, DEV, nan_padding=True)
    S = api.sketch(layers, lens)
    K, s, t2 = api.gram(S[:n], S[n:])
    wc, r2c, itc, kktc, infoc = api.project_cone(K, s, t2, cfg["iters"], 0.0)
    ws, le, r2s, infos = api.project_span(K, s, t2, 1e-3, RIDGE_REL_TRACE)
    idx, wt, infot = api.select_topk(s, n // 2)
    u = api.combine(S[:n], wc)
    torch.cuda.synchronize()
    Sg = host64(S)
    assert np.isfinite(Sg).all()
    K_ref, s_ref, t2_ref = oracle.gram_ref(Sg[:n], Sg[n:])
    assert rel(host64(K[0]), K_ref[0]) <= TOL_GRAM
    assert rel(host64(s[0]), s_ref[0]) <= TOL_GRAM
    Kh, sh = host64(K[0]), host64(s[0])
    w_ref = oracle.nnls_active_set(Kh, sh)
    assert int(infoc[0]) == 0 and int(itc[0]) == cfg["iters"]
    assert rel(host64(wc[0]), w_ref) <= TOL_SOLVE
    assert rel(host64(u), oracle.combine_ref(Sg[:n], w_ref)) <= TOL_SOLVE
    wsr, _, _ = oracle.span_ref(Kh, sh, 1e-3, RIDGE_REL_TRACE, lam_eff=float(le[0]))
    assert int(infos[0]) == 0 and rel(host64(ws[0]), wsr) <= TOL_SOLVE
    assert np.array_equal(idx[0].cpu().numpy(), oracle.topk_ref(host64(s[0]), n // 2))


def test_small_block_layerwise_groups():
    """Layer-wise mode (one group per layer, P = 8 groups of 4096 columns) on
    the benchmark's sketches: batched Gram, cone, span, top-k and combine,
    every group against the oracle on the GPU's own sketches."""
    cfg = workloads.CONFIGS["small"]
    n, m = cfg["n"], cfg["m"]
    layers, lens, kt = workloads.sketch_inputs(cfg, DEV)
    goff = [int(L["col_offset"]) for L in layers] + [kt]
    P = len(layers)
    S = api.sketch(layers, lens)
    K, s, t2 = api.gram(S[:n], S[n:], goff)
    wc, r2c, itc, kktc, infoc = api.project_cone(K, s, t2, cfg["iters"], 0.0)
    ws, le, r2s, infos = api.project_span(K, s, t2, 1e-3, RIDGE_REL_TRACE)
    idx, wt, infot = api.select_topk(s, n // 2)
    u = api.combine(S[:n], wc, goff)
    torch.cuda.synchronize()
    Sg = host64(S)
    K_ref, s_ref, t2_ref = oracle.gram_ref(Sg[:n], Sg[n:], goff)
    u_h = host64(u)
    for p in range(P):
        Kh, sh = host64(K[p]), host64(s[p])
        assert rel(Kh, K_ref[p]) <= TOL_GRAM and rel(sh, s_ref[p]) <= TOL_GRAM
        assert int(infoc[p]) == 0 and int(infos[p]) == 0 and int(infot[p]) == 0
        w_ref = oracle.nnls_active_set(Kh, sh)
        assert rel(host64(wc[p]), w_ref) <= TOL_SOLVE
        wsr, _, _ = oracle.span_ref(Kh, sh, 1e-3, RIDGE_REL_TRACE, lam_eff=float(le[p]))
        assert rel(host64(ws[p]), wsr) <= TOL_SOLVE
        assert np.array_equal(idx[p].cpu().numpy(), oracle.topk_ref(sh, n // 2))
        c0, c1 = goff[p], goff[p + 1]
        assert rel(u_h[c0:c1], oracle.combine_ref(Sg[:n, c0:c1], w_ref)) <= TOL_SOLVE


def test_llama_shaped_layerwise_projection():
    """Layer-wise mode at the Llama-shaped scale: 224 groups (one per matrix)
    of 1024 sketch columns, n = 256 general + 16 target rows; the Gram runs
    as two launches of at most 128 groups; span at lam = 0 and top-64 on
    every group, sampled groups against the oracle."""
    n, m, P, width = 256, 16, 224, 1024
    g = torch.Generator(device=DEV)
    g.manual_seed(4242)
    rows = torch.randn(n + m, P * width, generator=g, device=DEV)
    goff = [p * width for p in range(P + 1)]
    K, s, t2 = api.gram(rows[:n], rows[n:], goff)
    w, le, r2, info = api.project_span(K, s, t2, 0.0, 0)
    idx, wt, infot = api.select_topk(s, 64)
    torch.cuda.synchronize()
    assert torch.all(info == 0) and torch.all(infot == 0)
    Rh = host64(rows)
    for p in (0, 127, 128, 223):
        c0, c1 = goff[p], goff[p + 1]
        K_ref, s_ref, _ = oracle.gram_ref(Rh[:n, c0:c1], Rh[n:, c0:c1])
        assert rel(host64(K[p]), K_ref[0]) <= TOL_GRAM and rel(host64(s[p]), s_ref[0]) <= TOL_GRAM
        w_ref, _, info_ref = oracle.span_ref(host64(K[p]), host64(s[p]), 0.0, 0)
        assert info_ref == 0 and rel(host64(w[p]), w_ref) <= TOL_SOLVE
        assert np.array_equal(idx[p].cpu().numpy(), oracle.topk_ref(host64(s[p]), 64))


def test_long_context_layerwise_cone():
    """Long-context layer-wise mode: 16 groups with n = 32 general rows, cone
    to KKT residual 1e-6 in every group."""
    n, m, P, width = 32, 4, 16, 4096
    g = torch.Generator(device=DEV)
    g.manual_seed(777)
    rows = torch.randn(n + m, P * width, generator=g, device=DEV)
    rows[n:] += 0.3 * rows[: m]   # targets partly aligned with some general rows
    goff = [p * width for p in range(P + 1)]
    K, s, t2 = api.gram(rows[:n], rows[n:], goff)
    w, r2, it, kkt, info = api.project_cone(K, s, t2, 100000, 1e-6)
    torch.cuda.synchronize()
    for p in range(P):
        assert int(info[p]) == 0 and float(kkt[p]) <= 1e-6
        w_ref = oracle.nnls_active_set(host64(K[p]), host64(s[p]))
        assert rel(host64(w[p]), w_ref) <= TOL_SOLVE
