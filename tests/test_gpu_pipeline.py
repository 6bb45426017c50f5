"""End-to-end hot path on the GPU (sketch -> Gram -> projection -> combine),
each stage checked against the oracle on the stage's exact inputs, and the
end-to-end result checked against the oracle run from the raw inputs."""

import numpy as np
import pytest
import torch

import oracle
from oracle.span import RIDGE_REL_TRACE
from paper_2605_07063_amd import api, workloads
from gpu_helpers import (TOL_GRAM, TOL_SKETCH_BF16, TOL_SKETCH_F32, TOL_SOLVE, block_errors, host64, layers_to_host,
                         rel)

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


def _topk_consistent(idx_gpu, s_ref, k):
    """The GPU's top-k index set against the oracle's scores: identical
    whenever the k-th and (k+1)-th scores differ by more than 1e-6 of the
    largest |score|; otherwise differences only among near-tied indices."""
    ref = oracle.topk_ref(s_ref, k)
    if np.array_equal(idx_gpu, ref):
        return True
    order = np.lexsort((np.arange(s_ref.shape[0]), -s_ref))
    gap = s_ref[order[k - 1]] - s_ref[order[k]] if k < s_ref.shape[0] else np.inf
    tol = 1e-6 * np.abs(s_ref).max()
    if gap > tol:
        return False
    diff = np.setxor1d(idx_gpu, ref)
    return bool(np.all(np.abs(s_ref[diff] - s_ref[order[k - 1]]) <= tol))


def test_llama_shaped_step_global_group_on_its_own_sketches():
    """The whole Llama-shaped step at full size, launched as the benchmark
    launches it: 32 block calls (two resident blocks of activations, each
    block with its own projectors and column range), then one group over all
    229376 columns -- the Gram (many column-chunk partials), the span at
    lambda = 0 (Eq. (proj) exactly), top-64 and the combine -- each checked
    against the oracle on the GPU's own sketches; sampled sketch blocks of
    blocks 0 and 31 against the explicit-gradient oracle; and the strict
    orthogonality of the span residual to every general sketch."""
    cfg = workloads.CONFIGS["llama"]
    n, m, T, k = cfg["n"], cfg["m"], cfg["T"], cfg["topk"]
    N = n + m
    print("llama step: drawing two blocks of activations", flush=True)
    blocks, lens, ktot = workloads.llama_step_inputs(cfg, DEV)
    assert len(blocks) == 32 and ktot == 229376
    S = torch.empty(N, ktot, device=DEV)
    ws = torch.empty(max(1, api.dr_sketch_workspace_size(blocks[0], N, T, torch.bfloat16)), dtype=torch.uint8,
                     device=DEV)
    for blk in blocks:
        api.dr_sketch_grads(blk, N, T, lens, S, workspace=ws)
    K, s, t2 = api.gram(S[:n], S[n:])
    w, le, r2, info = api.project_span(K, s, t2, 0.0, 0)
    idx, wt, infot = api.select_topk(s, k)
    u = api.combine(S[:n], w)
    torch.cuda.synchronize()
    print("llama step: GPU done, checking", flush=True)
    assert int(info[0]) == 0 and int(infot[0]) == 0
    Sg = host64(S)
    assert np.isfinite(Sg).all()
    # sketch: two examples (a general and a target row) x 7 maps x blocks 0 and 31
    rows = [0, 271]
    for b in (0, 31):
        ref = oracle.sketch_ref(layers_to_host(blocks[b], rows), lens.cpu().numpy()[rows])
        errs = block_errors(Sg[rows], ref, blocks[b], range(len(rows)))
        print(f"llama step: block {b} sampled max block rel err {errs.max():.2e}", flush=True)
        assert errs.max() <= TOL_SKETCH_BF16
    # Gram, scores, target norm
    K_ref, s_ref, t2_ref = oracle.gram_ref(Sg[:n], Sg[n:])
    Kh, sh = host64(K[0]), host64(s[0])
    assert np.array_equal(Kh, Kh.T)
    assert rel(Kh, K_ref[0]) <= TOL_GRAM and rel(sh, s_ref[0]) <= TOL_GRAM
    assert abs(float(t2[0]) - t2_ref[0]) <= TOL_GRAM * t2_ref[0]
    # span at lambda = 0: stage-wise on the GPU's (K, s), then end to end
    w_stage, _, inf = oracle.span_ref(Kh, sh, 0.0, 0)
    wh = host64(w[0])
    assert inf == 0 and rel(wh, w_stage) <= TOL_SOLVE
    w_e2e, _, _ = oracle.span_ref(K_ref[0], s_ref[0], 0.0, 0)
    print(f"llama step: span stage err {rel(wh, w_stage):.2e}, end-to-end {rel(wh, w_e2e):.2e}", flush=True)
    assert rel(wh, w_e2e) <= 1e-4
    # the residual r = gbar - G^T w is orthogonal to every general sketch
    gbar = Sg[n:].mean(axis=0)
    r = gbar - Sg[:n].T @ wh
    cos = np.abs(Sg[:n] @ r) / (np.linalg.norm(Sg[:n], axis=1) * np.linalg.norm(r))
    print(f"llama step: max |cos(g_i, r)| {cos.max():.2e}", flush=True)
    assert cos.max() <= 1e-5
    assert abs(float(r2[0]) - r @ r) <= 1e-5 * (r @ r)
    # combine and top-64
    assert rel(host64(u), oracle.combine_ref(Sg[:n], wh)) <= TOL_SOLVE
    ig = idx[0].cpu().numpy()
    assert np.array_equal(ig, oracle.topk_ref(sh, k))
    assert _topk_consistent(ig, s_ref[0], k)
    assert np.all(wt[0].cpu().numpy()[ig] == np.float32(1.0 / k))
    # layer-wise mode on the same sketches: one group per map (224 x 1024 columns)
    goff = [p * 1024 for p in range(225)]
    Kl, sl, t2l = api.gram(S[:n], S[n:], goff)
    wl, lel, r2l, infol = api.project_span(Kl, sl, t2l, 0.0, 0)
    idxl, wtl, inftl = api.select_topk(sl, k)
    torch.cuda.synchronize()
    assert torch.all(infol == 0) and torch.all(inftl == 0)
    for p in (0, 6, 127, 128, 223):
        c0, c1 = goff[p], goff[p + 1]
        Kr, sr, _ = oracle.gram_ref(Sg[:n, c0:c1], Sg[n:, c0:c1])
        Kp, sp_ = host64(Kl[p]), host64(sl[p])
        assert rel(Kp, Kr[0]) <= TOL_GRAM and rel(sp_, sr[0]) <= TOL_GRAM
        wr, _, ir = oracle.span_ref(Kp, sp_, 0.0, 0)
        assert ir == 0 and rel(host64(wl[p]), wr) <= TOL_SOLVE
        assert np.array_equal(idxl[p].cpu().numpy(), oracle.topk_ref(sp_, k))


def test_long_context_step_on_its_own_sketches():
    """The long-context step at full size: 16 layers 4096 x 4096, 36
    examples x 4096 tokens of Student-t(3) activations with NaN padding
    after each length; sketch -> Gram -> cone to KKT residual 1e-6 ->
    combine, each against the oracle on the GPU's own sketches, sampled
    sketch blocks against the explicit-gradient oracle."""
    cfg = workloads.CONFIGS["long"]
    n, m, T = cfg["n"], cfg["m"], cfg["T"]
    print("long step: drawing inputs", flush=True)
    layers, lens, ktot = workloads.sketch_inputs(cfg, DEV, nan_padding=True)
    S = api.sketch(layers, lens)
    K, s, t2 = api.gram(S[:n], S[n:])
    w, r2, it, kkt, info = api.project_cone(K, s, t2, 10000, cfg["kkt_tol"])
    u = api.combine(S[:n], w)
    torch.cuda.synchronize()
    print("long step: GPU done, checking", flush=True)
    Sg = host64(S)
    assert np.isfinite(Sg).all()
    lh = lens.cpu().numpy()
    padded = [int(i) for i in np.flatnonzero(lh < T)]
    rows = sorted({0, padded[0], n + m - 1})
    sub = [layers[0], layers[15]]
    ref = oracle.sketch_ref(layers_to_host(sub, rows), lh[rows])
    errs = block_errors(Sg[rows], ref, sub, range(len(rows)))
    assert errs.max() <= TOL_SKETCH_BF16, errs.max()
    K_ref, s_ref, t2_ref = oracle.gram_ref(Sg[:n], Sg[n:])
    Kh, sh = host64(K[0]), host64(s[0])
    assert rel(Kh, K_ref[0]) <= TOL_GRAM and rel(sh, s_ref[0]) <= TOL_GRAM
    assert int(info[0]) == 0 and float(kkt[0]) <= cfg["kkt_tol"]
    wh = host64(w[0])
    assert oracle.cone_kkt_residual(Kh, sh, wh) <= 2 * cfg["kkt_tol"]
    w_ref = oracle.nnls_active_set(Kh, sh)
    print(f"long step: cone {int(it[0])} steps, kkt {float(kkt[0]):.2e}, w err {rel(wh, w_ref):.2e}, "
          f"support {int((w_ref > 0).sum())} of {n}", flush=True)
    assert rel(wh, w_ref) <= TOL_SOLVE
    assert rel(host64(u), oracle.combine_ref(Sg[:n], w_ref)) <= TOL_SOLVE
    _, r2_ref = oracle.cone_ref(K_ref[0], s_ref[0], t2_ref[0])
    assert abs(float(r2[0]) - r2_ref) <= 1e-4 * t2_ref[0]
