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
