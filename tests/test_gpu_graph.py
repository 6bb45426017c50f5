"""A projection step captured in a HIP graph and replayed.

The library enqueues kernels only (no memsets, allocations or host
synchronisations), so a whole step -- sketch, Gram, cone and combine on one
stream, span and top-k on a second one joined by events -- can be captured
once and replayed.  Every replay, with the program's own eager work and
synchronisations between replays, must reproduce the eager step bit for
bit (all reductions run in a fixed order).
"""
import pytest
import torch

from paper_2605_07063_amd import _lib, api, workloads

DEV = "cuda:0"


@pytest.mark.gpu
def test_graph_replay_of_a_projection_step_matches_eager():
    cfg = workloads.CONFIGS["small"]
    n, m, T = 16, 4, 256
    N = n + m
    layers, lens, ktot = workloads.sketch_inputs(cfg, DEV, layers=[0, 1], N=N, T=T)
    k_top = n // 2
    goff = [0, ktot]
    S = torch.empty(N, ktot, dtype=torch.float32, device=DEV)
    G, Gt = S[:n], S[n:]
    sk_ws = torch.empty(max(1, api.dr_sketch_workspace_size(layers, N, T, torch.bfloat16)), dtype=torch.uint8,
                        device=DEV)
    gr_ws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, goff, torch.float32)), dtype=torch.uint8,
                        device=DEV)
    sp_ws = torch.empty(max(1, api.dr_span_workspace_size(n, 1)), dtype=torch.uint8, device=DEV)
    cb_ws = torch.empty(max(1, api.dr_combine_workspace_size(n, goff)), dtype=torch.uint8, device=DEV)
    K = torch.empty(1, n, n, device=DEV)
    s = torch.empty(1, n, device=DEV)
    t2 = torch.empty(1, device=DEV)
    wc = torch.empty(1, n, device=DEV)
    r2c = torch.empty(1, device=DEV)
    itc = torch.empty(1, dtype=torch.int32, device=DEV)
    kktc = torch.empty(1, device=DEV)
    infoc = torch.empty(1, dtype=torch.int32, device=DEV)
    u = torch.empty(ktot, device=DEV)
    ws_ = torch.empty(1, n, device=DEV)
    le = torch.empty(1, device=DEV)
    r2s = torch.empty(1, device=DEV)
    infos = torch.empty(1, dtype=torch.int32, device=DEV)
    idx = torch.empty(1, k_top, dtype=torch.int32, device=DEV)
    wt = torch.empty(1, n, device=DEV)
    infot = torch.empty(1, dtype=torch.int32, device=DEV)
    side = torch.cuda.Stream()
    gram_done, side_done = torch.cuda.Event(), torch.cuda.Event()

    def step():
        cur = torch.cuda.current_stream()
        api.dr_sketch_grads(layers, N, T, lens, S, workspace=sk_ws)
        api.dr_gram(G, Gt, goff, K, s, t2, workspace=gr_ws)
        gram_done.record(cur)
        side.wait_event(gram_done)
        api.dr_project_cone(K, s, t2, 200, 0.0, wc, r2c, itc, kktc, infoc)
        api.dr_combine(G, goff, wc, u, workspace=cb_ws)
        api.dr_project_span(K, s, t2, 1e-3, _lib.DR_RIDGE_REL_TRACE, ws_, le, r2s, infos, workspace=sp_ws,
                            stream=side)
        api.dr_select_topk(s, k_top, idx, wt, infot, stream=side)
        side_done.record(side)
        cur.wait_event(side_done)

    outs = [S, K, s, t2, wc, r2c, itc, infoc, u, ws_, le, r2s, infos, idx, wt, infot]
    step()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    assert int(infoc[0]) == 0 and int(infos[0]) == 0 and int(infot[0]) == 0

    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=cap):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs:   # eager work between the replays
            o.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, ref):
            assert torch.equal(o, e), f"replay {rep} differs from the eager step"
