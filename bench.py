"""Benchmark of the hot path on one MI355X: one step = every stage of the
path over one batch of the small-block workload --
  sketch   : 8 linear layers 2048x2048, 64 general + 8 target examples,
             T = 512 with lengths U{128..512}, 64x64 Gaussian sketches (bf16)
  gram     : K = G G^T, scores s = G gbar, t2 = |gbar|^2 over 32768 columns
  cone     : NNLS by 200 projected-gradient steps
  span     : ridge solve (relative ridge 1e-3)
  top-k    : k = n/2 = 32
  combine  : u = G^T w for the cone weights
After the Gram, the cone and the combine run on the main stream while the
span and then the top-k run on a second stream.  Inputs are resident in HBM
before the timed region.
Prints one JSON line.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sketched per-example grads/sec + projection steps/sec; % of MFMA/HBM peak"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--groups", choices=["global", "layer"], default="global",
                    help="one group over all sketch columns (default), or one group per layer (P = 8)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle's sketch sample")
    ap.add_argument("--no-gram-dominated", action="store_true",
                    help="skip the Gram-dominated stage timings (16384 x 8192 Gram, span, top-1024)")
    ap.add_argument("--no-scale-configs", action="store_true",
                    help="skip the Llama-shaped block and long-context sketch timings")
    ap.add_argument("--gram-dominated-only", action="store_true",
                    help="time only the Gram-dominated stages and print their JSON object (for profiling)")
    ap.add_argument("--no-next-rows", action="store_true",
                    help="skip the separately timed widening rows (update, scorers, selection rules, simplex, "
                         "back-projection)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run three 1 GiB device-to-device copies first (known bytes, to scale HBM counters)")
    ap.add_argument("--summarize-gram-profile", metavar="KT_DIR",
                    help="write the Gram-dominated kernel-trace summary under profiles/ from rocprofv3 csv output")
    ap.add_argument("--summarize-profiles", nargs=3, metavar=("KT_DIR", "FETCH_DIR", "WRITE_DIR"),
                    help="write the profiles/ summaries from the csv output of a rocprofv3 kernel-trace run "
                         "and the FETCH_SIZE / WRITE_SIZE counter runs of this script (no GPU needed)")
    return ap.parse_args()


def main():
    args = parse()
    if args.summarize_profiles:
        summarize_profiles(*args.summarize_profiles)
        return
    if args.summarize_gram_profile:
        summarize_gram_profile(args.summarize_gram_profile)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: this build has no multi-GPU path "
              "(the per-GPU share is the single-GPU workload; see the design notes on sharding)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2605_07063_amd import _lib, api, workloads

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.gram_dominated_only:
        print(json.dumps(time_gram_dominated(api, _lib, workloads, dev)), flush=True)
        return
    cfg = workloads.CONFIGS["small"]
    n, m, T = cfg["n"], cfg["m"], cfg["T"]
    N = n + m
    layers, lens, ktot = workloads.sketch_inputs(cfg, dev)
    k_top = n // 2
    lam = 1e-3
    torch.cuda.synchronize()

    # every output and workspace allocated once, outside the timed region
    S = torch.empty(N, ktot, dtype=torch.float32, device=dev)
    sk_ws = torch.empty(max(1, api.dr_sketch_workspace_size(layers, N, T, torch.bfloat16)), dtype=torch.uint8,
                        device=dev)
    # groups: one over the concatenated sketch, or one per layer (layer-wise mode)
    goff = [0, ktot] if args.groups == "global" else [int(L["col_offset"]) for L in layers] + [ktot]
    P = len(goff) - 1
    K = torch.empty(P, n, n, device=dev)
    s = torch.empty(P, n, device=dev)
    t2 = torch.empty(P, device=dev)
    gr_ws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, goff, torch.float32)), dtype=torch.uint8, device=dev)
    wc = torch.empty(P, n, device=dev)
    r2c = torch.empty(P, device=dev)
    itc = torch.empty(P, dtype=torch.int32, device=dev)
    kktc = torch.empty(P, device=dev)
    infoc = torch.empty(P, dtype=torch.int32, device=dev)
    ws_ = torch.empty(P, n, device=dev)
    le = torch.empty(P, device=dev)
    r2s = torch.empty(P, device=dev)
    infos = torch.empty(P, dtype=torch.int32, device=dev)
    idx = torch.empty(P, k_top, dtype=torch.int32, device=dev)
    wt = torch.empty(P, n, device=dev)
    infot = torch.empty(P, dtype=torch.int32, device=dev)
    u = torch.empty(ktot, device=dev)
    cb_ws = torch.empty(max(1, api.dr_combine_workspace_size(n, goff)), dtype=torch.uint8, device=dev)

    G, Gt = S[:n], S[n:]
    stages = ["sketch", "gram", "cone", "combine", "span", "topk"]
    # the projections depend only on (K, s, t2): after the Gram the cone and
    # the combine run on the main stream while the span and then the top-k
    # run on a second one (both at the default priority)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    gram_done = torch.cuda.Event()
    side_done = torch.cuda.Event()

    def step(ev=None, marks=range(9)):
        def mark(i, stream):
            if ev is not None and i in marks:
                ev[i].record(stream)
        mark(0, main)
        api.dr_sketch_grads(layers, N, T, lens, S, workspace=sk_ws)
        mark(1, main)
        api.dr_gram(G, Gt, goff, K, s, t2, workspace=gr_ws)
        mark(2, main)
        gram_done.record(main)
        side.wait_event(gram_done)
        api.dr_project_cone(K, s, t2, cfg["iters"], 0.0, wc, r2c, itc, kktc, infoc, stream=main)
        mark(3, main)
        api.dr_combine(G, goff, wc, u, workspace=cb_ws, stream=main)
        mark(4, main)
        mark(5, side)
        api.dr_project_span(K, s, t2, lam, _lib.DR_RIDGE_REL_TRACE, ws_, le, r2s, infos, stream=side)
        mark(6, side)
        mark(7, side)
        api.dr_select_topk(s, k_top, idx, wt, infot, stream=side)
        mark(8, side)
        side_done.record(side)
        main.wait_event(side_done)

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # An event recorded between two kernels costs the stream about 4-5 us
    # here (a memory release for the host), so the timed steps carry the two
    # events around the sketch call (the roofline's live duration) on every
    # SAMPLE-th step only, and the per-stage breakdown comes from a second,
    # untimed run of the same number of steps with all nine marks.
    SAMPLE = 5
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(9)] for _ in range(args.steps)]
    sampled = [i for i in range(args.steps) if i % SAMPLE == 0]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i] if i % SAMPLE == 0 else None, marks=(0, 1))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    sketch_live_ms = float(np.mean([events[i][0].elapsed_time(events[i][1]) for i in sampled]))
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    spans = {"sketch": (0, 1), "gram": (1, 2), "cone": (2, 3), "combine": (3, 4), "span": (5, 6), "topk": (7, 8)}
    stage_ms = {nm: float(np.mean([events[i][a].elapsed_time(events[i][b]) for i in range(args.steps)]))
                for nm, (a, b) in spans.items()}
    stage_ms["sketch"] = sketch_live_ms
    # Gram end to the last projection's end (the three overlap)
    proj_wall = float(np.mean([max(events[i][2].elapsed_time(events[i][j]) for j in (4, 6, 8))
                               + events[i][1].elapsed_time(events[i][2]) for i in range(args.steps)]))
    if bool((infoc != 0).any()) or bool((infos != 0).any()) or bool((infot != 0).any()):
        raise RuntimeError("a projection reported a non-zero info code")

    # algorithmic bytes of one sketch call: valid tokens' x and dy rows, the
    # projectors and the fp32 sketch output
    lh = lens.cpu().numpy().astype(np.int64)
    es = 2
    alg_bytes = 0
    for L in layers:
        di, do = L["x"].shape[2], L["dy"].shape[2]
        alg_bytes += int(lh.sum()) * (di + do) * es
        alg_bytes += (L["p_in"].numel() + L["p_out"].numel()) * es
    alg_bytes += N * ktot * 4
    traffic = measured_traffic()
    sk_ms = stage_ms["sketch"]
    achieved = alg_bytes / (sk_ms * 1e-3) / 1e9
    proj_ms = proj_wall

    out = {
        "metric": METRIC,
        "value": N / (ms_per_step * 1e-3),
        "unit": "sketched per-example grads/s (each over all 8 layers, whole path per step)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "small-block: 8 linear layers 2048x2048, 64 general + 8 target examples, seq 512 with "
                        "lengths U{128..512}, 64x64 Gaussian sketches per layer (32768 columns), cone NNLS 200 "
                        "iterations + ridge span + top-32 + combine on the same Gram",
            "layers": 8, "d_in": 2048, "d_out": 2048, "n": n, "m": m, "seq_len": T, "sketch": "64x64",
            "valid_tokens": int(lh.sum()), "accumulate": "fp32", "solver_arithmetic": "fp64 on fp32 K",
            "groups": "one over all columns" if P == 1 else f"{P} (one per layer)",
        },
        "projection_steps_per_s": 1e3 / proj_ms,
        "projection_ms": proj_ms,
        "stages_ms": stage_ms,
        "roofline": {
            "kernel": "dr_sketch_grads (sketch_plan_kernel + sketch_packed_kernel + sketch_packed_reduce_kernel)",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes": alg_bytes,
            "avg_launch_ms": sk_ms,
            "timed_calls": len(sampled),
        },
    }

    if not args.no_next_rows:
        out["next_rows"] = time_next_rows(api, layers, lens, n, T, wt, wc, goff, dev, K=K, s=s)
    if not args.no_gram_dominated:
        out["gram_dominated"] = time_gram_dominated(api, _lib, workloads, dev)
    if not args.no_scale_configs:
        out.update(time_scale_configs(api, _lib, workloads, dev))

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(layers, lens, S, K, s, t2, n, m, k_top, lam, cfg, args.cpu_seconds, goff)
    print(json.dumps(out), flush=True)


def _event_ms(fn, reps):
    """GPU milliseconds per call of fn: a spin kernel keeps the stream busy
    while the host enqueues every call, so the two events bracket the calls'
    GPU execution and not the host's launch rate."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(100_000_000)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def time_next_rows(api, layers, lens, n, T, wt, wc, goff, dev, K=None, s=None, reps=20):
    """Stages after the path, timed on their own (not part of `value`): the
    update assembly in parameter space for the step's top-k weights (the
    paper's subset mean) and for its cone weights; the thresholding
    (negative score filtering) and greedy subset rules on the step's K, s."""
    import numpy as np
    import torch
    ul = [dict(x=L["x"], dy=L["dy"]) for L in layers]
    sizes = [L["dy"].shape[2] * L["x"].shape[2] for L in layers]
    offs = [int(v) for v in np.cumsum([0] + sizes[:-1])]
    U = torch.empty(sum(sizes), device=dev)
    P = wt.shape[0]
    gol = None if P == 1 else list(range(len(layers)))
    ws = torch.empty(max(1, api.dr_update_workspace_size(ul, n, T, torch.bfloat16)), dtype=torch.uint8, device=dev)
    lh = lens[:n].cpu().numpy().astype(np.int64)
    res = {}
    for name, w in (("update_topk", wt), ("update_cone", wc)):
        wh = w.cpu().numpy()
        flops = 0.0
        for li, L in enumerate(layers):
            row = 0 if P == 1 else li
            flops += 2.0 * float(lh[wh[row] != 0].sum()) * L["x"].shape[2] * L["dy"].shape[2]
        ms = _event_ms(lambda: api.dr_assemble_update(ul, n, T, lens, w, U, offs, group_of_layer=gol,
                                                       workspace=ws), reps)
        tf = flops / (ms * 1e-3) / 1e12
        res[name] = {"ms": ms, "examples": int((wh != 0).any(axis=0).sum()),
                     "roofline": {"kernel": "dr_assemble_update (update_plan_kernel + update_sort_kernel + "
                                            "update_bf16_kernel)",
                                  "bound": "mfma", "achieved": tf, "peak": BF16_MFMA_PEAK_TFLOPS,
                                  "unit": "TFLOP/s", "frac": tf / BF16_MFMA_PEAK_TFLOPS,
                                  "algorithmic_flops": flops}}
    if K is not None:
        P, nn = s.shape
        idx = torch.empty(P, nn, dtype=torch.int32, device=dev)
        cnt = torch.empty(P, dtype=torch.int32, device=dev)
        wq = torch.empty(P, nn, device=dev)
        info = torch.empty(P, dtype=torch.int32, device=dev)
        res["select_negative_filter_ms"] = _event_ms(
            lambda: api.dr_select_threshold(s, 0.0, True, idx, cnt, wq, info), reps)
        kk = nn // 2
        gidx = torch.empty(P, kk, dtype=torch.int32, device=dev)
        gws = torch.empty(max(1, api.dr_greedy_workspace_size(nn, P)), dtype=torch.uint8, device=dev)
        res["select_greedy_ms"] = _event_ms(lambda: api.dr_select_greedy(K, s, kk, gidx, wq, info, workspace=gws), reps)
    # exact per-layer scores of the 64 general rows against the 8 targets, by
    # the three contraction orders; algorithmic flops: the leading terms
    # (2 tokens d_in d_out for Direct / PIP, 4 sum_i sum_j len_i len_j (d_in
    # + d_out) / 2 for GIP's two cross-correlations)
    m = lens.shape[0] - n
    la = lens.cpu().numpy().astype(np.int64)
    sc = torch.empty(len(layers), n, device=dev)
    lead = {"direct": 0.0, "pip": 0.0, "gip": 0.0}
    for L in layers:
        di, do = L["x"].shape[2], L["dy"].shape[2]
        lead["direct"] += 2.0 * float(la.sum()) * di * do
        lead["pip"] += 2.0 * float(la.sum()) * di * do
        lead["gip"] += 2.0 * float(la[:n].sum()) * float(la[n:].sum()) * (di + do)
    scores = {}
    for meth in ("direct", "gip", "pip"):
        sws = torch.empty(max(1, api.dr_score_workspace_size(ul, n, m, T, meth)), dtype=torch.uint8, device=dev)
        ms = _event_ms(lambda: api.dr_score_exact(ul, n, m, T, lens, meth, sc, workspace=sws), max(3, reps // 4))
        scores[meth] = {"ms": ms, "algorithmic_tflops": lead[meth] / (ms * 1e-3) / 1e12}
    res["score_exact"] = scores
    if K is not None:
        # soft weighting over the simplex on the step's K, s (to a step residual of 1e-7)
        P, nn = s.shape
        t2 = torch.zeros(P, device=dev)
        wsx = torch.empty(P, nn, device=dev)
        r2 = torch.empty(P, device=dev)
        its = torch.empty(P, dtype=torch.int32, device=dev)
        rs = torch.empty(P, device=dev)
        inf = torch.empty(P, dtype=torch.int32, device=dev)
        res["simplex_ms"] = _event_ms(lambda: api.dr_project_simplex(K, s, t2, 5000, 1e-7, wsx, r2, its, rs, inf), reps)
        res["simplex_steps"] = its.cpu().tolist()
        # back-projection of a sketch-space vector to the 8 layers: writes
        # 8 x 2048 x 2048 fp32 (the HBM-bound part)
        u = torch.empty(int(layers[-1]["col_offset"]) + layers[-1]["p_in"].shape[0] * layers[-1]["p_out"].shape[0],
                        device=dev)
        bws = torch.empty(max(1, api.dr_backproject_workspace_size(layers)), dtype=torch.uint8, device=dev)
        u.normal_()
        ms = _event_ms(lambda: api.dr_back_project(layers, u, U, offs, workspace=bws), reps)
        wbytes = 4.0 * sum(sizes)
        res["back_project"] = {"ms": ms, "roofline": {"bound": "hbm", "achieved": wbytes / (ms * 1e-3) / 1e9,
                                                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                                      "frac": wbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                                      "algorithmic_bytes": wbytes}}
    return res


def time_gram_dominated(api, _lib, workloads, dev, reps=3):
    """The Gram-dominated workload's projection step, stage by stage: the
    16384 x 16384 Gram of 16384 bf16 rows of dimension 8192 (+ 32 target
    rows: scores and the target's squared norm), the ridge span at n = 16384
    (blocked Cholesky + refinement) and top-1024.  The Gram is the one stage
    of the path whose algorithmic work can reach the bf16 MFMA roofline:
    n (n + 1) / 2 entries of K and n scores, kappa MACs (2 FLOP) each."""
    import torch
    cfg = workloads.CONFIGS["gram"]
    rows = workloads.gram_rows(cfg, dev)
    n, kappa = cfg["n"], rows.shape[1]
    G, Gt = rows[:n], rows[n:]
    K = torch.empty(1, n, n, device=dev)
    s = torch.empty(1, n, device=dev)
    t2 = torch.empty(1, device=dev)
    gws = torch.empty(max(1, api.dr_gram_workspace_size(n, Gt.shape[0], [0, kappa], torch.bfloat16)),
                      dtype=torch.uint8, device=dev)
    w = torch.empty(1, n, device=dev)
    le = torch.empty(1, device=dev)
    r2 = torch.empty(1, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    sws = torch.empty(api.dr_span_workspace_size(n, 1), dtype=torch.uint8, device=dev)
    k = cfg["topk"]
    idx = torch.empty(1, k, dtype=torch.int32, device=dev)
    wt = torch.empty(1, n, device=dev)
    it = torch.empty(1, dtype=torch.int32, device=dev)
    gram_ms = _event_ms(lambda: api.dr_gram(G, Gt, [0, kappa], K, s, t2, workspace=gws), reps)
    span_ms = _event_ms(lambda: api.dr_project_span(K, s, t2, cfg["lam"], _lib.DR_RIDGE_REL_TRACE, w, le, r2, info,
                                                     workspace=sws), reps)
    topk_ms = _event_ms(lambda: api.dr_select_topk(s, k, idx, wt, it), 10 * reps)
    if int(info[0]) != 0 or int(it[0]) != 0:
        raise RuntimeError("Gram-dominated projection reported a non-zero info code")
    flops = float(n) * (n + 1) * kappa + 2.0 * n * kappa   # lower triangle of K, then the scores
    tf = flops / (gram_ms * 1e-3) / 1e12
    del K, sws, rows
    torch.cuda.empty_cache()
    return {
        "workload": "Gram-dominated: 16384 general + 32 target pre-sketched bf16 rows of dimension 8192 "
                    "(N(0,1) plus a rank-32 component of scale 3), ridge span lambda = 1e-2 relative, top-1024",
        "gram_ms": gram_ms, "span_ms": span_ms, "topk_ms": topk_ms,
        "projection_steps_per_s": 1e3 / (gram_ms + span_ms + topk_ms),
        "gram_roofline": {"kernel": "dr_gram (gram_big_kernel + target mean + scores)",
                          "bound": "mfma", "achieved": tf, "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                          "frac": tf / BF16_MFMA_PEAK_TFLOPS, "algorithmic_flops": flops},
        "span_fp32_factor_tflops": (n ** 3 / 3.0) / (span_ms * 1e-3) / 1e12,
    }


def _sketch_bytes(layers, lens, N, ktot):
    """Algorithmic bytes of one sketch call: the valid tokens' x and dy rows,
    the projectors and the fp32 sketch output."""
    tok = int(lens.sum())
    b = sum(tok * (L["x"].shape[2] + L["dy"].shape[2]) * L["x"].element_size()
            + (L["p_in"].numel() + L["p_out"].numel()) * L["p_in"].element_size() for L in layers)
    return b + N * ktot * 4


def time_scale_configs(api, _lib, workloads, dev, reps=3):
    """The two largest workloads, timed on their own (not part of `value`):
    * llama_block: one full Llama-3-8B-shaped block (q, k, v, o, gate, up,
      down; 256 + 16 examples x 1024 tokens, bf16, 32 x 32 sketches) -- the
      whole step streams 32 such blocks (46 GB each, 1.46 TB in all, more
      than the HBM holds), so the step's sketch time is 32 block calls; the
      Gram, span (lambda = 0) and top-64 run on a [272, 229376] fp32 sketch
      matrix of random N(0, 1) entries (their cost does not depend on the
      values);
    * long_context: the whole long-context workload (16 layers 4096 x 4096,
      32 + 4 examples x 4096 tokens, Student-t(3) activations, 30% of the
      examples padded), sketch, Gram and the cone to a KKT residual of 1e-6."""
    import torch
    res = {}
    # Llama-shaped block
    cfg = workloads.CONFIGS["llama"]
    n, m, T = cfg["n"], cfg["m"], cfg["T"]
    N = n + m
    layers, lens, kb = workloads.sketch_inputs(cfg, dev, layers=range(7))
    Sb = torch.empty(N, kb, device=dev)
    ws = torch.empty(max(1, api.dr_sketch_workspace_size(layers, N, T, torch.bfloat16)), dtype=torch.uint8, device=dev)
    ms = _event_ms(lambda: api.dr_sketch_grads(layers, N, T, lens, Sb, workspace=ws), reps)
    by = _sketch_bytes(layers, lens, N, kb)
    del layers, Sb, ws
    torch.cuda.empty_cache()
    ktot = 32 * kb
    S = torch.randn(N, ktot, device=dev)
    G, Gt = S[:n], S[n:]
    K = torch.empty(1, n, n, device=dev)
    sc = torch.empty(1, n, device=dev)
    t2 = torch.empty(1, device=dev)
    gws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, [0, ktot], torch.float32)), dtype=torch.uint8, device=dev)
    gram_ms = _event_ms(lambda: api.dr_gram(G, Gt, [0, ktot], K, sc, t2, workspace=gws), reps)
    w = torch.empty(1, n, device=dev)
    le = torch.empty(1, device=dev)
    r2 = torch.empty(1, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    span_ms = _event_ms(lambda: api.dr_project_span(K, sc, t2, 0.0, _lib.DR_RIDGE_ABS, w, le, r2, info), 10 * reps)
    idx = torch.empty(1, cfg["topk"], dtype=torch.int32, device=dev)
    wt = torch.empty(1, n, device=dev)
    it = torch.empty(1, dtype=torch.int32, device=dev)
    topk_ms = _event_ms(lambda: api.dr_select_topk(sc, cfg["topk"], idx, wt, it), 10 * reps)
    if int(info[0]) != 0 or int(it[0]) != 0:
        raise RuntimeError("Llama-shaped projection reported a non-zero info code")
    step_sketch_ms = 32 * ms
    res["llama_block"] = {
        "workload": "Llama-3-8B-shaped: one block of 7 maps (q 4096->4096, k/v 4096->1024, o 4096->4096, "
                    "gate/up 4096->14336, down 14336->4096), 256 + 16 examples x 1024 tokens, bf16 N(0, 0.02^2), "
                    "32x32 sketches; the step is 32 such blocks",
        "block_sketch_ms": ms,
        "sketch_roofline": {"bound": "hbm", "achieved": by / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": by / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": by},
        "step_sketch_ms": step_sketch_ms,
        "sketched_grads_per_s": N / (step_sketch_ms * 1e-3),
        "gram_ms": gram_ms, "span_ms": span_ms, "topk_ms": topk_ms,
        "projection_steps_per_s": 1e3 / (gram_ms + span_ms + topk_ms),
    }
    del S, G, Gt, K, gws
    torch.cuda.empty_cache()
    # long context
    cfg = workloads.CONFIGS["long"]
    n, m, T = cfg["n"], cfg["m"], cfg["T"]
    N = n + m
    layers, lens, ktot = workloads.sketch_inputs(cfg, dev)
    S = torch.empty(N, ktot, device=dev)
    ws = torch.empty(max(1, api.dr_sketch_workspace_size(layers, N, T, torch.bfloat16)), dtype=torch.uint8, device=dev)
    ms = _event_ms(lambda: api.dr_sketch_grads(layers, N, T, lens, S, workspace=ws), reps)
    by = _sketch_bytes(layers, lens, N, ktot)
    G, Gt = S[:n], S[n:]
    K = torch.empty(1, n, n, device=dev)
    sc = torch.empty(1, n, device=dev)
    t2 = torch.empty(1, device=dev)
    gws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, [0, ktot], torch.float32)), dtype=torch.uint8, device=dev)
    gram_ms = _event_ms(lambda: api.dr_gram(G, Gt, [0, ktot], K, sc, t2, workspace=gws), reps)
    w = torch.empty(1, n, device=dev)
    r2 = torch.empty(1, device=dev)
    its = torch.empty(1, dtype=torch.int32, device=dev)
    kkt = torch.empty(1, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    cone_ms = _event_ms(lambda: api.dr_project_cone(K, sc, t2, 10000, cfg["kkt_tol"], w, r2, its, kkt, info),
                        10 * reps)
    if int(info[0]) != 0:
        raise RuntimeError("long-context cone reported a non-zero info code")
    res["long_context"] = {
        "workload": "long-context: 16 layers 4096x4096, 32 + 4 examples x 4096 tokens, bf16 Student-t(3) "
                    "activations at unit variance, 30% of the examples padded to random lengths >= 256, 64x64 "
                    "sketches, cone to KKT 1e-6",
        "sketch_ms": ms, "valid_tokens": int(lens.sum()),
        "sketch_roofline": {"bound": "hbm", "achieved": by / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": by / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": by},
        "sketched_grads_per_s": N / (ms * 1e-3),
        "gram_ms": gram_ms, "cone_ms": cone_ms, "cone_steps": int(its[0]), "cone_kkt": float(kkt[0]),
        "projection_steps_per_s": 1e3 / (gram_ms + cone_ms),
    }
    del layers, S, G, Gt, K, ws, gws
    torch.cuda.empty_cache()
    return res


SKETCH_SOURCES = ["paper_2605_07063_amd/csrc/sketch.hip", "paper_2605_07063_amd/csrc/common.h"]
SKETCH_KERNELS = ("sketch_plan_kernel", "sketch_packed_kernel", "sketch_packed_reduce_kernel")
KT_CMD = ("rocprofv3 --kernel-trace --stats --output-format csv -d prof_out/kt -o small -- "
          "python -u bench.py --steps 50 --warmup 10 --no-cpu-baseline --no-scale-configs")
PMC_CMD = ("rocprofv3 --pmc {c} --output-format csv -d prof_out/{d} -o small -- "
           "python -u bench.py --steps 5 --warmup 2 --no-cpu-baseline --no-next-rows --no-gram-dominated "
           "--no-scale-configs --copy-calibration")
SUM_CMD = "python bench.py --summarize-profiles prof_out/kt prof_out/fetch prof_out/write"
GD_KT_CMD = ("rocprofv3 --kernel-trace --stats --output-format csv -d prof_out/gd -o gd -- "
             "python -u bench.py --gram-dominated-only")
GD_SUM_CMD = "python bench.py --summarize-gram-profile prof_out/gd"


def sketch_sources_sha():
    import hashlib
    h = hashlib.sha256()
    for rel in SKETCH_SOURCES:
        h.update(open(os.path.join(ROOT, rel), "rb").read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per sketch call from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE passes (scaled by a known-size copy), or None when the kernel
    sources have changed since those counters were taken."""
    path = os.path.join(ROOT, "profiles", "sketch_small_block_traffic.json")
    try:
        rec = json.load(open(path))
        sha = sketch_sources_sha()
    except (OSError, ValueError, KeyError):
        return None
    if sha != rec.get("sources_sha256"):
        return None
    return rec["traffic_bytes_per_call"]


def _short_name(name):
    import re
    n = re.sub(r"\(anonymous namespace\)::", "", name).replace("dr::", "")
    if n.startswith("void "):
        n = n[5:]
    return n.split("(")[0].strip()


def _kernel_rows(stats_csv):
    """Markdown rows (name, calls, avg / min / max us, share) of a rocprofv3
    kernel_stats.csv, and the average duration of each kernel."""
    import csv
    stats = list(csv.DictReader(open(stats_csv)))
    tot = sum(float(r["TotalDurationNs"]) for r in stats)
    rows, avg = [], {}
    for r in stats:
        nm = _short_name(r["Name"])
        if nm.startswith("Cijk_"):
            nm = "hipBLASLt GEMM " + nm[:24] + "..."
        ours = not r["Name"].startswith(("void at::", "at::", "__amd", "Cijk_"))
        avg[nm] = avg.get(nm, 0.0) + float(r["AverageNs"]) / 1e3
        rows.append(f"| `{nm}`{'' if ours else ' (input generation, untimed)'} | {int(r['Calls'])} | "
                    f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                    f"{float(r['MaxNs']) / 1e3:.2f} | {100 * float(r['TotalDurationNs']) / tot:.1f}% |")
    return rows, avg


def summarize_gram_profile(kt_dir):
    """profiles/gram_dominated_kernel_trace.md from the rocprofv3 kernel
    trace of `bench.py --gram-dominated-only`."""
    import glob
    f = sorted(glob.glob(os.path.join(kt_dir, "**", "*_kernel_stats.csv"), recursive=True))
    if not f:
        raise SystemExit(f"no kernel_stats.csv under {kt_dir}")
    rows, avg = _kernel_rows(f[0])
    gram = sum(v for k, v in avg.items() if k.startswith(("gram_big_kernel", "score_kernel", "target_mean_kernel")))
    kt = ["# Kernel trace: Gram-dominated workload (Gram, span, top-1024)", "",
          "Command (run from the repository root with `TMPDIR=/tmp`), summarised by", "",
          "```", GD_KT_CMD, GD_SUM_CMD, "```", "",
          "`bench.py --gram-dominated-only` times each stage once untimed and 3 times timed (top-k 30 times): "
          "4 `dr_gram` calls (16416 x 8192 bf16 rows) and 4 `dr_project_span` calls at n = 16384. "
          "Durations in microseconds. The span's kernels run on two streams (the diagonal-block chain "
          "overlaps the trailing updates), so their durations add up to more than the call's wall time.", "",
          "| Kernel | Calls | Avg (us) | Min | Max | Share |", "|---|---|---|---|---|---|"] + rows + [
          "", f"One `dr_gram` call = gram_big_kernel + target_mean_kernel + score_kernel = "
          f"**{gram:.1f} us** (average kernel durations)."]
    open(os.path.join(ROOT, "profiles", "gram_dominated_kernel_trace.md"), "w").write("\n".join(kt) + "\n")


def summarize_profiles(kt_dir, fetch_dir, write_dir):
    """profiles/ summaries (kernel trace, HBM traffic, the traffic record
    bench.py reads) from rocprofv3 csv output of this script's commands."""
    import csv
    import glob

    def one(pattern, d):
        f = sorted(glob.glob(os.path.join(d, "**", pattern), recursive=True))
        if not f:
            raise SystemExit(f"no {pattern} under {d}")
        return f[0]

    rows, avg = _kernel_rows(one("*_kernel_stats.csv", kt_dir))
    sk_avg = sum(v for k, v in avg.items() if k.startswith(SKETCH_KERNELS))
    kt = ["# Kernel trace: small-block workload, bench step", "",
          "Command (run from the repository root with `TMPDIR=/tmp`), summarised by", "",
          "```", KT_CMD, SUM_CMD, "```", "",
          "110 calls per kernel of the step = 10 warmup + 50 timed steps + 50 steps of the per-stage "
          "breakdown. The widening-row kernels (update "
          "assembly, exact scorers, subset rules, simplex, back-projection) and the Gram-dominated stages "
          "(gram_big_kernel, the blocked span's lg_* kernels, top-1024) run after the step in their own timed "
          "loops, with their own call counts. Durations in microseconds.", "",
          "| Kernel | Calls | Avg (us) | Min | Max | Share |", "|---|---|---|---|---|---|"] + rows + [
          "", f"The sketch call (`dr_sketch_grads`) = {' + '.join(SKETCH_KERNELS)} = **{sk_avg:.1f} us** per call "
          "(average kernel durations; bench.py's HIP-event time of the same call also spans the launch gaps)."]
    open(os.path.join(ROOT, "profiles", "small_block_kernel_trace.md"), "w").write("\n".join(kt) + "\n")

    def counters(d, cname):
        recs = list(csv.DictReader(open(one("*_counter_collection.csv", d))))
        per = {}
        for r in recs:
            if r["Counter_Name"] != cname:
                continue
            per.setdefault(_short_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
        return per

    fetch, write = counters(fetch_dir, "FETCH_SIZE"), counters(write_dir, "WRITE_SIZE")
    copy = "rocclr_copyBuffer"
    ck = [k for k in fetch if copy in k]
    # three 1 GiB copies: each reads and writes 1,048,576 KiB
    f_cal = max(fetch[ck[0]]) if ck else None
    w_cal = max(write[[k for k in write if copy in k][0]]) if ck else None
    ffac = 1048576.0 / f_cal if f_cal else 1.0
    wfac = 1048576.0 / w_cal if w_cal else 1.0
    lines, sk_bytes = [], 0.0
    for k in fetch:
        if copy in k or k.startswith(("at::", "void at::")):
            continue
        fa = sum(fetch[k]) / len(fetch[k])
        wa = sum(write.get(k, [0.0])) / max(1, len(write.get(k, [0.0])))
        lines.append(f"| `{k}` | {len(fetch[k])} | {fa:,.1f} | {fa * ffac * 1024 / 1e6:,.1f} MB | {wa:,.1f} | "
                     f"{wa * wfac * 1024 / 1e6:,.1f} MB |")
        if k.startswith(SKETCH_KERNELS):
            sk_bytes += (fa * ffac + wa * wfac) * 1024
    tr = ["# HBM traffic: small-block workload, bench step", "",
          "Two counter passes, each in its own run (from the repository root, `TMPDIR=/tmp`), summarised by the "
          "last command:", "", "```",
          PMC_CMD.format(c="FETCH_SIZE", d="fetch"), PMC_CMD.format(c="WRITE_SIZE", d="write"), SUM_CMD, "```", "",
          "Calibration: `--copy-calibration` makes three 1 GiB device-to-device copies (1,048,576 KiB read and "
          "written).",
          f"- FETCH_SIZE reads {f_cal:,.1f} KiB for such a copy: scale factor **{ffac:.4f}**." if f_cal else
          "- no copy kernel found: FETCH_SIZE unscaled.",
          f"- WRITE_SIZE reads {w_cal:,.1f} KiB: scale factor **{wfac:.4f}**." if w_cal else
          "- no copy kernel found: WRITE_SIZE unscaled.", "",
          "| Kernel | dispatches | FETCH_SIZE (KiB, raw avg) | fetched (scaled) | WRITE_SIZE (KiB avg) | "
          "written (scaled) |", "|---|---|---|---|---|---|"] + lines + [
          "", f"Sketch call total (plan + packed + reduce kernels): **{sk_bytes / 1e9:.4f} GB** of HBM traffic "
          "per call."]
    open(os.path.join(ROOT, "profiles", "small_block_hbm_traffic.md"), "w").write("\n".join(tr) + "\n")
    rec = {"kernel": "dr_sketch_grads", "workload": "small-block", "sources": SKETCH_SOURCES,
           "sources_sha256": sketch_sources_sha(), "traffic_bytes_per_call": sk_bytes,
           "fetch_factor": ffac, "write_factor": wfac}
    json.dump(rec, open(os.path.join(ROOT, "profiles", "sketch_small_block_traffic.json"), "w"), indent=1)
    print(f"sketch call {sk_avg:.1f} us, {sk_bytes / 1e9:.4f} GB per call")


def cpu_baseline(layers, lens, S, K, s, t2, n, m, k_top, lam, cfg, budget_s, goff):
    """The oracle, as it stands, on the host cores: explicit-gradient sketches
    on a bounded sample of (example, layer) blocks of the same inputs
    (extrapolated linearly to all 72 x 8 blocks), then Gram, cone, span,
    top-k and combine in full on the GPU's sketches."""
    import numpy as np
    import torch

    import oracle

    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threadpool_limits(cores)
        used = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        used = cores
    f64 = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
    N = n + m
    lh = lens.cpu().numpy()
    blocks = [(i, l) for i in range(N) for l in range(len(layers))]
    rng = np.random.default_rng(0)
    order = rng.permutation(len(blocks))
    host = {}
    done = 0
    t_sk = 0.0
    for bi in order:
        i, l = blocks[bi]
        L = layers[l]
        if l not in host:
            host[l] = (f64(L["p_in"]), f64(L["p_out"]))
        x = f64(L["x"][i])
        dy = f64(L["dy"][i])
        t0 = time.perf_counter()
        Gi = oracle.per_example_gradient(x, dy, lh[i])
        oracle.sketch_block(Gi, host[l][0], host[l][1])
        t_sk += time.perf_counter() - t0
        done += 1
        if t_sk >= budget_s:
            break
    t_sketch_full = t_sk * len(blocks) / done
    Sg = f64(S)
    t0 = time.perf_counter()
    Kr, sr, t2r = oracle.gram_ref(Sg[:n], Sg[n:], goff)
    t_gram = time.perf_counter() - t0
    t_cone = t_span = t_top = t_comb = 0.0
    for p in range(len(goff) - 1):
        t0 = time.perf_counter()
        wc = oracle.nnls_active_set(Kr[p], sr[p])
        t_cone += time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.span_ref(Kr[p], sr[p], lam, 1)
        t_span += time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.topk_ref(sr[p], k_top)
        t_top += time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.combine_ref(Sg[:n, goff[p]:goff[p + 1]], wc)
        t_comb += time.perf_counter() - t0
    t_step = t_sketch_full + t_gram + t_cone + t_span + t_top + t_comb
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {
        "value": N / t_step,
        "unit": "sketched per-example grads/s (each over all 8 layers, whole path per step)",
        "cores": used,
        "kind": "oracle",
        "sample": f"explicit-gradient sketches of {done} of the {len(blocks)} (example, layer) blocks "
                  f"({t_sk:.1f} s, extrapolated linearly); Gram, cone (exact active set), span, top-k and "
                  f"combine in full on the GPU's sketches ({t_step - t_sketch_full:.2f} s)",
        "cpu_model": cpu_model,
        "affinity_cores": cores,
        "seconds_per_step": t_step,
    }


if __name__ == "__main__":
    main()
