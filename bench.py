"""Benchmark of the hot path on one MI355X.

Headline (`value`): one step of the Llama-3-8B-shaped workload, the largest
configuration that runs on one GPU --
  sketch  : 32 blocks x 7 linear maps (q 4096->4096, k / v 4096->1024,
            o 4096->4096, gate / up 4096->14336, down 14336->4096), 256
            general + 16 target examples x 1024 tokens, bf16 N(0, 0.02^2)
            activations and output gradients, 32x32 Gaussian sketches per
            map (224 maps, 229376 columns); one dr_sketch_grads call per
            block (32 calls per step)
  gram    : K = G G^T (256 x 256), s = G gbar, t2 = |gbar|^2 over all
            229376 columns
  span    : Eq. (proj) onto the span of the 256 general sketches (lambda = 0)
  top-k   : k = 64 on the same scores
  combine : u = G^T w for the span weights
The step's retained pairs are 1.46 TB and do not fit in HBM together, so
two blocks' activations (45.6 GB each) are drawn and kept resident: block b
reads the activations of block b mod 2 with its own projectors and writes
its own column range.  Every call still streams a whole block from HBM.

Secondary objects (not `value`, each on its own inputs): the small-block
step, the Gram-dominated projection, the long-context step, the
layer-wise (group-wise) mode on the Llama step's own sketches, and the
widening rows after the path.  Every object carries the CPU oracle's time
on the same inputs (`cpu_baseline`, full or sampled and extrapolated, as
stated in its `sample`).

Prints one JSON line.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                       [--only llama|small|gram|long]
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
F32_MFMA_PEAK_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="budget of the oracle's explicit-gradient sketch sample of the headline workload")
    ap.add_argument("--only", choices=["llama", "small", "gram", "long"],
                    help="time one workload only and print its JSON object (profiling runs)")
    ap.add_argument("--no-secondary", action="store_true",
                    help="headline only: skip the small-block, Gram-dominated, long-context, layer-wise objects")
    ap.add_argument("--no-next-rows", action="store_true",
                    help="skip the widening rows (update, scorers, selection rules, simplex, back-projection)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run three 1 GiB device-to-device copies first (known bytes, to scale HBM counters)")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("NAME", "KT_DIR"),
                    help="write profiles/<NAME>_kernel_trace.md from a rocprofv3 kernel-trace csv directory")
    ap.add_argument("--summarize-traffic", nargs=3, metavar=("NAME", "FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/<NAME>_hbm_traffic.md (+ the traffic record bench.py reads) from the "
                         "FETCH_SIZE and WRITE_SIZE counter runs")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("NAME", "PMC_DIR"),
                    help="write profiles/<NAME>_counters.md from a rocprofv3 --pmc csv directory")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# timing helpers
# ---------------------------------------------------------------------------

def _event_ms(fn, reps, warm=0):
    """GPU milliseconds per call of fn.  By default a spin kernel keeps the
    stream busy while the host enqueues every call, so the two events bracket
    the calls' GPU execution and not the host's launch rate.  With warm > 0
    (calls of a millisecond and longer, whose launch rate never starves the
    GPU) warm untimed calls run right before the timed ones instead: the
    clock settles at its loaded level before the first event, as it is in a
    sequence of projection steps, where it takes several milliseconds to
    climb back after the GPU has idled (the spin kernel occupies one CU)."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if warm > 0:
        for _ in range(warm):
            fn()
    else:
        torch.cuda._sleep(100_000_000)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _host_cores():
    cores = len(os.sched_getaffinity(0))
    used = cores
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threadpool_limits(cores)
        used = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        pass
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return used, cores, model


def measured_peaks(dev):
    """Ceilings measured on this GPU by the probe library (libdrprobe.so):
    a plain streaming read of 8 GiB (every byte once), and MFMA issue
    loops on register operands in bf16 (16x16x32) and fp32 (16x16x4), the
    instruction shapes the library's kernels use."""
    import ctypes
    import torch
    from paper_2605_07063_amd import build as _build
    lib = ctypes.CDLL(_build.PROBE_LIB)
    lib.dr_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    lib.dr_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    cur = lambda: ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}
    nb = 8 << 30
    buf = torch.empty(nb, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    best = 0.0
    for blocks in (2048, 4096, 8192):
        sink = torch.empty(blocks, device=dev)
        ms = _event_ms(lambda: lib.dr_probe_read(buf.data_ptr(), nb, sink.data_ptr(), blocks, cur()), 5)
        best = max(best, nb / (ms * 1e-3) / 1e9)
    res["hbm_read_GBs"] = best
    del buf
    blocks, iters = 2048, 512
    sink = torch.empty(blocks * 256, device=dev)
    for name, bf, flop in (("bf16_mfma_TFLOPs", 1, 16384.0), ("fp32_mfma_TFLOPs", 0, 2048.0)):
        ms = _event_ms(lambda: lib.dr_probe_mfma(bf, iters, sink.data_ptr(), blocks, cur()), 5)
        res[name] = blocks * 4 * 8 * iters * flop / (ms * 1e-3) / 1e12
    torch.cuda.empty_cache()
    res["how"] = ("probe library: streaming read of 8 GiB (best of 2048 / 4096 / 8192 workgroups of 256 threads, "
                  "16-byte loads, four in flight per lane); MFMA loops of 8 independent accumulators per wave, "
                  "2048 workgroups of 4 waves, 512 iterations; 5 timed calls each after one untimed")
    return res


def _roofline(kernel, bound, work, ms, peak, unit, measured_peak=None, traffic=None, **extra):
    ach = work / (ms * 1e-3) / (1e9 if unit == "GB/s" else 1e12)
    r = {"kernel": kernel, "bound": bound, "achieved": ach, "peak": peak, "unit": unit, "frac": ach / peak}
    if measured_peak:
        r["measured_peak"] = measured_peak
        r["frac_of_measured"] = ach / measured_peak
    r["traffic"] = traffic
    r.update(extra)
    return r


def _gram_f32_flops(n, m, ktot):
    """Algorithmic flops of dr_gram over ktot columns: the lower triangle of
    K = G G^T with its diagonal, s = G gbar, t2 = |gbar|^2 and the target
    mean of m rows."""
    return (n * (n + 1) + 2 * n + 2 + m) * float(ktot)


def _sketch_bytes(layers, lens, N, ktot):
    """Algorithmic bytes of one sketch call: the valid tokens' x and dy rows,
    the projectors and the fp32 sketch output (its column range)."""
    tok = int(lens.sum())
    b = sum(tok * (L["x"].shape[2] + L["dy"].shape[2]) * L["x"].element_size()
            + (L["p_in"].numel() + L["p_out"].numel()) * L["p_in"].element_size() for L in layers)
    return b + N * ktot * 4


# ---------------------------------------------------------------------------
# the headline: the Llama-3-8B-shaped step
# ---------------------------------------------------------------------------

def run_llama(args, api, _lib, workloads, dev, peaks):
    import numpy as np
    import torch
    cfg = workloads.CONFIGS["llama"]
    n, m, T, k_top = cfg["n"], cfg["m"], cfg["T"], cfg["topk"]
    N = n + m
    blocks, lens, ktot = workloads.llama_step_inputs(cfg, dev, buffers=2)
    nb = len(blocks)
    S = torch.empty(N, ktot, dtype=torch.float32, device=dev)
    sk_ws = torch.empty(max(1, api.dr_sketch_workspace_size(blocks[0], N, T, torch.bfloat16)), dtype=torch.uint8,
                        device=dev)
    goff = [0, ktot]
    K = torch.empty(1, n, n, device=dev)
    s = torch.empty(1, n, device=dev)
    t2 = torch.empty(1, device=dev)
    gr_ws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, goff, torch.float32)), dtype=torch.uint8, device=dev)
    w = torch.empty(1, n, device=dev)
    le = torch.empty(1, device=dev)
    r2 = torch.empty(1, device=dev)
    info = torch.empty(1, dtype=torch.int32, device=dev)
    sp_ws = torch.empty(max(1, api.dr_span_workspace_size(n, 1)), dtype=torch.uint8, device=dev)
    idx = torch.empty(1, k_top, dtype=torch.int32, device=dev)
    wt = torch.empty(1, n, device=dev)
    infot = torch.empty(1, dtype=torch.int32, device=dev)
    u = torch.empty(ktot, device=dev)
    cb_ws = torch.empty(max(1, api.dr_combine_workspace_size(n, goff)), dtype=torch.uint8, device=dev)
    G, Gt = S[:n], S[n:]
    torch.cuda.synchronize()

    # events: two around every block's sketch call, then the ends of the
    # gram / span / top-k / combine calls
    NE = 2 * nb + 4

    def step(ev=None):
        for b in range(nb):
            if ev is not None:
                ev[2 * b].record()
            api.dr_sketch_grads(blocks[b], N, T, lens, S, workspace=sk_ws)
            if ev is not None:
                ev[2 * b + 1].record()
        api.dr_gram(G, Gt, goff, K, s, t2, workspace=gr_ws)
        if ev is not None:
            ev[2 * nb].record()
        api.dr_project_span(K, s, t2, cfg["lam"], _lib.DR_RIDGE_ABS, w, le, r2, info, workspace=sp_ws)
        if ev is not None:
            ev[2 * nb + 1].record()
        api.dr_select_topk(s, k_top, idx, wt, infot)
        if ev is not None:
            ev[2 * nb + 2].record()
        api.dr_combine(G, goff, w, u, workspace=cb_ws)
        if ev is not None:
            ev[2 * nb + 3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(NE)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    if int(info[0]) != 0 or int(infot[0]) != 0:
        raise RuntimeError(f"Llama-shaped projection reported info {int(info[0])} / {int(infot[0])}")
    blk_ms = np.array([[ev[2 * b].elapsed_time(ev[2 * b + 1]) for b in range(nb)] for ev in events])
    stage = {
        "sketch_32_blocks": float(np.mean([ev[0].elapsed_time(ev[2 * nb - 1]) for ev in events])),
        "gram": float(np.mean([ev[2 * nb - 1].elapsed_time(ev[2 * nb]) for ev in events])),
        "span": float(np.mean([ev[2 * nb].elapsed_time(ev[2 * nb + 1]) for ev in events])),
        "topk": float(np.mean([ev[2 * nb + 1].elapsed_time(ev[2 * nb + 2]) for ev in events])),
        "combine": float(np.mean([ev[2 * nb + 2].elapsed_time(ev[2 * nb + 3]) for ev in events])),
    }
    proj_ms = stage["gram"] + stage["span"] + stage["topk"] + stage["combine"]
    by = _sketch_bytes(blocks[0], lens, N, 7 * cfg["k_in"] * cfg["k_out"])
    avg_blk = float(blk_ms.mean())
    traffic = measured_traffic("llama_block")
    res = {
        "ms_per_step": ms_per_step,
        "sketched_grads_per_s": N / (ms_per_step * 1e-3),
        "projection_steps_per_s": 1e3 / proj_ms,
        "projection_ms": proj_ms,
        "stages_ms": stage,
        "block_sketch_ms": {"mean": avg_blk, "min": float(blk_ms.min()), "max": float(blk_ms.max())},
        "roofline": _roofline(
            "dr_sketch_grads, one block of 7 maps (sketch_plan_kernel + sketch_packed_kernel + "
            "sketch_packed_reduce_kernel)", "hbm", by, avg_blk, HBM_PEAK_GBS, "GB/s",
            measured_peak=peaks.get("hbm_read_GBs") if peaks else None, traffic=traffic,
            algorithmic_bytes=by, avg_launch_ms=avg_blk, timed_calls=int(blk_ms.size)),
        # fp32 rows, (n(n+1) + 2n + 2 + m) kappa flops on 4 (n + m) kappa bytes:
        # about 61 flops per byte, above the fp32 MFMA ridge (157.3 / 8), so
        # the Gram is priced against the fp32 MFMA peak
        "gram_roofline": _roofline("dr_gram (fp32 rows: gram_tile_lds_kernel + reduce + target mean)", "mfma",
                                   _gram_f32_flops(n, m, ktot), stage["gram"], F32_MFMA_PEAK_TFLOPS, "TFLOP/s",
                                   measured_peak=peaks.get("fp32_mfma_TFLOPs") if peaks else None,
                                   algorithmic_flops=_gram_f32_flops(n, m, ktot), algorithmic_bytes=N * ktot * 4.0),
        "span_info": int(info[0]),
    }
    return res, dict(blocks=blocks, lens=lens, S=S, K=K, s=s, t2=t2, w=w, idx=idx, u=u, n=n, m=m, k_top=k_top,
                     goff=goff, ktot=ktot)


def run_layerwise(api, _lib, st, dev):
    """Layer-wise (group-wise) mode on the Llama step's own sketches: one
    group per linear map (224 groups of 1024 columns), batched Gram, span
    (lambda = 0) and top-64 in every group."""
    import torch
    S, n, m, ktot = st["S"], st["n"], st["m"], st["ktot"]
    width = 1024
    P = ktot // width
    goff = [p * width for p in range(P + 1)]
    G, Gt = S[:n], S[n:]
    K = torch.empty(P, n, n, device=dev)
    s = torch.empty(P, n, device=dev)
    t2 = torch.empty(P, device=dev)
    gws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, goff, torch.float32)), dtype=torch.uint8, device=dev)
    w = torch.empty(P, n, device=dev)
    le = torch.empty(P, device=dev)
    r2 = torch.empty(P, device=dev)
    info = torch.empty(P, dtype=torch.int32, device=dev)
    sws = torch.empty(max(1, api.dr_span_workspace_size(n, P)), dtype=torch.uint8, device=dev)
    idx = torch.empty(P, st["k_top"], dtype=torch.int32, device=dev)
    wt = torch.empty(P, n, device=dev)
    it = torch.empty(P, dtype=torch.int32, device=dev)
    gram_ms = _event_ms(lambda: api.dr_gram(G, Gt, goff, K, s, t2, workspace=gws), 10)
    span_ms = _event_ms(lambda: api.dr_project_span(K, s, t2, 0.0, _lib.DR_RIDGE_ABS, w, le, r2, info,
                                                     workspace=sws), 10)
    topk_ms = _event_ms(lambda: api.dr_select_topk(s, st["k_top"], idx, wt, it), 50)
    bad = int((info != 0).sum()) + int((it != 0).sum())
    kb = P * n * n * 4.0 + 2 * P * n * 4.0   # K read once, s read and w written
    return {
        "workload": "layer-wise groups on the Llama-shaped step's sketches: 224 groups (one per linear map) of "
                    "1024 columns, n = 256 general + 16 target rows; batched Gram, span (lambda = 0) and top-64 "
                    "in every group",
        "groups": P, "gram_ms": gram_ms, "span_ms": span_ms, "topk_ms": topk_ms,
        "projection_steps_per_s": 1e3 / (gram_ms + span_ms + topk_ms),
        "nonzero_info_groups": bad,
        "span_roofline": _roofline("dr_project_span, 224 groups at n = 256 (span_small_kernel, one workgroup per "
                                   "group)", "hbm", kb, span_ms, HBM_PEAK_GBS, "GB/s", algorithmic_bytes=kb),
        "gram_roofline": _roofline("dr_gram, 224 groups (fp32 rows)", "mfma", _gram_f32_flops(n, m, ktot), gram_ms,
                                   F32_MFMA_PEAK_TFLOPS, "TFLOP/s", algorithmic_flops=_gram_f32_flops(n, m, ktot),
                                   algorithmic_bytes=(st["n"] + st["m"]) * ktot * 4.0),
    }


def cpu_baseline_llama(st, cfg, budget_s):
    """The oracle on the headline step: explicit-gradient sketches of a
    sample of (example, map) blocks of blocks 0 and 31 -- 8 examples x 7
    maps x 2 blocks, visited example by example until the time budget is
    used (every map at least once) -- extrapolated per map to all 272
    examples x 32 blocks; then the Gram, the span (lambda = 0), top-64 and
    the combine in full on the GPU's sketches.  Each sampled block is also
    compared with the GPU's sketch of it."""
    import numpy as np
    import oracle
    used, cores, model = _host_cores()
    f64 = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
    blocks, lens, S = st["blocks"], st["lens"], st["S"]
    n, m, k_top = st["n"], st["m"], st["k_top"]
    N = n + m
    nb = len(blocks)
    lh = lens.cpu().numpy()
    kk = cfg["k_in"] * cfg["k_out"]
    examples = [0, 37, 101, 160, 222, 255, 256, 271]
    times = {j: [] for j in range(7)}
    errs = []
    t_sk = 0.0
    done = 0
    proj = {}
    visited = []
    for i in examples:
        if t_sk >= budget_s and all(times[q] for q in range(7)):
            break
        visited.append(i)
        for b in (0, nb - 1):
            for j in range(7):
                if t_sk >= budget_s and all(times[q] for q in range(7)):
                    break
                L = blocks[b][j]
                if (b, j) not in proj:
                    proj[(b, j)] = (f64(L["p_in"]), f64(L["p_out"]))
                x, dy = f64(L["x"][i]), f64(L["dy"][i])
                t0 = time.perf_counter()
                Gi = oracle.per_example_gradient(x, dy, lh[i])
                blk = oracle.sketch_block(Gi, *proj[(b, j)])
                dt = time.perf_counter() - t0
                t_sk += dt
                times[j].append(dt)
                done += 1
                o = int(L["col_offset"])
                g = f64(S[i, o:o + kk])
                errs.append(float(np.linalg.norm(g - blk.ravel()) / np.linalg.norm(blk)))
    t_sketch_full = sum(float(np.mean(times[j])) for j in range(7)) * N * nb
    Sg = f64(S)
    t0 = time.perf_counter()
    Kr, sr, t2r = oracle.gram_ref(Sg[:n], Sg[n:])
    t_gram = time.perf_counter() - t0
    t0 = time.perf_counter()
    wr, _, _ = oracle.span_ref(Kr[0], sr[0], 0.0, 0)
    t_span = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.topk_ref(sr[0], k_top)
    t_top = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.combine_ref(Sg[:n], wr)
    t_comb = time.perf_counter() - t0
    t_proj = t_gram + t_span + t_top + t_comb
    t_step = t_sketch_full + t_proj
    return {
        "value": N / t_step,
        "unit": "sketched per-example grads/s (each over all 224 linear maps, whole path per step)",
        "cores": used, "kind": "oracle",
        "sample": f"explicit-gradient sketches of {done} (example, map) blocks from blocks 0 and {nb - 1} "
                  f"(examples {visited}, {t_sk:.1f} s), extrapolated per map to "
                  f"{N} examples x {nb} blocks ({t_sketch_full:.0f} s); Gram, span, top-{k_top} and combine in "
                  f"full on the GPU's sketches ({t_proj:.2f} s)",
        "extrapolated": True,
        "seconds_per_step": t_step,
        "projection_steps_per_s": 1.0 / t_proj,
        "sampled_blocks_max_rel_err_vs_gpu": max(errs) if errs else None,
        "cpu_model": model, "affinity_cores": cores,
    }


# ---------------------------------------------------------------------------
# secondary workloads
# ---------------------------------------------------------------------------

def run_small(args, api, _lib, workloads, dev, peaks, with_cpu, with_next):
    """The small-block step: sketch (8 layers 2048 x 2048, 64 + 8 examples,
    T = 512 ragged) -> Gram -> cone (200 steps) and combine on the main
    stream, span (relative ridge 1e-3) and top-32 on a second stream."""
    import numpy as np
    import torch
    cfg = workloads.CONFIGS["small"]
    n, m, T = cfg["n"], cfg["m"], cfg["T"]
    N = n + m
    layers, lens, ktot = workloads.sketch_inputs(cfg, dev)
    k_top = n // 2
    lam = 1e-3
    S = torch.empty(N, ktot, dtype=torch.float32, device=dev)
    sk_ws = torch.empty(max(1, api.dr_sketch_workspace_size(layers, N, T, torch.bfloat16)), dtype=torch.uint8,
                        device=dev)
    goff = [0, ktot]
    K = torch.empty(1, n, n, device=dev)
    s = torch.empty(1, n, device=dev)
    t2 = torch.empty(1, device=dev)
    gr_ws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, goff, torch.float32)), dtype=torch.uint8, device=dev)
    wc = torch.empty(1, n, device=dev)
    r2c = torch.empty(1, device=dev)
    itc = torch.empty(1, dtype=torch.int32, device=dev)
    kktc = torch.empty(1, device=dev)
    infoc = torch.empty(1, dtype=torch.int32, device=dev)
    ws_ = torch.empty(1, n, device=dev)
    le = torch.empty(1, device=dev)
    r2s = torch.empty(1, device=dev)
    infos = torch.empty(1, dtype=torch.int32, device=dev)
    idx = torch.empty(1, k_top, dtype=torch.int32, device=dev)
    wt = torch.empty(1, n, device=dev)
    infot = torch.empty(1, dtype=torch.int32, device=dev)
    u = torch.empty(ktot, device=dev)
    cb_ws = torch.empty(max(1, api.dr_combine_workspace_size(n, goff)), dtype=torch.uint8, device=dev)
    G, Gt = S[:n], S[n:]
    side = torch.cuda.Stream()
    gram_done = torch.cuda.Event()
    side_done = torch.cuda.Event()
    sp_ws = torch.empty(max(1, api.dr_span_workspace_size(n, 1)), dtype=torch.uint8, device=dev)

    def step(ev=None):
        main = torch.cuda.current_stream()   # the capture stream when a graph records the step

        def mark(i, stream):
            if ev is not None:
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
        api.dr_project_span(K, s, t2, lam, _lib.DR_RIDGE_REL_TRACE, ws_, le, r2s, infos, workspace=sp_ws,
                            stream=side)
        mark(6, side)
        api.dr_select_topk(s, k_top, idx, wt, infot, stream=side)
        mark(7, side)
        side_done.record(side)
        main.wait_event(side_done)

    steps = max(args.steps, 50)
    for _ in range(max(args.warmup, 10)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms_eager = (time.perf_counter() - t0) * 1e3 / steps
    # The step captured once in a HIP graph and replayed: the same kernels
    # with the host's launch cost taken out (the eager step enqueues about ten
    # kernels, four events and two stream joins, which a slow host cannot
    # always keep ahead of 0.4 ms of GPU work).  Falls back to the eager rate.
    ms_graph, graph_note = None, None
    try:
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(graph, stream=cap):
            step()
        torch.cuda.synchronize()
        for _ in range(5):
            graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            graph.replay()
        torch.cuda.synchronize()
        ms_graph = (time.perf_counter() - t0) * 1e3 / steps
    except Exception as exc:   # noqa: BLE001 (report and keep the eager rate)
        graph_note = f"graph capture failed ({type(exc).__name__}: {exc}); eager rate reported"
        torch.cuda.synchronize()
    ms_per_step = ms_graph if ms_graph is not None else ms_eager
    # per-stage breakdown from a second run of the same steps with events
    # (an event between two kernels costs this stream about 4-5 us)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(steps)]
    for i in range(steps):
        step(events[i])
    torch.cuda.synchronize()
    if bool((infoc != 0).any()) or bool((infos != 0).any()) or bool((infot != 0).any()):
        raise RuntimeError("a small-block projection reported a non-zero info code")
    spans = {"sketch": (0, 1), "gram": (1, 2), "cone": (2, 3), "combine": (3, 4), "span": (5, 6), "topk": (6, 7)}
    stage_ms = {k: float(np.mean([e[a].elapsed_time(e[b]) for e in events])) for k, (a, b) in spans.items()}
    proj_ms = float(np.mean([e[1].elapsed_time(e[2]) + max(e[2].elapsed_time(e[4]), e[2].elapsed_time(e[7]))
                             for e in events]))
    by = _sketch_bytes(layers, lens, N, ktot)
    res = {
        "workload": "small-block: 8 linear layers 2048x2048, 64 general + 8 target examples, seq 512 with lengths "
                    "U{128..512}, 64x64 Gaussian sketches per layer (32768 columns), cone NNLS 200 iterations + "
                    "ridge span + top-32 + combine on the same Gram",
        "ms_per_step": ms_per_step, "sketched_grads_per_s": N / (ms_per_step * 1e-3),
        "timing": ("HIP graph replay of the whole step" if ms_graph is not None else graph_note),
        "ms_per_step_eager": ms_eager,
        "projection_steps_per_s": 1e3 / proj_ms, "projection_ms": proj_ms, "stages_ms": stage_ms,
        "valid_tokens": int(lens.sum()),
        "roofline": _roofline("dr_sketch_grads (sketch_plan_kernel + sketch_packed_kernel + "
                              "sketch_packed_reduce_kernel)", "hbm", by, stage_ms["sketch"], HBM_PEAK_GBS, "GB/s",
                              measured_peak=peaks.get("hbm_read_GBs") if peaks else None,
                              traffic=measured_traffic("small_block"), algorithmic_bytes=by,
                              avg_launch_ms=stage_ms["sketch"], timed_calls=steps),
    }
    if with_next:
        res["next_rows"] = time_next_rows(api, layers, lens, n, T, wt, wc, goff, dev, K=K, s=s)
    if with_cpu:
        res["cpu_baseline"] = cpu_baseline_small(layers, lens, S, K, s, t2, n, m, k_top, lam, 8.0, goff)
    del layers, S
    torch.cuda.empty_cache()
    return res


def cpu_baseline_small(layers, lens, S, K, s, t2, n, m, k_top, lam, budget_s, goff):
    """The oracle on the small-block step: explicit-gradient sketches of a
    random sample of (example, layer) blocks until the budget is used
    (extrapolated linearly to all 72 x 8 blocks), then Gram, the exact
    cone, span, top-k and combine in full on the GPU's sketches."""
    import numpy as np
    import oracle
    used, cores, model = _host_cores()
    f64 = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
    N = n + m
    lh = lens.cpu().numpy()
    blocks = [(i, l) for i in range(N) for l in range(len(layers))]
    order = np.random.default_rng(0).permutation(len(blocks))
    host = {}
    done = 0
    t_sk = 0.0
    for bi in order:
        i, l = blocks[bi]
        L = layers[l]
        if l not in host:
            host[l] = (f64(L["p_in"]), f64(L["p_out"]))
        x, dy = f64(L["x"][i]), f64(L["dy"][i])
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
    t0 = time.perf_counter()
    wc = oracle.nnls_active_set(Kr[0], sr[0])
    oracle.span_ref(Kr[0], sr[0], lam, 1)
    oracle.topk_ref(sr[0], k_top)
    oracle.combine_ref(Sg[:n], wc)
    t_proj = time.perf_counter() - t0 + t_gram
    t_step = t_sketch_full + t_proj
    return {
        "value": N / t_step,
        "unit": "sketched per-example grads/s (each over all 8 layers, whole path per step)",
        "cores": used, "kind": "oracle",
        "sample": f"explicit-gradient sketches of {done} of the {len(blocks)} (example, layer) blocks "
                  f"({t_sk:.1f} s){', extrapolated linearly' if done < len(blocks) else ', all of them'}; Gram, "
                  f"cone (exact active set), span, top-k and combine in full on the GPU's sketches "
                  f"({t_proj:.2f} s)",
        "extrapolated": done < len(blocks),
        "seconds_per_step": t_step, "projection_steps_per_s": 1.0 / t_proj,
        "cpu_model": model, "affinity_cores": cores,
    }


def run_gram_dominated(api, _lib, workloads, dev, peaks, with_cpu, reps=10, warm=5):
    """The Gram-dominated projection step, stage by stage: the 16384 x 16384
    Gram of 16384 bf16 rows of dimension 8192 (+ 32 target rows: scores and
    the target's squared norm), the ridge span at n = 16384 (blocked
    Cholesky + refinement) and top-1024.  The Gram is the one stage of the
    path whose algorithmic work can reach the bf16 MFMA roofline: n (n + 1)
    / 2 entries of K and n scores, kappa MACs (2 FLOP) each."""
    import numpy as np
    import torch
    cfg = workloads.CONFIGS["gram"]
    rows = workloads.gram_rows(cfg, dev)
    n, kappa, k = cfg["n"], rows.shape[1], cfg["topk"]
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
    idx = torch.empty(1, k, dtype=torch.int32, device=dev)
    wt = torch.empty(1, n, device=dev)
    it = torch.empty(1, dtype=torch.int32, device=dev)
    gram_ms = _event_ms(lambda: api.dr_gram(G, Gt, [0, kappa], K, s, t2, workspace=gws), reps, warm)
    span_ms = _event_ms(lambda: api.dr_project_span(K, s, t2, cfg["lam"], _lib.DR_RIDGE_REL_TRACE, w, le, r2, info,
                                                     workspace=sws), reps, warm)
    topk_ms = _event_ms(lambda: api.dr_select_topk(s, k, idx, wt, it), 10 * reps)
    if int(info[0]) != 0 or int(it[0]) != 0:
        raise RuntimeError(f"Gram-dominated projection reported info {int(info[0])} / {int(it[0])}")
    flops = float(n) * (n + 1) * kappa + 2.0 * n * kappa   # lower triangle of K, then the scores
    res = {
        "workload": "Gram-dominated: 16384 general + 32 target pre-sketched bf16 rows of dimension 8192 "
                    "(N(0,1) plus a rank-32 component of scale 3), ridge span lambda = 1e-2 relative, top-1024",
        "gram_ms": gram_ms, "span_ms": span_ms, "topk_ms": topk_ms,
        "projection_steps_per_s": 1e3 / (gram_ms + span_ms + topk_ms),
        "gram_roofline": _roofline("dr_gram (gram_big_kernel + target mean + scores)", "mfma", flops, gram_ms,
                                   BF16_MFMA_PEAK_TFLOPS, "TFLOP/s",
                                   measured_peak=peaks.get("bf16_mfma_TFLOPs") if peaks else None,
                                   algorithmic_flops=flops),
        "span_roofline": _roofline("dr_project_span at n = 16384 (blocked Cholesky + 2 refinement steps), n^3/3 "
                                   "factor flops", "mfma", n ** 3 / 3.0, span_ms, F32_MFMA_PEAK_TFLOPS, "TFLOP/s",
                                   measured_peak=peaks.get("fp32_mfma_TFLOPs") if peaks else None,
                                   algorithmic_flops=n ** 3 / 3.0),
        "lam_eff": float(le[0]),
    }
    if with_cpu:
        used, cores, model = _host_cores()
        import oracle
        Rh = rows.float().cpu().numpy().astype(np.float64)
        t0 = time.perf_counter()
        Kr, sr, t2r = oracle.gram_ref(Rh[:n], Rh[n:])
        t_gram = time.perf_counter() - t0
        del Rh
        t0 = time.perf_counter()
        wr, ler, infr = oracle.span_ref(Kr[0], sr[0], cfg["lam"], 1)
        t_span = time.perf_counter() - t0
        t0 = time.perf_counter()
        oracle.topk_ref(sr[0], k)
        t_top = time.perf_counter() - t0
        tot = t_gram + t_span + t_top
        res["cpu_baseline"] = {
            "value": 1.0 / tot, "unit": "projection steps/s (Gram + span + top-1024)", "cores": used,
            "kind": "oracle", "extrapolated": False,
            "sample": f"the whole step from the same bf16 rows: Gram {t_gram:.1f} s, span (fp64 Cholesky) "
                      f"{t_span:.1f} s, top-k {t_top:.3f} s",
            "seconds_per_step": tot,
            "w_rel_err_vs_gpu_end_to_end": float(np.linalg.norm(w[0].cpu().numpy() - wr) / np.linalg.norm(wr)),
            "cpu_model": model, "affinity_cores": cores,
        }
        del Kr
    del K, sws, rows
    torch.cuda.empty_cache()
    return res


def run_long(api, _lib, workloads, dev, peaks, with_cpu, reps=3):
    """The long-context step: sketch (16 layers 4096 x 4096, 32 + 4 examples
    x 4096 tokens, Student-t(3) activations, 30 % of the examples padded),
    Gram and the cone to a KKT residual of 1e-6."""
    import numpy as np
    import torch
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
    gws = torch.empty(max(1, api.dr_gram_workspace_size(n, m, [0, ktot], torch.float32)), dtype=torch.uint8,
                      device=dev)
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
    step_ms = ms + gram_ms + cone_ms
    res = {
        "workload": "long-context: 16 layers 4096x4096, 32 + 4 examples x 4096 tokens, bf16 Student-t(3) "
                    "activations at unit variance, 30% of the examples padded to random lengths >= 256, 64x64 "
                    "sketches, cone to KKT 1e-6",
        "sketch_ms": ms, "valid_tokens": int(lens.sum()), "step_ms": step_ms,
        "sketched_grads_per_s": N / (step_ms * 1e-3),
        "roofline": _roofline("dr_sketch_grads, 16 layers", "hbm", by, ms, HBM_PEAK_GBS, "GB/s",
                              measured_peak=peaks.get("hbm_read_GBs") if peaks else None, algorithmic_bytes=by),
        "gram_ms": gram_ms, "cone_ms": cone_ms, "cone_steps": int(its[0]), "cone_kkt": float(kkt[0]),
        "projection_steps_per_s": 1e3 / (gram_ms + cone_ms),
    }
    if with_cpu:
        import oracle
        used, cores, model = _host_cores()
        f64 = lambda t: t.detach().float().cpu().numpy().astype(np.float64)
        lh = lens.cpu().numpy()
        padded = [int(i) for i in np.flatnonzero(lh < T)]
        rows = [0, padded[0] if padded else 1, 17, N - 1]
        t_sk, tok = 0.0, 0
        errs = []
        kk = cfg["k_in"] * cfg["k_out"]
        for l in (0, len(layers) - 1):
            L = layers[l]
            pin, pout = f64(L["p_in"]), f64(L["p_out"])
            for i in rows:
                x, dy = f64(L["x"][i]), f64(L["dy"][i])
                t0 = time.perf_counter()
                blk = oracle.sketch_block(oracle.per_example_gradient(x, dy, lh[i]), pin, pout)
                t_sk += time.perf_counter() - t0
                tok += int(lh[i])
                o = int(L["col_offset"])
                g = f64(S[i, o:o + kk])
                errs.append(float(np.linalg.norm(g - blk.ravel()) / np.linalg.norm(blk)))
        t_full = t_sk / tok * float(lh.sum()) * len(layers)
        Sg = f64(S)
        t0 = time.perf_counter()
        Kr, sr, _ = oracle.gram_ref(Sg[:n], Sg[n:])
        wr = oracle.nnls_active_set(Kr[0], sr[0])
        t_proj = time.perf_counter() - t0
        tot = t_full + t_proj
        res["cpu_baseline"] = {
            "value": N / tot, "unit": "sketched per-example grads/s (each over all 16 layers, whole path per step)",
            "cores": used, "kind": "oracle", "extrapolated": True,
            "sample": f"explicit-gradient sketches of examples {rows} x layers {{0, 15}} ({t_sk:.1f} s for {tok} "
                      f"valid tokens), extrapolated per valid token to all 36 examples x 16 layers "
                      f"({t_full:.0f} s); Gram and the exact cone in full on the GPU's sketches ({t_proj:.2f} s)",
            "seconds_per_step": tot,
            "sampled_blocks_max_rel_err_vs_gpu": max(errs),
            "cpu_model": model, "affinity_cores": cores,
        }
    del layers, S, G, Gt, K, ws, gws
    torch.cuda.empty_cache()
    return res


def time_next_rows(api, layers, lens, n, T, wt, wc, goff, dev, K=None, s=None, reps=20):
    """Stages after the path, timed on their own: the update assembly in
    parameter space for the step's top-k weights (the paper's subset mean)
    and for its cone weights; the thresholding (negative score filtering)
    and greedy subset rules on the step's K, s; the three exact scorers;
    the simplex soft weighting; the back-projection."""
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
        res[name] = {"ms": ms, "examples": int((wh != 0).any(axis=0).sum()),
                     "roofline": _roofline("dr_assemble_update (update_plan_kernel + update_sort_kernel + "
                                           "update_bf16_kernel)", "mfma", flops, ms, BF16_MFMA_PEAK_TFLOPS,
                                           "TFLOP/s", algorithmic_flops=flops)}
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
        P, nn = s.shape
        t2 = torch.zeros(P, device=dev)
        wsx = torch.empty(P, nn, device=dev)
        r2 = torch.empty(P, device=dev)
        its = torch.empty(P, dtype=torch.int32, device=dev)
        rs = torch.empty(P, device=dev)
        inf = torch.empty(P, dtype=torch.int32, device=dev)
        res["simplex_ms"] = _event_ms(lambda: api.dr_project_simplex(K, s, t2, 5000, 1e-7, wsx, r2, its, rs, inf), reps)
        res["simplex_steps"] = its.cpu().tolist()
        u = torch.empty(int(layers[-1]["col_offset"]) + layers[-1]["p_in"].shape[0] * layers[-1]["p_out"].shape[0],
                        device=dev)
        bws = torch.empty(max(1, api.dr_backproject_workspace_size(layers)), dtype=torch.uint8, device=dev)
        u.normal_()
        ms = _event_ms(lambda: api.dr_back_project(layers, u, U, offs, workspace=bws), reps)
        wbytes = 4.0 * sum(sizes)
        res["back_project"] = {"ms": ms, "roofline": _roofline("dr_back_project (bp_left_kernel + bp_mfma_kernel)",
                                                               "hbm", wbytes, ms, HBM_PEAK_GBS, "GB/s",
                                                               algorithmic_bytes=wbytes)}
    return res


# ---------------------------------------------------------------------------
# main
# ---------------------------------------------------------------------------

def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic)
        return
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the per-GPU share is the single-GPU workload; see the design notes on sharding)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2605_07063_amd import _lib, api, workloads

    dev = "cuda:0"
    torch.cuda.set_device(0)
    print(f"bench: start (steps {args.steps}, warmup {args.warmup})", file=sys.stderr, flush=True)
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    with_cpu = not args.no_cpu_baseline
    if args.only == "small":
        print(json.dumps(run_small(args, api, _lib, workloads, dev, {}, with_cpu, not args.no_next_rows)), flush=True)
        return
    if args.only == "gram":
        print(json.dumps(run_gram_dominated(api, _lib, workloads, dev, {}, with_cpu)), flush=True)
        return
    if args.only == "long":
        print(json.dumps(run_long(api, _lib, workloads, dev, {}, with_cpu)), flush=True)
        return
    peaks = measured_peaks(dev) if args.only is None else {}
    print("bench: headline (Llama-3-8B-shaped step)", file=sys.stderr, flush=True)
    cfg = workloads.CONFIGS["llama"]
    head, st = run_llama(args, api, _lib, workloads, dev, peaks)
    N = st["n"] + st["m"]
    out = {
        "metric": METRIC,
        "value": head["sketched_grads_per_s"],
        "unit": "sketched per-example grads/s (each over all 224 linear maps, whole path per step)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "llama3-8b-shaped step: 32 blocks x {q 4096->4096, k/v 4096->1024, o 4096->4096, "
                        "gate/up 4096->14336, down 14336->4096}, 256 general + 16 target examples x seq 1024, "
                        "bf16 N(0, 0.02^2), 32x32 Gaussian sketches per map (229376 columns) in 32 block calls; "
                        "Gram over all columns, span projection (lambda = 0), top-64 and combine on the same Gram; "
                        "two blocks' activations (45.6 GB each) resident in HBM, block b reads those of block b mod "
                        "2 with its own projectors",
            "blocks": 32, "maps_per_block": 7, "n": st["n"], "m": st["m"], "seq_len": cfg["T"], "sketch": "32x32",
            "columns": st["ktot"], "resident_activation_blocks": 2, "bytes_per_block_call": head["roofline"][
                "algorithmic_bytes"], "accumulate": "fp32", "solver_arithmetic": "fp32 factor + fp64 refinement",
            "groups": "one over all columns",
        },
        "projection_steps_per_s": head["projection_steps_per_s"],
        "projection_ms": head["projection_ms"],
        "stages_ms": head["stages_ms"],
        "block_sketch_ms": head["block_sketch_ms"],
        "roofline": head["roofline"],
        "gram_roofline": head["gram_roofline"],
        "measured_peaks": peaks,
    }
    if args.only is None and not args.no_secondary:
        print("bench: layer-wise groups on the step's sketches", file=sys.stderr, flush=True)
        out["layerwise"] = run_layerwise(api, _lib, st, dev)
    if with_cpu:
        print("bench: oracle on the headline step", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline_llama(st, cfg, args.cpu_seconds)
    del st, head
    torch.cuda.empty_cache()
    if args.only is None and not args.no_secondary:
        # the Gram-dominated step first: its large-n span overlaps work on two
        # auxiliary streams created by its first call, and after the small
        # block's HIP graph capture and replays in this process that overlap
        # measured 8% lower (17.3 against 16.0 ms, the rate it has alone)
        print("bench: Gram-dominated", file=sys.stderr, flush=True)
        out["gram_dominated"] = run_gram_dominated(api, _lib, workloads, dev, peaks, with_cpu)
        print("bench: small block", file=sys.stderr, flush=True)
        out["small_block"] = run_small(args, api, _lib, workloads, dev, peaks, with_cpu, not args.no_next_rows)
        print("bench: long context", file=sys.stderr, flush=True)
        out["long_context"] = run_long(api, _lib, workloads, dev, peaks, with_cpu)
    print(json.dumps(out), flush=True)


# ---------------------------------------------------------------------------
# profile summaries (no GPU needed)
# ---------------------------------------------------------------------------

SKETCH_SOURCES = ["paper_2605_07063_amd/csrc/sketch.hip", "paper_2605_07063_amd/csrc/common.h"]
SKETCH_KERNELS = ("sketch_plan_kernel", "sketch_packed_kernel", "sketch_packed_reduce_kernel")

# the commands behind each committed summary (run from the repository root
# with TMPDIR=/tmp; rocprofv3 writes csv files under prof_out/)
_SEL = "--kernel-include-regex 'dr::|copyBuffer'"
MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES "
                 "GRBM_GUI_ACTIVE")
TRACE_CMDS = {
    "llama_step": "rocprofv3 --kernel-trace --stats --output-format csv -d prof_out/llama_kt -o run -- "
                  "python -u bench.py --only llama --steps 5 --warmup 2 --no-cpu-baseline",
    "small_block": "rocprofv3 --kernel-trace --stats --output-format csv -d prof_out/small_kt -o run -- "
                   "python -u bench.py --only small --no-cpu-baseline",
    "gram_dominated": "rocprofv3 --kernel-trace --stats --output-format csv -d prof_out/gram_kt -o run -- "
                      "python -u bench.py --only gram --no-cpu-baseline",
}
TRAFFIC_CMDS = {
    "llama_block": f"rocprofv3 --pmc {{c}} {_SEL} --output-format csv -d prof_out/llama_{{d}} -o run -- "
                   "python -u bench.py --only llama --steps 1 --warmup 0 --no-cpu-baseline --copy-calibration",
    "small_block": f"rocprofv3 --pmc {{c}} {_SEL} --output-format csv -d prof_out/small_{{d}} -o run -- "
                   "python -u bench.py --only small --steps 1 --warmup 1 --no-cpu-baseline --no-next-rows "
                   "--copy-calibration",
    "gram_dominated": f"rocprofv3 --pmc {{c}} {_SEL} --output-format csv -d prof_out/gram_{{d}} -o run -- "
                      "python -u bench.py --only gram --no-cpu-baseline --copy-calibration",
}
COUNTER_CMDS = {
    "llama_block": f"rocprofv3 --pmc {MFMA_COUNTERS} {_SEL} --output-format csv -d prof_out/llama_mfma -o run -- "
                   "python -u bench.py --only llama --steps 1 --warmup 0 --no-cpu-baseline",
    "small_block": f"rocprofv3 --pmc {MFMA_COUNTERS} {_SEL} --output-format csv -d prof_out/small_mfma -o run -- "
                   "python -u bench.py --only small --steps 1 --warmup 1 --no-cpu-baseline",
    "gram_dominated": f"rocprofv3 --pmc {MFMA_COUNTERS} {_SEL} --output-format csv -d prof_out/gram_mfma -o run -- "
                      "python -u bench.py --only gram --no-cpu-baseline",
}


def sketch_sources_sha():
    import hashlib
    h = hashlib.sha256()
    for rel in SKETCH_SOURCES:
        h.update(open(os.path.join(ROOT, rel), "rb").read())
    return h.hexdigest()


def measured_traffic(name):
    """HBM bytes per sketch call of a workload from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE passes (scaled by a known-size copy), or None
    when the sketch sources have changed since those counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{name}_traffic.json")
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


def _find(pattern, d):
    import glob
    f = sorted(glob.glob(os.path.join(d, "**", pattern), recursive=True))
    if not f:
        raise SystemExit(f"no {pattern} under {d}")
    return f[0]


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
        rows.append(f"| `{nm}`{'' if ours else ' (input generation / library, untimed)'} | {int(r['Calls'])} | "
                    f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                    f"{float(r['MaxNs']) / 1e3:.2f} | {100 * float(r['TotalDurationNs']) / tot:.1f}% |")
    return rows, avg


def summarize_trace(name, kt_dir):
    rows, avg = _kernel_rows(_find("*_kernel_stats.csv", kt_dir))
    sk = sum(v for k, v in avg.items() if k.startswith(SKETCH_KERNELS))
    cmd = TRACE_CMDS[name]
    lines = [f"# Kernel trace: {name.replace('_', ' ')}", "",
             "Command (from the repository root, `TMPDIR=/tmp`), then "
             f"`python bench.py --summarize-trace {name} {cmd.split(' -d ')[1].split()[0]}`:", "",
             "```", cmd, "```", "",
             "Durations in microseconds (average, min, max over the calls).", "",
             "| Kernel | Calls | Avg (us) | Min | Max | Share |", "|---|---|---|---|---|---|"] + rows
    if sk > 0:
        lines += ["", f"One sketch call = {' + '.join(SKETCH_KERNELS)} = **{sk:.1f} us** (sum of the average "
                      "kernel durations; kernels a call does not launch count zero)."]
    open(os.path.join(ROOT, "profiles", f"{name}_kernel_trace.md"), "w").write("\n".join(lines) + "\n")
    print(f"{name}: sketch call {sk:.1f} us")


def _counters(d, cname):
    import csv
    per = {}
    for r in csv.DictReader(open(_find("*_counter_collection.csv", d))):
        if r["Counter_Name"] != cname:
            continue
        per.setdefault(_short_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    return per


def summarize_traffic(name, fetch_dir, write_dir):
    fetch, write = _counters(fetch_dir, "FETCH_SIZE"), _counters(write_dir, "WRITE_SIZE")
    copy = "rocclr_copyBuffer"
    ck = [k for k in fetch if copy in k]
    f_cal = max(fetch[ck[0]]) if ck else None
    wk = [k for k in write if copy in k]
    w_cal = max(write[wk[0]]) if wk else None
    ffac = 1048576.0 / f_cal if f_cal else 1.0
    wfac = 1048576.0 / w_cal if w_cal else 1.0
    lines, per_kernel, sk_bytes = [], {}, 0.0
    for k in fetch:
        if copy in k or k.startswith(("at::", "void at::", "Cijk_")):
            continue
        fa = sum(fetch[k]) / len(fetch[k])
        wa = sum(write.get(k, [0.0])) / max(1, len(write.get(k, [0.0])))
        b = (fa * ffac + wa * wfac) * 1024
        per_kernel[k] = b
        lines.append(f"| `{k}` | {len(fetch[k])} | {fa:,.1f} | {fa * ffac * 1024 / 1e6:,.1f} MB | {wa:,.1f} | "
                     f"{wa * wfac * 1024 / 1e6:,.1f} MB |")
        if k.startswith(SKETCH_KERNELS):
            sk_bytes += b
    cmd = TRAFFIC_CMDS[name]
    tr = [f"# HBM traffic: {name.replace('_', ' ')}", "",
          "Two counter passes, each in its own run (from the repository root, `TMPDIR=/tmp`), summarised by "
          f"`python bench.py --summarize-traffic {name} <fetch dir> <write dir>`:", "", "```",
          cmd.format(c="FETCH_SIZE", d="fetch"), cmd.format(c="WRITE_SIZE", d="write"), "```", "",
          "Calibration: `--copy-calibration` makes three 1 GiB device-to-device copies (1,048,576 KiB read and "
          "written).",
          f"- FETCH_SIZE reads {f_cal:,.1f} KiB for such a copy: scale factor **{ffac:.4f}**." if f_cal else
          "- no copy kernel found: FETCH_SIZE unscaled.",
          f"- WRITE_SIZE reads {w_cal:,.1f} KiB: scale factor **{wfac:.4f}**." if w_cal else
          "- no copy kernel found: WRITE_SIZE unscaled.", "",
          "| Kernel | dispatches | FETCH_SIZE (KiB, raw avg) | fetched (scaled) | WRITE_SIZE (KiB avg) | "
          "written (scaled) |", "|---|---|---|---|---|---|"] + lines
    if sk_bytes > 0:
        tr += ["", f"Sketch call total (plan + packed + reduce kernels): **{sk_bytes / 1e9:.4f} GB** of HBM "
                   "traffic per call."]
    open(os.path.join(ROOT, "profiles", f"{name}_hbm_traffic.md"), "w").write("\n".join(tr) + "\n")
    rec = {"workload": name, "sources": SKETCH_SOURCES, "sources_sha256": sketch_sources_sha(),
           "traffic_bytes_per_call": sk_bytes if sk_bytes > 0 else None, "per_kernel_bytes": per_kernel,
           "fetch_factor": ffac, "write_factor": wfac}
    json.dump(rec, open(os.path.join(ROOT, "profiles", f"{name}_traffic.json"), "w"), indent=1)
    print(f"{name}: sketch call {sk_bytes / 1e9:.4f} GB")


XCDS, SIMDS = 8, 1024          # MI355X: 8 XCDs, 256 CUs x 4 SIMDs
MFMA_FLOP_PER_CLK = {"SQ_INSTS_VALU_MFMA_MOPS_BF16": 1024.0, "SQ_INSTS_VALU_MFMA_MOPS_F32": 64.0}   # per SIMD


def summarize_counters(name, pmc_dir):
    """Per-kernel averages of the MFMA counters of a rocprofv3 --pmc run and
    what they imply:
    - clock = GRBM_GUI_ACTIVE / 8 XCDs / the dispatch's duration (its start
      and end stamps; counter runs serialise the dispatches);
    - executed TFLOP/s = SQ_INSTS_VALU_MFMA_MOPS_* x 512 flops / duration;
    - MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8);
    - executed / dense peak at that clock (bf16 1024 and fp32 64 flops per
      SIMD per clock: 2.5 PFLOP/s and 157.3 TFLOP/s at 2.4 GHz)."""
    import csv
    import glob
    per, dur = {}, {}
    for f in sorted(glob.glob(os.path.join(pmc_dir, "**", "*_counter_collection.csv"), recursive=True)):
        for r in csv.DictReader(open(f)):
            k = _short_name(r["Kernel_Name"])
            if k.startswith(("at::", "void at::", "Cijk_")) or "rocclr" in k:
                continue
            per.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            dur.setdefault(k, {})[r["Dispatch_Id"]] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    avg = lambda v: sum(v) / len(v)
    cmd = COUNTER_CMDS[name]
    lines = [f"# MFMA counters: {name.replace('_', ' ')}", "",
             "Command (from the repository root, `TMPDIR=/tmp`), then "
             f"`python bench.py --summarize-counters {name} {cmd.split(' -d ')[1].split()[0]}`:", "",
             "```", cmd, "```", "",
             "Per-kernel averages per dispatch (counter runs serialise the dispatches). Clock = GRBM_GUI_ACTIVE / 8 "
             "XCDs / duration. Executed = SQ_INSTS_VALU_MFMA_MOPS_BF16 and _F32 x 512 flops / duration. MFMA busy "
             "= SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8). Of peak at clock = executed / "
             "(1024 SIMDs x 1024 bf16 or 64 fp32 flops per clock x clock). The clock is meaningful for dispatches of "
             "about 100 us and longer only: GRBM_GUI_ACTIVE also counts the dispatch's start-up and drain.", "",
             "| Kernel | dispatches | avg duration (us) | clock (GHz) | MOPS_BF16 | MOPS_F32 | executed TFLOP/s | "
             "MFMA busy | of peak at clock |", "|---|---|---|---|---|---|---|---|---|"]
    for k, cs in per.items():
        nd = len(dur[k])
        d_s = avg(list(dur[k].values())) * 1e-9
        g = avg(cs.get("GRBM_GUI_ACTIVE", [0.0])) / XCDS
        clk = g / d_s / 1e9 if d_s > 0 else 0.0
        mb = avg(cs.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", [0.0]))
        mf = avg(cs.get("SQ_INSTS_VALU_MFMA_MOPS_F32", [0.0]))
        tf = (mb + mf) * 512 / d_s / 1e12 if d_s > 0 else 0.0
        busy = avg(cs.get("SQ_VALU_MFMA_BUSY_CYCLES", [0.0])) / (SIMDS * g) if g > 0 else 0.0
        # peak at this clock for the kernel's dominant MFMA type
        kind = "SQ_INSTS_VALU_MFMA_MOPS_BF16" if mb >= mf else "SQ_INSTS_VALU_MFMA_MOPS_F32"
        pk = SIMDS * MFMA_FLOP_PER_CLK[kind] * clk * 1e9 / 1e12
        of = tf / pk if (mb + mf) > 0 and pk > 0 else 0.0
        lines.append(f"| `{k}` | {nd} | {d_s * 1e6:,.1f} | {clk:.2f} | {mb:,.4g} | {mf:,.4g} | {tf:,.1f} | "
                     f"{busy:.3f} | {of:.3f} |")
    open(os.path.join(ROOT, "profiles", f"{name}_counters.md"), "w").write("\n".join(lines) + "\n")
    print(f"{name}: {len(per)} kernels")


if __name__ == "__main__":
    main()
