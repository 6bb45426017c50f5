"""GPU parity of dr_assemble_update against the oracle's explicit gradients.

Tolerance: the inputs are bf16 or fp32 and every product is exact in fp32,
so the only error is fp32 accumulation over the valid tokens of the
weighted examples (about sqrt(tokens) * 2^-24 relative for random signs:
< 3e-5 for 10^6 tokens).  Each layer block must match the float64 oracle to
a relative Frobenius error of 1e-4 -- tighter than the 2e-3 allowed for bf16
sketches -- and no NaN from padding, from zero-weight rows or from the
target rows may reach it.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2605_07063_amd import api, workloads
from gpu_helpers import host64, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL_UPDATE = 1e-4


def make_layers(specs, N, T, dtype, lens, seed, nan_rows=()):
    """specs: list of (d_in, d_out); NaN in padding and in the given rows."""
    g = torch.Generator(device=DEV)
    g.manual_seed(4321 + seed)
    mask = torch.arange(T, device=DEV)[None, :] >= lens[:, None]
    out = []
    for di, do in specs:
        x = torch.randn(N, T, di, generator=g, device=DEV).to(dtype)
        dy = torch.randn(N, T, do, generator=g, device=DEV).to(dtype)
        x[mask] = float("nan")
        dy[mask] = float("nan")
        for r in nan_rows:
            x[r] = float("nan")
            dy[r] = float("nan")
        out.append(dict(x=x, dy=dy))
    return out


def check(layers, w, n, lens, group_of_layer=None, rows=None, cols=None):
    """Compare every layer block (or its rows x cols sample) with the oracle."""
    U = api.assemble_update(layers, w, n=n, lengths=lens, group_of_layer=group_of_layer)
    torch.cuda.synchronize()
    lens_h = None if lens is None else lens[:n].cpu().numpy()
    w_h = host64(w.reshape(-1, w.shape[-1]))
    errs = []
    for li, (L, Ul) in enumerate(zip(layers, U)):
        x, dy = L["x"][:n], L["dy"][:n]
        if cols is not None:
            x = x[:, :, cols]
        if rows is not None:
            dy = dy[:, :, rows]
        hl = [dict(x=host64(x), dy=host64(dy))]
        gl = None if group_of_layer is None else [group_of_layer[li]]
        (ref,) = oracle.update_ref(hl, w_h, lens_h, group_of_layer=gl)
        got = Ul
        if rows is not None:
            got = got[rows]
        if cols is not None:
            got = got[:, cols]
        got = host64(got)
        assert np.isfinite(got).all(), f"layer {li}: non-finite values leaked"
        if np.linalg.norm(ref) == 0.0:
            assert np.all(got == 0.0), f"layer {li}: expected an all-zero block"
            errs.append(0.0)
        else:
            errs.append(rel(got, ref))
    errs = np.array(errs)
    assert errs.max() <= TOL_UPDATE, f"max layer error {errs.max():.3e} > {TOL_UPDATE}"
    return U, errs


def mixed_weights(n, seed, zero_rows=()):
    g = torch.Generator(device=DEV)
    g.manual_seed(99 + seed)
    w = torch.randn(n, generator=g, device=DEV)
    w[1:4] = 0.25                      # a run of equal weights (one flush)
    for r in zero_rows:
        w[r] = 0.0
    return w


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_ragged_tiles_tokens_and_weights(dtype):
    n, m, T = 13, 3, 100                # token tails of 32-token (bf16) and 16-token (f32) steps
    lens = torch.tensor([0, 1, 31, 32, 33, 64, 100, 99, 47, 5, 100, 2, 70, 100, 100, 100],
                        dtype=torch.int32, device=DEV)
    specs = [(136, 264), (200, 72), (64, 64)] if dtype == torch.bfloat16 else [(100, 72), (36, 132)]
    layers = make_layers(specs, n + m, T, dtype, lens, seed=1, nan_rows=(6, 13, 14, 15))
    w = mixed_weights(n, 1, zero_rows=(6, 9))
    _, errs = check(layers, w, n, lens)
    print(f"{dtype} ragged max layer rel err {errs.max():.2e}")


def test_groups_and_more_than_sixteen_layers():
    n, T = 20, 70
    lens = torch.randint(0, T + 1, (n,), dtype=torch.int32, device=DEV)
    specs = [(64, 128), (128, 64), (72, 136)] * 6          # 18 layers: two launches
    layers = make_layers(specs, n, T, torch.bfloat16, lens, seed=2)
    g = torch.Generator(device=DEV)
    g.manual_seed(7)
    w = torch.randn(3, n, generator=g, device=DEV)
    w[1, ::3] = 0.0
    w[2] = 0.0
    w[2, 5] = 2.0                                            # one example only
    gol = [i % 3 for i in range(len(specs))]
    check(layers, w, n, lens, group_of_layer=gol)


def test_topk_weights_are_the_subset_mean():
    n, T = 48, 96
    lens = torch.randint(1, T + 1, (n,), dtype=torch.int32, device=DEV)
    layers = make_layers([(256, 512), (512, 256)], n, T, torch.bfloat16, lens, seed=3)
    s = torch.randn(1, n, device=DEV)
    idx, w, info = api.select_topk(s, 12)
    assert int(info[0]) == 0
    U, _ = check(layers, w[0], n, lens)
    # the same update from the explicit subset with unit weights, scaled by 1/k
    sel = torch.zeros(n, device=DEV)
    sel[idx[0].long()] = 1.0
    U1 = api.assemble_update(layers, sel, n=n, lengths=lens)
    for a, b in zip(U, U1):
        assert rel(host64(a), host64(b) / 12.0) <= 1e-6


def test_split_path_and_f32_tiny_config():
    # one bf16 tile: the example list is split over many workgroups, then reduced
    n, T = 40, 50
    lens = torch.randint(0, T + 1, (n,), dtype=torch.int32, device=DEV)
    layers = make_layers([(64, 64)], n, T, torch.bfloat16, lens, seed=4)
    check(layers, mixed_weights(n, 4), n, lens)
    cfg = workloads.CONFIGS["tiny"]
    tl, tlens, _ = workloads.sketch_inputs(cfg, DEV)
    w = mixed_weights(cfg["n"], 5, zero_rows=(0,))
    check([dict(x=L["x"], dy=L["dy"]) for L in tl], w, cfg["n"], tlens)


def test_empty_and_degenerate_cases():
    n, T = 6, 40
    lens = torch.tensor([0, 40, 3, 0, 17, 40], dtype=torch.int32, device=DEV)
    layers = make_layers([(128, 256)], n, T, torch.bfloat16, lens, seed=6, nan_rows=(1, 2, 4, 5))
    zero = torch.zeros(n, device=DEV)
    w = torch.tensor([3.0, 0.0, 0.0, -1.0, 0.0, 0.0], device=DEV)   # only empty examples carry weight
    for ww in (zero, w):
        (U,) = api.assemble_update(layers, ww, n=n, lengths=lens)
        torch.cuda.synchronize()
        assert torch.all(U == 0.0)
    (U,) = api.assemble_update(layers, torch.ones(1, device=DEV), n=0, lengths=None)
    torch.cuda.synchronize()
    assert torch.all(U == 0.0)
    # T = 1 (rank-one update per example) and NULL lengths (all T)
    l1 = make_layers([(64, 72)], n, 1, torch.bfloat16, torch.ones(n, dtype=torch.int32, device=DEV), seed=7)
    check(l1, mixed_weights(n, 7), n, None)


def test_determinism():
    n, T = 30, 200
    lens = torch.randint(0, T + 1, (n,), dtype=torch.int32, device=DEV)
    layers = make_layers([(384, 512)], n, T, torch.bfloat16, lens, seed=8)
    w = mixed_weights(n, 8)
    (a,) = api.assemble_update(layers, w, n=n, lengths=lens)
    (b,) = api.assemble_update(layers, w, n=n, lengths=lens)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_small_block_full_size_sampled_rows():
    """The small-block workload at full size (8 layers 2048 x 2048, 64 general
    examples of up to 512 tokens): top-k and signed weights, 24 sampled
    output rows x 24 sampled columns of every layer against the oracle."""
    cfg = workloads.CONFIGS["small"]
    layers, lens, _ = workloads.sketch_inputs(cfg, DEV)
    n = cfg["n"]
    layers = [dict(x=L["x"], dy=L["dy"]) for L in layers]
    rows = [0, 1, 15, 16, 255, 256, 257, 511, 640, 1023, 1024, 1200, 1500, 1791, 1792, 1900, 2000, 2040,
            2041, 2042, 2043, 2045, 2046, 2047]
    cols = [2047 - r for r in rows]
    s = torch.randn(1, n, device=DEV)
    _, wt, _ = api.select_topk(s, 32)
    _, errs = check(layers, wt[0], n, lens, rows=rows, cols=cols)
    print(f"small-block top-k max layer rel err {errs.max():.2e}")
    _, errs = check(layers, mixed_weights(n, 9, zero_rows=(3, 4, 60)), n, lens, rows=rows, cols=cols)
    print(f"small-block signed max layer rel err {errs.max():.2e}")


def test_llama_down_proj_full_size_sampled_entries():
    """One Llama-shaped down projection (d_in 14336 -> d_out 4096) with the
    full 256 general examples of 1024 tokens: sampled rows x columns."""
    n, T = 256, 1024
    g = torch.Generator(device=DEV)
    g.manual_seed(11)
    x = (0.02 * torch.randn(n, T, 14336, generator=g, device=DEV)).to(torch.bfloat16)
    dy = (0.02 * torch.randn(n, T, 4096, generator=g, device=DEV)).to(torch.bfloat16)
    w = mixed_weights(n, 10, zero_rows=tuple(range(0, n, 5)))
    rows = [0, 1, 255, 256, 2047, 2048, 4000, 4095]
    cols = [0, 7, 127, 128, 8191, 8192, 14000, 14335]
    _, errs = check([dict(x=x, dy=dy)], w, n, None, rows=rows, cols=cols)
    print(f"llama down_proj max rel err {errs.max():.2e}")


def test_weights_spanning_sixty_orders_of_magnitude():
    """The kernel rescales one accumulator by w_prev / w_next in |w| order:
    weights from 1e-30 to 1e30 with both signs must neither overflow nor
    lose the large terms."""
    n, T = 24, 64
    lens = torch.randint(1, T + 1, (n,), dtype=torch.int32, device=DEV)
    layers = make_layers([(256, 256), (64, 200)], n, T, torch.bfloat16, lens, seed=12)
    mags = torch.logspace(-30, 30, n, device=DEV)
    signs = torch.tensor([1.0, -1.0] * (n // 2), device=DEV)
    perm = torch.randperm(n, generator=torch.Generator().manual_seed(3)).to(DEV)
    w = (mags * signs)[perm].contiguous()
    w[5] = w[7]                                       # a tie in |w| and sign
    _, errs = check(layers, w, n, lens)
    print(f"wide-range weights max layer rel err {errs.max():.2e}")
    # the largest weights dominate: the same update from the top 3 alone is close
    top = torch.zeros_like(w)
    big = torch.argsort(w.abs(), descending=True)[:3]
    top[big] = w[big]
    Ua = api.assemble_update(layers, w, n=n, lengths=lens)
    Ub = api.assemble_update(layers, top, n=n, lengths=lens)
    for a, b in zip(Ua, Ub):
        assert rel(host64(a), host64(b)) <= 1e-5
