"""Seeded synthetic inputs shaped like the paper's post-training workloads.

This module only draws random tensors (with torch generators on the target
device) and holds none of the method's arithmetic; both the HIP path and the
CPU oracle are fed from it (the oracle always receives host copies of the
exact tensors the device consumed).

Every workload is a merged batch of n general + m target examples
(Sec. 4.2, "merging training and target batch"), with per-layer retained
pairs x = a (layer inputs) and dy = dL/de (output gradients) of shape
[N, T, d], loss-masked padding after len_i tokens, and per-layer Gaussian
projectors P_in [k_in, d_in], P_out [k_out, d_out] with N(0, 1/k) entries
(so the sketch preserves inner products in expectation).  Low-precision
tensors are drawn in fp32 and rounded to bf16 once (round to nearest even).
"""

import math

import torch

# (d_in, d_out) of the seven linear maps of one Llama-3-8B block
LLAMA_BLOCK = [
    ("q", 4096, 4096), ("k", 4096, 1024), ("v", 4096, 1024), ("o", 4096, 4096),
    ("gate", 4096, 14336), ("up", 4096, 14336), ("down", 14336, 4096),
]

CONFIGS = {
    # one 256x256 layer, fp32, 16 + 4 examples of 32 tokens, 16x16 sketch, span (ridge 1e-3)
    "tiny": dict(cid=0, layers=[(256, 256)], k_in=16, k_out=16, n=16, m=4, T=32, dtype=torch.float32,
                 dist="normal", std=1.0, lengths="full", solver="span", lam=1e-3),
    # 8 layers 2048x2048, bf16, 64 + 8 examples, T=512 with lengths U{128..512}, 64x64 sketches, cone 200 iters
    "small": dict(cid=1, layers=[(2048, 2048)] * 8, k_in=64, k_out=64, n=64, m=8, T=512, dtype=torch.bfloat16,
                  dist="normal", std=1.0, lengths=("uniform_all", 128, 512), solver="cone", iters=200),
    # 32 Llama-3-8B-shaped blocks (7 maps each), bf16 N(0, 0.02^2), 256 + 16 examples, T=1024, 32x32 sketches
    "llama": dict(cid=2, layers=[(di, do) for _ in range(32) for (_, di, do) in LLAMA_BLOCK], k_in=32, k_out=32,
                  n=256, m=16, T=1024, dtype=torch.bfloat16, dist="normal", std=0.02, lengths="full",
                  solver="span", lam=0.0, topk=64),
    # 16384 + 32 pre-sketched rows of dim 8192: N(0, I) plus a rank-32 component of scale 3
    "gram": dict(cid=3, rows=16384 + 32, dim=8192, n=16384, m=32, rank=32, scale=3.0, dtype=torch.bfloat16,
                 lam=1e-2, topk=1024),
    # 16 layers 4096x4096, 32 + 4 examples at T=4096, Student-t(3) scaled to unit variance, 30 % padded
    "long": dict(cid=4, layers=[(4096, 4096)] * 16, k_in=64, k_out=64, n=32, m=4, T=4096, dtype=torch.bfloat16,
                 dist="student_t3", std=1.0, lengths=("pad_fraction", 0.3, 256), solver="cone", kkt_tol=1e-6),
}

# generator streams
S_PIN, S_POUT, S_X, S_DY, S_LEN, S_NOISE, S_FACTOR = range(7)


def seed_of(cid, stream, layer=0):
    return (int(cid) * 1_000_003 + int(stream) * 10_007 + int(layer) * 7 + 12_345) % (2 ** 31 - 1)


def _gen(device, cid, stream, layer=0):
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(cid, stream, layer))
    return g


def _draw(shape, dist, std, g, device, dtype, chunk_rows=8):
    """Draw [N, ...] in chunks along dim 0 (bounded fp32 temporaries)."""
    out = torch.empty(shape, dtype=dtype, device=device)
    for r0 in range(0, shape[0], chunk_rows):
        r1 = min(shape[0], r0 + chunk_rows)
        sub = (r1 - r0,) + tuple(shape[1:])
        z = torch.randn(sub, generator=g, device=device, dtype=torch.float32)
        if dist == "student_t3":
            # t_3 = Z / sqrt(chi2_3 / 3); Var(t_3) = 3, so divide by sqrt(3) for unit variance
            chi2 = torch.zeros_like(z)
            for _ in range(3):
                e = torch.randn(sub, generator=g, device=device, dtype=torch.float32)
                chi2.addcmul_(e, e)
            z = z / torch.sqrt(chi2 / 3.0) / math.sqrt(3.0)
            del chi2
        elif dist != "normal":
            raise ValueError(dist)
        if std != 1.0:
            z.mul_(std)
        out[r0:r1] = z.to(dtype)
        del z
    return out


def lengths(cfg, device, cid=None):
    """Valid-token counts [N] (int32) following the workload's length mix."""
    cid = cfg["cid"] if cid is None else cid
    N, T = cfg["n"] + cfg["m"], cfg["T"]
    spec = cfg["lengths"]
    g = _gen("cpu", cid, S_LEN)
    if spec == "full":
        L = torch.full((N,), T, dtype=torch.int32)
    elif spec[0] == "uniform_all":
        L = torch.randint(spec[1], spec[2] + 1, (N,), generator=g, dtype=torch.int64).to(torch.int32)
    elif spec[0] == "pad_fraction":
        npad = int(round(spec[1] * N))
        rows = torch.randperm(N, generator=g)[:npad]
        L = torch.full((N,), T, dtype=torch.int32)
        L[rows] = torch.randint(spec[2], T, (npad,), generator=g, dtype=torch.int64).to(torch.int32)
    else:
        raise ValueError(spec)
    return L.to(device)


def projector(k, d, dtype, device, cid, stream, layer):
    g = _gen(device, cid, stream, layer)
    p = torch.randn(k, d, generator=g, device=device, dtype=torch.float32) / math.sqrt(k)
    return p.to(dtype)


def layer_inputs(cfg, layer, device, N=None, T=None, d_in=None, d_out=None, nan_padding=False, lens=None,
                 cid=None):
    """Retained pair and projectors of one layer: dict(x, dy, p_in, p_out).

    N, T, d_in, d_out override the workload's sizes (scaled-down parity
    cases); with nan_padding the positions t >= lens[i] are set to NaN.
    """
    cid = cfg["cid"] if cid is None else cid
    N = cfg["n"] + cfg["m"] if N is None else N
    T = cfg["T"] if T is None else T
    di, do = cfg["layers"][layer % len(cfg["layers"])]
    d_in = di if d_in is None else d_in
    d_out = do if d_out is None else d_out
    dt = cfg["dtype"]
    x = _draw((N, T, d_in), cfg["dist"], cfg["std"], _gen(device, cid, S_X, layer), device, dt)
    dy = _draw((N, T, d_out), cfg["dist"], cfg["std"], _gen(device, cid, S_DY, layer), device, dt)
    if nan_padding:
        if lens is None:
            raise ValueError("nan_padding needs lens")
        mask = torch.arange(T, device=device)[None, :] >= lens.to(device)[:, None]
        x[mask] = float("nan")
        dy[mask] = float("nan")
    p_in = projector(cfg["k_in"], d_in, dt, device, cid, S_PIN, layer)
    p_out = projector(cfg["k_out"], d_out, dt, device, cid, S_POUT, layer)
    return dict(x=x, dy=dy, p_in=p_in, p_out=p_out)


def sketch_inputs(cfg, device, layers=None, nan_padding=False, **over):
    """All layers of a workload (or the given layer indices) with column offsets."""
    idx = list(range(len(cfg["layers"]))) if layers is None else list(layers)
    lens = lengths(cfg, device)
    if "T" in over and over["T"] is not None:
        lens = lens.clamp(max=over["T"])
    if "N" in over and over["N"] is not None:
        lens = lens[: over["N"]]
    out, off = [], 0
    for l in idx:
        L = layer_inputs(cfg, l, device, nan_padding=nan_padding, lens=lens, **over)
        L["col_offset"] = off
        off += cfg["k_in"] * cfg["k_out"]
        out.append(L)
    return out, lens, off


def llama_step_inputs(cfg, device, buffers=2, blocks=None):
    """The whole Llama-shaped step: 32 blocks x 7 maps, 224 sketch column
    blocks of 32 x 32 (229376 columns in all).

    One block's retained pairs are 45.6 GB of bf16 (272 examples x 1024
    tokens over the seven maps), and the step's 32 blocks (1.46 TB) do not
    fit in HBM at once, so `buffers` blocks of activations are drawn and
    kept resident: block b reads the activations of block b % buffers.  Its
    projectors are its own (seeded by the map index 7 b + j) and it writes
    its own column range.  Every sketch call still streams a whole block
    from HBM (far above the last-level cache), so the reuse changes the
    values, not the traffic.  Returns (blocks: list of 7-layer lists with
    col_offset set, lens, k_tot)."""
    nb = len(cfg["layers"]) // len(LLAMA_BLOCK)
    blocks = list(range(nb)) if blocks is None else list(blocks)
    lens = lengths(cfg, device)
    kk = cfg["k_in"] * cfg["k_out"]
    acts = {}
    out = []
    for b in blocks:
        src = b % buffers
        if src not in acts:
            acts[src] = []
            for j in range(len(LLAMA_BLOCK)):
                L = layer_inputs(cfg, 7 * src + j, device, lens=lens)
                acts[src].append((L["x"], L["dy"]))
        blk = []
        for j in range(len(LLAMA_BLOCK)):
            l = 7 * b + j
            di, do = cfg["layers"][l]
            x, dy = acts[src][j]
            blk.append(dict(x=x, dy=dy,
                            p_in=projector(cfg["k_in"], di, cfg["dtype"], device, cfg["cid"], S_PIN, l),
                            p_out=projector(cfg["k_out"], do, cfg["dtype"], device, cfg["cid"], S_POUT, l),
                            col_offset=l * kk))
        out.append(blk)
    return out, lens, len(cfg["layers"]) * kk


def gram_rows(cfg, device, rows=None, dim=None):
    """Pre-sketched rows Z + scale * C B (rank-r shared component), bf16."""
    cid = cfg["cid"]
    rows = cfg["rows"] if rows is None else rows
    dim = cfg["dim"] if dim is None else dim
    r = cfg["rank"]
    gz = _gen(device, cid, S_NOISE)
    gf = _gen(device, cid, S_FACTOR)
    C = torch.randn(rows, r, generator=gf, device=device, dtype=torch.float32)
    B = torch.randn(r, dim, generator=gf, device=device, dtype=torch.float32) / math.sqrt(r)
    out = torch.empty(rows, dim, dtype=cfg["dtype"], device=device)
    step = 2048
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        z = torch.randn(r1 - r0, dim, generator=gz, device=device, dtype=torch.float32)
        z.addmm_(C[r0:r1], B, alpha=cfg["scale"])
        out[r0:r1] = z.to(cfg["dtype"])
    return out
