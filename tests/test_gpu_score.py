"""GPU parity of the exact scorers (Direct, GIP, PIP) against the oracle.

The oracle's Direct scorer (explicit fp64 gradients; pinned against GIP, PIP
and autograd) is the reference for all three methods.  Inputs are bf16,
every product is exact in fp32 and the target-mean gradient enters PIP as a
bf16 hi + lo pair (relative rounding ~2^-17), so each layer's score vector
must match to a relative error of 1e-4 (tighter than the 2e-3 allowed for
bf16 sketches).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2605_07063_amd import api
from gpu_helpers import host64, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL_SCORE = 1e-4
METHODS = ["direct", "gip", "pip"]


def make(specs, N, T, lens, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(777 + seed)
    mask = torch.arange(T, device=DEV)[None, :] >= lens[:, None]
    out = []
    for di, do in specs:
        x = torch.randn(N, T, di, generator=g, device=DEV).to(torch.bfloat16)
        dy = torch.randn(N, T, do, generator=g, device=DEV).to(torch.bfloat16)
        x[mask] = float("nan")
        dy[mask] = float("nan")
        out.append(dict(x=x, dy=dy))
    return out


def reference(layers, n, m, lens):
    lh = lens.cpu().numpy()
    refs = []
    for L in layers:
        x, dy = host64(L["x"]), host64(L["dy"])
        refs.append(oracle.score_direct(x[:n], dy[:n], lh[:n], x[n:n + m], dy[n:n + m], lh[n:n + m]))
    return refs


@pytest.mark.parametrize("method", METHODS)
def test_ragged_lengths_and_dimension_tails(method):
    n, m, T = 7, 3, 150
    lens = torch.tensor([150, 0, 1, 127, 128, 129, 60, 150, 0, 77], dtype=torch.int32, device=DEV)
    layers = make([(136, 264), (64, 200)], n + m, T, lens, seed=1)
    s = api.score_exact(layers, n, m, lens, method=method)
    torch.cuda.synchronize()
    for l, ref in enumerate(reference(layers, n, m, lens)):
        got = host64(s[l])
        assert np.isfinite(got).all()
        assert got[1] == 0.0                              # an empty example scores exactly 0
        assert rel(got, ref) <= TOL_SCORE, f"{method} layer {l}: {rel(got, ref):.2e}"


def test_methods_agree_at_full_layer_width():
    """One 2048 x 2048 layer of the small-block workload's shape, 16 general
    and 4 target examples of up to 512 tokens."""
    n, m, T = 16, 4, 512
    lens = torch.randint(128, T + 1, (n + m,), generator=torch.Generator().manual_seed(2),
                         dtype=torch.int32).to(DEV)
    layers = make([(2048, 2048)], n + m, T, lens, seed=2)
    (ref,) = reference(layers, n, m, lens)
    outs = {}
    for method in METHODS:
        s = api.score_exact(layers, n, m, lens, method=method)
        torch.cuda.synchronize()
        outs[method] = host64(s[0])
        assert rel(outs[method], ref) <= TOL_SCORE, f"{method}: {rel(outs[method], ref):.2e}"
    # the orderings agree with each other (top-4 sets too)
    for method in METHODS:
        assert set(np.argsort(-outs[method])[:4]) == set(np.argsort(-ref)[:4])


def test_null_lengths_and_no_general_examples():
    n, m, T = 4, 2, 40
    full = torch.full((n + m,), T, dtype=torch.int32, device=DEV)
    layers = make([(64, 64)], n + m, T, full, seed=3)
    for method in METHODS:
        a = api.score_exact(layers, n, m, None, method=method)
        b = api.score_exact(layers, n, m, full, method=method)
        torch.cuda.synchronize()
        assert torch.equal(a, b)
        s = torch.empty(1, 0, device=DEV)
        api.dr_score_exact(layers, 0, m, T, None, method, s)
