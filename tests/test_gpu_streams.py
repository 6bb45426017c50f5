"""Calls enqueued on a stream other than the current one: buffers that the
Python binding allocates itself (workspaces and outputs) stay reserved until
that stream's work has finished."""

import numpy as np
import pytest
import torch

import oracle
from paper_2605_07063_amd import api
from gpu_helpers import TOL_SOLVE, host64, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_side_stream_blocked_span_keeps_its_workspace():
    """The blocked span (n = 512 > 256) runs on a side stream held back by a
    spin kernel while the current stream allocates and overwrites memory of
    the span workspace's size: the result equals the same call on the
    current stream, and the oracle's."""
    n = 512
    g = torch.Generator(device=DEV)
    g.manual_seed(99)
    A = torch.randn(n, 2 * n, generator=g, device=DEV)
    K = (A @ A.T).unsqueeze(0).contiguous()
    s = torch.randn(1, n, generator=g, device=DEV)
    t2 = torch.ones(1, device=DEV)
    w0, le0, r20, info0 = api.project_span(K, s, t2, 1e-3, 1)
    torch.cuda.synchronize()
    assert int(info0[0]) == 0
    nbytes = api.dr_span_workspace_size(n, 1)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        torch.cuda._sleep(50_000_000)
    w, le, r2, info = api.project_span(K, s, t2, 1e-3, 1, stream=side)
    junk = [torch.full((nbytes,), 255, dtype=torch.uint8, device=DEV) for _ in range(3)]
    torch.cuda.synchronize()
    del junk
    assert int(info[0]) == 0
    assert torch.equal(w, w0) and torch.equal(r2, r20)
    w_ref, _, _ = oracle.span_ref(host64(K[0]), host64(s[0]), 1e-3, 1, lam_eff=float(le[0]))
    assert rel(host64(w[0]), w_ref) <= TOL_SOLVE


def test_side_stream_raw_handle_and_combine_order():
    """A raw stream handle (int) works like a torch stream, and the
    allocating combine orders its zero fill before the side-stream kernel."""
    n, kappa = 64, 4096
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    G = torch.randn(n, kappa, generator=g, device=DEV)
    w = torch.randn(1, n, generator=g, device=DEV)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        torch.cuda._sleep(20_000_000)
    u = api.combine(G, w, stream=side.cuda_stream)
    torch.cuda.synchronize()
    ref = oracle.combine_ref(host64(G), host64(w[0]))
    assert rel(host64(u), ref) <= TOL_SOLVE
    assert np.isfinite(host64(u)).all()
