"""dr_gram_noalloc (the Gram with the library's fixed per-device scratch)
called through the C ABI, against dr_gram with a caller workspace and
against the oracle, on consecutive calls of shrinking size that take the
three Gram paths."""

import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2605_07063_amd import _lib, api
from gpu_helpers import TOL_GRAM, host64, rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _rows(n, m, cols, dtype, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    R = torch.randn(n + m, cols, generator=g, device=DEV)
    return R.to(dtype)


def _noalloc(G, Gt, goff, K, s, t2):
    """The raw C call: device pointers, host group offsets, the current stream."""
    lib = _lib.load()
    ga = (ctypes.c_int64 * len(goff))(*goff)
    dt = _lib.DR_BF16 if Gt.dtype == torch.bfloat16 else _lib.DR_F32
    return lib.dr_gram_noalloc(ctypes.c_void_p(G.data_ptr()), G.shape[0], G.stride(0), ctypes.c_void_p(Gt.data_ptr()),
                               Gt.shape[0], Gt.stride(0), dt, ga, len(goff) - 1, ctypes.c_void_p(K.data_ptr()),
                               ctypes.c_void_p(s.data_ptr()), ctypes.c_void_p(t2.data_ptr()),
                               ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


CASES = [
    # (n, m, columns, groups, dtype): fp32 tall-skinny tiles with many chunk
    # partials (the largest scratch), then smaller: the one-pass small path
    # with several groups, then bf16 rows
    (256, 16, 98304, 1, torch.float32),
    (64, 8, 32768, 8, torch.float32),
    (40, 4, 4096, 2, torch.bfloat16),
]


@pytest.mark.parametrize("order", ["shrinking", "growing_back"])
def test_noalloc_matches_workspace_call_on_consecutive_calls(order):
    cases = CASES if order == "shrinking" else CASES[::-1] + CASES[:1]
    for i, (n, m, cols, P, dt) in enumerate(cases):
        print(f"no-alloc call {i}: n={n} m={m} cols={cols} P={P} {dt}", flush=True)
        R = _rows(n, m, cols, dt, 1000 + i)
        G, Gt = R[:n], R[n:]
        goff = [p * cols // P for p in range(P + 1)]
        need = api.dr_gram_workspace_size(n, m, goff, dt)
        assert 0 < need <= _lib.DR_GRAM_NOALLOC_MAX_BYTES
        K0, s0, t20 = api.gram(G, Gt, goff)
        K1 = torch.full_like(K0, float("nan"))
        s1 = torch.full_like(s0, float("nan"))
        t21 = torch.full_like(t20, float("nan"))
        assert _noalloc(G, Gt, goff, K1, s1, t21) == _lib.DR_OK
        torch.cuda.synchronize()
        assert torch.equal(K1, K0) and torch.equal(s1, s0) and torch.equal(t21, t20)
        Rh = host64(R)
        K_ref, s_ref, t2_ref = oracle.gram_ref(Rh[:n], Rh[n:], goff)
        for p in range(P):
            assert rel(host64(K1[p]), K_ref[p]) <= TOL_GRAM and rel(host64(s1[p]), s_ref[p]) <= TOL_GRAM
        assert np.allclose(host64(t21), t2_ref, rtol=TOL_GRAM, atol=0)


def test_noalloc_python_binding():
    n, m, cols = 64, 8, 8192
    R = _rows(n, m, cols, torch.float32, 7)
    K0, s0, t20 = api.gram(R[:n], R[n:])
    K1, s1, t21 = torch.empty_like(K0), torch.empty_like(s0), torch.empty_like(t20)
    api.dr_gram_noalloc(R[:n], R[n:], [0, cols], K1, s1, t21)
    torch.cuda.synchronize()
    assert torch.equal(K1, K0) and torch.equal(s1, s0) and torch.equal(t21, t20)
