"""Python face of the C ABI: the same calls, taking torch tensors.

Each function checks device / dtype / contiguity, turns tensors into device
pointers, passes torch's current HIP stream and raises DrError on a non-OK
status.  Workspaces are allocated with torch when the caller passes none.
No arithmetic of the method happens here.
"""

import ctypes

import torch

from . import _lib
from ._lib import DrLayer, check

_DTYPES = {torch.float32: _lib.DR_F32, torch.bfloat16: _lib.DR_BF16}


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _side_stream(stream, device):
    """The launch stream as a torch stream when it is not the current stream
    of `device` (None otherwise)."""
    if stream is None:
        return None
    if isinstance(stream, torch.cuda.Stream):
        ts = stream
    else:
        ts = torch.cuda.ExternalStream(int(stream), device=device)
    if ts.cuda_stream == torch.cuda.current_stream(device).cuda_stream:
        return None
    return ts


def _keep(stream, *tensors):
    """Tensors allocated here on the current stream but used by work enqueued
    on another stream: tell the caching allocator, so that their memory is
    not handed out again before that stream's work has finished."""
    for t in tensors:
        if t is None:
            continue
        ts = _side_stream(stream, t.device)
        if ts is not None:
            t.record_stream(ts)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _dev(t, name, dtype=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def _contig(t, name):
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _workspace(nbytes, device, workspace, stream=None):
    if nbytes == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _keep(stream, workspace)
    if workspace.numel() * workspace.element_size() < nbytes:
        raise ValueError("workspace too small")
    return workspace, workspace.numel() * workspace.element_size()


def _goff_array(goff):
    arr = (ctypes.c_int64 * len(goff))(*[int(v) for v in goff])
    return arr


def make_layer_array(layers):
    """Host array of dr_layer descriptors from dicts of device tensors.

    Each dict: x [N, T, d_in], dy [N, T, d_out] (row stride may exceed d),
    p_in [k_in, d_in], p_out [k_out, d_out], col_offset.
    """
    arr = (DrLayer * len(layers))()
    for i, L in enumerate(layers):
        x, dy, p_in, p_out = L["x"], L["dy"], L["p_in"], L["p_out"]
        for t, nm in ((x, "x"), (dy, "dy")):
            if t.numel() > 0 and (t.stride(-1) != 1 or t.stride(0) != t.shape[1] * t.stride(1)):
                raise ValueError(f"{nm} must be [N][T][ld] with unit element stride")
        _contig(p_in, "p_in")
        _contig(p_out, "p_out")
        arr[i] = DrLayer(x.data_ptr(), max(x.stride(1), x.shape[2]), dy.data_ptr(), max(dy.stride(1), dy.shape[2]),
                         p_in.data_ptr(), p_out.data_ptr(),
                         x.shape[2], dy.shape[2], p_in.shape[0], p_out.shape[0], int(L["col_offset"]))
    return arr


def dr_sketch_workspace_size(layers, N, T, dtype):
    arr = make_layer_array(layers)
    return _lib.load().dr_sketch_workspace_size(arr, len(layers), N, T, _DTYPES[dtype])


def dr_sketch_grads(layers, N, T, lengths, S, workspace=None, stream=None):
    """S[i, off_l + a*k_in + b] = sum_{t<len_i} (P_out dy_{i,t})[a] (P_in x_{i,t})[b]."""
    lib = _lib.load()
    dtype = layers[0]["x"].dtype
    if dtype not in _DTYPES:
        raise ValueError("x must be float32 or bfloat16")
    for L in layers:
        for nm in ("x", "dy", "p_in", "p_out"):
            _dev(L[nm], nm, dtype)
    _dev(S, "S", torch.float32)
    if S.dim() != 2 or S.stride(1) != 1:
        raise ValueError("S must be [N][ldS] with unit column stride")
    if lengths is not None:
        _dev(lengths, "lengths", torch.int32)
        _contig(lengths, "lengths")
    arr = make_layer_array(layers)
    nbytes = lib.dr_sketch_workspace_size(arr, len(layers), N, T, _DTYPES[dtype])
    ws, wsb = _workspace(nbytes, S.device, workspace, stream)
    check("dr_sketch_grads", lib.dr_sketch_grads(arr, len(layers), N, T, _ptr(lengths), _DTYPES[dtype], _ptr(S),
                                                 S.stride(0), _ptr(ws), wsb, _stream(stream)))
    return S


def dr_gram_workspace_size(n, m, goff, dtype):
    return _lib.load().dr_gram_workspace_size(n, m, _goff_array(goff), len(goff) - 1, _DTYPES[dtype])


def dr_gram(G, Gt, goff, K, s, t2, workspace=None, stream=None):
    """Per group: K_p = G_p G_p^T, s_p = G_p gbar_p, t2_p = |gbar_p|^2 (gbar = target mean)."""
    lib = _lib.load()
    dtype = Gt.dtype
    _dev(Gt, "Gt", dtype)
    n, m = G.shape[0], Gt.shape[0]
    if n > 0:
        _dev(G, "G", dtype)
    for t, nm in ((K, "K"), (s, "s"), (t2, "t2")):
        _dev(t, nm, torch.float32)
        _contig(t, nm)
    P = len(goff) - 1
    ga = _goff_array(goff)
    nbytes = lib.dr_gram_workspace_size(n, m, ga, P, _DTYPES[dtype])
    ws, wsb = _workspace(nbytes, Gt.device, workspace, stream)
    check("dr_gram", lib.dr_gram(_ptr(G), n, G.stride(0) if n > 0 else 0, _ptr(Gt), m, Gt.stride(0),
                                 _DTYPES[dtype], ga, P, _ptr(K), _ptr(s), _ptr(t2), _ptr(ws), wsb,
                                 _stream(stream)))


def dr_gram_noalloc(G, Gt, goff, K, s, t2, stream=None):
    """dr_gram with the library's fixed per-device scratch instead of a workspace."""
    lib = _lib.load()
    dtype = Gt.dtype
    _dev(Gt, "Gt", dtype)
    n, m = G.shape[0], Gt.shape[0]
    if n > 0:
        _dev(G, "G", dtype)
    for t, nm in ((K, "K"), (s, "s"), (t2, "t2")):
        _dev(t, nm, torch.float32)
        _contig(t, nm)
    ga = _goff_array(goff)
    check("dr_gram_noalloc", lib.dr_gram_noalloc(_ptr(G), n, G.stride(0) if n > 0 else 0, _ptr(Gt), m, Gt.stride(0),
                                                 _DTYPES[dtype], ga, len(goff) - 1, _ptr(K), _ptr(s), _ptr(t2),
                                                 _stream(stream)))


def dr_span_workspace_size(n, P):
    return _lib.load().dr_span_workspace_size(n, P)


def dr_project_span(K, s, t2, lam, mode, w, lam_eff, resid2, info, workspace=None, stream=None):
    """(K_p + lam_eff_p I) w_p = s_p per group."""
    lib = _lib.load()
    P = t2.shape[0]
    n = s.shape[-1] if s.numel() > 0 else 0
    for t, nm in ((K, "K"), (s, "s"), (t2, "t2"), (w, "w"), (lam_eff, "lam_eff"), (resid2, "resid2")):
        _dev(t, nm, torch.float32)
        _contig(t, nm)
    _dev(info, "info", torch.int32)
    nbytes = lib.dr_span_workspace_size(n, P)
    ws, wsb = _workspace(nbytes, t2.device, workspace, stream)
    check("dr_project_span", lib.dr_project_span(_ptr(K), _ptr(s), _ptr(t2), n, P, float(lam), int(mode), _ptr(w),
                                                 _ptr(lam_eff), _ptr(resid2), _ptr(info), _ptr(ws), wsb,
                                                 _stream(stream)))


def dr_project_cone(K, s, t2, max_iter, kkt_tol, w, resid2, iters, kkt, info, stream=None):
    """w_p = argmin_{w >= 0} 1/2 w^T K_p w - s_p^T w per group."""
    lib = _lib.load()
    P = t2.shape[0]
    n = s.shape[-1] if s.numel() > 0 else 0
    for t, nm in ((K, "K"), (s, "s"), (t2, "t2"), (w, "w"), (resid2, "resid2"), (kkt, "kkt")):
        _dev(t, nm, torch.float32)
        _contig(t, nm)
    for t, nm in ((iters, "iters"), (info, "info")):
        _dev(t, nm, torch.int32)
    check("dr_project_cone", lib.dr_project_cone(_ptr(K), _ptr(s), _ptr(t2), n, P, int(max_iter), float(kkt_tol),
                                                 _ptr(w), _ptr(resid2), _ptr(iters), _ptr(kkt), _ptr(info), None,
                                                 0, _stream(stream)))


def dr_project_simplex(K, s, t2, max_iter, tol, w, resid2, iters, res, info, stream=None):
    """Soft weighting: w = argmin over the simplex of w^T K w - 2 s^T w, per group."""
    lib = _lib.load()
    P, n = s.shape
    for t, nm in ((K, "K"), (s, "s"), (t2, "t2"), (w, "w"), (resid2, "resid2"), (res, "res")):
        _dev(t, nm, torch.float32)
        _contig(t, nm)
    _dev(iters, "iters", torch.int32)
    _dev(info, "info", torch.int32)
    check("dr_project_simplex", lib.dr_project_simplex(_ptr(K), _ptr(s), _ptr(t2), n, P, int(max_iter), float(tol),
                                                       _ptr(w), _ptr(resid2), _ptr(iters), _ptr(res), _ptr(info),
                                                       _stream(stream)))


def _projector_layer_array(layers):
    arr = (DrLayer * len(layers))()
    for i, L in enumerate(layers):
        arr[i] = DrLayer(None, 0, None, 0, L["p_in"].data_ptr(), L["p_out"].data_ptr(), L["p_in"].shape[1],
                         L["p_out"].shape[1], L["p_in"].shape[0], L["p_out"].shape[0], int(L["col_offset"]))
    return arr


def dr_backproject_workspace_size(layers):
    return _lib.load().dr_backproject_workspace_size(_projector_layer_array(layers), len(layers))


def dr_back_project(layers, u, U, u_offset, workspace=None, stream=None):
    """U[u_offset[l]:] (as [d_out][d_in]) = P_out^T X'_l P_in for every layer."""
    lib = _lib.load()
    dtype = layers[0]["p_in"].dtype
    if dtype not in _DTYPES:
        raise ValueError("p_in must be float32 or bfloat16")
    for L in layers:
        for nm in ("p_in", "p_out"):
            _dev(L[nm], nm, dtype)
            _contig(L[nm], nm)
    _dev(u, "u", torch.float32)
    _dev(U, "U", torch.float32)
    arr = _projector_layer_array(layers)
    ws, wsb = _workspace(lib.dr_backproject_workspace_size(arr, len(layers)), U.device, workspace, stream)
    check("dr_back_project", lib.dr_back_project(arr, len(layers), _DTYPES[dtype], _ptr(u), _ptr(U),
                                                 _goff_array(u_offset), _ptr(ws), wsb, _stream(stream)))
    return U


def dr_select_topk(s, k, idx, w, info, stream=None):
    """idx_p = the k largest s_p (ties -> lowest index), ascending; w_p = 1/k on idx_p."""
    lib = _lib.load()
    P, n = s.shape
    _dev(s, "s", torch.float32)
    _contig(s, "s")
    _dev(idx, "idx", torch.int32)
    _dev(info, "info", torch.int32)
    if w is not None:
        _dev(w, "w", torch.float32)
    check("dr_select_topk", lib.dr_select_topk(_ptr(s), n, P, int(k), _ptr(idx), _ptr(w), _ptr(info),
                                               _stream(stream)))


def dr_select_threshold(s, tau, inclusive, idx, count, w, info, stream=None):
    """Keep s_i > tau (or >= tau when inclusive) per group; idx ascending then -1."""
    lib = _lib.load()
    _dev(s, "s", torch.float32)
    _contig(s, "s")
    P, n = s.shape
    for t, nm, dt in ((count, "count", torch.int32), (info, "info", torch.int32)):
        _dev(t, nm, dt)
    if idx is not None:
        _dev(idx, "idx", torch.int32)
    if w is not None:
        _dev(w, "w", torch.float32)
    check("dr_select_threshold", lib.dr_select_threshold(_ptr(s), n, P, float(tau), 1 if inclusive else 0, _ptr(idx),
                                                         _ptr(count), _ptr(w), _ptr(info), _stream(stream)))


def dr_greedy_workspace_size(n, P):
    return _lib.load().dr_greedy_workspace_size(n, P)


def dr_select_greedy(K, s, k, idx, w, info, workspace=None, stream=None):
    """Greedy subset of size k on the full objective, per group (ascending idx)."""
    lib = _lib.load()
    _dev(K, "K", torch.float32)
    _dev(s, "s", torch.float32)
    _contig(K, "K")
    _contig(s, "s")
    P, n = s.shape
    _dev(idx, "idx", torch.int32)
    _dev(info, "info", torch.int32)
    if w is not None:
        _dev(w, "w", torch.float32)
    ws, wsb = _workspace(lib.dr_greedy_workspace_size(n, P), s.device, workspace, stream)
    check("dr_select_greedy", lib.dr_select_greedy(_ptr(K), _ptr(s), n, P, k, _ptr(idx), _ptr(w), _ptr(info), _ptr(ws),
                                                   wsb, _stream(stream)))


def dr_combine_workspace_size(n, goff):
    return _lib.load().dr_combine_workspace_size(n, _goff_array(goff), len(goff) - 1)


def dr_combine(G, goff, w, u, workspace=None, stream=None):
    """u[cols_p] = G[:, cols_p]^T w_p per group."""
    lib = _lib.load()
    dtype = G.dtype
    n = G.shape[0]
    if n > 0:
        _dev(G, "G", dtype)
    _dev(w, "w", torch.float32)
    _dev(u, "u", torch.float32)
    P = len(goff) - 1
    ga = _goff_array(goff)
    nbytes = lib.dr_combine_workspace_size(n, ga, P)
    ws, wsb = _workspace(nbytes, u.device, workspace, stream)
    check("dr_combine", lib.dr_combine(_ptr(G), n, G.stride(0) if n > 0 else 0, _DTYPES[dtype], ga, P, _ptr(w),
                                       _ptr(u), _ptr(ws), wsb, _stream(stream)))


def make_update_layer_array(layers):
    """Host dr_layer descriptors for dr_assemble_update: dicts with x [N, T, d_in]
    and dy [N, T, d_out] (projector fields are not used by the call)."""
    arr = (DrLayer * len(layers))()
    for i, L in enumerate(layers):
        x, dy = L["x"], L["dy"]
        for t, nm in ((x, "x"), (dy, "dy")):
            if t.numel() > 0 and (t.stride(-1) != 1 or t.stride(0) != t.shape[1] * t.stride(1)):
                raise ValueError(f"{nm} must be [N][T][ld] with unit element stride")
        arr[i] = DrLayer(x.data_ptr(), max(x.stride(1), x.shape[2]), dy.data_ptr(), max(dy.stride(1), dy.shape[2]),
                         None, None, x.shape[2], dy.shape[2], 0, 0, 0)
    return arr


def dr_update_workspace_size(layers, n, T, dtype):
    arr = make_update_layer_array(layers)
    return _lib.load().dr_update_workspace_size(arr, len(layers), n, T, _DTYPES[dtype])


def dr_assemble_update(layers, n, T, lengths, w, U, u_offset, group_of_layer=None, workspace=None, stream=None):
    """U[u_offset[l]:] (as [d_out][d_in]) = sum_{i<n, w[g_l][i] != 0} w[g_l][i] sum_{t<len_i} dy_{i,t} x_{i,t}^T."""
    lib = _lib.load()
    dtype = layers[0]["x"].dtype
    if dtype not in _DTYPES:
        raise ValueError("x must be float32 or bfloat16")
    for L in layers:
        for nm in ("x", "dy"):
            _dev(L[nm], nm, dtype)
    _dev(U, "U", torch.float32)
    _contig(U, "U")
    _dev(w, "w", torch.float32)
    if w.dim() == 1:
        w = w.unsqueeze(0)
    if w.dim() != 2 or w.stride(1) != 1:
        raise ValueError("w must be [P][ldw] with unit column stride")
    if lengths is not None:
        _dev(lengths, "lengths", torch.int32)
        _contig(lengths, "lengths")
    arr = make_update_layer_array(layers)
    offs = _goff_array(u_offset)
    gol = None
    if group_of_layer is not None:
        gol = (ctypes.c_int32 * len(layers))(*[int(v) for v in group_of_layer])
    nbytes = lib.dr_update_workspace_size(arr, len(layers), n, T, _DTYPES[dtype])
    ws, wsb = _workspace(nbytes, U.device, workspace, stream)
    check("dr_assemble_update", lib.dr_assemble_update(
        arr, len(layers), n, T, _ptr(lengths), _DTYPES[dtype], _ptr(w), w.shape[0], w.stride(0), gol, _ptr(U), offs,
        _ptr(ws), wsb, _stream(stream)))
    return U


_SCORE_METHODS = {"direct": _lib.DR_SCORE_DIRECT, "gip": _lib.DR_SCORE_GIP, "pip": _lib.DR_SCORE_PIP}


def dr_score_workspace_size(layers, n, m, T, method):
    arr = make_update_layer_array(layers)
    return _lib.load().dr_score_workspace_size(arr, len(layers), n, m, T, _lib.DR_BF16, _SCORE_METHODS[method])


def dr_score_exact(layers, n, m, T, lengths, method, s, workspace=None, stream=None):
    """s[l, i] = <gbar*_l, G_i^(l)> by the Direct, GIP or PIP contraction order."""
    lib = _lib.load()
    for L in layers:
        for nm in ("x", "dy"):
            _dev(L[nm], nm, torch.bfloat16)
    _dev(s, "s", torch.float32)
    _contig(s, "s")
    if lengths is not None:
        _dev(lengths, "lengths", torch.int32)
        _contig(lengths, "lengths")
    arr = make_update_layer_array(layers)
    meth = _SCORE_METHODS[method]
    nbytes = lib.dr_score_workspace_size(arr, len(layers), n, m, T, _lib.DR_BF16, meth)
    ws, wsb = _workspace(nbytes, s.device, workspace, stream)
    check("dr_score_exact", lib.dr_score_exact(arr, len(layers), n, m, T, _ptr(lengths), _lib.DR_BF16, meth, _ptr(s),
                                               _ptr(ws), wsb, _stream(stream)))
    return s


# ---------------------------------------------------------------------------
# allocating conveniences (outputs created with torch on the inputs' device)
# ---------------------------------------------------------------------------

def sketch(layers, lengths=None, stream=None):
    N, T = layers[0]["x"].shape[:2]
    kt = max(int(L["col_offset"]) + L["p_in"].shape[0] * L["p_out"].shape[0] for L in layers)
    S = torch.empty(N, kt, dtype=torch.float32, device=layers[0]["x"].device)
    _keep(stream, S)
    return dr_sketch_grads(layers, N, T, lengths, S, stream=stream)


def gram(G, Gt, goff=None, stream=None):
    if goff is None:
        goff = [0, Gt.shape[1]]
    P, n = len(goff) - 1, G.shape[0]
    dev = Gt.device
    K = torch.empty(P, n, n, dtype=torch.float32, device=dev)
    s = torch.empty(P, n, dtype=torch.float32, device=dev)
    t2 = torch.empty(P, dtype=torch.float32, device=dev)
    _keep(stream, K, s, t2)
    dr_gram(G, Gt, goff, K, s, t2, stream=stream)
    return K, s, t2


def project_span(K, s, t2, lam, mode=_lib.DR_RIDGE_REL_TRACE, stream=None):
    P, n = s.shape
    dev = t2.device
    w = torch.empty(P, n, dtype=torch.float32, device=dev)
    lam_eff = torch.empty(P, dtype=torch.float32, device=dev)
    resid2 = torch.empty(P, dtype=torch.float32, device=dev)
    info = torch.empty(P, dtype=torch.int32, device=dev)
    _keep(stream, w, lam_eff, resid2, info)
    dr_project_span(K, s, t2, lam, mode, w, lam_eff, resid2, info, stream=stream)
    return w, lam_eff, resid2, info


def project_cone(K, s, t2, max_iter, kkt_tol=0.0, stream=None):
    P, n = s.shape
    dev = t2.device
    w = torch.empty(P, n, dtype=torch.float32, device=dev)
    resid2 = torch.empty(P, dtype=torch.float32, device=dev)
    iters = torch.empty(P, dtype=torch.int32, device=dev)
    kkt = torch.empty(P, dtype=torch.float32, device=dev)
    info = torch.empty(P, dtype=torch.int32, device=dev)
    _keep(stream, w, resid2, iters, kkt, info)
    dr_project_cone(K, s, t2, max_iter, kkt_tol, w, resid2, iters, kkt, info, stream=stream)
    return w, resid2, iters, kkt, info


def select_topk(s, k, with_weights=True, stream=None):
    P, n = s.shape
    dev = s.device
    idx = torch.empty(P, k, dtype=torch.int32, device=dev)
    w = torch.empty(P, n, dtype=torch.float32, device=dev) if with_weights else None
    info = torch.empty(P, dtype=torch.int32, device=dev)
    _keep(stream, idx, w, info)
    dr_select_topk(s, k, idx, w, info, stream=stream)
    return idx, w, info


def combine(G, w, goff=None, stream=None):
    if goff is None:
        goff = [0, G.shape[1]]
    u = torch.zeros(goff[-1], dtype=torch.float32, device=w.device)
    _keep(stream, u)
    ts = _side_stream(stream, u.device)
    if ts is not None:
        # the zero fill runs on the current stream: order the combine after it
        ts.wait_stream(torch.cuda.current_stream(u.device))
    dr_combine(G, goff, w, u, stream=stream)
    return u


def assemble_update(layers, w, n=None, lengths=None, group_of_layer=None, stream=None):
    """Per-layer updates [d_out, d_in] (views of one flat fp32 buffer)."""
    N, T = layers[0]["x"].shape[:2]
    n = w.shape[-1] if n is None else n
    sizes = [L["dy"].shape[2] * L["x"].shape[2] for L in layers]
    offs, o = [], 0
    for sz in sizes:
        offs.append(o)
        o += sz
    U = torch.empty(o, dtype=torch.float32, device=w.device)
    _keep(stream, U)
    dr_assemble_update(layers, n, T, lengths, w, U, offs, group_of_layer=group_of_layer, stream=stream)
    return [U[a:a + sz].view(L["dy"].shape[2], L["x"].shape[2]) for a, sz, L in zip(offs, sizes, layers)]


def select_threshold(s, tau=0.0, inclusive=True, stream=None):
    """Kept indices [P, n] (ascending, then -1), counts [P], weights [P, n], info [P]."""
    P, n = s.shape
    dev = s.device
    idx = torch.empty(P, n, dtype=torch.int32, device=dev)
    count = torch.empty(P, dtype=torch.int32, device=dev)
    w = torch.empty(P, n, dtype=torch.float32, device=dev)
    info = torch.empty(P, dtype=torch.int32, device=dev)
    _keep(stream, idx, count, w, info)
    dr_select_threshold(s, tau, inclusive, idx, count, w, info, stream=stream)
    return idx, count, w, info


def select_greedy(K, s, k, stream=None):
    P, n = s.shape
    dev = s.device
    idx = torch.empty(P, k, dtype=torch.int32, device=dev)
    w = torch.empty(P, n, dtype=torch.float32, device=dev)
    info = torch.empty(P, dtype=torch.int32, device=dev)
    _keep(stream, idx, w, info)
    dr_select_greedy(K, s, k, idx, w, info, stream=stream)
    return idx, w, info


def score_exact(layers, n, m, lengths=None, method="pip", stream=None):
    """Per-layer exact scores [num_layers, n] of the first n rows against the mean of the next m."""
    T = layers[0]["x"].shape[1]
    s = torch.empty(len(layers), n, dtype=torch.float32, device=layers[0]["x"].device)
    _keep(stream, s)
    return dr_score_exact(layers, n, m, T, lengths, method, s, stream=stream)


def project_simplex(K, s, t2, max_iter=2000, tol=1e-7, stream=None):
    P, n = s.shape
    dev = t2.device
    w = torch.empty(P, n, dtype=torch.float32, device=dev)
    resid2 = torch.empty(P, dtype=torch.float32, device=dev)
    iters = torch.empty(P, dtype=torch.int32, device=dev)
    res = torch.empty(P, dtype=torch.float32, device=dev)
    info = torch.empty(P, dtype=torch.int32, device=dev)
    _keep(stream, w, resid2, iters, res, info)
    dr_project_simplex(K, s, t2, max_iter, tol, w, resid2, iters, res, info, stream=stream)
    return w, resid2, iters, res, info


def back_project(layers, u, stream=None):
    """Per-layer parameter-space blocks [d_out, d_in] of a sketch-space vector."""
    sizes = [L["p_out"].shape[1] * L["p_in"].shape[1] for L in layers]
    offs, o = [], 0
    for sz in sizes:
        offs.append(o)
        o += sz
    U = torch.empty(o, dtype=torch.float32, device=u.device)
    _keep(stream, U)
    dr_back_project(layers, u, U, offs, stream=stream)
    return [U[a:a + sz].view(L["p_out"].shape[1], L["p_in"].shape[1]) for a, sz, L in zip(offs, sizes, layers)]
