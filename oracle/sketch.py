"""Oracle: explicit per-example gradients and their factorised sketches.

Test infrastructure only (see the package header).

Definitions followed
--------------------
* Per-sample weight gradient of a linear layer (Sec. 4.1, "Backward pass";
  App. C.3 "Per-Sample Gradient Compression"):
      G_i = sum over tokens tau of  dL/de_{i,tau}  (outer)  a_{i,tau},
  a d_out x d_in matrix.  Only the valid tokens tau < len_i enter the sum:
  padded positions are loss-masked and contribute nothing (they are sliced
  away, never multiplied by zero, so NaN padding cannot leak).
* Factorised projector Pi = P_final (P_in kron P_out) applied to an
  outer-product sum (App. C.3 "Forward projection"): each token contributes
  the small outer product (P_out b)(P_in a)^T.  With P_final = I this is
      S_i = P_out G_i P_in^T   (kappa_out x kappa_in),
  stored row-major, i.e. element (a, b) at position a*kappa_in + b.
  (The paper writes the Kronecker factors in both orders; the two readings
  differ only by transposing this small block, and every downstream quantity
  is an inner product, so the stored order only has to be the same for all
  rows.  Row-major [kappa_out][kappa_in] is the reading used everywhere.)

The oracle forms G_i explicitly as a full d_out x d_in matrix (a matmul of the
token-major factors is exactly the sum of the per-token outer products) and
only then sketches it.  The GPU path never forms G_i.

Parity: pinned by tests (identity projectors reproduce torch.func per-sample
gradients and the autograd weight gradient; explicit Kronecker matrix; exact
scorers; rank-one and empty cases; NaN padding).
"""

import numpy as np


def per_example_gradient(x, dy, length):
    """Explicit per-sample weight gradient of one linear layer.

    x:  [T, d_in]  layer inputs a_{i,tau} (token-major).
    dy: [T, d_out] output gradients dL/de_{i,tau}.
    length: number of valid tokens; rows >= length are padding.
    Returns G = sum_{tau < length} dy[tau] x[tau]^T as float64 [d_out, d_in].
    """
    length = int(length)
    xv = np.asarray(x, dtype=np.float64)[:length]
    dv = np.asarray(dy, dtype=np.float64)[:length]
    return dv.T @ xv


def sketch_block(G, p_in, p_out):
    """Factorised compression of one explicit gradient: P_out G P_in^T."""
    p_in = np.asarray(p_in, dtype=np.float64)
    p_out = np.asarray(p_out, dtype=np.float64)
    return p_out @ np.asarray(G, dtype=np.float64) @ p_in.T


def sketch_ref(layers, lengths=None, rows=None):
    """Sketches of every example of a merged batch, concatenated over layers.

    layers: sequence of dicts with keys
        x     [N, T, d_in], dy [N, T, d_out],
        p_in  [k_in, d_in], p_out [k_out, d_out],
        col_offset (optional; defaults to the running sum of k_out*k_in).
    lengths: [N] valid-token counts (None: every example is full length).
    rows: optional subset of example indices to compute (others left zero).
    Returns S as float64 [N, kappa_tot] where row i holds, for each layer,
    the flattened block P_out G_i P_in^T at that layer's column offset.
    """
    N, T = np.asarray(layers[0]["x"]).shape[:2]
    if lengths is None:
        lengths = np.full(N, T, dtype=np.int64)
    offsets = []
    off = 0
    for L in layers:
        k_out, k_in = np.asarray(L["p_out"]).shape[0], np.asarray(L["p_in"]).shape[0]
        offsets.append(int(L.get("col_offset", off)))
        off = max(off, offsets[-1] + k_out * k_in)
    kappa_tot = off
    S = np.zeros((N, kappa_tot), dtype=np.float64)
    row_list = range(N) if rows is None else rows
    for L, o in zip(layers, offsets):
        k_out, k_in = np.asarray(L["p_out"]).shape[0], np.asarray(L["p_in"]).shape[0]
        for i in row_list:
            G = per_example_gradient(L["x"][i], L["dy"][i], lengths[i])
            S[i, o:o + k_out * k_in] = sketch_block(G, L["p_in"], L["p_out"]).reshape(-1)
    return S
