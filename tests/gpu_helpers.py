"""Shared helpers of the GPU parity tests (no arithmetic of the method)."""

import numpy as np
import torch

# tolerances: bf16-input sketches rel 2e-3 (per example and layer block);
# fp32-input sketches, Gram / scores and the fp32 solves rel 1e-5
TOL_SKETCH_BF16 = 2e-3
TOL_SKETCH_F32 = 1e-5
TOL_GRAM = 1e-5
TOL_SOLVE = 1e-5


def host64(t):
    """Exact float64 host copy of a device tensor (bf16 / fp32 upcast exactly)."""
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    if nb == 0.0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b) / nb)


def layers_to_host(layers, rows=None):
    """Host float64 copies of the layers (only the given example rows, if any)."""
    def pick(t):
        return host64(t if rows is None else t[list(rows)])
    return [dict(x=pick(L["x"]), dy=pick(L["dy"]), p_in=host64(L["p_in"]), p_out=host64(L["p_out"]),
                 col_offset=int(L["col_offset"])) for L in layers]


def block_errors(S_gpu, S_ref, layers, rows):
    """Relative Frobenius error of each (example, layer) sketch block."""
    errs = []
    for L in layers:
        k = L["p_in"].shape[0] * L["p_out"].shape[0]
        o = int(L["col_offset"])
        for i in rows:
            g, r = S_gpu[i, o:o + k], S_ref[i, o:o + k]
            if np.linalg.norm(r) == 0.0:
                errs.append(0.0 if np.all(g == 0.0) else np.inf)
            else:
                errs.append(rel(g, r))
    return np.array(errs)
