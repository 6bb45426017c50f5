"""Oracle: assembly of the update in full parameter space.

Test infrastructure only (see the package header).

Definition followed
-------------------
Once the weights w of the general examples are known, the update of every
linear layer is assembled from the retained pairs (a, dL/de) as the weighted
sum of the explicit per-example weight gradients (Sec. 4.2, the post-hoc
assembly step of the Global Subset Update algorithm and the per-layer
assembly of the Layer-Wise Subset Update algorithm):
    U_l = sum_i w_i G_i^(l),   G_i^(l) = sum_{tau < len_i} dL/de_{i,tau} (outer) a_{i,tau}.
The paper states it for the top-k rule, w_i = 1/k on the selected set S
(u = g_S, Sec. 3.3.2); the same sum with the span or cone weights is the
update u = G^T w of Eq. (proj) in parameter space.  With group-wise
weights (Sec. 3.3.3) layer l uses the weight row of the group it belongs to.

Readings
--------
* Examples with w_i = 0 are not part of the update: they are skipped, not
  multiplied by zero (like padded tokens), so whatever their rows hold
  (NaN included) cannot leak.
* Only the first n rows of a merged batch carry weights (the general
  examples); the target rows after them never enter the update.

Parity: pinned by tests (one-hot weights reproduce torch.func per-sample
gradients; unit weights reproduce the autograd weight gradient; subset-mean
weights reproduce autograd of the subset-mean loss; sketching the update
equals the weighted sum of the pinned sketches; a hand fixture).
"""

import numpy as np

from .sketch import per_example_gradient


def update_ref(layers, w, lengths=None, group_of_layer=None):
    """Assembled update of every layer, as a list of float64 [d_out, d_in].

    layers: sequence of dicts with keys x [N, T, d_in] and dy [N, T, d_out].
    w:      [P, n] (or [n]) weights of the first n examples, n <= N.
    lengths: [N] valid tokens per example (None = all T).
    group_of_layer: [num_layers] row of w used by each layer (None = row 0).
    """
    w = np.atleast_2d(np.asarray(w, dtype=np.float64))
    n = w.shape[1]
    out = []
    for li, layer in enumerate(layers):
        x, dy = layer["x"], layer["dy"]
        T = x.shape[1]
        g = 0 if group_of_layer is None else int(group_of_layer[li])
        U = np.zeros((dy.shape[2], x.shape[2]))
        for i in range(n):
            wi = w[g, i]
            if wi == 0.0:
                continue
            L = T if lengths is None else int(lengths[i])
            U += wi * per_example_gradient(x[i], dy[i], L)
        out.append(U)
    return out
