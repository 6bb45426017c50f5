"""Oracle: top-k selection by alignment score.

Test infrastructure only (see the package header).

Definition followed: the top-k rule of Sec. 3.3.2 keeps the k training
examples with the largest scores s_i = <g_i, g_star_hat>, ignoring the
redundancy term; the Select-S step of the one-pass Global Subset and
Layer-Wise algorithms (Sec. 4.2) applies it.  With w_i = 1/k on the selected
set the update is the subset average g_S (Sec. 3.3.2).

Conventions (readings): ties go to the lowest index; -0.0 equals +0.0;
+-inf order normally; any NaN score is an error.  The selected indices are
returned in ascending index order.

Parity: pinned by tests (exhaustive search over all k-subsets with exact
rational sums, k = n, K = cI equivalence with the exact subset projection).
"""

import numpy as np


def topk_ref(s, k):
    """Indices of the k largest scores (ties -> lowest index), ascending.

    Raises ValueError on NaN or on k outside [0, n].
    """
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    if not 0 <= k <= n:
        raise ValueError("k must satisfy 0 <= k <= n")
    if np.isnan(s).any():
        raise ValueError("NaN score")
    order = sorted(range(n), key=lambda i: (-s[i], i))
    return np.array(sorted(order[:k]), dtype=np.int64)
