"""CPU oracle for the Dr. Post-Training sketch / Gram / projection path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports, calls or
links this package; only the test suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP path.

Everything here is plain NumPy (SciPy for two textbook routines) in float64,
written for a reader who checks it against the paper by eye:

* ``sketch``  -- explicit per-example linear-layer gradients (sum of outer
  products over valid tokens, Sec. 4.1 "Backward pass"), compressed by the
  factorised projector of App. C.3 ("Factorized Projection", "Per-Sample
  Gradient Compression").
* ``scores``  -- the three exact scorers of Sec. 4.3 (Direct, Ghost Inner
  Product, Per-Token Inner Product); used to pin the sketch oracle.
* ``gram``    -- target mean, Gram matrix and alignment scores
  (Sec. 3.2 batch gradients; Sec. 3.3.2 alignment / redundancy split).
* ``span``    -- Euclidean projection, Eq. (proj), onto the span of the
  general-data gradients, with a Tikhonov ridge.
* ``cone``    -- Eq. (proj) onto the convex cone of the general-data
  gradients (non-negative least squares, exact active-set solver).
* ``topk``    -- the top-k rule of Sec. 3.3.2 with lowest-index tie break.
* ``select``  -- thresholding / negative filtering and greedy construction,
  the other subset rules of Sec. 3.3.2.
* ``simplex`` -- soft weighting over the probability simplex (Sec. 6) and
  the back-projection Pi^T of App. C.3.
* ``update``  -- the weighted assembly of the update in parameter space
  (Sec. 4.2, post-hoc assembly from the retained pairs).
* ``brute``   -- exhaustive enumeration for tiny inputs.

Parity status of every function is stated in its module header.
"""

from .sketch import per_example_gradient, sketch_block, sketch_ref
from .scores import score_direct, score_gip, score_pip, score_compressed
from .gram import gram_ref
from .span import ridge_lambda, span_ref, span_residual2, combine_ref
from .cone import nnls_active_set, cone_ref, cone_kkt_residual, cone_pg_replay
from .topk import topk_ref
from .update import update_ref
from .select import threshold_ref, greedy_ref, subset_objective
from .simplex import simplex_ref, simplex_residual, simplex_objective, backproject_ref
from . import brute

__all__ = [
    "per_example_gradient", "sketch_block", "sketch_ref",
    "score_direct", "score_gip", "score_pip", "score_compressed",
    "gram_ref",
    "ridge_lambda", "span_ref", "span_residual2", "combine_ref",
    "nnls_active_set", "cone_ref", "cone_kkt_residual", "cone_pg_replay",
    "topk_ref", "update_ref", "threshold_ref", "greedy_ref", "subset_objective", "simplex_ref", "simplex_residual", "simplex_objective", "backproject_ref", "brute",
]
