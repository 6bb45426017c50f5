"""MI355X-native hot path of Dr. Post-Training (arXiv 2605.07063).

The work runs in libdr.so (hand-written HIP for gfx950, C ABI in
include/dr_api.h).  `api` is its Python face; `workloads` draws seeded
synthetic inputs.  Importing the package does not load the library; the
first call into `api` does, and fails loudly if it has not been built.
"""

__all__ = ["api", "workloads", "build"]
