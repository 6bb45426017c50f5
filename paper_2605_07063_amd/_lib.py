"""ctypes binding of libdr.so (the C ABI declared in include/dr_api.h).

Argument marshalling only: every step of the path runs in the library's
HIP kernels.  PyTorch supplies device memory and the current stream.  If the
shared library is missing the import fails loudly; there is no fallback.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdr.so")

DR_OK, DR_ERR_ARG, DR_ERR_DTYPE, DR_ERR_NOT_SPD, DR_ERR_NOT_CONVERGED = 0, 1, 2, 3, 4
DR_ERR_NONFINITE, DR_ERR_WORKSPACE, DR_ERR_HIP, DR_ERR_UNSUPPORTED, DR_ERR_TOO_LARGE = 5, 6, 7, 8, 9
DR_GRAM_NOALLOC_MAX_BYTES = 64 << 20
DR_INFO_NOT_CONVERGED, DR_INFO_NONFINITE = -2, -3
DR_F32, DR_BF16 = 0, 1
DR_RIDGE_ABS, DR_RIDGE_REL_TRACE = 0, 1
DR_SCORE_DIRECT, DR_SCORE_GIP, DR_SCORE_PIP = 0, 1, 2

c_i64, c_int, c_size, c_vp, c_float = ctypes.c_int64, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_float


class DrLayer(ctypes.Structure):
    _fields_ = [
        ("x", c_vp), ("ldx", c_i64),
        ("dy", c_vp), ("lddy", c_i64),
        ("p_in", c_vp), ("p_out", c_vp),
        ("d_in", c_i64), ("d_out", c_i64), ("k_in", c_i64), ("k_out", c_i64),
        ("col_offset", c_i64),
    ]


# name -> (restype, argtypes); the exported symbols of dr_api.h
SIGNATURES = {
    "dr_abi_version": (c_int, []),
    "dr_status_string": (ctypes.c_char_p, [c_int]),
    "dr_sketch_grads": (c_int, [ctypes.POINTER(DrLayer), c_int, c_i64, c_i64, c_vp, c_int, c_vp, c_i64,
                                c_vp, c_size, c_vp]),
    "dr_sketch_workspace_size": (c_size, [ctypes.POINTER(DrLayer), c_int, c_i64, c_i64, c_int]),
    "dr_gram": (c_int, [c_vp, c_i64, c_i64, c_vp, c_i64, c_i64, c_int, ctypes.POINTER(c_i64), c_int,
                        c_vp, c_vp, c_vp, c_vp, c_size, c_vp]),
    "dr_gram_workspace_size": (c_size, [c_i64, c_i64, ctypes.POINTER(c_i64), c_int, c_int]),
    "dr_gram_noalloc": (c_int, [c_vp, c_i64, c_i64, c_vp, c_i64, c_i64, c_int, ctypes.POINTER(c_i64), c_int,
                                c_vp, c_vp, c_vp, c_vp]),
    "dr_project_span": (c_int, [c_vp, c_vp, c_vp, c_i64, c_int, c_float, c_int, c_vp, c_vp, c_vp, c_vp,
                                c_vp, c_size, c_vp]),
    "dr_span_workspace_size": (c_size, [c_i64, c_int]),
    "dr_project_cone": (c_int, [c_vp, c_vp, c_vp, c_i64, c_int, c_int, c_float, c_vp, c_vp, c_vp, c_vp, c_vp,
                                c_vp, c_size, c_vp]),
    "dr_cone_workspace_size": (c_size, [c_i64, c_int]),
    "dr_select_topk": (c_int, [c_vp, c_i64, c_int, c_i64, c_vp, c_vp, c_vp, c_vp]),
    "dr_combine": (c_int, [c_vp, c_i64, c_i64, c_int, ctypes.POINTER(c_i64), c_int, c_vp, c_vp, c_vp, c_size,
                           c_vp]),
    "dr_combine_workspace_size": (c_size, [c_i64, ctypes.POINTER(c_i64), c_int]),
    "dr_project_simplex": (c_int, [c_vp, c_vp, c_vp, c_i64, c_int, c_int, c_float, c_vp, c_vp, c_vp, c_vp, c_vp,
                                   c_vp]),
    "dr_back_project": (c_int, [ctypes.POINTER(DrLayer), c_int, c_int, c_vp, c_vp, ctypes.POINTER(c_i64), c_vp, c_size,
                                c_vp]),
    "dr_backproject_workspace_size": (c_size, [ctypes.POINTER(DrLayer), c_int]),
    "dr_select_threshold": (c_int, [c_vp, c_i64, c_int, c_float, c_int, c_vp, c_vp, c_vp, c_vp, c_vp]),
    "dr_select_greedy": (c_int, [c_vp, c_vp, c_i64, c_int, c_i64, c_vp, c_vp, c_vp, c_vp, c_size, c_vp]),
    "dr_greedy_workspace_size": (c_size, [c_i64, c_int]),
    "dr_assemble_update": (c_int, [ctypes.POINTER(DrLayer), c_int, c_i64, c_i64, c_vp, c_int, c_vp, c_int, c_i64,
                                   ctypes.POINTER(ctypes.c_int32), c_vp, ctypes.POINTER(c_i64), c_vp, c_size, c_vp]),
    "dr_score_exact": (c_int, [ctypes.POINTER(DrLayer), c_int, c_i64, c_i64, c_i64, c_vp, c_int, c_int, c_vp, c_vp,
                               c_size, c_vp]),
    "dr_score_workspace_size": (c_size, [ctypes.POINTER(DrLayer), c_int, c_i64, c_i64, c_i64, c_int, c_int]),
    "dr_update_workspace_size": (c_size, [ctypes.POINTER(DrLayer), c_int, c_i64, c_i64, c_int]),
}

_lib = None


def load():
    """Load libdr.so (once) and declare every exported function's signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2605_07063_amd.build` "
            "(there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class DrError(RuntimeError):
    def __init__(self, fn, status):
        lib = load()
        msg = lib.dr_status_string(status).decode()
        super().__init__(f"{fn} returned {status} ({msg})")
        self.status = status


def check(fn, status):
    if status != DR_OK:
        raise DrError(fn, status)
