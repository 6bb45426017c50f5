"""The C ABI library loads on a host without a GPU, exports every symbol the
header declares, and rejects invalid arguments before any HIP call."""

import ctypes
import os
import re

import pytest

from paper_2605_07063_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dr_api.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2605_07063_amd import build
        build.build()
    return _lib.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\*?\s+\*?(dr_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported_and_bound(lib):
    names = declared_functions()
    assert len(names) >= 12
    for nm in names:
        assert hasattr(lib, nm), nm
        assert nm in _lib.SIGNATURES, f"{nm} missing from the Python binding"
    assert set(_lib.SIGNATURES) == set(names)


def test_version_and_status_strings(lib):
    assert lib.dr_abi_version() == 1
    for code in range(10):
        assert lib.dr_status_string(code) != b"unknown status"
    assert lib.dr_status_string(0) == b"ok"


FAKE = 0x1000_0000   # 16-byte aligned, never dereferenced: validation fails first


def layer(**kw):
    d = dict(x=FAKE, ldx=256, dy=FAKE, lddy=256, p_in=FAKE, p_out=FAKE, d_in=256, d_out=256, k_in=16, k_out=16,
             col_offset=0)
    d.update(kw)
    return _lib.DrLayer(**d)


def sketch_call(lib, layers, N=4, T=8, dtype=_lib.DR_F32, S=FAKE, ldS=256, ws=None, wsb=0):
    arr = (_lib.DrLayer * max(1, len(layers)))(*layers)
    return lib.dr_sketch_grads(arr, len(layers), N, T, None, dtype, S, ldS, ws, wsb, None)


def test_sketch_argument_errors(lib):
    E = _lib
    assert sketch_call(lib, []) == E.DR_ERR_ARG
    assert sketch_call(lib, [layer(k_in=48)]) == E.DR_ERR_ARG
    assert sketch_call(lib, [layer(k_out=8)]) == E.DR_ERR_ARG
    assert sketch_call(lib, [layer()], dtype=7) == E.DR_ERR_DTYPE
    assert sketch_call(lib, [layer(d_in=254, ldx=256)]) == E.DR_ERR_ARG        # not a multiple of 4
    assert sketch_call(lib, [layer(ldx=128)]) == E.DR_ERR_ARG                   # ld < d
    assert sketch_call(lib, [layer(x=FAKE + 4)]) == E.DR_ERR_ARG                # misaligned
    assert sketch_call(lib, [layer(col_offset=250)]) == E.DR_ERR_ARG            # block beyond ldS
    assert sketch_call(lib, [layer()], N=-1) == E.DR_ERR_ARG
    assert sketch_call(lib, [layer()], S=None) == E.DR_ERR_ARG
    assert sketch_call(lib, [layer(d_in=12, ldx=12)], dtype=E.DR_BF16) == E.DR_ERR_ARG   # bf16 needs multiples of 8
    assert sketch_call(lib, [layer()], N=0) == E.DR_OK                          # nothing to do, no HIP call


def test_sketch_workspace_query_and_check(lib):
    layers = [layer(d_in=2048, d_out=2048, ldx=2048, lddy=2048, k_in=64, k_out=64, col_offset=4096 * i)
              for i in range(8)]
    arr = (_lib.DrLayer * 8)(*layers)
    ws = lib.dr_sketch_workspace_size(arr, 8, 72, 512, _lib.DR_BF16)
    assert ws > 0 and ws % 4 == 0
    assert ws == lib.dr_sketch_workspace_size(arr, 8, 72, 512, _lib.DR_BF16)   # deterministic plan
    st = lib.dr_sketch_grads(arr, 8, 72, 512, None, _lib.DR_BF16, FAKE, 32768, None, 0, None)
    assert st == _lib.DR_ERR_WORKSPACE
    st = lib.dr_sketch_grads(arr, 8, 72, 512, None, _lib.DR_BF16, FAKE, 32768, FAKE, ws - 1, None)
    assert st == _lib.DR_ERR_WORKSPACE


def goff(*v):
    return (ctypes.c_int64 * len(v))(*v)


def test_gram_argument_errors(lib):
    E = _lib
    g = goff(0, 64)
    call = lambda **kw: lib.dr_gram(kw.get("G", FAKE), kw.get("n", 8), kw.get("ldG", 64), kw.get("Gt", FAKE),
                                    kw.get("m", 2), kw.get("ldGt", 64), kw.get("dtype", E.DR_F32),
                                    kw.get("goff", g), kw.get("P", 1), FAKE, FAKE, FAKE, kw.get("ws", FAKE),
                                    kw.get("wsb", 1 << 30), None)
    assert call(P=0) == E.DR_ERR_ARG
    assert call(m=0) == E.DR_ERR_ARG
    assert call(ldG=32) == E.DR_ERR_ARG
    assert call(goff=goff(8, 4), P=1) == E.DR_ERR_ARG
    assert call(goff=goff(0, 6), P=1) == E.DR_ERR_ARG          # group edge not a multiple of 4
    assert call(dtype=3) == E.DR_ERR_DTYPE
    assert call(ws=None) == E.DR_ERR_WORKSPACE
    assert call(wsb=16) == E.DR_ERR_WORKSPACE
    assert lib.dr_gram_workspace_size(64, 8, goff(0, 32768), 1, E.DR_F32) > 0


def test_gram_noalloc_argument_errors_and_scratch_limit(lib):
    """The no-allocation Gram validates like dr_gram, and refuses a problem
    whose workspace exceeds its fixed scratch, all before any HIP call."""
    E = _lib
    g = goff(0, 64)
    call = lambda **kw: lib.dr_gram_noalloc(FAKE, kw.get("n", 8), kw.get("ldG", 64), FAKE, 2, kw.get("ldGt", 64),
                                            kw.get("dtype", E.DR_F32), kw.get("goff", g), kw.get("P", 1), FAKE, FAKE,
                                            FAKE, None)
    assert call(P=0) == E.DR_ERR_ARG
    assert call(ldG=32) == E.DR_ERR_ARG
    assert call(dtype=3) == E.DR_ERR_DTYPE
    n, cols = 8000, 1 << 20
    need = lib.dr_gram_workspace_size(n, 2, goff(0, cols), 1, E.DR_F32)
    assert need > E.DR_GRAM_NOALLOC_MAX_BYTES
    assert call(n=n, ldG=cols, ldGt=cols, goff=goff(0, cols)) == E.DR_ERR_TOO_LARGE
    assert lib.dr_status_string(E.DR_ERR_TOO_LARGE).startswith(b"problem needs more scratch")
    hdr = open(HEADER).read()
    assert re.search(r"#define DR_GRAM_NOALLOC_MAX_BYTES \(\(size_t\)64 << 20\)", hdr)


def test_solver_and_select_argument_errors(lib):
    E = _lib
    span = lambda n=8, P=1, lam=0.0, mode=0: lib.dr_project_span(FAKE, FAKE, FAKE, n, P, lam, mode, FAKE, FAKE,
                                                                 FAKE, FAKE, None, 0, None)
    assert span(n=-1) == E.DR_ERR_ARG
    assert span(lam=-1.0) == E.DR_ERR_ARG
    assert span(lam=float("nan")) == E.DR_ERR_ARG
    assert span(mode=5) == E.DR_ERR_ARG
    assert span(n=257) == E.DR_ERR_WORKSPACE                 # the blocked path needs its workspace
    assert span(n=65537) == E.DR_ERR_UNSUPPORTED
    assert lib.dr_span_workspace_size(256, 1) == 0
    assert lib.dr_span_workspace_size(16384, 3) >= 16384 * 16384 * 4
    assert span(P=0) == E.DR_OK
    cone = lambda n=8, P=1, it=10, tol=0.0: lib.dr_project_cone(FAKE, FAKE, FAKE, n, P, it, tol, FAKE, FAKE, FAKE,
                                                                FAKE, FAKE, None, 0, None)
    assert cone(it=-1) == E.DR_ERR_ARG
    assert cone(n=300) == E.DR_ERR_UNSUPPORTED
    assert cone(tol=float("nan")) == E.DR_ERR_ARG
    assert cone(P=0) == E.DR_OK
    top = lambda n=8, P=1, k=2: lib.dr_select_topk(FAKE, n, P, k, FAKE, None, FAKE, None)
    assert top(k=9) == E.DR_ERR_ARG
    assert top(k=-1) == E.DR_ERR_ARG
    assert top(P=0) == E.DR_OK
    g = goff(0, 64)
    assert lib.dr_combine(FAKE, 8, 64, 9, g, 1, FAKE, FAKE, None, 0, None) == E.DR_ERR_DTYPE
    assert lib.dr_combine(FAKE, 8, 32, E.DR_F32, g, 1, FAKE, FAKE, None, 0, None) == E.DR_ERR_ARG
    assert lib.dr_combine_workspace_size(8, g, 1) == 0          # n <= 256: one pass, no partials
    need = lib.dr_combine_workspace_size(1000, g, 1)
    assert need > 0
    assert lib.dr_combine(FAKE, 1000, 64, E.DR_F32, g, 1, FAKE, FAKE, None, 0, None) == E.DR_ERR_WORKSPACE


def update_call(lib, layers, n=4, T=8, dtype=_lib.DR_F32, w=FAKE, P=1, ldw=4, gol=None, U=FAKE, offs=None,
                ws=None, wsb=0):
    arr = (_lib.DrLayer * max(1, len(layers)))(*layers)
    if offs is None:
        offs = [0] * max(1, len(layers))
    oa = (ctypes.c_int64 * len(offs))(*offs)
    ga = None if gol is None else (ctypes.c_int32 * len(gol))(*gol)
    return lib.dr_assemble_update(arr, len(layers), n, T, None, dtype, w, P, ldw, ga, U, oa, ws, wsb, None)


def test_update_argument_errors(lib):
    E = _lib
    assert update_call(lib, []) == E.DR_ERR_ARG
    assert update_call(lib, [layer()], dtype=5) == E.DR_ERR_DTYPE
    assert update_call(lib, [layer()], n=-1) == E.DR_ERR_ARG
    assert update_call(lib, [layer()], ldw=3) == E.DR_ERR_ARG                   # ldw < n
    assert update_call(lib, [layer()], w=None) == E.DR_ERR_ARG
    assert update_call(lib, [layer()], U=None) == E.DR_ERR_ARG
    assert update_call(lib, [layer()], P=0) == E.DR_ERR_ARG
    assert update_call(lib, [layer(), layer()], P=2, gol=[0, 2]) == E.DR_ERR_ARG   # group row out of range
    assert update_call(lib, [layer()], offs=[-4]) == E.DR_ERR_ARG
    assert update_call(lib, [layer(d_in=254, ldx=256)]) == E.DR_ERR_ARG
    assert update_call(lib, [layer(d_in=12, ldx=12)], dtype=E.DR_BF16) == E.DR_ERR_ARG
    assert update_call(lib, [layer(dy=FAKE + 8)]) == E.DR_ERR_ARG
    # one example spanning 4 GiB of rows cannot be addressed with 32-bit offsets
    big = layer(d_in=8192, ldx=8192, d_out=8192, lddy=8192)
    assert update_call(lib, [big], T=1 << 18, dtype=E.DR_BF16) == E.DR_ERR_UNSUPPORTED
    # the projector fields are ignored
    assert update_call(lib, [layer(p_in=None, p_out=None, k_in=3, k_out=0)]) == E.DR_ERR_WORKSPACE


def test_update_workspace_query(lib):
    layers = [layer(d_in=2048, d_out=2048, ldx=2048, lddy=2048) for _ in range(8)]
    arr = (_lib.DrLayer * 8)(*layers)
    ws = lib.dr_update_workspace_size(arr, 8, 64, 512, _lib.DR_BF16)
    assert ws > 0 and ws % 256 == 0
    assert update_call(lib, layers, n=64, T=512, ldw=64, dtype=_lib.DR_BF16, ws=FAKE, wsb=ws - 1) == \
        _lib.DR_ERR_WORKSPACE
    assert lib.dr_update_workspace_size(arr, 8, -1, 512, _lib.DR_BF16) == 0


def test_threshold_and_greedy_argument_errors(lib):
    E = _lib
    cnt, info = FAKE, FAKE
    assert lib.dr_select_threshold(FAKE, -1, 1, 0.0, 1, None, cnt, None, info, None) == E.DR_ERR_ARG
    assert lib.dr_select_threshold(FAKE, 8, 1, float("nan"), 1, None, cnt, None, info, None) == E.DR_ERR_ARG
    assert lib.dr_select_threshold(FAKE, 8, 1, 0.0, 1, None, None, None, info, None) == E.DR_ERR_ARG
    assert lib.dr_select_threshold(None, 8, 1, 0.0, 1, None, cnt, None, info, None) == E.DR_ERR_ARG
    assert lib.dr_select_threshold(FAKE, 8, 0, 0.0, 1, None, cnt, None, info, None) == E.DR_OK
    ws = lib.dr_greedy_workspace_size(100, 2)
    assert ws >= 2 * 100 * 4
    assert lib.dr_select_greedy(FAKE, FAKE, 100, 2, 101, FAKE, None, info, FAKE, ws, None) == E.DR_ERR_ARG
    assert lib.dr_select_greedy(FAKE, FAKE, 16385, 1, 5, FAKE, None, info, FAKE, 1 << 30, None) == \
        E.DR_ERR_UNSUPPORTED
    assert lib.dr_select_greedy(FAKE, FAKE, 100, 2, 5, FAKE, None, info, FAKE, ws - 1, None) == E.DR_ERR_WORKSPACE
    assert lib.dr_select_greedy(FAKE, FAKE, 100, 2, 5, None, None, info, FAKE, ws, None) == E.DR_ERR_ARG


def test_score_argument_errors(lib):
    E = _lib
    arr = (_lib.DrLayer * 1)(layer(ldx=256, lddy=256))
    call = lambda **kw: lib.dr_score_exact(arr, kw.get("nl", 1), kw.get("n", 4), kw.get("m", 2), kw.get("T", 8), None,
                                           kw.get("dtype", E.DR_BF16), kw.get("method", E.DR_SCORE_PIP),
                                           kw.get("s", FAKE), kw.get("ws", None), kw.get("wsb", 0), None)
    assert call(m=0) == E.DR_ERR_ARG
    assert call(method=7) == E.DR_ERR_ARG
    assert call(dtype=E.DR_F32) == E.DR_ERR_UNSUPPORTED
    assert call(dtype=9) == E.DR_ERR_DTYPE
    assert call(s=None) == E.DR_ERR_ARG
    assert call(nl=0) == E.DR_ERR_ARG
    for meth in (E.DR_SCORE_DIRECT, E.DR_SCORE_GIP, E.DR_SCORE_PIP):
        ws = lib.dr_score_workspace_size(arr, 1, 4, 2, 8, E.DR_BF16, meth)
        assert ws > 0
        assert call(method=meth, ws=FAKE, wsb=ws - 1) == E.DR_ERR_WORKSPACE


def test_simplex_and_backprojection_argument_errors(lib):
    E = _lib
    args = lambda **kw: (kw.get("K", FAKE), FAKE, FAKE, kw.get("n", 8), kw.get("P", 1), kw.get("it", 10),
                         kw.get("tol", 0.0), FAKE, FAKE, FAKE, kw.get("res", FAKE), FAKE, None)
    assert lib.dr_project_simplex(*args(n=-1)) == E.DR_ERR_ARG
    assert lib.dr_project_simplex(*args(it=-1)) == E.DR_ERR_ARG
    assert lib.dr_project_simplex(*args(tol=float("nan"))) == E.DR_ERR_ARG
    assert lib.dr_project_simplex(*args(res=None)) == E.DR_ERR_ARG
    assert lib.dr_project_simplex(*args(K=None)) == E.DR_ERR_ARG
    assert lib.dr_project_simplex(*args(n=257)) == E.DR_ERR_UNSUPPORTED
    assert lib.dr_project_simplex(*args(P=0)) == E.DR_OK
    L = [layer(k_in=16, k_out=16)]
    arr = (_lib.DrLayer * 1)(*L)
    offs = (ctypes.c_int64 * 1)(0)
    ws = lib.dr_backproject_workspace_size(arr, 1)
    assert ws >= 16 * 256 * 4
    assert lib.dr_back_project(arr, 1, 9, FAKE, FAKE, offs, FAKE, ws, None) == E.DR_ERR_DTYPE
    assert lib.dr_back_project(arr, 1, E.DR_F32, None, FAKE, offs, FAKE, ws, None) == E.DR_ERR_ARG
    assert lib.dr_back_project(arr, 1, E.DR_F32, FAKE, FAKE, offs, FAKE, ws - 1, None) == E.DR_ERR_WORKSPACE
    big = (_lib.DrLayer * 1)(layer(k_in=128))
    assert lib.dr_back_project(big, 1, E.DR_F32, FAKE, FAKE, offs, FAKE, 1 << 30, None) == E.DR_ERR_ARG


def test_probe_library_exports_its_header():
    """The measurement probes' library exports what dr_probe.h declares and
    rejects invalid arguments before any HIP call."""
    from paper_2605_07063_amd import build
    if not os.path.exists(build.PROBE_LIB):
        build.build()
    plib = ctypes.CDLL(build.PROBE_LIB)
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "dr_probe.h")).read(), flags=re.S)
    names = re.findall(r"^\s*int\s+(dr_probe_\w+)\s*\(", text, flags=re.M)
    assert sorted(names) == ["dr_probe_mfma", "dr_probe_read"]
    for nm in names:
        assert hasattr(plib, nm)
    plib.dr_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    plib.dr_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    assert plib.dr_probe_read(FAKE, 24, FAKE, 16, None) == 1        # not a multiple of 16 bytes
    assert plib.dr_probe_read(FAKE, 4096, FAKE, 0, None) == 1
    assert plib.dr_probe_mfma(1, 0, FAKE, 16, None) == 1
    assert plib.dr_probe_mfma(1, 16, None, 16, None) == 1
