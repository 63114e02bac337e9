"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point declared in include/*.h, and rejects invalid arguments
before touching a device."""
import ctypes
import os
import re

import pytest

from paper_2402_03994_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if h.endswith(".h"):
            src = open(os.path.join(ROOT, "include", h)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b((?:sketch|sk_hvp)_[a-z_T]+)\s*\(", src))
    return sorted(names)


def test_header_and_binding_agree():
    assert declared_functions() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = _lib.load()
    for name in declared_functions():
        assert hasattr(L, name), name


def shapes(*ss):
    arr = (_lib.LayerShape * len(ss))()
    for i, s in enumerate(ss):
        arr[i].rows, arr[i].cols = s[0], s[1]
        arr[i].qk_da = s[2] if len(s) > 2 else 0
        arr[i].qk_db = s[3] if len(s) > 3 else 0
    return arr


@pytest.mark.parametrize("kind,shp,D,flags,code", [
    (9, [(1, 10)], 64, 0, -1),            # unknown kind
    (3, [(1, 10)], 63, 0, -1),            # D not a power of two
    (3, [(1, 10)], 0, 0, -1),
    (3, [(1, 10)], 8, 0, -5),             # below the kernels' minimum
    (3, [(1, 10)], 1 << 21, 0, -5),       # above the kernels' maximum
    (3, [(0, 10)], 64, 0, -1),            # empty layer
    (3, [(1, 10)], 64, 2, -1),            # unknown flags
    (4, [(4, 5, 2, 2)], 5, 0, -1),        # QK: sum dA*dB != D
    (4, [(4, 5, 5, 2)], 10, 0, -1),       # QK: dA > rows
    (4, [(4, 5, 0, 2)], 0, 0, -1),        # QK: dA < 1
    (5, [(1, 10)], 1024, 0, -5),          # QKH: D below 2048
    (6, [(1, 10)], 1 << 21, 0, -5),       # AFJLQ: D above 2^20
    (6, [(1, 10)], 3000, 0, -1),          # AFJLQ: D not a power of two
    (10, [(1, 10)], 4096, 0, -1),         # unknown kind
    (7, [(1, 1 << 27)], 4096, 0, -5),     # AFFDQ: N' above 2^26
    (0, [(2, (1 << 31) + 1)], 4096, 0, -5),  # FJL: N' above 2^32 (positions are 32-bit words)
    (8, [(1, 10)], 1024, 0, -5),          # AFJLF: D below 2048
    (8, [(1, 40000)], 1 << 17, 0, -5),    # AFJLF: N' = D with more than 16384 entries and 2^15 outputs per residue
    (8, [(1, 1 << 21)], 1 << 20, 0, -5),  # AFJLF: N' = 2D: 2^18 outputs per residue
    (9, [(1, 10)], 4096, 0, -1),          # unknown kind
])
def test_create_rejects_invalid_arguments(kind, shp, D, flags, code):
    L = _lib.load()
    h = ctypes.c_void_p(1234)
    rc = L.sketch_create(kind, shapes(*shp), len(shp), D, 0, flags, 0, ctypes.byref(h))
    assert rc == code, L.sketch_last_error()
    assert h.value is None  # *out cleared on failure
    assert len(L.sketch_last_error()) > 0


def test_null_arguments():
    L = _lib.load()
    assert L.sketch_create(3, None, 1, 64, 0, 0, 0, ctypes.byref(ctypes.c_void_p())) == -1
    assert L.sketch_create(3, shapes((1, 4)), 1, 64, 0, 0, 0, None) == -1
    assert L.sketch_apply(None, None, 0, 1, None, 0, 1, 0, None) == -1
    assert L.sketch_apply_T(None, None, 1, None, 0, None, 0, 1, None) == -1
    assert L.sketch_query(None, None) == -1
    L.sketch_destroy(None)  # no-op


def test_status_strings():
    L = _lib.load()
    for code in [0, -1, -2, -3, -4, -5]:
        assert L.sketch_status_string(code).decode() != "unknown status"


def test_hvp_entry_points_reject_invalid_arguments():
    L = _lib.load()
    lam = (ctypes.c_float * 2)(1.0, 2.0)
    h = ctypes.c_void_p(99)
    assert L.sk_hvp_create(shapes((1, 10)), 1, 0, lam, 0.0, 0, 1, 0, ctypes.byref(h)) == -1   # rank 0
    assert h.value is None
    assert L.sk_hvp_create(shapes((1, 10)), 1, 33, lam, 0.0, 0, 1, 0, ctypes.byref(h)) == -1  # rank > 32
    assert L.sk_hvp_create(shapes((1, 10)), 1, 2, None, 0.0, 0, 1, 0, ctypes.byref(h)) == -1  # no lambdas
    assert L.sk_hvp_create(shapes((1, 10)), 1, 2, lam, 0.0, 0, 0, 0, ctypes.byref(h)) == -1   # max_batch 0
    assert L.sk_hvp_create(shapes((0, 10)), 1, 2, lam, 0.0, 0, 1, 0, ctypes.byref(h)) == -1   # empty layer
    assert L.sk_hvp_apply(None, None, 1, None, None) == -1
    assert L.sketch_hvp(None, None, None, 1, None, None) == -1
    assert L.sketch_arnoldi(None, None, None, 4, None, None, None) == -1
    assert L.sketch_arnoldi_step(None, 16, 0, None, 4, None, None) == -1
    assert L.sketch_arnoldi_work_floats(0, 4) == 0
    assert L.sketch_arnoldi_work_floats(4096, 10) == 2 * 12 + 12 + 4
    L.sk_hvp_destroy(None)  # no-op


def test_id_search_rejects_invalid_arguments():
    L = _lib.load()
    res = _lib.IdResult()
    assert L.sketch_id_search(None, None, None, 1, 0.9, 0.05, 4, 4, None, None, None, ctypes.byref(res), None) == -1
    assert L.sketch_id_search_work_floats(0) == 0
    assert L.sketch_id_search_work_floats(1024) == 6 * 1024 + 32
