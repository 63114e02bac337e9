"""ctypes declarations of the C ABI in include/sketch.h and include/sketch_hvp.h (argument
marshalling only)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsketch.so")

SK_FJL, SK_FFD, SK_AFFD, SK_AFJL, SK_QK, SK_QKH, SK_AFJLQ, SK_AFFDQ, SK_AFJLF = range(9)
SK_F32, SK_BF16 = 0, 1
STATUS = {0: "SK_OK", -1: "SK_EINVAL", -2: "SK_EDTYPE", -3: "SK_ENOMEM", -4: "SK_EHIP", -5: "SK_EUNSUPPORTED"}
STREAMS = {"sign": 1, "gauss": 2, "index": 3, "ffdperm": 4, "pi1": 5, "pi2": 6, "qka": 7, "qkb": 8, "qh": 9,
           "hvp": 10}
EXPORTS = ("sketch_create", "sketch_apply", "sketch_apply_noalloc", "sketch_apply_T", "sketch_destroy", "sketch_query",
           "sketch_debug_stream", "sketch_profile", "sketch_profile_read", "sketch_last_error",
           "sketch_status_string", "sk_hvp_create", "sk_hvp_apply", "sk_hvp_destroy", "sketch_hvp",
           "sketch_arnoldi_work_floats", "sketch_arnoldi_step", "sketch_arnoldi", "sk_hvp_profile",
           "sk_hvp_profile_read", "sketch_id_search_work_floats", "sketch_id_search")
HVP_PROF_CLASSES = ["hvp_dots", "hvp_combine", "arnoldi_orth"]
HVP_MAX_RANK = 32
PROF_CLASSES = ["afjl_fold", "afjl_tail", "fwht", "prolog", "affd_fold", "gather", "ffd", "qk", "other",
                "affd_rows", "qk_xb", "qh_first", "qh_second", "qh_t", "ffd_t", "ff_rows", "ff_res",
                "ff_small", "fjl_t"]


class IdResult(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int64), ("status", ctypes.c_int32), ("rounds", ctypes.c_int32),
                ("L0", ctypes.c_double)]


class LayerShape(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("qk_da", ctypes.c_int32),
                ("qk_db", ctypes.c_int32)]


class Info(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("D", ctypes.c_int64),
                ("seed", ctypes.c_uint64), ("total_numel", ctypes.c_int64), ("total_padded", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_int64), ("rng_version", ctypes.c_int32), ("device", ctypes.c_int32)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libsketch.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2402_03994_amd.build` "
                           "(or __graft_entry__.build()); there is no non-HIP fallback")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u32, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
    L.sketch_create.argtypes = [ctypes.c_int, ctypes.POINTER(LayerShape), i32, i64, u64, u32, i32,
                                ctypes.POINTER(P)]
    L.sketch_create.restype = ctypes.c_int
    L.sketch_apply.argtypes = [P, ctypes.POINTER(P), ctypes.c_int, i64, P, i32, i32, i32, P]
    L.sketch_apply.restype = ctypes.c_int
    L.sketch_apply_noalloc.argtypes = [P, ctypes.POINTER(P), ctypes.c_int, i64, P, i32, i32, i32, P]
    L.sketch_apply_noalloc.restype = ctypes.c_int
    L.sketch_apply_T.argtypes = [P, P, i64, ctypes.POINTER(P), ctypes.c_int, ctypes.POINTER(P), i32, i32, P]
    L.sketch_apply_T.restype = ctypes.c_int
    L.sketch_destroy.argtypes = [P]
    L.sketch_destroy.restype = None
    L.sketch_query.argtypes = [P, ctypes.POINTER(Info)]
    L.sketch_query.restype = ctypes.c_int
    L.sketch_debug_stream.argtypes = [P, i32, i32, u64, u64, u64, P]
    L.sketch_debug_stream.restype = ctypes.c_int
    L.sketch_profile.argtypes = [P, ctypes.c_uint32]
    L.sketch_profile.restype = ctypes.c_int
    L.sketch_profile_read.argtypes = [P, P, P, P]
    L.sketch_profile_read.restype = ctypes.c_int
    L.sketch_last_error.argtypes = []
    L.sketch_last_error.restype = ctypes.c_char_p
    L.sketch_status_string.argtypes = [ctypes.c_int]
    L.sketch_status_string.restype = ctypes.c_char_p
    f32 = ctypes.c_float
    L.sk_hvp_create.argtypes = [ctypes.POINTER(LayerShape), i32, i32, P, f32, u64, i64, i32, ctypes.POINTER(P)]
    L.sk_hvp_create.restype = ctypes.c_int
    L.sk_hvp_apply.argtypes = [P, ctypes.POINTER(P), i64, ctypes.POINTER(P), P]
    L.sk_hvp_apply.restype = ctypes.c_int
    L.sk_hvp_destroy.argtypes = [P]
    L.sk_hvp_destroy.restype = None
    L.sketch_hvp.argtypes = [P, P, P, i64, P, P]
    L.sketch_hvp.restype = ctypes.c_int
    L.sketch_arnoldi_work_floats.argtypes = [i64, i32]
    L.sketch_arnoldi_work_floats.restype = i64
    L.sketch_arnoldi_step.argtypes = [P, i64, i32, P, i32, P, P]
    L.sketch_arnoldi_step.restype = ctypes.c_int
    L.sketch_arnoldi.argtypes = [P, P, P, i32, P, P, P]
    L.sketch_arnoldi.restype = ctypes.c_int
    L.sk_hvp_profile.argtypes = [P, u32]
    L.sk_hvp_profile.restype = ctypes.c_int
    L.sk_hvp_profile_read.argtypes = [P, P, P, P]
    L.sk_hvp_profile_read.restype = ctypes.c_int
    L.sketch_id_search_work_floats.argtypes = [i64]
    L.sketch_id_search_work_floats.restype = i64
    L.sketch_id_search.argtypes = [P, P, ctypes.POINTER(P), i64, f32, f32, i32, i32, P, P, P,
                                   ctypes.POINTER(IdResult), P]
    L.sketch_id_search.restype = ctypes.c_int
    _lib = L
    return L


class SketchError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


def check(rc: int) -> None:
    if rc != 0:
        raise SketchError(rc, load().sketch_last_error().decode())
