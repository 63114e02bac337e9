"""fp64 CPU oracle for the structured sketches (FJL, FFD, AFFD, AFJL, QK, QKH, AFJLQ, AFFDQ, AFJLF).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library never imports it; the two share no code.

The arithmetic lives in ``sk_oracle.c`` (plain C, double precision, textbook
Walsh-Hadamard transform, literal operator chains of the paper's equations
ailon_chazelle, fastfood, bami, frikadel and straight).  This module only
marshals numpy arrays into that library.  The kinds with the random-orthogonal
Kronecker pre-conditioner (QKH, AFJLQ, AFFDQ) are in ``qhaar.py`` (numpy, fp64);
the kind with the Fourier pre-conditioner (AFJLF) is in ``fourier.py`` (numpy,
fp64); the synthetic Hessian, the sketched HVP operator and the Arnoldi
iteration on it are in ``krylov.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sk_oracle.c")
_LIB = os.path.join(_HERE, "libsk_oracle.so")

KINDS = {"fjl": 0, "ffd": 1, "affd": 2, "afjl": 3, "qk": 4}
# kinds with the random-orthogonal Kronecker pre-conditioner (numpy, qhaar.py)
QKINDS = ("qkh", "afjlq", "affdq")
# kinds with the Fourier pre-conditioner (numpy, fourier.py)
FKINDS = ("afjlf",)
DTYPES = {"f32": 0, "bf16": 1}
STREAMS = {"sign": 1, "gauss": 2, "index": 3, "ffdperm": 4, "pi1": 5, "pi2": 6, "qka": 7, "qkb": 8, "qh": 9,
           "hvp": 10}


def build() -> str:
    """Compile the oracle with gcc (OpenMP, -O2, strict IEEE: no fast-math)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off", "-o", _LIB, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        u32, u64, i32, i64 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64
        P = ctypes.c_void_p
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_sign.argtypes = [u64, u32, u64]
        L.orc_sign.restype = ctypes.c_int
        L.orc_gauss.argtypes = [u64, u32, u32, u64]
        L.orc_gauss.restype = ctypes.c_double
        L.orc_index.argtypes = [u64, u32, u64, u64]
        L.orc_index.restype = u64
        L.orc_perm.argtypes = [u64, u32, u32, u32, u32, u32]
        L.orc_perm.restype = u32
        L.orc_perm_inv.argtypes = [u64, u32, u32, u32, u32, u32]
        L.orc_perm_inv.restype = u32
        L.orc_kron_shapes.argtypes = [u64, P]
        L.orc_kron_shapes.restype = ctypes.c_int
        L.orc_fwht.argtypes = [P, u64]
        L.orc_padded.argtypes = [u64, u64]
        L.orc_padded.restype = u64
        L.orc_round_bf16.argtypes = [ctypes.c_double]
        L.orc_round_bf16.restype = ctypes.c_double
        L.orc_digit_perm_table.argtypes = [u64, u32, u32, u64, P]
        L.orc_apply.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P, P, P, i64, u64, i64,
                                ctypes.c_int, P, P, ctypes.c_int, ctypes.c_int]
        L.orc_apply.restype = ctypes.c_int
        L.orc_apply_T.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P, P, P, i64, u64, i64,
                                  P, P, ctypes.c_int, ctypes.c_int]
        L.orc_apply_T.restype = ctypes.c_int
        L.orc_signs.argtypes = [u64, u32, u64, u64, P]
        L.orc_gauss_range.argtypes = [u64, u32, u32, u64, u64, P]
        L.orc_index_range.argtypes = [u64, u32, u64, u64, u64, P]
        L.orc_perm_table.argtypes = [u64, u32, u32, u32, u32, P]
        L.orc_hvp_sign.argtypes = [u64, u32, u32, u64]
        L.orc_hvp_sign.restype = ctypes.c_int
        L.orc_hvp_signs.argtypes = [u64, u32, u32, u64, u64, P]
        L.orc_hvp_dots.argtypes = [u64, u32, ctypes.c_int, u64, P, P]
        L.orc_hvp_combine.argtypes = [u64, u32, ctypes.c_int, u64, ctypes.c_double, P, P, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# --- random streams ---------------------------------------------------------
def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    o = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(o))
    return o


def signs(seed: int, layer: int, start: int, count: int) -> np.ndarray:
    o = np.zeros(count, dtype=np.int8)
    lib().orc_signs(seed, layer, start, count, _ptr(o))
    return o


def gauss(seed: int, layer: int, stream: str, start: int, count: int) -> np.ndarray:
    o = np.zeros(count, dtype=np.float64)
    lib().orc_gauss_range(seed, layer, STREAMS[stream], start, count, _ptr(o))
    return o


def indices(seed: int, layer: int, start: int, count: int, np_len: int) -> np.ndarray:
    o = np.zeros(count, dtype=np.uint64)
    lib().orc_index_range(seed, layer, start, count, np_len, _ptr(o))
    return o


def perm(seed: int, layer: int, stream: str, pid: int, w: int) -> np.ndarray:
    o = np.zeros(1 << w, dtype=np.uint32)
    lib().orc_perm_table(seed, layer, STREAMS[stream], pid, w, _ptr(o))
    return o


def perm_inv(seed: int, layer: int, stream: str, pid: int, w: int, y: int) -> int:
    return int(lib().orc_perm_inv(seed, layer, STREAMS[stream], pid, w, y))


def digit_perm(seed: int, layer: int, stream: str, np_len: int) -> np.ndarray:
    o = np.zeros(np_len, dtype=np.uint64)
    lib().orc_digit_perm_table(seed, layer, STREAMS[stream], np_len, _ptr(o))
    return o


def kron_shapes(n: int) -> tuple:
    o = np.zeros(8, dtype=np.uint64)
    k = lib().orc_kron_shapes(n, _ptr(o))
    return tuple(int(v) for v in o[:k])


def padded(n: int, d: int) -> int:
    return int(lib().orc_padded(n, d))


def fwht(v: np.ndarray) -> np.ndarray:
    a = np.array(v, dtype=np.float64, copy=True)
    lib().orc_fwht(_ptr(a), a.size)
    return a


def round_bf16(v: float) -> float:
    return float(lib().orc_round_bf16(v))


# --- sketches ---------------------------------------------------------------
def _shape_arrays(shapes):
    rows = np.array([s[0] for s in shapes], dtype=np.int64)
    cols = np.array([s[1] for s in shapes], dtype=np.int64)
    da = np.array([s[2] if len(s) > 2 else 0 for s in shapes], dtype=np.int32)
    db = np.array([s[3] if len(s) > 3 else 0 for s in shapes], dtype=np.int32)
    return rows, cols, da, db


def apply(kind: str, shapes, D: int, seed: int, xs, dtype: str = "f32", layer0: int = 0,
          nthreads: int = 0, qk_bf16: bool = False) -> np.ndarray:
    """Forward sketch y = S x of a batch.

    shapes: per layer (rows, cols[, dA, dB]); xs: per layer an array [batch, rows*cols]
    (float32 for "f32", uint16 bf16 bit patterns for "bf16").  Layers carry RNG
    layer ids layer0, layer0+1, ...  Returns fp64 [batch, D]."""
    if kind in QKINDS:
        from . import qhaar
        return qhaar.apply(kind, shapes, D, seed, xs, dtype, layer0)
    if kind in FKINDS:
        from . import fourier
        return fourier.apply(kind, shapes, D, seed, xs, dtype, layer0, nthreads)
    rows, cols, da, db = _shape_arrays(shapes)
    want = np.float32 if dtype == "f32" else np.uint16
    arrs = [np.ascontiguousarray(x, dtype=want) for x in xs]
    batch = arrs[0].shape[0]
    for a, r, c in zip(arrs, rows, cols):
        assert a.shape == (batch, r * c), (a.shape, r, c)
    ptrs = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    y = np.zeros((batch, D), dtype=np.float64)
    rc = lib().orc_apply(KINDS[kind], layer0, len(arrs), _ptr(rows), _ptr(cols), _ptr(da), _ptr(db), D, seed,
                         batch, DTYPES[dtype], ptrs, _ptr(y), nthreads, int(qk_bf16))
    if rc != 0:
        raise RuntimeError(f"orc_apply failed ({rc})")
    return y


def apply_T(kind: str, shapes, D: int, seed: int, z: np.ndarray, layer0: int = 0, nthreads: int = 0,
            qk_bf16: bool = False, theta0=None):
    """Transpose S^T z of a batch z [batch, D]; returns a list of fp64 [batch, rows*cols].
    With theta0 (a list of per-layer vectors or None entries) the result is theta0 + S^T z."""
    if kind in QKINDS:
        from . import qhaar
        return qhaar.apply_T(kind, shapes, D, seed, z, layer0, theta0)
    if kind in FKINDS:
        from . import fourier
        return fourier.apply_T(kind, shapes, D, seed, z, layer0, theta0, nthreads)
    rows, cols, da, db = _shape_arrays(shapes)
    z = np.ascontiguousarray(z, dtype=np.float64)
    batch = z.shape[0]
    outs = [np.zeros((batch, int(r * c)), dtype=np.float64) for r, c in zip(rows, cols)]
    ptrs = (ctypes.c_void_p * len(outs))(*[o.ctypes.data for o in outs])
    rc = lib().orc_apply_T(KINDS[kind], layer0, len(outs), _ptr(rows), _ptr(cols), _ptr(da), _ptr(db), D, seed,
                           batch, _ptr(z), ptrs, nthreads, int(qk_bf16))
    if rc != 0:
        raise RuntimeError(f"orc_apply_T failed ({rc})")
    if theta0 is not None:
        for o, t in zip(outs, theta0):
            if t is not None:
                o += np.asarray(t, dtype=np.float64)[None, :]
    return outs
