"""Thin Python binding of the sketch C ABI for torch tensors on a ROCm device.

Only argument marshalling lives here: every step of a sketch runs in the HIP
kernels of libsketch.so, queued on torch's current stream.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import torch

from . import _lib

KINDS = {"fjl": _lib.SK_FJL, "ffd": _lib.SK_FFD, "affd": _lib.SK_AFFD, "afjl": _lib.SK_AFJL, "qk": _lib.SK_QK,
         "qkh": _lib.SK_QKH, "afjlq": _lib.SK_AFJLQ, "affdq": _lib.SK_AFFDQ, "afjlf": _lib.SK_AFJLF}
_DT = {torch.float32: _lib.SK_F32, torch.bfloat16: _lib.SK_BF16}


def _stream_ptr(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


class Sketch:
    """A seeded structured sketch S: R^N -> R^D over a list of parameter shapes.

    shapes: per layer (rows, cols) or (rows, cols, qk_da, qk_db) for QK.
    flags: sketch_create flags (AFFD_NO_MTAB: regenerate the AFFD Gaussians on
    every call instead of storing the per-layer M tables).
    """

    AFFD_NO_MTAB = 1

    def __init__(self, kind: str, shapes: Sequence[Sequence[int]], D: int, seed: int, device=None, flags: int = 0):
        self.lib = _lib.load()
        self.kind = kind
        self.D = int(D)
        self.seed = int(seed)
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None else
                                   torch.device(device).index or 0)
        self.shapes = [tuple(int(v) for v in s) for s in shapes]
        arr = (_lib.LayerShape * len(self.shapes))()
        for i, s in enumerate(self.shapes):
            arr[i].rows, arr[i].cols = s[0], s[1]
            arr[i].qk_da = s[2] if len(s) > 2 else 0
            arr[i].qk_db = s[3] if len(s) > 3 else 0
        h = ctypes.c_void_p()
        _lib.check(self.lib.sketch_create(KINDS[kind], arr, len(self.shapes), self.D, self.seed, int(flags),
                                          self.device.index, ctypes.byref(h)))
        self._h = h

    @property
    def numels(self):
        return [s[0] * s[1] for s in self.shapes]

    def close(self):
        if getattr(self, "_h", None):
            self.lib.sketch_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> dict:
        inf = _lib.Info()
        _lib.check(self.lib.sketch_query(self._h, ctypes.byref(inf)))
        return {k: getattr(inf, k) for k, _ in _lib.Info._fields_}

    def apply(self, grads: Sequence[torch.Tensor], out: Optional[torch.Tensor] = None, first_layer: int = 0,
              accumulate: bool = False, noalloc: bool = False) -> torch.Tensor:
        """out[batch, D] (+)= sum over layers first_layer.. of S_l grads[l] (grads[l]: [batch, numel]).

        noalloc: call sketch_apply_noalloc (scratch in the library's static device array, not the handle's
        workspace); pass `out` as well for a call that allocates nothing at all."""
        grads = list(grads)
        dt = grads[0].dtype
        batch = grads[0].shape[0]
        for g, n in zip(grads, self.numels[first_layer:first_layer + len(grads)]):
            if g.dtype != dt or g.device != self.device or not g.is_contiguous() or tuple(g.shape) != (batch, n):
                raise ValueError(f"gradient tensor must be contiguous {dt} [{batch}, {n}] on {self.device}")
        if out is None:
            out = torch.empty((batch, self.D), dtype=torch.float32, device=self.device)
        elif out.dtype != torch.float32 or tuple(out.shape) != (batch, self.D) or not out.is_contiguous():
            raise ValueError("out must be contiguous float32 [batch, D]")
        ptrs = (ctypes.c_void_p * len(grads))(*[g.data_ptr() for g in grads])
        fn = self.lib.sketch_apply_noalloc if noalloc else self.lib.sketch_apply
        _lib.check(fn(self._h, ptrs, _DT[dt], batch, out.data_ptr(), first_layer, len(grads), int(accumulate),
                      _stream_ptr(self.device)))
        return out

    def apply_T(self, z: torch.Tensor, out_dtype=torch.float32, theta0: Optional[Sequence] = None,
                first_layer: int = 0, n_layers: Optional[int] = None, outs=None):
        """[S_l^T z (+ theta0_l)] for layers first_layer..; z: [batch, D] float32."""
        n_layers = len(self.shapes) - first_layer if n_layers is None else n_layers
        if z.dtype != torch.float32 or z.dim() != 2 or z.shape[1] != self.D or not z.is_contiguous():
            raise ValueError("z must be contiguous float32 [batch, D]")
        batch = z.shape[0]
        if outs is None:
            outs = [torch.empty((batch, n), dtype=out_dtype, device=self.device)
                    for n in self.numels[first_layer:first_layer + n_layers]]
        optr = (ctypes.c_void_p * n_layers)(*[o.data_ptr() for o in outs])
        tptr = None
        if theta0 is not None:
            tptr = (ctypes.c_void_p * n_layers)(*[0 if t is None else t.data_ptr() for t in theta0])
        _lib.check(self.lib.sketch_apply_T(self._h, z.data_ptr(), batch, optr, _DT[out_dtype], tptr, first_layer,
                                           n_layers, _stream_ptr(self.device)))
        return outs

    def profile(self, enable: bool = True, classes=None) -> None:
        """Start (clearing earlier records) or stop per-kernel-class event timing.

        classes: names from PROF_CLASSES to time (default: all of them)."""
        if not enable:
            mask = 0
        elif classes is None:
            mask = (1 << len(_lib.PROF_CLASSES)) - 1
        else:
            mask = 0
            for c in classes:
                mask |= 1 << _lib.PROF_CLASSES.index(c)
        _lib.check(self.lib.sketch_profile(self._h, mask))

    def profile_read(self) -> dict:
        """{class: (ms, groups, algorithmic bytes)} recorded since profile(True); clears the record."""
        import numpy as np
        n = len(_lib.PROF_CLASSES)
        ms, cnt, by = np.zeros(n), np.zeros(n, dtype=np.int64), np.zeros(n, dtype=np.int64)
        _lib.check(self.lib.sketch_profile_read(self._h, ms.ctypes.data_as(ctypes.c_void_p),
                                                cnt.ctypes.data_as(ctypes.c_void_p),
                                                by.ctypes.data_as(ctypes.c_void_p)))
        return {c: (float(ms[i]), int(cnt[i]), int(by[i])) for i, c in enumerate(_lib.PROF_CLASSES) if cnt[i]}

    def debug_stream(self, layer: int, stream: str, start: int, count: int, aux: int = 0):
        import numpy as np
        dt = {"sign": np.int8, "gauss": np.float32, "qka": np.float32, "qkb": np.float32}.get(stream, np.uint32)
        buf = np.zeros(count, dtype=dt)
        _lib.check(self.lib.sketch_debug_stream(self._h, layer, _lib.STREAMS[stream], start, count, aux,
                                                buf.ctypes.data_as(ctypes.c_void_p)))
        return buf
