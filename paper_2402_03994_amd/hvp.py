"""Binding of the sketched-HVP entry points (include/sketch_hvp.h) for torch tensors.

Argument marshalling only: the synthetic Hessian, the sketched operator
v -> S H S^T v and the Arnoldi steps run in the HIP kernels of libsketch.so on
torch's current stream.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import numpy as np
import torch

from . import _lib
from .sketch import Sketch, _stream_ptr


class SyntheticHessian:
    """H = shift I + sum_j lambdas[j] v_j v_j^T over the concatenated parameters of `shapes`
    (v_j = s_j / sqrt(N_tot), s_j regenerated Rademacher vectors; rank <= 32).

    max_batch: the most vectors one apply / sketch_hvp call takes (the handle owns
    2 * max_batch * N_tot floats of workspace)."""

    def __init__(self, shapes: Sequence[Sequence[int]], rank: int, lambdas, shift: float, seed: int,
                 max_batch: int = 1, device=None):
        self.lib = _lib.load()
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None else
                                   torch.device(device).index or 0)
        self.shapes = [tuple(int(v) for v in s[:2]) for s in shapes]
        self.rank = int(rank)
        self.lambdas = np.ascontiguousarray(lambdas, dtype=np.float32)
        if self.lambdas.shape != (self.rank,):
            raise ValueError("lambdas must hold `rank` values")
        self.shift = float(shift)
        self.seed = int(seed)
        self.max_batch = int(max_batch)
        arr = (_lib.LayerShape * len(self.shapes))()
        for i, (r, c) in enumerate(self.shapes):
            arr[i].rows, arr[i].cols = r, c
        h = ctypes.c_void_p()
        _lib.check(self.lib.sk_hvp_create(arr, len(self.shapes), self.rank,
                                          self.lambdas.ctypes.data_as(ctypes.c_void_p), self.shift, self.seed,
                                          self.max_batch, self.device.index, ctypes.byref(h)))
        self._h = h

    @property
    def numels(self):
        return [r * c for r, c in self.shapes]

    def close(self):
        if getattr(self, "_h", None):
            self.lib.sk_hvp_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def apply(self, xs: Sequence[torch.Tensor], ys: Optional[Sequence[torch.Tensor]] = None):
        """[H x] per layer for xs[l]: float32 [batch, numel_l] (contiguous, on the device)."""
        xs = list(xs)
        batch = xs[0].shape[0]
        for x, n in zip(xs, self.numels):
            if x.dtype != torch.float32 or x.device != self.device or not x.is_contiguous() or \
                    tuple(x.shape) != (batch, n):
                raise ValueError(f"x must be contiguous float32 [{batch}, {n}] on {self.device}")
        if len(xs) != len(self.shapes):
            raise ValueError("one tensor per layer")
        if ys is None:
            ys = [torch.empty_like(x) for x in xs]
        xp = (ctypes.c_void_p * len(xs))(*[x.data_ptr() for x in xs])
        yp = (ctypes.c_void_p * len(ys))(*[y.data_ptr() for y in ys])
        _lib.check(self.lib.sk_hvp_apply(self._h, xp, batch, yp, _stream_ptr(self.device)))
        return ys

    def profile(self, enable: bool = True, classes=None) -> None:
        """Start (clearing earlier records) or stop event timing of this handle's kernel classes
        (names from HVP_PROF_CLASSES; default all)."""
        mask = 0
        if enable:
            names = _lib.HVP_PROF_CLASSES if classes is None else classes
            for c in names:
                mask |= 1 << _lib.HVP_PROF_CLASSES.index(c)
        _lib.check(self.lib.sk_hvp_profile(self._h, mask))

    def profile_read(self) -> dict:
        n = len(_lib.HVP_PROF_CLASSES)
        ms, cnt, by = np.zeros(n), np.zeros(n, dtype=np.int64), np.zeros(n, dtype=np.int64)
        _lib.check(self.lib.sk_hvp_profile_read(self._h, ms.ctypes.data_as(ctypes.c_void_p),
                                                cnt.ctypes.data_as(ctypes.c_void_p),
                                                by.ctypes.data_as(ctypes.c_void_p)))
        return {c: (float(ms[i]), int(cnt[i]), int(by[i])) for i, c in enumerate(_lib.HVP_PROF_CLASSES) if cnt[i]}


def _check_vec(t: torch.Tensor, shape, device, name):
    if t.dtype != torch.float32 or t.device != device or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be contiguous float32 {tuple(shape)} on {device}")


def sketch_hvp(sk: Sketch, hess: SyntheticHessian, v: torch.Tensor, out: Optional[torch.Tensor] = None):
    """S H S^T v for v: float32 [batch, D] (Sec. 2, the sketch of the HVP operator)."""
    if v.dim() != 2:
        raise ValueError("v must be [batch, D]")
    _check_vec(v, (v.shape[0], sk.D), sk.device, "v")
    if out is None:
        out = torch.empty_like(v)
    _check_vec(out, v.shape, sk.device, "out")
    _lib.check(sk.lib.sketch_hvp(sk._h, hess._h, v.data_ptr(), v.shape[0], out.data_ptr(), _stream_ptr(sk.device)))
    return out


def arnoldi_work_floats(D: int, k: int) -> int:
    return int(_lib.load().sketch_arnoldi_work_floats(D, k))


def arnoldi_step(Q: torch.Tensor, j: int, Hbar: torch.Tensor, work: torch.Tensor) -> None:
    """One Arnoldi step on Q [k+1, D] and Hbar [k+1, k] (row j+1 of Q holds A q_j on entry; j = -1
    normalises row 0); work: float32 of arnoldi_work_floats(D, k) entries."""
    k1, D = Q.shape
    k = k1 - 1
    _check_vec(Q, (k + 1, D), Q.device, "Q")
    _check_vec(Hbar, (k + 1, k), Q.device, "Hbar")
    if work.dtype != torch.float32 or work.numel() < arnoldi_work_floats(D, k) or work.device != Q.device:
        raise ValueError("work too small")
    _lib.check(_lib.load().sketch_arnoldi_step(Q.data_ptr(), D, j, Hbar.data_ptr(), k, work.data_ptr(),
                                               _stream_ptr(Q.device)))


def arnoldi(sk: Sketch, hess: SyntheticHessian, v0: torch.Tensor, k: int, Q: Optional[torch.Tensor] = None,
            Hbar: Optional[torch.Tensor] = None):
    """k Arnoldi steps with full re-orthogonalisation on v -> S H S^T v from v0 [D] (Sec. 4).
    Returns (Q [k+1, D], Hbar [k+1, k]) on the device."""
    _check_vec(v0, (sk.D,), sk.device, "v0")
    if Q is None:
        Q = torch.empty((k + 1, sk.D), dtype=torch.float32, device=sk.device)
    if Hbar is None:
        Hbar = torch.empty((k + 1, k), dtype=torch.float32, device=sk.device)
    _check_vec(Q, (k + 1, sk.D), sk.device, "Q")
    _check_vec(Hbar, (k + 1, k), sk.device, "Hbar")
    _lib.check(sk.lib.sketch_arnoldi(sk._h, hess._h, v0.data_ptr(), k, Q.data_ptr(), Hbar.data_ptr(),
                                     _stream_ptr(sk.device)))
    return Q, Hbar


def ritz_values(Hbar: torch.Tensor) -> np.ndarray:
    """Eigenvalues of the leading k x k block of Hbar (a small host eigenproblem), by decreasing real part."""
    h = Hbar.detach().cpu().double().numpy()
    k = h.shape[1]
    ev = np.linalg.eigvals(h[:k, :k])
    return ev[np.argsort(-ev.real)]


def id_search(sk: Sketch, hess: SyntheticHessian, theta0: Sequence[torch.Tensor], d_min: int, tau_target: float,
              delta: float, c: int, max_rounds: int, work: Optional[torch.Tensor] = None) -> dict:
    """Intrinsic-dimension search (Sec. 4) on L(theta) = 1/2 theta^T H theta over theta0 + S^T omega:
    rounds of c conjugate-gradient steps on omega[:d], d doubled when a round improves
    tau = 1 - L/L(theta0) by less than delta, stop at tau >= tau_target.  theta0: per layer float32
    [numel] on the device.  Returns dict(d, status, rounds, L0, taus, ds, omega)."""
    theta0 = list(theta0)
    for t, n in zip(theta0, hess.numels):
        if t.dtype != torch.float32 or t.device != sk.device or not t.is_contiguous() or t.numel() != n:
            raise ValueError(f"theta0 tensors must be contiguous float32 with {n} entries on {sk.device}")
    nw = int(sk.lib.sketch_id_search_work_floats(sk.D))
    if work is None:
        work = torch.empty(nw, dtype=torch.float32, device=sk.device)
    if work.dtype != torch.float32 or work.numel() < nw or work.device != sk.device:
        raise ValueError("work too small")
    taus = np.zeros(max_rounds, dtype=np.float64)
    ds = np.zeros(max_rounds, dtype=np.int64)
    res = _lib.IdResult()
    tp = (ctypes.c_void_p * len(theta0))(*[t.data_ptr() for t in theta0])
    _lib.check(sk.lib.sketch_id_search(sk._h, hess._h, tp, int(d_min), float(tau_target), float(delta), int(c),
                                       int(max_rounds), work.data_ptr(), taus.ctypes.data_as(ctypes.c_void_p),
                                       ds.ctypes.data_as(ctypes.c_void_p), ctypes.byref(res),
                                       _stream_ptr(sk.device)))
    k = res.rounds
    return dict(d=int(res.d), status=int(res.status), rounds=k, L0=float(res.L0), taus=taus[:k].tolist(),
                ds=ds[:k].tolist(), omega=work[:sk.D])
