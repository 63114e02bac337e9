"""fp64 oracle for the sketch with the Fourier pre-conditioner (Sec. 3,
paragraph "Alternative pre-conditioners": H_N replaced by the FFT; Table
tab:gains_design_choices, rows "H_N -> FFT"; Table
tab:gradient_computation_full, rows F = 1).

TEST INFRASTRUCTURE ONLY (see the package docstring): the product never
imports this module and shares no code with it.

The paper does not say how a real gradient goes through a complex transform.
The reading used here (parity target of the GPU kind SK_AFJLF):

* F_N is the real orthonormal Fourier matrix of even size N: with
  X_k = sum_n v_n exp(-2 pi i k n / N) the DFT of v,
      (F_N v)_0      = X_0 / sqrt(N)
      (F_N v)_1      = X_{N/2} / sqrt(N)
      (F_N v)_{2k}   = sqrt(2/N) Re X_k      (1 <= k < N/2)
      (F_N v)_{2k+1} = sqrt(2/N) Im X_k
  i.e. the rows are the cosine and sine basis vectors, the two real ones
  first, then one (cos, sin) pair per frequency.  F_N is orthogonal, and any
  even number D of its leading rows gives every column the squared norm D/N,
  which keeps E||S x||^2 = ||x||^2 exactly (the role the flat entries of H_N
  play).
* AFJLF (eq. frikadel with H^{pi1}_N -> F_N): per layer l with N = N'_l,
      y = sqrt(N / D) G R_D F_N B pad(x),
  B the layer's sign stream, G = diag(g_0 .. g_{D-1}) its Gaussian stream
  (the streams of AFJL).  The FFT has no Kronecker factors, so there are no
  digit permutations.
* Several layers: the sum of the per-layer sketches; transposes are the exact
  adjoints truncated to the layer's n entries.

The arithmetic is the definition written out: scipy's real FFT (fp64, the
vectors of a batch transformed together on `workers` threads) is the one
library step, the packing is spelled out, and the pins check the result
against the dense cos / sin matrix and numpy's complex FFT.
"""
from __future__ import annotations

import os

import numpy as np
import scipy.fft

from . import gauss, padded, signs

FKINDS = ("afjlf",)


def _workers(nthreads: int = 0) -> int:
    return nthreads or int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))


def packed_rfft(v: np.ndarray, nthreads: int = 0) -> np.ndarray:
    """F_N v for real fp64 vectors of even length N (the last axis)."""
    v = np.asarray(v, dtype=np.float64)
    N = v.shape[-1]
    X = scipy.fft.rfft(v, axis=-1, workers=_workers(nthreads))
    out = np.empty(v.shape, dtype=np.float64)
    out[..., 0] = X[..., 0].real
    out[..., 1] = X[..., N // 2].real
    out[..., 2::2] = np.sqrt(2.0) * X[..., 1:N // 2].real
    out[..., 3::2] = np.sqrt(2.0) * X[..., 1:N // 2].imag
    return out / np.sqrt(N)


def packed_irfft(p: np.ndarray, N: int, nthreads: int = 0) -> np.ndarray:
    """F_N^T p for coefficient vectors p holding the first p.shape[-1] <= N packed coordinates (zero beyond)."""
    p = np.asarray(p, dtype=np.float64)
    q = np.zeros(p.shape[:-1] + (N,), dtype=np.float64)
    q[..., :p.shape[-1]] = p
    Y = np.empty(p.shape[:-1] + (N // 2 + 1,), dtype=np.complex128)
    Y[..., 0] = q[..., 0]
    Y[..., N // 2] = q[..., 1]
    Y[..., 1:N // 2] = (q[..., 2::2] + 1j * q[..., 3::2]) / np.sqrt(2.0)
    # irfft(Y)_n = (Y_0 + Y_{N/2} (-1)^n + 2 sum_k Re(Y_k e^{2 pi i k n / N})) / N
    return scipy.fft.irfft(Y * np.sqrt(N), n=N, axis=-1, workers=_workers(nthreads))


def layer_forward(kind: str, x: np.ndarray, n: int, D: int, seed: int, layer: int, nthreads: int = 0) -> np.ndarray:
    """The layer's sketch of a batch x [batch, n]: [batch, D]."""
    assert kind == "afjlf"
    N = padded(n, D)
    v = np.zeros((x.shape[0], N), dtype=np.float64)
    v[:, :n] = signs(seed, layer, 0, n)[None, :] * x
    g = gauss(seed, layer, "gauss", 0, D)
    return np.sqrt(N / D) * g[None, :] * packed_rfft(v, nthreads)[:, :D]


def layer_transpose(kind: str, z: np.ndarray, n: int, D: int, seed: int, layer: int, nthreads: int = 0):
    """The layer's transpose of a batch z [batch, D]: [batch, n]."""
    assert kind == "afjlf"
    N = padded(n, D)
    g = gauss(seed, layer, "gauss", 0, D)
    w = packed_irfft(g[None, :] * np.asarray(z, dtype=np.float64), N, nthreads)
    return np.sqrt(N / D) * signs(seed, layer, 0, n)[None, :] * w[:, :n]


def _to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    u = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def apply(kind: str, shapes, D: int, seed: int, xs, dtype: str = "f32", layer0: int = 0,
          nthreads: int = 0) -> np.ndarray:
    """Forward sketch of a batch: the sum over layers of the per-layer sketches; fp64 [batch, D]."""
    batch = np.asarray(xs[0]).shape[0]
    y = np.zeros((batch, D), dtype=np.float64)
    for i, (s, x) in enumerate(zip(shapes, xs)):
        n = int(s[0]) * int(s[1])
        y += layer_forward(kind, _to_f64(x, dtype).reshape(batch, n), n, D, seed, layer0 + i, nthreads)
    return y


def apply_T(kind: str, shapes, D: int, seed: int, z: np.ndarray, layer0: int = 0, theta0=None, nthreads: int = 0):
    """Transpose of a batch z [batch, D]: per layer fp64 [batch, n] (plus theta0 where given)."""
    z = np.asarray(z, dtype=np.float64)
    outs = []
    for i, s in enumerate(shapes):
        n = int(s[0]) * int(s[1])
        o = layer_transpose(kind, z, n, D, seed, layer0 + i, nthreads)
        if theta0 is not None and theta0[i] is not None:
            o = o + np.asarray(theta0[i], dtype=np.float64)[None, :]
        outs.append(o)
    return outs
