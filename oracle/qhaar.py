"""fp64 oracle for the sketches with the random-orthogonal Kronecker
pre-conditioner Q (Sec. 3, paragraphs "Alternative pre-conditioners" and
"Direct usage of the pre-conditioner Q"; eq. straight; Table
tab:gains_design_choices, rows "H_N -> Q").

TEST INFRASTRUCTURE ONLY (see the package docstring): the product never
imports this module and shares no code with it.

Definitions, per parameter tensor (layer) l with N = N'_l (the padded length
of the other kinds) and Kronecker factor sizes (b_0, ..., b_{K-1}) = ks(N):

* Factor k is Haar-distributed on the orthogonal group of size b_k: the Q of
  the QR factorisation of a b_k x b_k matrix A of N(0, 1) entries, with the
  signs fixed so that R has a positive diagonal (the QR factor of a Gaussian
  matrix is Haar only with that normalisation).  A[r][c] is number
  k 2^20 + r b_k + c of the layer's "qh" Gaussian stream.
* Q_N = Q_0 (x) Q_1 (x) ... (x) Q_{K-1} (Kronecker product, row-major digit
  order: digit 0 most significant), applied as y = Q_N x.
* QKH ("QK" of eq. straight, on the flattened layer):
      y = sqrt(N / D) R_D Q_N pad(x)
  R_D keeps the first D coordinates; in row-major digit order that equals the
  Kronecker product of the factors restricted to their first D_k rows, with
  D_k = b_k for the trailing factors that fit in D, one partial factor, and
  D_k = 1 for the leading ones (the D_i x B_i factors of eq. straight).
* AFJLQ (eq. frikadel with H_N -> Q; the text notes that Q needs no sign
  diagonal B, and a Haar factor needs no digit permutation):
      y = sqrt(N / D) G R_D Q_N pad(x),  G = diag(g_0 .. g_{D-1})
  with g the layer's "gauss" stream (the same g as AFJL).
* AFFDQ (eq. bami with both H_N -> Q):
      y = sqrt(N / D) R_D Q'_N G Q_N pad(x),  G = diag(g_0 .. g_{N-1})
  with Q_N the factors above and Q'_N an independent set (factor k of Q'_N is
  factor 8 + k of the layer's stream), g the layer's "gauss" stream over N.
* Several layers: the sum of the per-layer sketches (as for AFFD / AFJL).
* Transposes: the exact adjoints, truncated to the layer's n entries.

The arithmetic below is the definition written out with numpy: QR (LAPACK),
matrix products and reshapes.  No blocking or fusion beyond the restriction
of R_D to the factors, which the pins check against the dense R_D Q_N.
"""
from __future__ import annotations

import numpy as np

from . import gauss, kron_shapes, padded, round_bf16  # noqa: F401  (round_bf16 re-exported for tests)

QH_STREAM = "qh"
_FACTOR_STRIDE = 1 << 20  # Gaussian numbers reserved per factor (b_k <= 1024)

_cache: dict = {}


def haar_factor(seed: int, layer: int, k: int, b: int) -> np.ndarray:
    """Factor k (b x b, fp64) of layer `layer`: QR of the Gaussian matrix with R's diagonal made positive."""
    key = (seed, layer, k, b)
    if key not in _cache:
        a = gauss(seed, layer, QH_STREAM, k * _FACTOR_STRIDE, b * b).reshape(b, b)
        q, r = np.linalg.qr(a, mode="complete")
        s = np.sign(np.diag(r))
        s[s == 0] = 1.0
        if len(_cache) >= 4096:
            _cache.clear()
        _cache[key] = q * s[None, :]
    return _cache[key]


def restriction(dims, D: int):
    """Rows kept per factor: D_k with prod D_k = D, trailing factors first."""
    out = [1] * len(dims)
    rem = D
    for k in range(len(dims) - 1, -1, -1):
        out[k] = min(dims[k], rem)
        rem //= out[k]
    assert rem == 1, (dims, D)
    return out


def layer_plan(n: int, D: int):
    np_len = padded(n, D)
    dims = kron_shapes(np_len)
    return np_len, dims, restriction(dims, D)


def _mode_product(t: np.ndarray, m: np.ndarray, axis: int) -> np.ndarray:
    """Multiply tensor t along `axis` by matrix m (new axis length = m.shape[0])."""
    return np.moveaxis(np.tensordot(m, t, axes=([1], [axis])), 0, axis)


SECOND = 8  # factor index offset of the second set (AFFDQ)


def layer_forward(kind: str, x: np.ndarray, n: int, D: int, seed: int, layer: int) -> np.ndarray:
    """One layer, one vector (fp64 x of length n): the D-vector of the layer's sketch."""
    np_len, dims, dk = layer_plan(n, D)
    t = np.zeros(np_len, dtype=np.float64)
    t[:n] = x
    t = t.reshape(dims)
    if kind == "affdq":
        for k, b in enumerate(dims):
            t = _mode_product(t, haar_factor(seed, layer, k, b), k)
        t = t * gauss(seed, layer, "gauss", 0, np_len).reshape(dims)
        for k, b in enumerate(dims):
            t = _mode_product(t, haar_factor(seed, layer, SECOND + k, b)[: dk[k], :], k)
        return t.reshape(-1) * np.sqrt(np_len / D)
    for k, b in enumerate(dims):
        t = _mode_product(t, haar_factor(seed, layer, k, b)[: dk[k], :], k)
    y = t.reshape(-1) * np.sqrt(np_len / D)
    if kind == "afjlq":
        y = y * gauss(seed, layer, "gauss", 0, D)
    return y


def layer_transpose(kind: str, z: np.ndarray, n: int, D: int, seed: int, layer: int) -> np.ndarray:
    """One layer, one vector: the adjoint applied to z (length D), truncated to n entries."""
    np_len, dims, dk = layer_plan(n, D)
    u = np.array(z, dtype=np.float64) * np.sqrt(np_len / D)
    if kind == "affdq":
        t = u.reshape(dk)
        for k, b in enumerate(dims):
            t = _mode_product(t, haar_factor(seed, layer, SECOND + k, b)[: dk[k], :].T, k)
        t = t * gauss(seed, layer, "gauss", 0, np_len).reshape(dims)
        for k, b in enumerate(dims):
            t = _mode_product(t, haar_factor(seed, layer, k, b).T, k)
        return t.reshape(-1)[:n]
    if kind == "afjlq":
        u = u * gauss(seed, layer, "gauss", 0, D)
    t = u.reshape(dk)
    for k, b in enumerate(dims):
        t = _mode_product(t, haar_factor(seed, layer, k, b)[: dk[k], :].T, k)
    return t.reshape(-1)[:n]


def _to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    u = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def apply(kind: str, shapes, D: int, seed: int, xs, dtype: str = "f32", layer0: int = 0) -> np.ndarray:
    """Forward sketch of a batch: sum over layers of the per-layer sketches; fp64 [batch, D]."""
    batch = np.asarray(xs[0]).shape[0]
    y = np.zeros((batch, D), dtype=np.float64)
    for i, (s, x) in enumerate(zip(shapes, xs)):
        n = int(s[0]) * int(s[1])
        xv = _to_f64(x, dtype).reshape(batch, n)
        for b in range(batch):
            y[b] += layer_forward(kind, xv[b], n, D, seed, layer0 + i)
    return y


def apply_T(kind: str, shapes, D: int, seed: int, z: np.ndarray, layer0: int = 0, theta0=None):
    """Transpose of a batch z [batch, D]: per layer fp64 [batch, n] (plus theta0 where given)."""
    z = np.asarray(z, dtype=np.float64)
    outs = []
    for i, s in enumerate(shapes):
        n = int(s[0]) * int(s[1])
        o = np.stack([layer_transpose(kind, z[b], n, D, seed, layer0 + i) for b in range(z.shape[0])])
        if theta0 is not None and theta0[i] is not None:
            o = o + np.asarray(theta0[i], dtype=np.float64)[None, :]
        outs.append(o)
    return outs


def dense(kind: str, n: int, D: int, seed: int, layer: int) -> np.ndarray:
    """The layer's D x n matrix built densely: sqrt(N/D) [G] R_D (Q_0 (x) ... (x) Q_{K-1}), n columns kept.
    For small N only (a pin of the restricted-factor evaluation above)."""
    np_len, dims, _ = layer_plan(n, D)
    m = np.ones((1, 1))
    for k, b in enumerate(dims):
        m = np.kron(m, haar_factor(seed, layer, k, b))
    if kind == "affdq":
        m2 = np.ones((1, 1))
        for k, b in enumerate(dims):
            m2 = np.kron(m2, haar_factor(seed, layer, SECOND + k, b))
        g = gauss(seed, layer, "gauss", 0, np_len)
        return (m2[:D, :] * g[None, :]) @ m[:, :n] * np.sqrt(np_len / D)
    s = m[:D, :n] * np.sqrt(np_len / D)
    if kind == "afjlq":
        s = s * gauss(seed, layer, "gauss", 0, D)[:, None]
    return s
