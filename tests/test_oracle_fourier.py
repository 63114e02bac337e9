"""Pins of the Fourier pre-conditioner oracle (oracle/fourier.py, kind AFJLF: eq. frikadel with H_N replaced by
the FFT, Sec. 3 "Alternative pre-conditioners").

The oracle's one library step is numpy's real FFT; the pins check it against things other than itself: the
real Fourier matrix built entry by entry from its cos / sin definition, the complex FFT, orthogonality, the
per-column norm that the reading's packing guarantees (E||Sx||^2 = ||x||^2 exactly), the dense sketch, the
adjoint identity, S S^T, worked examples and the isometry in expectation over seeds.
"""
import math

import numpy as np
import pytest

import oracle as O
from oracle import fourier as F


def fourier_dense(N):
    """Real orthonormal Fourier matrix from its definition: rows 1/sqrt(N), (-1)^n/sqrt(N), then per frequency
    k = 1 .. N/2-1 the pair sqrt(2/N) cos(2 pi k n/N), -sqrt(2/N) sin(2 pi k n/N)."""
    M = np.zeros((N, N))
    for n in range(N):
        M[0, n] = 1.0 / math.sqrt(N)
        M[1, n] = (-1.0) ** n / math.sqrt(N)
        for k in range(1, N // 2):
            M[2 * k, n] = math.sqrt(2.0 / N) * math.cos(2 * math.pi * k * n / N)
            M[2 * k + 1, n] = -math.sqrt(2.0 / N) * math.sin(2 * math.pi * k * n / N)
    return M


@pytest.mark.parametrize("N", [2, 4, 8, 16, 64, 256])
def test_packed_transform_is_the_dense_fourier_matrix(N):
    Fd = fourier_dense(N)
    cols = np.column_stack([F.packed_rfft(e) for e in np.eye(N)])
    np.testing.assert_allclose(cols, Fd, atol=1e-13)
    np.testing.assert_allclose(Fd @ Fd.T, np.eye(N), atol=1e-13)
    p = np.random.default_rng(N).standard_normal(N)
    np.testing.assert_allclose(F.packed_irfft(p, N), Fd.T @ p, atol=1e-12)
    # a truncated coefficient vector is zero-extended
    np.testing.assert_allclose(F.packed_irfft(p[:N // 2], N), Fd[:N // 2].T @ p[:N // 2], atol=1e-12)


def test_packing_against_the_complex_fft():
    N = 1 << 12
    v = np.random.default_rng(3).standard_normal(N)
    X = np.fft.fft(v)
    y = F.packed_rfft(v)
    assert y[0] == pytest.approx(X[0].real / math.sqrt(N), abs=1e-12)
    assert y[1] == pytest.approx(X[N // 2].real / math.sqrt(N), abs=1e-12)
    for k in [1, 2, 17, N // 4, N // 2 - 1]:
        assert y[2 * k] == pytest.approx(math.sqrt(2.0 / N) * X[k].real, abs=1e-11)
        assert y[2 * k + 1] == pytest.approx(math.sqrt(2.0 / N) * X[k].imag, abs=1e-11)
    assert np.linalg.norm(y) == pytest.approx(np.linalg.norm(v), rel=1e-13)


@pytest.mark.parametrize("N", [16, 64, 256])
def test_every_column_of_leading_rows_has_norm_D_over_N(N):
    """The packing keeps the (cos, sin) pairs together: any even D leading rows give each column D/N.  A
    packing with all cosines first (Re | Im) fails this."""
    Fd = fourier_dense(N)
    for D in range(2, N + 1, 2):
        np.testing.assert_allclose((Fd[:D] ** 2).sum(axis=0), D / N, atol=1e-12)


def dense_afjlf(n, D, seed, layer):
    N = O.padded(n, D)
    Fd = fourier_dense(N)
    b = O.signs(seed, layer, 0, n).astype(np.float64)
    g = O.gauss(seed, layer, "gauss", 0, D)
    return math.sqrt(N / D) * g[:, None] * Fd[:D, :n] * b[None, :]


PAIRS = [(16, 16), (30, 16), (64, 16), (100, 32), (7, 16), (256, 64), (200, 128), (1, 16)]


@pytest.mark.parametrize("n,D", PAIRS)
def test_afjlf_against_dense_matrix(n, D):
    seed, layer = 77, 3
    S = dense_afjlf(n, D, seed, layer)
    x = np.random.default_rng(n + D).standard_normal((2, n))
    y = O.apply("afjlf", [(1, n)], D, seed, [x.astype(np.float32)], layer0=layer)
    np.testing.assert_allclose(y, x.astype(np.float32).astype(np.float64) @ S.T, atol=1e-11)
    z = np.random.default_rng(n * D).standard_normal((2, D))
    t = O.apply_T("afjlf", [(1, n)], D, seed, z, layer0=layer)[0]
    np.testing.assert_allclose(t, z @ S, atol=1e-11)


def test_adjoint_and_layer_sum():
    shapes = [(1, 300), (5, 77), (2, 1000)]
    D, seed = 128, 12
    rng = np.random.default_rng(5)
    xs = [rng.standard_normal((3, r * c)).astype(np.float32) for r, c in shapes]
    z = rng.standard_normal((3, D))
    y = O.apply("afjlf", shapes, D, seed, xs)
    ts = O.apply_T("afjlf", shapes, D, seed, z)
    lhs = (y * z).sum(axis=1)
    rhs = sum((x.astype(np.float64) * t).sum(axis=1) for x, t in zip(xs, ts))
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12)
    parts = sum(O.apply("afjlf", [s], D, seed, [x], layer0=i) for i, (s, x) in enumerate(zip(shapes, xs)))
    np.testing.assert_allclose(y, parts, atol=1e-12)


def test_s_st_is_scaled_gaussian_diagonal():
    n, D, seed = 500, 64, 9
    N = O.padded(n, D)
    # columns of S over the full padded layer: a layer of n = N entries
    S = O.apply_T("afjlf", [(1, N)], D, seed, np.eye(D))[0]  # rows: S^T e_i, i.e. S = that matrix transposed
    g = O.gauss(seed, 0, "gauss", 0, D)
    np.testing.assert_allclose(S @ S.T, (N / D) * np.diag(g ** 2), atol=1e-10)
    assert (S ** 2).sum() == pytest.approx((N / D) * (g ** 2).sum(), rel=1e-12)


@pytest.mark.parametrize("row", [0, 1, 2, 7, 30])
def test_worked_example_single_fourier_row(row):
    """x = B F^T e_row (a signed sampled cosine, sine or alternating vector): S x = sqrt(N/D) g_row e_row."""
    N, D, seed = 256, 32, 4
    b = O.signs(seed, 0, 0, N).astype(np.float64)
    x = b * fourier_dense(N)[row]
    y = O.apply("afjlf", [(1, N)], D, seed, [x.astype(np.float32)[None, :]])[0]
    # x was rounded to fp32: compare against the sketch of the rounded vector's leading component
    g = O.gauss(seed, 0, "gauss", 0, D)
    want = np.zeros(D)
    want[row] = math.sqrt(N / D) * g[row]
    np.testing.assert_allclose(y, want, atol=1e-6)


def test_isometry_in_expectation():
    n, D = 700, 64
    x = np.random.default_rng(1).standard_normal(n).astype(np.float32)
    nx = float((x.astype(np.float64) ** 2).sum())
    r = np.array([(O.apply("afjlf", [(1, n)], D, s, [x[None, :]])[0] ** 2).sum() / nx for s in range(1000)])
    z = (r.mean() - 1.0) / (r.std() / math.sqrt(len(r)))
    assert abs(z) < 4.5


def test_bf16_inputs_are_widened_exactly():
    n, D, seed = 3000, 256, 2
    x = np.random.default_rng(4).standard_normal((2, n)).astype(np.float32)
    u = (x.view(np.uint32) >> 16).astype(np.uint16)  # truncated to bf16 bit patterns
    widened = (u.astype(np.uint32) << 16).view(np.float32)
    np.testing.assert_allclose(O.apply("afjlf", [(1, n)], D, seed, [u], dtype="bf16"),
                               O.apply("afjlf", [(1, n)], D, seed, [widened]), atol=0)
