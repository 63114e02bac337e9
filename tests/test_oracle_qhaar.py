"""Pins of the fp64 oracle for the kinds with the random-orthogonal Kronecker
pre-conditioner (QKH: eq. straight on the flattened layer; AFJLQ: eq. frikadel
with H_N -> Q; AFFDQ: eq. bami with both H_N -> Q; Table tab:gains_design_choices).

Each pin checks the oracle against something other than itself: the QR
identity and its uniqueness, Haar statistics, the dense Kronecker product,
exact Gram identities, a worked example and the isometry in expectation."""
import numpy as np
import pytest

import oracle as O
from oracle import qhaar as Q

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


@pytest.mark.parametrize("b", [2, 16, 64, 1024])
def test_factor_is_the_qr_factor_with_positive_r(b):
    """Q^T Q = I and Q^T A is upper triangular with a positive diagonal: by uniqueness of that QR
    factorisation, Q is the normalised QR factor of the stream's Gaussian matrix."""
    seed, layer, k = 11, 3, 1
    a = O.gauss(seed, layer, "qh", k << 20, b * b).reshape(b, b)
    q = Q.haar_factor(seed, layer, k, b)
    assert np.abs(q.T @ q - np.eye(b)).max() < 1e-12
    r = q.T @ a
    scale = np.abs(a).max()
    assert np.abs(np.tril(r, -1)).max() < 1e-11 * scale * b
    assert (np.diag(r) > 0).all()
    assert np.abs(q @ np.triu(r) - a).max() < 1e-11 * scale * b


def test_factor_streams_are_distinct():
    f0 = Q.haar_factor(1, 0, 0, 8)
    assert not np.allclose(f0, Q.haar_factor(1, 0, 1, 8))   # factor index
    assert not np.allclose(f0, Q.haar_factor(1, 1, 0, 8))   # layer
    assert not np.allclose(f0, Q.haar_factor(2, 0, 0, 8))   # seed


def test_haar_statistics():
    """Over many draws of a 3 x 3 factor: E[Q00] = 0, E[Q00^2] = 1/3, E[det] = 0 (Haar on O(3)).
    Without the sign normalisation the QR factor has E[Q00] far from 0."""
    b, m = 3, 3000
    q00, det = np.empty(m), np.empty(m)
    for i in range(m):
        q = Q.haar_factor(5, i, 0, b)
        q00[i], det[i] = q[0, 0], np.linalg.det(q)
    se = 1.0 / np.sqrt(m)
    assert abs(q00.mean()) < 4.5 * np.sqrt(1.0 / 3.0) * se
    # Q00^2 ~ Beta(1/2, 1): variance 2 (b - 1) / (b^2 (b + 2))
    assert abs((q00 ** 2).mean() - 1.0 / 3.0) < 4.5 * np.sqrt(2 * 2 / (9 * 5)) * se
    assert abs(det.mean()) < 4.5 * se
    assert np.allclose(np.abs(det), 1.0)


@pytest.mark.parametrize("kind", ["qkh", "afjlq", "affdq"])
@pytest.mark.parametrize("n,D", [(1, 16), (100, 16), (3000, 64), (4096, 4096), (4096, 1024), (5000, 1024),
                                 (2048, 4096), (1500, 2)])
def test_restricted_factors_equal_dense_restriction(kind, n, D):
    """The factor-by-factor evaluation equals R_D of the dense Kronecker product, forward and transpose."""
    seed, layer = 7, 2
    S = Q.dense(kind, n, D, seed, layer)
    rng = np.random.default_rng(n + D)
    x, z = rng.standard_normal(n), rng.standard_normal(D)
    y = Q.layer_forward(kind, x, n, D, seed, layer)
    assert np.abs(S @ x - y).max() <= 1e-12 * max(1.0, np.abs(y).max())
    xt = Q.layer_transpose(kind, z, n, D, seed, layer)
    assert np.abs(S.T @ z - xt).max() <= 1e-12 * max(1.0, np.abs(xt).max())


@pytest.mark.parametrize("n,D", [(4096, 1024), (3000, 64), (100, 128)])
def test_gram_identities(n, D):
    """S S^T = (N/D) I for QKH and (N/D) diag(g^2) for AFJLQ, exactly (orthonormal restricted rows),
    when n = N' (no truncation)."""
    seed, layer = 3, 0
    np_len, _, _ = Q.layer_plan(n, D)
    S = Q.dense("qkh", np_len, D, seed, layer)
    assert np.abs(S @ S.T - (np_len / D) * np.eye(D)).max() < 1e-11 * np_len / D
    g = O.gauss(seed, layer, "gauss", 0, D)
    S = Q.dense("afjlq", np_len, D, seed, layer)
    assert np.abs(S @ S.T - (np_len / D) * np.diag(g * g)).max() < 1e-11 * np_len / D * (g * g).max()


@pytest.mark.parametrize("n,D", [(70000, 4096), (2 ** 20, 2 ** 16), (4096, 4096)])
def test_worked_example_first_row(n, D):
    """x* = the first row of Q_N (the Kronecker product of the factors' first rows): Q_N x* = e_0,
    so QKH(x*) = sqrt(N/D) e_0 and AFJLQ(x*) = sqrt(N/D) g_0 e_0 (analogue of the worked example
    of Thm. fastfood_bad_inputs)."""
    seed, layer = 9, 4
    np_len, dims, _ = Q.layer_plan(n, D)
    row = np.ones(1)
    for k, b in enumerate(dims):
        row = np.kron(row, Q.haar_factor(seed, layer, k, b)[0])
    x = row[:n]
    if n < np_len:  # a truncated first row is no longer exact: pad the layer instead
        x = row
        n = np_len
    want = np.zeros(D)
    want[0] = np.sqrt(np_len / D)
    y = Q.layer_forward("qkh", x, n, D, seed, layer)
    assert np.abs(y - want).max() < 1e-12 * np.sqrt(np_len / D)
    g0 = O.gauss(seed, layer, "gauss", 0, 1)[0]
    y = Q.layer_forward("afjlq", x, n, D, seed, layer)
    assert np.abs(y - g0 * want).max() < 1e-12 * np.sqrt(np_len / D) * max(1.0, abs(g0))


@pytest.mark.parametrize("n,D", [(70000, 4096), (4096, 4096), (3000, 64)])
def test_affdq_worked_example(n, D):
    """AFFDQ(Q_N^T e_0) = sqrt(N/D) g_0 (first column of Q'_N)[:D]: the first transform maps x* to e_0,
    G scales it by g_0, the second transform's restriction keeps D rows of its first column."""
    seed, layer = 4, 1
    np_len, dims, _ = Q.layer_plan(n, D)
    row, col2 = np.ones(1), np.ones(1)
    for k, b in enumerate(dims):
        row = np.kron(row, Q.haar_factor(seed, layer, k, b)[0])
        col2 = np.kron(col2, Q.haar_factor(seed, layer, Q.SECOND + k, b)[:, 0])
    g0 = O.gauss(seed, layer, "gauss", 0, 1)[0]
    want = np.sqrt(np_len / D) * g0 * col2[:D]
    y = Q.layer_forward("affdq", row, np_len, D, seed, layer)
    assert np.abs(y - want).max() < 1e-12 * max(1.0, np.abs(want).max())


def test_isometry_in_expectation():
    """E ||S x||^2 = ||x||^2 over seeds (QKH; AFJLQ and AFFDQ add E g^2 = 1), as a z-test on the mean ratio."""
    n, D, m = 200, 32, 600
    x = np.random.default_rng(0).standard_normal(n)
    for kind in ("qkh", "afjlq", "affdq"):
        r = np.array([np.sum(Q.layer_forward(kind, x, n, D, s, 0) ** 2) for s in range(m)]) / np.dot(x, x)
        assert abs(r.mean() - 1.0) < 4.5 * r.std() / np.sqrt(m), (kind, r.mean(), r.std())


def test_layers_sum_and_batch():
    """Several layers: the sum of per-layer sketches with layer ids layer0, layer0+1, ...; bf16 input."""
    shapes = [(3, 100), (1, 7), (64, 64)]
    D, seed = 256, 4
    rng = np.random.default_rng(1)
    xs = [rng.standard_normal((2, r * c)).astype(np.float32) for r, c in shapes]
    y = O.apply("qkh", shapes, D, seed, xs, layer0=5)
    for b in range(2):
        want = sum(Q.layer_forward("qkh", xs[i][b].astype(np.float64), r * c, D, seed, 5 + i)
                   for i, (r, c) in enumerate(shapes))
        assert np.abs(y[b] - want).max() < 1e-13 * np.abs(want).max()
    xb = [(x.view(np.uint32) >> 16).astype(np.uint16) for x in xs]
    yb = O.apply("afjlq", shapes, D, seed, xb, dtype="bf16")
    for b in range(2):
        want = sum(Q.layer_forward("afjlq", (xb[i][b].astype(np.uint32) << 16).view(np.float32).astype(np.float64),
                                   r * c, D, seed, i) for i, (r, c) in enumerate(shapes))
        assert np.abs(yb[b] - want).max() < 1e-13 * np.abs(want).max()
    z = rng.standard_normal((2, D))
    outs = O.apply_T("afjlq", shapes, D, seed, z, theta0=[None, np.ones(7), None])
    assert [o.shape for o in outs] == [(2, 300), (2, 7), (2, 4096)]
    t1 = Q.layer_transpose("afjlq", z[1], 7, D, seed, 1) + 1.0
    assert np.abs(outs[1][1] - t1).max() < 1e-13 * np.abs(t1).max()
