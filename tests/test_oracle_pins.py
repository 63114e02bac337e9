"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: published
known-answer vectors, dense matrices built from their definitions
(scipy.linalg.hadamard, explicit permutation and diagonal matrices), the
paper's Kronecker-einsum formulation of permuted Hadamard factors, closed
forms (Frobenius norms, S S^T), the worked example of Thm. fastfood_bad_inputs
and the norm-preservation property of eq. jl_prob.
"""
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.stats

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def H(n):
    """Normalised Sylvester Hadamard matrix (Appendix, Walsh-Hadamard definition)."""
    return scipy.linalg.hadamard(n).astype(np.float64) / np.sqrt(n)


# --------------------------------------------------------------------- RNG
def test_philox_known_answers():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) if not l.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(t, 16) for t in r]
        got = O.philox(v[0:4], v[4:6])
        assert [int(g) for g in got] == v[6:10]


def test_sign_stream_layout_and_balance():
    # bit j%32 of word (j/32)%4 of block j/128 (bit 1 -> -1)
    seed, layer = 123456789012345, 7
    s = O.signs(seed, layer, 0, 1 << 16)
    for j in [0, 1, 31, 32, 127, 128, 5000, 65535]:
        w = O.philox([j >> 7, 0, layer, O.STREAMS["sign"]], [seed & 0xFFFFFFFF, seed >> 32])
        bit = (int(w[(j >> 5) & 3]) >> (j & 31)) & 1
        assert s[j] == (-1 if bit else 1)
    z = s.sum() / np.sqrt(s.size)
    assert abs(z) < 5


def test_gaussian_stream_moments_and_ks():
    g = O.gauss(3, 1, "gauss", 0, 400000)
    assert abs(g.mean()) < 5 / np.sqrt(g.size)
    assert abs(g.var() - 1) < 5 * np.sqrt(2 / g.size)
    assert abs(scipy.stats.kurtosis(g)) < 0.05
    assert scipy.stats.kstest(g, "norm").pvalue > 1e-4


def test_gaussian_box_muller_values():
    # g = sqrt(-2 ln u1) * (cos | sin)(2 pi u2) on the 24-bit uniforms of a word pair
    seed, layer = 99, 4
    g = O.gauss(seed, layer, "gauss", 0, 8)
    for blk in range(2):
        w = O.philox([blk, 0, layer, O.STREAMS["gauss"]], [seed, 0])
        for pair in range(2):
            u1 = ((int(w[2 * pair]) >> 8) + 1) / 2.0**24
            u2 = (int(w[2 * pair + 1]) >> 8) / 2.0**24
            r = np.sqrt(-2 * np.log(u1))
            assert g[4 * blk + 2 * pair] == pytest.approx(r * np.cos(2 * np.pi * u2), abs=1e-15)
            assert g[4 * blk + 2 * pair + 1] == pytest.approx(r * np.sin(2 * np.pi * u2), abs=1e-15)


def test_index_stream_uniform():
    np_len = 1 << 10
    idx = O.indices(5, 2, 0, 200000, np_len)
    assert idx.max() < np_len
    counts = np.bincount(idx.astype(np.int64), minlength=np_len)
    assert scipy.stats.chisquare(counts).pvalue > 1e-4


@pytest.mark.parametrize("np_len", [16, 1 << 20, 1 << 32])
def test_index_stream_layout(np_len):
    # position i: word i%4 of the block with counter (i/4, 0, layer, stream 3), masked to N' - 1
    seed, layer = 0xFEEDFACE0BADF00D, 11
    idx = O.indices(seed, layer, 0, 4096, np_len)
    for i in [0, 1, 2, 3, 4, 7, 1001, 4095]:
        w = O.philox([i >> 2, 0, layer, O.STREAMS["index"]], [seed & 0xFFFFFFFF, seed >> 32])
        assert int(idx[i]) == int(w[i & 3]) & (np_len - 1)
    # a start offset reads the same positions
    assert np.array_equal(O.indices(seed, layer, 1001, 7, np_len), idx[1001:1008])


def test_oracle_rejects_fjl_beyond_32bit_positions():
    import ctypes
    L = O.lib()
    rows = np.array([2], dtype=np.int64)
    cols = np.array([(1 << 31) + 1], dtype=np.int64)
    zero = np.zeros(1, dtype=np.int32)
    y = np.zeros(16, dtype=np.float64)
    ptrs = (ctypes.c_void_p * 1)(None)
    assert L.orc_apply(0, 0, 1, O._ptr(rows), O._ptr(cols), O._ptr(zero), O._ptr(zero), 16, 0, 1, 0, ptrs,
                       O._ptr(y), 1, 0) == -1
    assert L.orc_apply_T(0, 0, 1, O._ptr(rows), O._ptr(cols), O._ptr(zero), O._ptr(zero), 16, 0, 1, O._ptr(y),
                         ptrs, 1, 0) == -1


@pytest.mark.parametrize("w", list(range(0, 17)))
def test_feistel_is_a_bijection_with_inverse(w):
    t = O.perm(11, 3, "pi1", 2, w)
    assert sorted(t.tolist()) == list(range(1 << w))
    for y in [0, (1 << w) - 1, (1 << w) // 3]:
        assert t[O.perm_inv(11, 3, "pi1", 2, w, y)] == y


def test_feistel_position_uniform_over_seeds():
    # chi-square of pi(0) over many keys on a 6-bit domain
    vals = [int(O.perm(s, 0, "ffdperm", 0, 6)[0]) for s in range(6400)]
    counts = np.bincount(vals, minlength=64)
    assert scipy.stats.chisquare(counts).pvalue > 1e-4


# ---------------------------------------------------------- Hadamard / shapes
@pytest.mark.parametrize("n", [1, 2, 4, 8, 64, 1024, 4096])
def test_fwht_matches_dense_hadamard(n):
    v = np.random.default_rng(n).standard_normal(n)
    np.testing.assert_allclose(O.fwht(v), H(n) @ v, rtol=0, atol=1e-12 * max(1, np.abs(v).sum()))


def test_hadamard_definition_small():
    np.testing.assert_allclose(np.column_stack([O.fwht(e) for e in np.eye(2)]), [[1, 1], [1, -1]] / np.sqrt(2))
    n = 16
    Hd = np.column_stack([O.fwht(e) for e in np.eye(n)])
    # (H_n)_{ij} = n^{-1/2} (-1)^{popcount(i & j)}
    ref = np.array([[(-1) ** bin(i & j).count("1") for j in range(n)] for i in range(n)]) / np.sqrt(n)
    np.testing.assert_allclose(Hd, ref, atol=1e-15)
    np.testing.assert_allclose(Hd @ Hd.T, np.eye(n), atol=1e-14)
    # H_{AB} = H_A kron H_B (Sec. 3, lookup removal)
    np.testing.assert_allclose(Hd, np.kron(H(4), H(4)), atol=1e-15)


def test_kron_shapes_golden():
    for l in open(os.path.join(GOLDEN, "kron_shapes.txt")):
        if l.startswith("#") or not l.strip():
            continue
        mb, n, sh = l.split()
        assert int(mb) == 1024
        want = () if sh == "-" else tuple(int(t) for t in sh.split(","))
        assert O.kron_shapes(int(n)) == want
        assert int(np.prod(want)) == int(n) if want else int(n) == 1


# ------------------------------------------------------ dense-matrix pins
def kron_apply_first_index(x, mats):
    """Apply the Kronecker product of factor matrices by contracting each
    factor's FIRST index along its axis of x reshaped row-major (the einsum
    convention of the paper's Kronecker listing)."""
    shape = tuple(m.shape[0] for m in mats)
    y = x.reshape(shape)
    for ax, m in enumerate(mats):
        y = np.moveaxis(np.tensordot(y, m, axes=([ax], [0])), -1, ax)
    return y.reshape(-1)


def digit_tables(seed, layer, stream, np_len):
    dims = O.kron_shapes(np_len)
    return dims, [O.perm(seed, layer, stream, k, int(np.log2(d))) for k, d in enumerate(dims)]


def dense_perm_factor(np_len, seed, layer, stream, permute_col):
    """sqrt(N) H^pi_N as a dense matrix, built from row- or column-permuted
    unnormalised Hadamard factors through the first-index contraction."""
    dims, tabs = digit_tables(seed, layer, stream, np_len)
    mats = []
    for d, t in zip(dims, tabs):
        h = scipy.linalg.hadamard(d).astype(np.float64)
        mats.append(h[:, t] if permute_col else h[t, :])
    return np.column_stack([kron_apply_first_index(e, mats) for e in np.eye(np_len)])


def scatter_matrix(perm):
    P = np.zeros((perm.size, perm.size))
    P[perm.astype(np.int64), np.arange(perm.size)] = 1.0  # y[pi(i)] = x[i]
    return P


def gather_matrix(perm):
    P = np.zeros((perm.size, perm.size))
    P[np.arange(perm.size), perm.astype(np.int64)] = 1.0  # y[c] = x[pi(c)]
    return P


def dense_S(kind, n, D, seed, layer):
    """Dense D x n sketch matrix from the paper's definitions."""
    np_len = O.padded(n, D)
    sc = np.sqrt(np_len / D)
    b = O.signs(seed, layer, 0, np_len).astype(np.float64)
    if kind == "afjl":
        g = O.gauss(seed, layer, "gauss", 0, D)
        P1 = scatter_matrix(O.digit_perm(seed, layer, "pi1", np_len))
        S = sc * (np.diag(g) @ (H(np_len) @ P1 @ np.diag(b))[:D])
    elif kind == "affd":
        g = O.gauss(seed, layer, "gauss", 0, np_len)
        P1 = scatter_matrix(O.digit_perm(seed, layer, "pi1", np_len))
        P2 = gather_matrix(O.digit_perm(seed, layer, "pi2", np_len))
        S = sc * (P2 @ H(np_len) @ np.diag(g) @ H(np_len) @ P1 @ np.diag(b))[:D]
    elif kind == "fjl":
        g = O.gauss(seed, layer, "gauss", 0, D)
        idx = O.indices(seed, layer, 0, D, np_len).astype(np.int64)
        E = np.zeros((D, np_len))
        E[np.arange(D), idx] = 1.0
        S = sc * (np.diag(g) @ E @ H(np_len) @ np.diag(b))
    elif kind == "ffd":
        S = np.zeros((D, np_len))
        wd = int(np.log2(D))
        for blk in range(np_len // D):
            gb = O.gauss(seed, layer, "gauss", blk * D, D)
            bb = b[blk * D:(blk + 1) * D]
            Pi = gather_matrix(O.perm(seed, layer, "ffdperm", blk, wd))
            S[:, blk * D:(blk + 1) * D] = np.diag(bb) @ H(D) @ Pi.T @ np.diag(gb) @ H(D)
    else:
        raise ValueError(kind)
    return S[:, :n]


CASES = [(n, D) for n, D in [(1, 4), (5, 8), (64, 16), (100, 32), (256, 256), (300, 64), (1000, 128),
                             (1024, 1024), (2048, 4), (2500, 512), (4096, 64)]]


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
@pytest.mark.parametrize("n,D", CASES)
def test_chain_matches_dense_matrix(kind, n, D):
    seed, layer = 17 + n, 3
    S = dense_S(kind, n, D, seed, layer)
    rng = np.random.default_rng(n * 7 + D)
    x = rng.standard_normal((2, n)).astype(np.float32)
    y = O.apply(kind, [(1, n)], D, seed, [x], layer0=layer)
    np.testing.assert_allclose(y, x.astype(np.float64) @ S.T, rtol=0, atol=1e-12 * np.abs(S).sum(1).max() * 4)
    z = rng.standard_normal((2, D))
    (xt,) = O.apply_T(kind, [(1, n)], D, seed, z, layer0=layer)
    np.testing.assert_allclose(xt, z @ S, rtol=0, atol=1e-12 * np.abs(S).sum(0).max() * 4)


@pytest.mark.parametrize("np_len", [2, 8, 64, 2048, 4096])
def test_digit_permutation_matches_paper_einsum_semantics(np_len):
    """H^{pi1} (row-permuted factors) is H o Scatter_pi1 and H^{pi2}
    (column-permuted factors) is Gather_pi2 o H, both as the paper's
    first-index contraction of permuted unnormalised Hadamard factors."""
    seed, layer = 5, 1
    Hn = scipy.linalg.hadamard(np_len).astype(np.float64)
    row = dense_perm_factor(np_len, seed, layer, "pi1", permute_col=False)
    col = dense_perm_factor(np_len, seed, layer, "pi2", permute_col=True)
    np.testing.assert_allclose(row, Hn @ scatter_matrix(O.digit_perm(seed, layer, "pi1", np_len)), atol=1e-9)
    np.testing.assert_allclose(col, gather_matrix(O.digit_perm(seed, layer, "pi2", np_len)) @ Hn, atol=1e-9)


def test_affd_matches_paper_einsum_formulation():
    """AFFD chain against the paper's formulation: B, first-index contraction
    with row-permuted factors, /sqrt(N), G, contraction with column-permuted
    factors, /sqrt(N), sigma * first D coordinates (eq. bami)."""
    n, D, seed, layer = 3000, 256, 8, 0
    np_len = O.padded(n, D)
    x = np.random.default_rng(1).standard_normal((1, n)).astype(np.float32)
    v = np.zeros(np_len)
    v[:n] = x[0]
    v = v * O.signs(seed, layer, 0, np_len)
    dims, t1 = digit_tables(seed, layer, "pi1", np_len)
    _, t2 = digit_tables(seed, layer, "pi2", np_len)
    m1 = [scipy.linalg.hadamard(d)[t, :].astype(np.float64) for d, t in zip(dims, t1)]
    m2 = [scipy.linalg.hadamard(d)[:, t].astype(np.float64) for d, t in zip(dims, t2)]
    v = kron_apply_first_index(v, m1) / np.sqrt(np_len)
    v = v * O.gauss(seed, layer, "gauss", 0, np_len)
    v = kron_apply_first_index(v, m2) / np.sqrt(np_len)
    want = np.sqrt(np_len / D) * v[:D]
    got = O.apply("affd", [(1, n)], D, seed, [x], layer0=layer)[0]
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-10)


def test_qk_kronecker_identity():
    """(A kron B) vec_r(X) = vec_r(A X B^T) (eq. qk_proof_tensor_dec), with A, B
    the N(0,1/dA), N(0,1/dB) factors of the QK streams."""
    m, n, da, db, seed, layer = 12, 20, 3, 5, 4, 2
    A = O.gauss(seed, layer, "qka", 0, da * m).reshape(da, m) / np.sqrt(da)
    B = O.gauss(seed, layer, "qkb", 0, db * n).reshape(db, n) / np.sqrt(db)
    x = np.random.default_rng(0).standard_normal((2, m * n)).astype(np.float32)
    y = O.apply("qk", [(m, n, da, db)], da * db, seed, [x], layer0=layer)
    np.testing.assert_allclose(y, x.astype(np.float64) @ np.kron(A, B).T, atol=1e-12)
    z = np.random.default_rng(1).standard_normal((2, da * db))
    (xt,) = O.apply_T("qk", [(m, n, da, db)], da * db, seed, z, layer0=layer)
    np.testing.assert_allclose(xt, z @ np.kron(A, B), atol=1e-12)


def test_qk_bf16_factor_rounding():
    assert O.round_bf16(1.0) == 1.0
    assert O.round_bf16(1.0 + 2**-9) == 1.0          # tie -> even
    assert O.round_bf16(1.0 + 3 * 2**-9) == 1.0 + 2**-7  # tie -> even (up)
    assert O.round_bf16(1.0 + 2**-8 + 2**-12) == 1.0 + 2**-7


# ------------------------------------------------------------ closed forms
def multi_layer_dense(kind, sizes, D, seed):
    return np.hstack([dense_S(kind, n, D, seed, l) for l, n in enumerate(sizes)])


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
def test_frobenius_closed_forms(kind):
    """||S||_F^2 from the oracle chain applied to every basis vector against the
    closed forms: sum g^2 over N' (AFFD), over live blocks (FFD), and
    (N'/D) sum_{i<D} g_i^2 (AFJL, FJL)."""
    n, D, seed, layer = 700, 128, 21, 0
    np_len = O.padded(n, D)
    cols = O.apply(kind, [(1, n)], D, seed, [np.eye(n, dtype=np.float32)], layer0=layer)  # rows S e_j
    fro = (cols**2).sum()
    if kind == "affd":
        # padding columns of S are dropped: sum over the n kept columns only
        S_full = dense_S(kind, np_len, D, seed, layer)
        want = (S_full[:, :n] ** 2).sum()
        assert (S_full**2).sum() == pytest.approx((O.gauss(seed, layer, "gauss", 0, np_len) ** 2).sum(), rel=1e-12)
    elif kind == "ffd":
        g = O.gauss(seed, layer, "gauss", 0, np_len)
        S_full = dense_S(kind, np_len, D, seed, layer)
        assert (S_full**2).sum() == pytest.approx((g**2).sum(), rel=1e-12)
        want = (S_full[:, :n] ** 2).sum()
    else:
        g = O.gauss(seed, layer, "gauss", 0, D)
        want_full = np_len / D * (g**2).sum()
        S_full = dense_S(kind, np_len, D, seed, layer)
        assert (S_full**2).sum() == pytest.approx(want_full, rel=1e-12)
        want = (S_full[:, :n] ** 2).sum()
    assert fro == pytest.approx(want, rel=1e-12)


def test_afjl_gram_is_diagonal():
    """AFJL on the padded space: S S^T = (N/D) diag(g_{<D}^2) exactly."""
    n, D, seed = 512, 64, 2
    S = O.apply("afjl", [(1, n)], D, seed, [np.eye(n, dtype=np.float32)]).T
    g = O.gauss(seed, 0, "gauss", 0, D)
    np.testing.assert_allclose(S @ S.T, np.diag(n / D * g**2), atol=1e-10)


def test_fjl_gram_collisions():
    """FJL: S S^T = (N/D) G C G with C_ij = [idx_i == idx_j]."""
    n, D, seed = 64, 32, 9
    S = O.apply("fjl", [(1, n)], D, seed, [np.eye(n, dtype=np.float32)]).T
    g = O.gauss(seed, 0, "gauss", 0, D)
    idx = O.indices(seed, 0, 0, D, n)
    C = (idx[:, None] == idx[None, :]).astype(np.float64)
    np.testing.assert_allclose(S @ S.T, n / D * np.outer(g, g) * C, atol=1e-10)


def test_fastfood_bad_input_worked_example():
    """Thm. fastfood_bad_inputs: x with block b = H e_1 (zeros elsewhere) gives
    ||FFD(x)||^2 = sigma^2 g_{b,1}^2 with sigma = 1."""
    D, nb, seed = 64, 4, 13
    for blk in range(nb):
        x = np.zeros((1, nb * D), dtype=np.float64)
        x[0, blk * D:(blk + 1) * D] = H(D)[:, 0]
        y = O.apply("ffd", [(1, nb * D)], D, seed, [x.astype(np.float32)])
        g0 = O.gauss(seed, 0, "gauss", blk * D, 1)[0]
        # x is exactly representable (entries +-1/8), so equality holds to rounding
        assert (y**2).sum() == pytest.approx(g0**2, rel=1e-12)


def test_afjl_affd_bad_input_analogs():
    """Same argument for x* = B Gather_pi1 H_N e_0: AFJL(x*) = sqrt(N/D) g_0 e_0 and
    AFFD(x*) = (g_0 / sqrt(D)) 1_D."""
    np_len, D, seed = 1024, 64, 31
    b = O.signs(seed, 0, 0, np_len).astype(np.float64)
    p1 = O.digit_perm(seed, 0, "pi1", np_len).astype(np.int64)
    h0 = H(np_len)[:, 0]
    xstar = b * h0[p1]  # entries +-1/32: exact in fp32
    x = xstar[None, :].astype(np.float32)
    ya = O.apply("afjl", [(1, np_len)], D, seed, [x])[0]
    g = O.gauss(seed, 0, "gauss", 0, np_len)
    want = np.zeros(D)
    want[0] = np.sqrt(np_len / D) * g[0]
    np.testing.assert_allclose(ya, want, atol=1e-12)
    yf = O.apply("affd", [(1, np_len)], D, seed, [x])[0]
    np.testing.assert_allclose(yf, np.full(D, g[0] / np.sqrt(D)), atol=1e-12)


def test_fold_identity():
    """R_D H_N w = sqrt(D/N) H_D fold_D(w), fold summing the N/D consecutive
    length-D chunks (from the Hadamard definition)."""
    N, D = 2048, 128
    w = np.random.default_rng(3).standard_normal(N)
    np.testing.assert_allclose((H(N) @ w)[:D], np.sqrt(D / N) * H(D) @ w.reshape(-1, D).sum(0), atol=1e-12)


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd", "qk"])
def test_adjoint_multilayer(kind):
    """<S x, z> = <x, S^T z> with several layers, including n < D and a ragged n."""
    rng = np.random.default_rng(5)
    if kind == "qk":
        shapes, D = [(9, 14, 3, 4), (1, 50, 1, 7), (33, 8, 5, 2)], 12 + 7 + 10
    else:
        shapes, D = [(1, 30), (7, 111), (1, 4096), (3, 1500)], 512
    xs = [rng.standard_normal((3, s[0] * s[1])).astype(np.float32) for s in shapes]
    y = O.apply(kind, shapes, D, 77, xs)
    z = rng.standard_normal((3, D))
    outs = O.apply_T(kind, shapes, D, 77, z)
    lhs = (y * z).sum(1)
    rhs = sum((x.astype(np.float64) * o).sum(1) for x, o in zip(xs, outs))
    np.testing.assert_allclose(lhs, rhs, rtol=1e-11, atol=1e-11)
    # the multi-layer sketch is the sum of single-layer sketches with their own layer ids
    if kind != "qk":
        parts = sum(O.apply(kind, [s], D, 77, [x], layer0=l) for l, (s, x) in enumerate(zip(shapes, xs)))
        np.testing.assert_allclose(y, parts, atol=1e-12)


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd", "qk"])
def test_norm_preservation_in_expectation(kind):
    """eq. jl_prob: E||S x||^2 = ||x||^2 over seeds (z-test on the mean ratio)."""
    n = 300
    D = 64
    rng = np.random.default_rng(0)
    x = rng.standard_normal((1, n)).astype(np.float32)
    x[0, :5] *= 10  # uneven mass
    nx = float((x.astype(np.float64) ** 2).sum())
    shape = (15, 20, 8, 8) if kind == "qk" else (1, n)
    r = np.array([(O.apply(kind, [shape], D, s, [x]) ** 2).sum() / nx for s in range(1500)])
    z = (r.mean() - 1.0) / (r.std(ddof=1) / np.sqrt(r.size))
    assert abs(z) < 4.5, (r.mean(), r.std())
