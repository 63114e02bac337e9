"""Pins of the fp64 oracle for the sketched HVP operator v -> S H S^T v and the Arnoldi
iteration on it (Sec. 2, sketch of the HVP; Sec. 4, "Scaling eigenvalue estimation";
Appendix "HVP in implicit vs explicit form").

Each pin checks the oracle against something other than itself: the Philox counter
layout of the synthetic Hessian's sign vectors, the dense definition of H, its closed-form
spectrum, symmetry, the Arnoldi relation, the exact spectrum after a full Krylov space,
the closed-form first Arnoldi step on diag(1..n), breakdown on a rank-r operator, and
the composition S H S^T = S V L (S V)^T when the shift is zero."""
import numpy as np
import pytest

import oracle as O
from oracle import krylov as K

SHAPES = [(1, 100), (30, 64), (1, 7), (5, 333)]
LAM = np.array([6.0, 3.5, -2.25, 1.0], dtype=np.float32)


def _hp(rank=4, shift=0.5, seed=3, lam=LAM):
    return dict(rank=rank, lambdas=lam[:rank], shift=shift, seed=seed)


def test_sign_layout_from_raw_philox():
    """Sign of coordinate e, layer l, vector j = bit (e & 31) of word ((e >> 5) & 3) of the Philox block with
    counter (lo32(e >> 7), hi32(e >> 7), (l << 6) | j, 10) under key (lo32 seed, hi32 seed)."""
    seed = 0x1234_5678_9ABC_DEF0
    for layer, j in [(0, 0), (3, 17), (200, 63)]:
        for e in [0, 31, 32, 127, 128, 5000, (1 << 33) + 77]:
            w = O.philox([e >> 7 & 0xFFFFFFFF, e >> 39, (layer << 6) | j, 10], [seed & 0xFFFFFFFF, seed >> 32])
            bit = (int(w[(e >> 5) & 3]) >> (e & 31)) & 1
            assert K.hvp_signs(seed, layer, j, e, 1)[0] == (-1 if bit else 1)


def test_signs_are_balanced_and_uncorrelated():
    n = 1 << 16
    s0 = K.hvp_signs(9, 0, 0, 0, n).astype(np.float64)
    s1 = K.hvp_signs(9, 0, 1, 0, n).astype(np.float64)
    s2 = K.hvp_signs(9, 1, 0, 0, n).astype(np.float64)
    bound = 4.5 / np.sqrt(n)
    assert abs(s0.mean()) < bound
    assert abs((s0 * s1).mean()) < bound  # vector index j changes the stream
    assert abs((s0 * s2).mean()) < bound  # layer index changes the stream


@pytest.mark.parametrize("rank,shift", [(1, 0.0), (4, 0.5), (4, -1.25)])
def test_hvp_equals_dense_definition(rank, shift):
    """The two-pass evaluation (all dots, then one combine) equals (shift I + V L V^T) x with V built
    column by column from the sign streams."""
    g = np.random.default_rng(0)
    xs = [g.standard_normal((2, r * c)) for r, c in SHAPES]
    ys = K.hvp(SHAPES, xs=xs, **_hp(rank, shift))
    V = K.hvp_vectors(SHAPES, rank, 3)
    H = shift * np.eye(V.shape[0]) + V @ np.diag(LAM[:rank].astype(np.float64)) @ V.T
    X, Y = np.concatenate(xs, axis=1), np.concatenate(ys, axis=1)
    assert np.abs(Y - X @ H.T).max() < 1e-12 * np.abs(Y).max()


def test_hvp_is_symmetric():
    g = np.random.default_rng(1)
    x = [g.standard_normal((1, r * c)) for r, c in SHAPES]
    y = [g.standard_normal((1, r * c)) for r, c in SHAPES]
    hx, hy = K.hvp(SHAPES, xs=x, **_hp()), K.hvp(SHAPES, xs=y, **_hp())
    a = sum(float((u * v).sum()) for u, v in zip(hx, y))
    b = sum(float((u * v).sum()) for u, v in zip(x, hy))
    assert abs(a - b) < 1e-12 * max(abs(a), 1.0)


def test_hvp_spectrum_closed_form():
    """eig(H) = {shift} (N - r times) and shift + eig(L^1/2 G L^1/2), G = V^T V: the operator is probed
    only through the two-pass hvp on the identity's columns."""
    shapes = [(1, 50), (3, 41)]
    n = sum(r * c for r, c in shapes)
    hp = _hp(4, 0.75)
    eye = np.eye(n)
    cols = K.hvp(shapes, xs=[eye[:, :50], eye[:, 50:]], **hp)
    Hd = np.concatenate(cols, axis=1)  # row i = H e_i
    ev = np.sort(np.linalg.eigvalsh(0.5 * (Hd + Hd.T)))[::-1]
    top = K.hessian_spectrum_top(shapes, **hp)
    spike = np.sort(np.concatenate([top, np.full(n - 4, 0.75)]))[::-1]
    assert np.abs(ev - spike).max() < 1e-12 * np.abs(spike).max()
    # the spikes are near lambda + shift because the sign vectors are nearly orthogonal
    assert np.abs(np.sort(top) - np.sort(LAM.astype(np.float64) + 0.75)).max() < 0.6


def _sym_matrix(n, seed):
    g = np.random.default_rng(seed)
    a = g.standard_normal((n, n))
    return a + a.T


def test_arnoldi_relation_and_orthonormal_basis():
    n, k = 60, 25
    A = _sym_matrix(n, 2)
    A[0, 1] += 0.3  # a nonsymmetric operator: the relation holds for any A
    v0 = np.random.default_rng(3).standard_normal(n)
    Q, Hb = K.arnoldi(lambda v: A @ v, v0, k)
    assert np.abs(A @ Q[:k].T - Q.T @ Hb).max() < 1e-12 * np.abs(A).max()
    assert np.abs(Q @ Q.T - np.eye(k + 1)).max() < 1e-13
    assert np.allclose(Q[0], v0 / np.linalg.norm(v0))
    assert np.abs(np.tril(Hb, -2)).max() == 0.0


def test_arnoldi_full_space_gives_the_spectrum():
    """After n steps on an n x n operator the Krylov space is R^n: the Ritz values are its eigenvalues and
    the last step breaks down (h[n, n-1] = 0)."""
    n = 14
    A = _sym_matrix(n, 4)
    Q, Hb = K.arnoldi(lambda v: A @ v, np.random.default_rng(5).standard_normal(n), n)
    assert Hb[n, n - 1] == 0.0
    ritz = np.sort(K.ritz_values(Hb).real)
    assert np.abs(ritz - np.sort(np.linalg.eigvalsh(A))).max() < 1e-10


def test_arnoldi_symmetric_operator_gives_tridiagonal():
    n, k = 80, 30
    A = _sym_matrix(n, 6)
    _, Hb = K.arnoldi(lambda v: A @ v, np.ones(n), k)
    T = Hb[:k, :k]
    scale = np.abs(T).max()
    assert np.abs(np.triu(T, 2)).max() < 1e-10 * scale
    assert np.abs(T - T.T).max() < 1e-10 * scale


def test_arnoldi_first_step_closed_form():
    """On diag(1..n) from the all-ones vector: h00 is the mean (n + 1)/2 of the diagonal and h10 its
    standard deviation sqrt((n^2 - 1)/12)."""
    n = 101
    d = np.arange(1, n + 1, dtype=np.float64)
    _, Hb = K.arnoldi(lambda v: d * v, np.ones(n), 1)
    assert abs(Hb[0, 0] - (n + 1) / 2) < 1e-12 * n
    assert abs(Hb[1, 0] - np.sqrt((n * n - 1) / 12.0)) < 1e-12 * n


def test_arnoldi_rank_r_operator_breaks_down():
    """A rank-3 symmetric operator and a start vector in its range: the Krylov space has dimension 3, so
    the step that forms q_3 breaks down and the three Ritz values are the nonzero eigenvalues."""
    n = 40
    U = np.linalg.qr(np.random.default_rng(7).standard_normal((n, 3)))[0]
    A = U @ np.diag([5.0, -2.0, 0.7]) @ U.T
    Q, Hb = K.arnoldi(lambda v: A @ v, U @ np.random.default_rng(8).standard_normal(3), 6)
    assert Hb[3, 2] == 0.0 and np.all(Q[3:] == 0.0) and np.all(Hb[:, 3:] == 0.0)
    assert np.allclose(np.sort(np.linalg.eigvals(Hb[:3, :3]).real), [-2.0, 0.7, 5.0], atol=1e-12)


def _dense_sketched(kind, shapes, D, seed, hp):
    return K.sketched_hvp(kind, shapes, D, seed, hp, np.eye(D))  # row i = S H S^T e_i


@pytest.mark.parametrize("kind", ["afjl", "affd", "fjl", "ffd"])
def test_sketched_operator_symmetric(kind):
    shapes, D = [(1, 300), (20, 40)], 64
    M = _dense_sketched(kind, shapes, D, 11, _hp())
    assert np.abs(M - M.T).max() < 1e-12 * np.abs(M).max()


@pytest.mark.parametrize("kind", ["afjl", "affd"])
def test_sketched_operator_composition(kind):
    """Shift 0: S H S^T = (S V) L (S V)^T with S V the sketches of the Hessian's own vectors (forward
    sketches only, no transpose), so the lift - HVP - sketch order is checked independently."""
    shapes, D = [(1, 300), (20, 40)], 64
    hp = _hp(4, 0.0)
    M = _dense_sketched(kind, shapes, D, 11, hp)
    V = K.hvp_vectors(shapes, 4, hp["seed"])
    n0 = 300
    SV = K._apply_fp64(kind, shapes, D, 11, [V[:n0].T, V[n0:].T]).T  # D x r
    ref = SV @ np.diag(LAM.astype(np.float64)) @ SV.T
    assert np.abs(M - ref).max() < 1e-12 * np.abs(ref).max()


def test_arnoldi_on_sketched_operator_full_space():
    shapes, D = [(1, 300), (20, 40)], 16
    hp = _hp(4, 0.5)
    M = _dense_sketched("afjl", shapes, D, 11, hp)
    op = lambda v: K.sketched_hvp("afjl", shapes, D, 11, hp, v)[0]
    _, Hb = K.arnoldi(op, np.random.default_rng(12).standard_normal(D), D)
    ritz = np.sort(K.ritz_values(Hb).real)
    assert np.abs(ritz - np.sort(np.linalg.eigvalsh(0.5 * (M + M.T)))).max() < 1e-10 * np.abs(M).max()


@pytest.mark.parametrize("kind,D", [("afjl", 2048), ("affd", 1024)])
def test_sketched_top_eigenvalues_near_hessian(kind, D):
    """Sanity check of the purpose (quality of sketches is not pinned by the paper): with a well separated
    rank-10 spike, the top Ritz values of the sketched operator are within 10% of H's spikes (the paper
    reports relative errors below 5% at D = 2^10 .. 2^12 on real models)."""
    shapes = [(64, 512), (1, 4000), (30, 300)]
    lam = np.array([40, 32, 25, 20, 16, 12.5, 10, 8, 6.5, 5], dtype=np.float32)
    hp = dict(rank=10, lambdas=lam, shift=0.0, seed=21)
    op = lambda v: K.sketched_hvp(kind, shapes, D, 5, hp, v)[0]
    _, Hb = K.arnoldi(op, np.random.default_rng(13).standard_normal(D), 14)
    truth = K.hessian_spectrum_top(shapes, **hp)
    assert K.top_rel_mae(K.ritz_values(Hb), truth, 10) < 0.1


# --- intrinsic-dimension search (Sec. 4, "Improving the search for the intrinsic dimension") -------------
def test_id_decide_rules():
    """The listing's rules: stop at the target; double d when a round improves the metric by less than delta
    (failing past D_max); otherwise keep d."""
    assert K.id_decide(0.95, 0.1, 8, 0.9, 0.05, 64) == ("done", 8)
    assert K.id_decide(0.30, 0.28, 8, 0.9, 0.05, 64) == ("go", 16)
    assert K.id_decide(0.30, 0.20, 8, 0.9, 0.05, 64) == ("go", 8)
    assert K.id_decide(0.30, 0.28, 64, 0.9, 0.05, 64) == ("fail", 128)
    assert K.id_decide(0.90, 0.89, 64, 0.9, 0.05, 64) == ("done", 64)  # the target wins over a small step


def _id_problem(rank=4, shift=0.0, shapes=((1, 3000), (20, 250))):
    hp = dict(rank=rank, lambdas=np.ones(rank, dtype=np.float32), shift=shift, seed=9)
    g = np.random.default_rng(0)
    x = [g.standard_normal((1, a * b)) for a, b in shapes]
    th0 = [t[0] for t in K.hvp(list(shapes), xs=x, **dict(hp, shift=0.0))]  # theta0 in the span of the v_j
    return list(shapes), hp, th0


def test_id_objective_gradient_by_finite_differences():
    """The finetuning gradient S H (theta0 + S^T omega) against central differences of
    L(theta0 + S^T omega) = 1/2 theta^T H theta, on a few coordinates of omega."""
    shapes, hp, th0 = _id_problem(shift=0.25)
    D, seed = 64, 3
    om = np.random.default_rng(1).standard_normal(D) * 0.1

    def loss(o):
        th = [t + u for t, u in zip([np.asarray(t)[None, :] for t in th0],
                                    O.apply_T("afjl", shapes, D, seed, o[None, :]))]
        return 0.5 * sum(float((a * b).sum()) for a, b in zip(th, K.hvp(shapes, xs=th, **hp)))

    th = [t[None, :] + u for t, u in zip(th0, O.apply_T("afjl", shapes, D, seed, om[None, :]))]
    g = K._apply_fp64("afjl", shapes, D, seed, K.hvp(shapes, xs=th, **hp))[0]
    eps = 1e-4
    for i in [0, 5, 63]:
        e = np.zeros(D)
        e[i] = eps
        fd = (loss(om + e) - loss(om - e)) / (2 * eps)
        assert abs(fd - g[i]) < 1e-6 * max(1.0, abs(g[i]))


def test_id_search_known_answer():
    """A rank-4 quadratic with theta0 in the span of its spikes and no bulk: a d-dimensional subspace
    removes all of the loss exactly when d >= 4 (CG converges in at most rank steps), so the search
    from d = 1 returns 4; the frozen coordinates of omega stay zero."""
    shapes, hp, th0 = _id_problem()
    res = K.id_search("afjl", shapes, 256, 3, hp, th0, 1, 0.9, 6, 0.05, 12)
    assert res["status"] == 0 and res["d"] == 4
    assert res["taus"][-1] > 1 - 1e-9
    assert all(t < 0.9 for t in res["taus"][:-1])
    assert np.all(res["omega"][4:] == 0.0)


def test_id_search_round_minimises_on_the_subspace():
    """With c >= rank CG steps a round reaches the minimum of L on theta0 + S^T span(e_0..e_{d-1}): the
    gradient's free components vanish."""
    shapes, hp, th0 = _id_problem(rank=3, shift=0.0)
    D, seed = 128, 4
    res = K.id_search("afjl", shapes, D, seed, hp, th0, 2, 1.1, 5, -1.0, 1)  # one round at d = 2
    om = res["omega"]
    th = [t[None, :] + u for t, u in zip(th0, O.apply_T("afjl", shapes, D, seed, om[None, :]))]
    g = K._apply_fp64("afjl", shapes, D, seed, K.hvp(shapes, xs=th, **hp))[0]
    g0 = K._apply_fp64("afjl", shapes, D, seed, K.hvp(shapes, xs=[t[None, :] for t in th0], **hp))[0]
    assert np.abs(g[:2]).max() < 1e-9 * np.abs(g0).max()


def test_id_search_fails_past_D_max():
    shapes, hp, th0 = _id_problem(rank=8)
    res = K.id_search("afjl", shapes, 16, 3, hp, th0, 4, 0.999999, 2, 0.5, 20)
    assert res["status"] == 1 and res["d"] == 0
