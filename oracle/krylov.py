"""fp64 oracle for the sketched Hessian-vector-product operator and the Arnoldi
iteration on it (Sec. 2: the sketch of the HVP is the map v -> Phi(HVP(Phi^T v))
of R^D to itself; Sec. 4, "Scaling eigenvalue estimation": Arnoldi with full
re-orthogonalisation builds the Krylov subspace in the sketched space, so the
stored basis vectors have D entries instead of N; Appendix "HVP in implicit vs
explicit form": the explicit form lifts v by Phi^T, applies the HVP in
parameter space and sketches the result).

TEST INFRASTRUCTURE ONLY (see the package docstring): the product never
imports this module and shares no code with it.

Synthetic Hessian (a stand-in for a model's HVP, which needs a trained model
and data):  H = shift I + sum_{j<r} lambda_j v_j v_j^T on the concatenated
parameters of the layer list (N_tot = sum of the element counts, no padding),
with v_j = s_j / sqrt(N_tot) and s_j the Rademacher vector of the "hvp" stream
(``orc_hvp_sign`` in sk_oracle.c).  Its spectrum is known in closed form: shift
with multiplicity N_tot - r and shift + eig(L^1/2 G L^1/2), G = V^T V.

Arnoldi (the textbook iteration, classical Gram-Schmidt applied twice per step
for the full re-orthogonalisation): q_0 = v0 / |v0|; for j = 0 .. k-1:
w = A q_j; two passes of c = Q_j^T w, w -= Q_j c with h[:j+1, j] the sum of the
two c; beta = |w|; h[j+1, j] = beta and q_{j+1} = w / beta, except when
beta <= BREAKDOWN_TOL |A q_j| (the Krylov space is exhausted to working
precision: the paper does not treat this case), where h[j+1, j] = 0 and
q_{j+1} = 0.  Then A Q_k = Q_{k+1} Hbar_k with Hbar_k the (k+1) x k upper
Hessenberg matrix, and the eigenvalues of its leading k x k block (the Ritz
values) estimate the operator's extreme eigenvalues.
"""
from __future__ import annotations

import numpy as np

from . import apply as _sk_apply
from . import apply_T as _sk_apply_T
from . import lib, _ptr

BREAKDOWN_TOL = 1e-5


# --- synthetic Hessian -------------------------------------------------------
def hvp_signs(seed: int, layer: int, j: int, start: int, count: int) -> np.ndarray:
    """Rademacher signs s_j of coordinates [start, start+count) of one layer (int8)."""
    o = np.zeros(count, dtype=np.int8)
    lib().orc_hvp_signs(seed, layer, j, start, count, _ptr(o))
    return o


def hvp(shapes, rank: int, lambdas, shift: float, seed: int, xs, layer0: int = 0):
    """y = H x for a batch given per layer ([batch, n_l] arrays); returns fp64 per layer.

    lambdas: the r eigen-weights; the product receives them as fp32, so callers
    comparing with it pass fp32-representable values."""
    lam = np.asarray(lambdas, dtype=np.float64)
    assert lam.shape == (rank,)
    ns = [int(s[0]) * int(s[1]) for s in shapes]
    ntot = float(sum(ns))
    xs = [np.ascontiguousarray(x, dtype=np.float64) for x in xs]
    batch = xs[0].shape[0]
    ys = [np.zeros((batch, n), dtype=np.float64) for n in ns]
    for b in range(batch):
        t = np.zeros(rank, dtype=np.float64)
        for li, (x, n) in enumerate(zip(xs, ns)):
            xb = np.ascontiguousarray(x[b])
            lib().orc_hvp_dots(seed, layer0 + li, rank, n, _ptr(xb), _ptr(t))
        coef = np.ascontiguousarray(lam * t / ntot)
        for li, (x, n) in enumerate(zip(xs, ns)):
            xb = np.ascontiguousarray(x[b])
            yb = np.zeros(n, dtype=np.float64)
            lib().orc_hvp_combine(seed, layer0 + li, rank, n, float(shift), _ptr(coef), _ptr(xb), _ptr(yb))
            ys[li][b] = yb
    return ys


def hvp_vectors(shapes, rank: int, seed: int) -> np.ndarray:
    """V = [v_0 .. v_{r-1}] as a dense N_tot x r fp64 matrix (small sizes only)."""
    cols = []
    for j in range(rank):
        parts = [hvp_signs(seed, li, j, 0, int(s[0]) * int(s[1])).astype(np.float64) for li, s in enumerate(shapes)]
        cols.append(np.concatenate(parts))
    V = np.stack(cols, axis=1)
    return V / np.sqrt(V.shape[0])


def hessian_spectrum_top(shapes, rank: int, lambdas, shift: float, seed: int) -> np.ndarray:
    """The r eigenvalues of H that differ from `shift`, descending: shift + eig(L^1/2 G L^1/2) with
    G = V^T V (H V = V (shift I + L G) and V has full column rank).  Streams over the layers, so it
    runs at full model size."""
    lam = np.asarray(lambdas, dtype=np.float64)
    gram = np.zeros((rank, rank), dtype=np.float64)
    ntot = 0
    for li, s in enumerate(shapes):
        n = int(s[0]) * int(s[1])
        ntot += n
        S = np.stack([hvp_signs(seed, li, j, 0, n).astype(np.float64) for j in range(rank)], axis=1)
        gram += S.T @ S
    gram /= ntot
    # eig(L G) = eig(G^1/2 L G^1/2) (similar matrices; G is positive definite)
    w, U = np.linalg.eigh(gram)
    gh = (U * np.sqrt(w)) @ U.T
    return np.sort(shift + np.linalg.eigvalsh(gh @ np.diag(lam) @ gh))[::-1]


# --- sketched HVP operator ---------------------------------------------------
def sketched_hvp(kind: str, shapes, D: int, seed: int, hvp_params: dict, v: np.ndarray) -> np.ndarray:
    """S H S^T v for v [batch, D]: the explicit form (lift, HVP, sketch)."""
    lifted = _sk_apply_T(kind, shapes, D, seed, np.atleast_2d(v))
    hx = hvp(shapes, xs=lifted, **hvp_params)
    return _apply_fp64(kind, shapes, D, seed, hx)


def _apply_fp64(kind, shapes, D, seed, xs):
    """Forward sketch of fp64 inputs: the oracle's fp64 chain, fed exactly by splitting each value into
    fp32 parts (the C chain reads fp32 or bf16) and summing the linear images."""
    rest = [np.asarray(x, dtype=np.float64) for x in xs]
    y = None
    for _ in range(3):  # three fp32 terms carry the 53-bit mantissa exactly
        part = [r.astype(np.float32) for r in rest]
        yy = _sk_apply(kind, shapes, D, seed, part)
        y = yy if y is None else y + yy
        rest = [r - p.astype(np.float64) for r, p in zip(rest, part)]
    return y


# --- Arnoldi -----------------------------------------------------------------
def arnoldi(op, v0: np.ndarray, k: int, tol: float = BREAKDOWN_TOL):
    """k steps of Arnoldi with two classical Gram-Schmidt passes per step.

    op: function R^D -> R^D (fp64).  Returns (Q [k+1, D], Hbar [(k+1), k])."""
    v0 = np.asarray(v0, dtype=np.float64)
    D = v0.size
    Q = np.zeros((k + 1, D), dtype=np.float64)
    Hb = np.zeros((k + 1, k), dtype=np.float64)
    nv = np.linalg.norm(v0)
    Q[0] = v0 / nv if nv > 0 else 0.0
    for j in range(k):
        w = np.asarray(op(Q[j]), dtype=np.float64).reshape(D)
        n0 = np.linalg.norm(w)
        for _ in range(2):
            c = Q[: j + 1] @ w
            w = w - Q[: j + 1].T @ c
            Hb[: j + 1, j] += c
        beta = np.linalg.norm(w)
        if beta > tol * n0:
            Hb[j + 1, j] = beta
            Q[j + 1] = w / beta
    return Q, Hb


def ritz_values(Hb: np.ndarray) -> np.ndarray:
    """Eigenvalues of the leading k x k block of Hbar, by decreasing real part."""
    k = Hb.shape[1]
    ev = np.linalg.eigvals(Hb[:k, :k])
    return ev[np.argsort(-ev.real)]


def top_rel_mae(est, truth, m: int = 10) -> float:
    """Relative mean absolute error of the m largest eigenvalues (the metric of the eigenvalue rows of
    the paper's quality tables): mean_i |est_i - truth_i| / |truth_i| over the m largest of each."""
    e = np.sort(np.real(np.asarray(est)))[::-1][:m]
    t = np.sort(np.asarray(truth, dtype=np.float64))[::-1][:m]
    return float(np.mean(np.abs(e - t) / np.abs(t)))


# --- intrinsic-dimension search ------------------------------------------------
def id_decide(tau_new: float, tau_old: float, d: int, tau_target: float, delta: float, D_max: int):
    """One decision of the search (Sec. 4, "Improving the search for the intrinsic dimension"): returns
    ("done", d) when the metric reached its target, ("fail", d) when doubling would pass D_max, else
    ("go", d') with d' = 2 d if the round improved the metric by less than delta, d otherwise."""
    if tau_new >= tau_target:
        return "done", d
    if tau_new - tau_old < delta:
        d = 2 * d
        if d > D_max:
            return "fail", d
    return "go", d


def id_search(kind: str, shapes, D: int, seed: int, hp: dict, theta0, d_min: int, tau_target: float, c: int,
              delta: float, max_rounds: int):
    """The intrinsic-dimension search on the synthetic quadratic objective L(theta) = 1/2 theta^T H theta
    (minimum 0 at theta* = 0), metric tau = 1 - L(theta) / L(theta0) (the fraction of the loss the
    finetuning removes; the full model reaches 1).

    Finetuning (the listing leaves it abstract): theta = theta0 + S^T omega with omega in R^D (D = D_max)
    and only omega[:d] free (the listing zeros the gradient's other components); c steps of linear
    conjugate gradients on omega[:d], restarted every round from the current omega.  For this objective
    f(omega) = L(theta0 + S^T omega) has gradient S H theta and Hessian M = S H S^T, so one CG step costs
    one sketched HVP.  A step with p.Mp <= 0 or r.r = 0 leaves the state unchanged.
    After each round: tau from the definition (lift, HVP, inner product) and id_decide.

    theta0: per layer a [n_l] array.  Returns dict(d, status, taus, ds, omega, L0) with status 0 (target
    reached, d the estimate), 1 (D_max exceeded) or 2 (max_rounds used)."""
    theta0 = [np.asarray(t, dtype=np.float64).reshape(1, -1) for t in theta0]
    omega = np.zeros(D, dtype=np.float64)

    def lift(om):
        st = _sk_apply_T(kind, shapes, D, seed, om[None, :])
        return [t + u for t, u in zip(theta0, st)]

    def loss_hx(th):
        hx = hvp(shapes, xs=th, **hp)
        return 0.5 * sum(float((a * b).sum()) for a, b in zip(th, hx)), hx

    def grad(om):
        _, hx = loss_hx(lift(om))
        return _apply_fp64(kind, shapes, D, seed, hx)[0]

    def M(p):
        return sketched_hvp(kind, shapes, D, seed, hp, p[None, :])[0]

    L0, _ = loss_hx(lift(omega))
    tau_old, d = 0.0, int(d_min)
    taus, ds = [], []
    for _ in range(max_rounds):
        r = grad(omega)
        r[d:] = 0.0
        p = -r
        rr = float(r @ r)
        for _ in range(c):
            q = M(p)
            q[d:] = 0.0
            pq = float(p @ q)
            if pq <= 0.0 or rr == 0.0:
                continue
            alpha = rr / pq
            omega += alpha * p
            r = r + alpha * q
            rr_new = float(r @ r)
            p = -r + (rr_new / rr) * p
            rr = rr_new
        L, _ = loss_hx(lift(omega))
        tau = 1.0 - L / L0
        taus.append(tau)
        ds.append(d)
        decision, d_next = id_decide(tau, tau_old, d, tau_target, delta, D)
        if decision == "done":
            return dict(d=d, status=0, taus=taus, ds=ds, omega=omega, L0=L0)
        if decision == "fail":
            return dict(d=0, status=1, taus=taus, ds=ds, omega=omega, L0=L0)
        d, tau_old = d_next, tau
    return dict(d=0, status=2, taus=taus, ds=ds, omega=omega, L0=L0)
