"""Pins for the CPU oracle: checks against facts the paper and mathematics fix.

Each ``pin_*`` takes a namespace ``o`` exposing the oracle's functions (the
real module, or a deliberately broken copy in the mutation tests) and raises
AssertionError when the oracle disagrees with the pinned fact.  None of the
pins re-types the oracle's own formula: each compares against an
independent route (closed form, brute force, another library algorithm, or a
lemma of the paper).
"""
from __future__ import annotations

import numpy as np

rng = np.random.default_rng


def _spd(n, cond, seed):
    r = rng(seed)
    Q, _ = np.linalg.qr(r.standard_normal((n, n)))
    lam = np.logspace(0, np.log10(cond), n)
    return (Q * lam) @ Q.T


def _relf(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


# ------------------------------------------------------------------ stats
def pin_stats_rank1(o):
    """G = u v^T gives G G^T = |v|^2 u u^T and G^T G = |u|^2 v v^T
    (rank-one gradients, appendix comparing with K-FAC)."""
    r = rng(1)
    u, v = r.standard_normal(7), r.standard_normal(5)
    L, R = o.stats_update(np.zeros((7, 7)), np.zeros((5, 5)), np.outer(u, v))
    assert _relf(L, (v @ v) * np.outer(u, u)) < 1e-14
    assert _relf(R, (u @ u) * np.outer(v, v)) < 1e-14


def pin_stats_trace(o):
    """tr L_t = tr R_t = sum_s ||G_s||_F^2 (both sides from zero)."""
    r = rng(2)
    L, R = np.zeros((6, 6)), np.zeros((9, 9))
    tot = 0.0
    for _ in range(4):
        G = r.standard_normal((6, 9))
        tot += float(np.sum(G * G))
        L, R = o.stats_update(L, R, G)
    assert abs(np.trace(L) - tot) < 1e-12 * tot
    assert abs(np.trace(R) - tot) < 1e-12 * tot


def pin_stats_integer_bruteforce(o):
    """Integer gradients: the sums are exact; compare with a pure-Python
    triple loop over the definition of L_t and R_t."""
    r = rng(3)
    m, n, T = 4, 3, 3
    Gs = [r.integers(-5, 6, size=(m, n)) for _ in range(T)]
    L, R = np.zeros((m, m)), np.zeros((n, n))
    for G in Gs:
        L, R = o.stats_update(L, R, G)
    Lb = [[sum(int(G[i, k]) * int(G[j, k]) for G in Gs for k in range(n))
           for j in range(m)] for i in range(m)]
    Rb = [[sum(int(G[k, i]) * int(G[k, j]) for G in Gs for k in range(m))
           for j in range(n)] for i in range(n)]
    assert np.array_equal(L, np.array(Lb, dtype=float))
    assert np.array_equal(R, np.array(Rb, dtype=float))


def pin_stats_onehot_embedding(o):
    """Embedding layer with one-hot inputs: G = dy x^T and x^T x = I give
    G G^T = dy dy^T; with multi-hot columns x^T x is diagonal (appendix
    "Shampoo for embedding layers")."""
    r = rng(4)
    d, N, m = 5, 40, 6
    dy = r.standard_normal((d, m))
    x = np.zeros((N, m))
    x[r.choice(N, m, replace=False), np.arange(m)] = 1.0
    L, _ = o.stats_update(np.zeros((d, d)), None, dy @ x.T)
    assert _relf(L, dy @ dy.T) < 1e-13
    # multi-hot: column j has c_j ones in rows no other column uses
    x = np.zeros((N, m))
    rows = r.permutation(N)
    counts = [1, 2, 3, 1, 2, 4]
    s = 0
    for j, c in enumerate(counts):
        x[rows[s:s + c], j] = 1.0
        s += c
    L, _ = o.stats_update(np.zeros((d, d)), None, dy @ x.T)
    assert _relf(L, dy @ np.diag(counts) @ dy.T) < 1e-13


def pin_embedding_lookup_matrix(o):
    """Row-major table: G = S dy with S[idx_e, feat_e] += w_e the dense
    lookup matrix (vocab x m); with distinct one-hot rows S^T S = I, so the
    right statistic G^T G equals dy^T dy (appendix "Shampoo for embedding
    layers"); with repeats it equals dy^T (S^T S) dy."""
    r = rng(30)
    V, d, m = 50, 4, 9
    dy = r.standard_normal((m, d))
    idx = r.choice(V, m, replace=False)
    G = o.embedding_grad(V, idx, None, None, dy)
    _, R = o.stats_update(None, np.zeros((d, d)), G)
    assert _relf(R, dy.T @ dy) < 1e-13
    # multi-hot with repeats and weights
    nnz = 25
    idx = r.integers(0, 12, nnz)
    feat = r.integers(0, m, nnz)
    w = r.standard_normal(nnz)
    S = np.zeros((V, m))
    for e in range(nnz):
        S[idx[e], feat[e]] += w[e]
    G = o.embedding_grad(V, idx, feat, w, dy)
    assert _relf(G, S @ dy) < 1e-13
    _, R = o.stats_update(None, np.zeros((d, d)), G)
    assert _relf(R, dy.T @ (S.T @ S) @ dy) < 1e-12
    rows, U = o.embedding_rows(V, idx, feat, w, dy)
    assert list(rows) == sorted(set(int(i) for i in idx))
    assert np.array_equal(U, G[rows])


def pin_embedding_worked_example(o):
    """5-row table, d = 2, dy rows (1,2), (3,4), (5,6); entries (row, feature,
    weight): (3,0,1), (1,1,1), (3,2,1/2), (1,0,2), plus three invalid ones
    (row 5, row -1, feature 3) that are dropped.  By hand: row 1 = dy1 +
    2 dy0 = (5, 8), row 3 = dy0 + dy2/2 = (3.5, 5), all other rows 0."""
    dy = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]])
    idx = [3, 1, 3, 1, 5, -1, 0]
    feat = [0, 1, 2, 0, 0, 1, 3]
    w = [1.0, 1.0, 0.5, 2.0, 1.0, 1.0, 1.0]
    G = o.embedding_grad(5, idx, feat, w, dy)
    want = np.zeros((5, 2))
    want[1] = [5.0, 8.0]
    want[3] = [3.5, 5.0]
    assert np.array_equal(G, want)
    rows, U = o.embedding_rows(5, idx, feat, w, dy)
    assert list(rows) == [1, 3] and np.array_equal(U, [[5.0, 8.0], [3.5, 5.0]])


def pin_stats_ema(o):
    """beta2 < 1 with a constant gradient: L_t = (1 - beta2^t) G G^T
    (geometric series of Algorithm 2's EMA from L_0 = 0)."""
    r = rng(5)
    G = r.standard_normal((4, 6))
    b2, t = 0.9, 7
    L, R = np.zeros((4, 4)), np.zeros((6, 6))
    for _ in range(t):
        L, R = o.stats_update(L, R, G, beta2=b2)
    f = 1.0 - b2 ** t
    assert _relf(L, f * G @ G.T) < 1e-13
    assert _relf(R, f * G.T @ G) < 1e-13


def pin_lemma1(o):
    """Lemma 1: with rank <= r gradients, H_hat <= r L^{1/p} (x) R^{1/q}
    for 1/p + 1/q = 1 (Loewner order); vec is row stacking."""
    r = rng(6)
    m, n, rank, eps = 3, 4, 2, 1e-3
    L, R = np.zeros((m, m)), np.zeros((n, n))
    H = eps * np.eye(m * n)
    for _ in range(3):
        G = r.standard_normal((m, rank)) @ r.standard_normal((rank, n))
        L, R = o.stats_update(L, R, G)
        g = G.reshape(-1)
        H += np.outer(g, g)
    L += eps * np.eye(m)
    R += eps * np.eye(n)
    for p in (2.0, 3.0, 1.5):
        q = p / (p - 1.0)
        Lp, _, _ = o.inv_root(L, -p)       # L^{1/p}
        Rq, _, _ = o.inv_root(R, -q)
        gap = rank * np.kron(Lp, Rq) - H
        assert np.linalg.eigvalsh(0.5 * (gap + gap.T)).min() > -1e-9


def pin_lemma2(o):
    """Lemma 2: H_hat <= k B_t with B_t block diagonal over k sub-vectors."""
    r = rng(7)
    m, k, eps = 3, 4, 1e-3
    H = eps * np.eye(m * k)
    blocks = [eps * np.eye(m) for _ in range(k)]
    for _ in range(5):
        g = r.standard_normal(m * k)
        H += np.outer(g, g)
        for j in range(k):
            gj = g[j * m:(j + 1) * m].reshape(m, 1)
            blocks[j], _ = o.stats_update(blocks[j], None, gj)
    B = np.zeros((m * k, m * k))
    for j in range(k):
        B[j * m:(j + 1) * m, j * m:(j + 1) * m] = blocks[j]
    gap = k * B - H
    assert np.linalg.eigvalsh(gap).min() > -1e-9


# ------------------------------------------------------------------ roots
def pin_root_diagonal(o):
    """diag(d) + eps I -> diag((d + eps)^(-1/p))."""
    d = np.array([0.5, 2.0, 7.0, 1e-3, 30.0])
    for p in (1, 2, 3, 4, 6, 8):
        X, st, _ = o.inv_root(np.diag(d), p, eps=1e-4)
        assert st == o.CONVERGED
        assert np.max(np.abs(X - np.diag((d + 1e-4) ** (-1.0 / p)))) < 1e-12 * np.max(X)


def pin_root_scaled_identity(o):
    """c I -> (c + eps)^(-1/p) I, also with eps relative to lambda_max = c."""
    n, c = 6, 3.7
    for p in (2, 4):
        X, _, _ = o.inv_root(c * np.eye(n), p, eps=0.1)
        assert np.allclose(X, (c + 0.1) ** (-1.0 / p) * np.eye(n), rtol=1e-13, atol=0)
        X, _, e = o.inv_root(c * np.eye(n), p, eps=0.1, eps_relative=True)
        assert abs(e - 0.1 * c) < 1e-12
        assert np.allclose(X, (c * 1.1) ** (-1.0 / p) * np.eye(n), rtol=1e-12, atol=0)


def pin_root_p1_inverse(o):
    """p = 1 is the ordinary inverse (LU-based numpy.linalg.inv)."""
    A = _spd(12, 1e3, 8)
    X, _, _ = o.inv_root(A, 1, eps=1e-3)
    assert _relf(X, np.linalg.inv(A + 1e-3 * np.eye(12))) < 1e-11


def pin_root_p2_square(o):
    """p = 2: X^2 (A + eps I) = I."""
    A = _spd(10, 1e4, 9)
    X, _, _ = o.inv_root(A, 2, eps=1e-2)
    assert np.linalg.norm(X @ X @ (A + 1e-2 * np.eye(10)) - np.eye(10)) < 1e-10


def pin_root_invariant(o):
    """||X^p (A + eps I) - I||_F <= 1e-6 at condition numbers up to 1e6."""
    for n, cond, p in ((64, 1e3, 4), (96, 1e6, 4), (80, 1e6, 2), (48, 1e5, 8), (40, 1e4, 3), (36, 1e4, 6)):
        A = _spd(n, cond, 10 + n)
        X, _, _ = o.inv_root(A, p, eps=1e-6)
        res = np.linalg.matrix_power(X, p) @ (A + 1e-6 * np.eye(n)) - np.eye(n)
        assert np.linalg.norm(res) <= 1e-6


def pin_root_mpmath_4x4(o):
    """4 x 4 brute force at 50 digits: mpmath powm(A + eps I, -1/p)."""
    import mpmath as mp
    mp.mp.dps = 50
    r = rng(11)
    B = r.standard_normal((4, 4))
    A = B @ B.T + 0.1 * np.eye(4)
    for p in (2, 4):
        X, _, _ = o.inv_root(A, p, eps=1e-3)
        Am = mp.matrix([[mp.mpf(float(A[i, j])) + (mp.mpf('1e-3') if i == j else 0)
                         for j in range(4)] for i in range(4)])
        Xm = mp.powm(Am, mp.mpf(-1) / p)
        Xb = np.array([[float(mp.re(Xm[i, j])) for j in range(4)] for i in range(4)])
        assert _relf(X, Xb) < 1e-13


def pin_root_2x2_closed_form(o):
    """2 x 2 SPD square root: sqrt(A) = (A + s I) / t, s = sqrt(det A),
    t = sqrt(tr A + 2 s); A^{-1/4} is the inverse of sqrt(sqrt(A))."""
    A = np.array([[3.0, 1.2], [1.2, 2.0]])

    def sqrt2(M):
        s = np.sqrt(np.linalg.det(M))
        return (M + s * np.eye(2)) / np.sqrt(np.trace(M) + 2 * s)
    X, _, _ = o.inv_root(A, 4)
    assert _relf(X, np.linalg.inv(sqrt2(sqrt2(A)))) < 1e-14
    X, _, _ = o.inv_root(A, 2)
    assert _relf(X, np.linalg.inv(sqrt2(A))) < 1e-14


def pin_root_schur_pade(o):
    """scipy's fractional_matrix_power (Schur-Pade, not eigh) agrees."""
    from scipy.linalg import fractional_matrix_power
    A = _spd(40, 1e4, 12)
    for p in (2, 4, 8):
        X, _, _ = o.inv_root(A, p, eps=1e-5)
        Y = np.real(fractional_matrix_power(A + 1e-5 * np.eye(40), -1.0 / p))
        assert _relf(X, Y) < 1e-10


def pin_root_kronecker(o):
    """(A (x) B)^a = A^a (x) B^a (Preliminaries)."""
    A, B = _spd(3, 20.0, 13), _spd(4, 50.0, 14)
    X, _, _ = o.inv_root(np.kron(A, B), 4)
    XA, _, _ = o.inv_root(A, 4)
    XB, _, _ = o.inv_root(B, 4)
    assert _relf(X, np.kron(XA, XB)) < 1e-12


def pin_root_not_pd(o):
    """A^alpha with alpha < 0 is undefined unless positive definite."""
    A = np.diag([1.0, 2.0, -0.5])
    X, st, _ = o.inv_root(A, 4, eps=0.1)
    assert st == o.NOT_PD and X is None


def pin_root_asymmetric_input(o):
    """An input that is symmetric up to a perturbation gives the root of its
    symmetric part: add a skew matrix and the result must not change."""
    A = _spd(8, 100.0, 15)
    S = rng(16).standard_normal((8, 8))
    X0, _, _ = o.inv_root(A, 4)
    X1, _, _ = o.inv_root(A + 1e-3 * (S - S.T), 4)
    assert _relf(X1, X0) < 1e-13


def pin_cond_damped(o):
    """Condition number of the damped matrix A + eps_eff I: for a rotated
    diagonal d it is (max d + eps_eff) / (min d + eps_eff), with eps_eff = eps
    (absolute) or eps * max d (relative, MaxSV of an isolated top eigenvalue);
    an indefinite damped matrix has no finite condition number."""
    r = rng(18)
    Q, _ = np.linalg.qr(r.standard_normal((9, 9)))
    d = np.array([1e-6, 3e-5, 0.01, 0.2, 0.5, 0.9, 1.0, 1.3, 40.0])
    A = (Q * d) @ Q.T
    for eps in (0.0, 1e-6, 1e-3):
        want = (d.max() + eps) / (d.min() + eps)
        assert abs(o.cond_damped(A, eps) - want) < 1e-6 * want
    for eps in (1e-6, 1e-8):
        e = eps * d.max()
        want = (d.max() + e) / (d.min() + e)
        assert abs(o.cond_damped(A, eps, eps_relative=True) - want) < 1e-6 * want
        # the lambda_max the GPU reports may be passed in instead of MaxSV's
        assert abs(o.cond_damped(A, eps, eps_relative=True, lam_max=2.0 * d.max())
                   - (d.max() + 2 * e) / (d.min() + 2 * e)) < 1e-6 * want
    # a slightly asymmetric input: condition of its symmetric part
    S = r.standard_normal((9, 9))
    want = (d.max() + 1e-3) / (d.min() + 1e-3)
    assert abs(o.cond_damped(A + 1e-7 * (S - S.T), 1e-3) - want) < 1e-6 * want
    assert o.cond_damped(np.diag([1.0, 2.0, -0.5]), 0.1) == np.inf


def pin_root_shared_eig(o):
    """One eigendecomposition reused for several orders and dampings gives
    exactly the results of separate calls (roots and condition numbers)."""
    A = _spd(30, 1e5, 19)
    eig = o.sym_eig(A)
    for p, eps, relative in ((2, 1e-6, True), (4, 1e-8, True), (4, 1e-3, False)):
        X0, s0, e0 = o.inv_root(A, p, eps, relative)
        X1, s1, e1 = o.inv_root(A, p, eps, relative, eig=eig)
        assert s0 == s1 and e0 == e1 and np.array_equal(X0, X1)
        assert o.cond_damped(A, eps, relative) == o.cond_damped(A, eps, relative, eig=eig)


# ------------------------------------------------------------------ MaxSV
def pin_maxsv(o):
    """Power iteration converges to the top eigenvalue when it is isolated."""
    r = rng(17)
    Q, _ = np.linalg.qr(r.standard_normal((30, 30)))
    lam = np.concatenate([np.linspace(0.1, 1.0, 29), [5.0]])
    A = (Q * lam) @ Q.T
    l, steps = o.max_sv(A, n_step=500, tol=1e-12)
    assert abs(l - 5.0) < 1e-9 and steps < 500


# ------------------------------------------------------------------ coupled Newton (Algorithm 1)
def pin_newton_vs_eigh(o):
    """The fp64 coupled iteration reaches the eigh-defined root to 1e-9."""
    for n, cond, p in ((64, 1e2, 4), (64, 1e6, 4), (48, 1e6, 2), (32, 1e4, 8), (40, 1e3, 1), (40, 1e4, 3),
                       (36, 1e3, 6), (30, 1e3, 7)):
        A = _spd(n, cond, 20 + n + p)
        res = o.coupled_newton(A, p, eps=1e-6, tol=1e-12)
        X, _, _ = o.inv_root(A, p, eps=1e-6)
        assert res['status'] in (o.CONVERGED, o.STAGNATED)
        assert _relf(res['X'], X) < 1e-9


def pin_newton_scalar_iters(o):
    """On a diagonal input every eigenvalue follows the scalar recurrence
    m <- ((p+1-m)/p)^p m from m0 = z lambda_i, so the iteration count is
    the largest count over the diagonal, and the iterate stays diagonal."""
    d = np.array([1e-3, 0.1, 1.0, 3.0, 50.0])
    for p in (2, 3, 4, 6):
        res = o.coupled_newton(np.diag(d), p, eps=0.0, tol=1e-12)
        z = (1.0 + p) / (2.0 * np.linalg.norm(d))
        want = max(o.scalar_newton_iters(z * x, p, 1e-12) for x in d)
        assert abs(res['iters'] - want) <= 1
        assert np.count_nonzero(res['X'] - np.diag(np.diag(res['X']))) == 0
        assert _relf(np.diag(res['X']), d ** (-1.0 / p)) < 1e-10
    # heavy damping: z is set by the damped matrix (Frobenius norm taken
    # after the ridge), which fixes the count through the same recurrence
    d2, eps = np.array([1e-3, 1.0, 3.0]), 100.0
    for p in (2, 4):
        res = o.coupled_newton(np.diag(d2), p, eps=eps, tol=1e-12)
        z = (1.0 + p) / (2.0 * np.linalg.norm(d2 + eps))
        want = max(o.scalar_newton_iters(z * (x + eps), p, 1e-12) for x in d2)
        assert res['status'] == o.CONVERGED and abs(res['iters'] - want) <= 1
        assert _relf(np.diag(res['X']), (d2 + eps) ** (-1.0 / p)) < 1e-12


def pin_newton_power4_scaling(o):
    """Power-bound start: z = (p+1) / (2 (sum_i lambda_i^8)^(1/8)) on a
    diagonal input (the bound from its eigenvalues directly), so the count is
    the scalar recurrence's from z lambda_i; the result is the eigh root, and
    a flat spectrum needs far fewer iterations than the Frobenius start."""
    d = np.array([0.7, 1.0, 1.3, 1.1, 0.9, 1.2] * 40)
    for p in (2, 4):
        res = o.coupled_newton(np.diag(d), p, eps=0.0, tol=1e-12, scaling='power4')
        z = (1.0 + p) / (2.0 * np.sum(d ** 8) ** 0.125)
        want = max(o.scalar_newton_iters(z * x, p, 1e-12) for x in d)
        assert abs(res['iters'] - want) <= 1
        assert _relf(np.diag(res['X']), d ** (-1.0 / p)) < 1e-10
        fro = o.coupled_newton(np.diag(d), p, eps=0.0, tol=1e-12)
        assert res['iters'] + 2 <= fro['iters']
    A = _spd(48, 1e4, 77)
    res = o.coupled_newton(A, 4, eps=1e-6, tol=1e-12, scaling='power4')
    X, _, _ = o.inv_root(A, 4, eps=1e-6)
    assert _relf(res['X'], X) < 1e-9


def pin_newton_status_rules(o):
    """MAXITER at a tiny cap, DIVERGED on an indefinite matrix, STAGNATED
    when the tolerance is below what fp64 can reach, MaxSV damping used."""
    A = _spd(16, 1e3, 30)
    assert o.coupled_newton(A, 4, eps=0.0, tol=1e-12, max_iters=1)['status'] == o.MAXITER
    assert o.coupled_newton(np.diag([1.0, 2.0, -1.0]), 4, tol=1e-10)['status'] == o.DIVERGED
    res = o.coupled_newton(A, 4, tol=0.0)
    assert res['status'] == o.STAGNATED and res['resid'] < 1e-12
    res = o.coupled_newton(A, 4, eps=1e-3, eps_relative=True, tol=1e-12)
    lmax = np.linalg.eigvalsh(A).max()
    assert abs(res['eps_eff'] - 1e-3 * lmax) < 1e-6 * lmax


def pin_newton_warm(o):
    """Warm start (coupled-Newton appendix): the exact previous root needs
    no iteration; a commuting diagonal start follows the scalar recurrence
    from m0 = x0^p d to the exact root; a non-commuting start converges to
    X0 (X0^p A)^{-1/p} (scipy's Schur-Pade power of a non-symmetric matrix);
    an ill-conditioned drift trips the commutator monitor and falls back to
    the cold root."""
    from scipy.linalg import fractional_matrix_power
    A = _spd(24, 1e2, 90)
    X, _, _ = o.inv_root(A, 4, eps=1e-6)
    res = o.coupled_newton_warm(A, 4, X, eps=1e-6, tol=1e-9)
    assert res['iters'] == 0 and not res['warm_aborted'] and np.array_equal(res['X'], X)
    d = np.array([0.5, 1.0, 2.0, 4.0])
    for p in (2, 4):
        x0 = d ** (-1.0 / p) * np.array([1.1, 0.9, 1.05, 0.8])
        res = o.coupled_newton_warm(np.diag(d), p, np.diag(x0), tol=1e-12)
        want = max(o.scalar_newton_iters(x ** p * y, p, 1e-12) for x, y in zip(x0, d))
        assert not res['warm_aborted'] and abs(res['iters'] - want) <= 1
        assert _relf(np.diag(res['X']), d ** (-1.0 / p)) < 1e-12
    B = A + 1e-3 * _spd(24, 10.0, 91)
    res = o.coupled_newton_warm(B, 4, X, eps=1e-6, tol=1e-12)
    Bd = B + 1e-6 * np.eye(24)
    lim = X @ np.real(fractional_matrix_power(np.linalg.matrix_power(X, 4) @ Bd, -0.25))
    assert not res['warm_aborted'] and _relf(res['X'], lim) < 1e-8
    # tol below the fp64 floor: the residual stops decreasing and the result
    # is accepted as STAGNATED (R3), still the warm limit
    res = o.coupled_newton_warm(B, 4, X, eps=1e-6, tol=0.0)
    assert res['status'] == o.STAGNATED and not res['warm_aborted'] and res['resid'] < 1e-12
    assert _relf(res['X'], lim) < 1e-8
    C = _spd(48, 1e6, 92)
    Xc, _, _ = o.inv_root(C, 4, eps=1e-6, eps_relative=True)
    C2 = C + 1e-3 * C.max() * _spd(48, 1e1, 93) / 48
    res = o.coupled_newton_warm(C2, 4, Xc, eps=1e-6, eps_relative=True, tol=1e-12)
    Xt, _, _ = o.inv_root(C2, 4, eps=1e-6, eps_relative=True, lam_max=res['lam_max'])
    assert res['warm_aborted'] and _relf(res['X'], Xt) < 1e-9
    # a drift whose warm iteration converges smoothly (no residual growth)
    # to a matrix 4% away: only the commutator (2.7e-2 after one iteration)
    # stops it
    C = _spd(48, 1e3, 92)
    Xc, _, _ = o.inv_root(C, 4, eps=1e-6)
    C2 = C + 1e-2 * 1e3 * _spd(48, 1e1, 93) / 48
    Xt, _, _ = o.inv_root(C2, 4, eps=1e-6)
    res = o.coupled_newton_warm(C2, 4, Xc, eps=1e-6, tol=1e-12)
    assert res['warm_aborted'] and res['warm_iters'] == 1 and _relf(res['X'], Xt) < 1e-9


# ------------------------------------------------------------------ precondition
def pin_precondition_kronecker(o):
    """vec(Lr G Rr) = (Lr (x) Rr^T) vec(G) with row-stacking vec, on
    non-symmetric factors so a transposed operand would show."""
    r = rng(40)
    Lr, Rr, G = r.standard_normal((6, 6)), r.standard_normal((5, 5)), r.standard_normal((6, 5))
    P = o.precondition(G, Lr, Rr)
    assert _relf(P.reshape(-1), np.kron(Lr, Rr.T) @ G.reshape(-1)) < 1e-13
    assert _relf(o.precondition(G, None, Rr), G @ Rr) < 1e-14
    assert _relf(o.precondition(G, Lr, None), Lr @ G) < 1e-14
    assert np.array_equal(o.precondition(G, None, None), G)


def pin_precondition_full_matrix_link(o):
    """With H = (L (x) R)^{1/2} formed and rooted as one mn x mn matrix,
    H^{-1/2} vec(G) equals vec(L^{-1/4} G R^{-1/4}) (Shampoo update from
    the full-matrix AdaGrad rule)."""
    r = rng(41)
    m, n = 4, 3
    L, R = np.zeros((m, m)), np.zeros((n, n))
    for _ in range(6):
        L, R = o.stats_update(L, R, r.standard_normal((m, n)))
    L += 1e-2 * np.eye(m)
    R += 1e-2 * np.eye(n)
    G = r.standard_normal((m, n))
    w, Q = np.linalg.eigh(np.kron(L, R))
    Hm12 = (Q * w ** -0.25) @ Q.T              # ((L (x) R)^{1/2})^{-1/2}
    Lr, _, _ = o.inv_root(L, 4)
    Rr, _, _ = o.inv_root(R, 4)
    assert _relf(o.precondition(G, Lr, Rr).reshape(-1), Hm12 @ G.reshape(-1)) < 1e-11


# ------------------------------------------------------------------ graft
def pin_graft_norm_identity(o):
    """beta1 = 0: ||dW||_F = eta0 ||D^{-1/2} o G||_F whatever the direction."""
    r = rng(50)
    W, D0 = r.standard_normal((7, 5)), r.random((7, 5))
    G, P = r.standard_normal((7, 5)), r.standard_normal((7, 5))
    out = o.graft_update(W, D0, G, P, eta0=0.3)
    want = 0.3 * np.linalg.norm(G / np.sqrt(D0 + G * G))
    assert abs(np.linalg.norm(out['W'] - W) - want) < 1e-13 * want
    assert _relf(out['D'], D0 + G * G) < 1e-15


def pin_graft_first_step(o):
    """t = 1 (D_0 = 0): D^{-1/2} o G = sign(G), so ||dW||_F = eta0 sqrt(nnz);
    zero entries of G stay zero (no 0/0)."""
    r = rng(51)
    G = r.standard_normal((6, 6))
    G[r.random((6, 6)) < 0.3] = 0.0
    P = r.standard_normal((6, 6))
    out = o.graft_update(np.zeros((6, 6)), np.zeros((6, 6)), G, P, eta0=0.5)
    nnz = np.count_nonzero(G)
    assert abs(np.linalg.norm(out['W']) - 0.5 * np.sqrt(nnz)) < 1e-13
    assert np.array_equal(out['Mg'], np.sign(G))


def pin_graft_identity_roots(o):
    """Roots proportional to I: the direction is G / ||G||_F."""
    r = rng(52)
    G, D0 = r.standard_normal((5, 4)), r.random((5, 4))
    P = o.precondition(G, 2.0 * np.eye(5), 0.5 * np.eye(4))
    out = o.graft_update(np.zeros((5, 4)), D0, G, P, eta0=1.0)
    mag = np.linalg.norm(G / np.sqrt(D0 + G * G))
    assert _relf(-out['W'], mag * G / np.linalg.norm(G)) < 1e-14


def pin_graft_adagrad_fallback(o):
    """Before the first roots (t <= tau1) the step is eta0 * M_t."""
    r = rng(53)
    W, D0, G = r.standard_normal((3, 3)), r.random((3, 3)), r.standard_normal((3, 3))
    out = o.graft_update(W, D0, G, None, eta0=0.1, use_shampoo=False)
    assert _relf(out['W'], W - 0.1 * G / np.sqrt(D0 + G * G)) < 1e-15


def pin_graft_momentum_1x1(o):
    """Two steps of Algorithm 2 on a 1 x 1 block, worked by hand:
    beta1 = 1/2, eta0 = 1, G = 3 then 4, P = 2 then 2.
      t=1: D=9,  D^-1/2 G = 1,   M = 1/2,  P_1 = 1,   eta = 1/2,  W -= 1/2
      t=2: D=25, D^-1/2 G = 4/5, M = 13/20, P_2 = 3/2, eta = 13/30, W -= 13/20
    so W ends at W0 - 23/20; a third step with P = -3/2 makes P_3 = 0 and
    then eta = 0 (no update)."""
    s = dict(W=np.array([[1.0]]), D=np.zeros((1, 1)), Mg=np.zeros((1, 1)), Ps=np.zeros((1, 1)))
    o1 = o.graft_update(s['W'], s['D'], np.array([[3.0]]), np.array([[2.0]]), 1.0, 0.5, s['Mg'], s['Ps'])
    assert abs(o1['eta'] - 0.5) < 1e-15 and abs(o1['W'][0, 0] - 0.5) < 1e-15
    o2 = o.graft_update(o1['W'], o1['D'], np.array([[4.0]]), np.array([[2.0]]), 1.0, 0.5, o1['Mg'], o1['Ps'])
    assert abs(o2['Mg'][0, 0] - 0.65) < 1e-15 and abs(o2['Ps'][0, 0] - 1.5) < 1e-15
    assert abs(o2['eta'] - 13.0 / 30.0) < 1e-15
    assert abs(o2['W'][0, 0] - (1.0 - 23.0 / 20.0)) < 1e-14
    o3 = o.graft_update(o2['W'], o2['D'], np.array([[1.0]]), np.array([[-1.5]]), 1.0, 0.5, o2['Mg'], o2['Ps'])
    assert o3['eta'] == 0.0 and o3['W'][0, 0] == o2['W'][0, 0]


def pin_lamb_step_norm(o):
    """LARS/LAMB magnitude: ||dW||_F = eta0 ||W||_F along -P/||P||_F (and
    along -G/||G||_F before the roots), unchanged when G or P is scaled."""
    r = rng(54)
    W, G, P = r.standard_normal((6, 4)), r.standard_normal((6, 4)), r.standard_normal((6, 4))
    nw = np.linalg.norm(W)
    out = o.lamb_graft_update(W, G, P, eta0=0.2)
    dW = out['W'] - W
    assert abs(np.linalg.norm(dW) - 0.2 * nw) < 1e-13 * nw
    assert _relf(dW, -0.2 * nw * P / np.linalg.norm(P)) < 1e-13
    out2 = o.lamb_graft_update(W, 7.0 * G, 3.0 * P, eta0=0.2)
    assert _relf(out2['W'], out['W']) < 1e-14
    out3 = o.lamb_graft_update(W, G, None, eta0=0.2, use_shampoo=False)
    assert _relf(out3['W'] - W, -0.2 * nw * G / np.linalg.norm(G)) < 1e-13


def pin_lamb_worked(o):
    """By hand: W = (3, 4), ||W|| = 5, G = (1, 0), P = (0, 2), eta0 = 0.1:
    Shampoo direction: eta = 0.1 * 5 / 2 = 0.25, W -> (3, 3.5);
    before the roots: eta = 0.5, W -> (2.5, 4); P = 0 gives no step.
    Momentum on a 1 x 1 block, beta1 = 1/2, eta0 = 1/2, W = 4:
      t=1: G = 4, P = 2:  Mg = 2,   Ps = 1,    eta = 2,   W = 2
      t=2: G = 1, P = -6: Mg = 1.5, Ps = -2.5, eta = 0.4, W = 3."""
    W, G, P = np.array([[3.0, 4.0]]), np.array([[1.0, 0.0]]), np.array([[0.0, 2.0]])
    a = o.lamb_graft_update(W, G, P, eta0=0.1)
    assert abs(a['eta'] - 0.25) < 1e-15 and np.allclose(a['W'], [[3.0, 3.5]], rtol=0, atol=1e-15)
    b = o.lamb_graft_update(W, G, None, eta0=0.1, use_shampoo=False)
    assert abs(b['eta'] - 0.5) < 1e-15 and np.allclose(b['W'], [[2.5, 4.0]], rtol=0, atol=1e-15)
    c = o.lamb_graft_update(W, G, np.zeros((1, 2)), eta0=0.1)
    assert c['eta'] == 0.0 and np.array_equal(c['W'], W)
    z = np.zeros((1, 1))
    s1 = o.lamb_graft_update(np.array([[4.0]]), np.array([[4.0]]), np.array([[2.0]]), 0.5, 0.5, z, z)
    assert abs(s1['eta'] - 2.0) < 1e-15 and abs(s1['W'][0, 0] - 2.0) < 1e-15 and s1['Mg'][0, 0] == 2.0
    s2 = o.lamb_graft_update(s1['W'], np.array([[1.0]]), np.array([[-6.0]]), 0.5, 0.5, s1['Mg'], s1['Ps'])
    assert abs(s2['Mg'][0, 0] - 1.5) < 1e-15 and abs(s2['Ps'][0, 0] + 2.5) < 1e-15
    assert abs(s2['eta'] - 0.4) < 1e-15 and abs(s2['W'][0, 0] - 3.0) < 1e-14


# ------------------------------------------------------------------ order-k tensors
def pin_tensor_stats_bruteforce(o):
    """Per-mode statistics of a 2 x 3 x 4 tensor by pure-Python loops over
    the other two indices; every mode's trace is ||G||_F^2; a rank-1 tensor
    u (x) v (x) w has H_1 = |v|^2 |w|^2 u u^T (and likewise per mode)."""
    r = np.random.default_rng(70)
    G = r.standard_normal((2, 3, 4))
    H = o.tensor_stats(None, G)
    d = G.shape
    for i in range(3):
        want = [[0.0] * d[i] for _ in range(d[i])]
        for a in range(d[i]):
            for b in range(d[i]):
                acc = 0.0
                for x in range(d[(i + 1) % 3]):
                    for y in range(d[(i + 2) % 3]):
                        ia, ib = [0] * 3, [0] * 3
                        ia[i], ib[i] = a, b
                        ia[(i + 1) % 3] = ib[(i + 1) % 3] = x
                        ia[(i + 2) % 3] = ib[(i + 2) % 3] = y
                        acc += G[tuple(ia)] * G[tuple(ib)]
                want[a][b] = acc
        assert np.allclose(H[i], np.array(want), rtol=1e-13, atol=1e-13)
        assert abs(np.trace(H[i]) - float(np.sum(G * G))) < 1e-12
    u, v, w = r.standard_normal(5), r.standard_normal(6), r.standard_normal(7)
    T = np.einsum('a,b,c->abc', u, v, w)
    H = o.tensor_stats(None, T)
    nu, nv, nw = u @ u, v @ v, w @ w
    assert np.allclose(H[0], nv * nw * np.outer(u, u), rtol=1e-12, atol=1e-12)
    assert np.allclose(H[1], nu * nw * np.outer(v, v), rtol=1e-12, atol=1e-12)
    assert np.allclose(H[2], nu * nv * np.outer(w, w), rtol=1e-12, atol=1e-12)
    # EMA: beta2 H + (1 - beta2) G_(i) G_(i)^T
    H2 = o.tensor_stats(H, T, beta2=0.5)
    assert np.allclose(H2[1], 0.5 * H[1] + 0.5 * nu * nw * np.outer(v, v), rtol=1e-12, atol=1e-12)


def pin_tensor_precondition_kronecker(o):
    """vec(G x_1 H_1 x_2 H_2 x_3 H_3) = (H_1 (x) H_2 (x) H_3) vec(G) with
    row-major vec and non-symmetric H (numpy's kron); for an order-2 tensor
    the mode products are H_1 G H_2^T."""
    r = np.random.default_rng(71)
    G = r.standard_normal((2, 3, 4))
    Hs = [r.standard_normal((n, n)) for n in G.shape]
    P = o.tensor_precondition(G, Hs)
    K = np.kron(np.kron(Hs[0], Hs[1]), Hs[2])
    assert np.allclose(P.reshape(-1), K @ G.reshape(-1), rtol=1e-12, atol=1e-12)
    P = o.tensor_precondition(G, [None, Hs[1], None])
    assert np.allclose(P.reshape(-1), np.kron(np.kron(np.eye(2), Hs[1]), np.eye(4)) @ G.reshape(-1),
                       rtol=1e-12, atol=1e-12)
    M = r.standard_normal((3, 5))
    A, B = r.standard_normal((3, 3)), r.standard_normal((5, 5))
    assert np.allclose(o.tensor_precondition(M, [A, B]), A @ M @ B.T, rtol=1e-12, atol=1e-12)



# ------------------------------------------------------------------ whole step (Algorithm 2)
def _stats_loops(Gs, m, n):
    """L_t = sum_s G_s G_s^T and R_t = sum_s G_s^T G_s by pure-Python loops."""
    L = [[sum(float(G[i, k]) * float(G[j, k]) for G in Gs for k in range(n)) for j in range(m)] for i in range(m)]
    R = [[sum(float(G[k, i]) * float(G[k, j]) for G in Gs for k in range(m)) for j in range(n)] for i in range(n)]
    return np.array(L), np.array(R)


def _kron_root_apply(Ld, Rd, G, p):
    """(Ld (x) Rd)^{-1/p} vec(G) from one eigendecomposition of the mn x mn
    Kronecker product (row-stacking vec): the full-matrix preconditioner of
    the Preliminaries, of which L^{-1/p} G R^{-1/p} is the factored form."""
    w, V = np.linalg.eigh(np.kron(Ld, Rd))
    return ((V * w ** (-1.0 / p)) @ V.T @ G.reshape(-1)).reshape(G.shape)


def pin_shampoo_step_kronecker(o):
    """Three steps of Algorithm 2 (beta1 = 0, beta2 = 1) on a non-square and
    a square block, against an independent route: statistics by loops, the
    direction from one eigh of the mn x mn Kronecker product of the damped
    statistics, the AdaGrad magnitude from the explicit sum of squares.
    Step 2 keeps step 1's roots (no refresh), step 3 refreshes them.  The
    step is eta0 ||D_t^{-1/2} o G_t||_F long along -dir / ||dir||; at t = 1
    D^{-1/2} o G = sign(G), so its length is eta0 sqrt(nnz(G))."""
    eps, p, eta0 = 1e-3, 4, 0.1
    for seed, (m, n) in ((60, (3, 2)), (61, (3, 3))):
        r = rng(seed)
        Gs = [r.standard_normal((m, n)) for _ in range(3)]
        W0 = r.standard_normal((m, n))
        s = dict(W=W0.copy(), D=np.zeros((m, n)), L=np.zeros((m, m)), R=np.zeros((n, n)))
        W = W0.copy()
        Ld = Rd = None
        for t, refresh in ((1, True), (2, False), (3, True)):
            G = Gs[t - 1]
            s = o.shampoo_step(s, G, p=p, eps=eps, eta0=eta0, refresh_roots=refresh)
            if refresh:
                L, R = _stats_loops(Gs[:t], m, n)
                Ld, Rd = L + eps * np.eye(m), R + eps * np.eye(n)
            dirn = _kron_root_apply(Ld, Rd, G, p)
            Dt = sum(g * g for g in Gs[:t])
            mag = eta0 * np.linalg.norm(G / np.sqrt(Dt))
            if t == 1:
                assert abs(mag - eta0 * np.sqrt(m * n)) < 1e-12
            W = W - mag * dirn / np.linalg.norm(dirn)
            assert _relf(s['W'], W) < 1e-10, (m, n, t)
            assert _relf(s['D'], Dt) < 1e-14


def pin_shampoo_step_variants(o):
    """The step's other branches against the same independent routes:
    the AdaGrad fallback before the first roots (W -= eta0 M_t, at t = 1
    eta0 sign(G)); a one-sided block (right side not tracked: the Kronecker
    factor on that side is the identity); and heavy-ball momentum beta1 =
    1/2 over two steps, unrolled from M_0 = P_0 = 0 as Algorithm 2 states."""
    eps, p = 1e-3, 4
    r = rng(62)
    G1, G2, W0 = r.standard_normal((3, 4)), r.standard_normal((3, 4)), r.standard_normal((3, 4))
    s0 = dict(W=W0, D=np.zeros((3, 4)), L=np.zeros((3, 3)), R=np.zeros((4, 4)))
    s = o.shampoo_step(s0, G1, p=p, eps=eps, eta0=0.2, use_shampoo=False)
    assert _relf(s['W'], W0 - 0.2 * np.sign(G1)) < 1e-15
    # one-sided
    s = o.shampoo_step(dict(W=W0, D=np.zeros((3, 4)), L=np.zeros((3, 3))), G1, p=p, eps=eps, eta0=0.2,
                       right=False)
    L, _ = _stats_loops([G1], 3, 4)
    dirn = _kron_root_apply(L + eps * np.eye(3), np.eye(4), G1, p)
    assert _relf(s['W'], W0 - 0.2 * np.sqrt(12) * dirn / np.linalg.norm(dirn)) < 1e-10
    assert s.get('R') is None and s.get('Rr') is None
    # momentum
    b1 = 0.5
    s = dict(W=W0, D=np.zeros((3, 4)), L=np.zeros((3, 3)), R=np.zeros((4, 4)), Mg=np.zeros((3, 4)),
             Ps=np.zeros((3, 4)))
    M, P, W = np.zeros((3, 4)), np.zeros((3, 4)), W0.copy()
    for t, G in ((1, G1), (2, G2)):
        s = o.shampoo_step(s, G, p=p, eps=eps, eta0=0.2, beta1=b1)
        L, R = _stats_loops([G1, G2][:t], 3, 4)
        Dt = sum(g * g for g in [G1, G2][:t])
        M = b1 * M + (1 - b1) * G / np.sqrt(Dt)
        P = b1 * P + (1 - b1) * _kron_root_apply(L + eps * np.eye(3), R + eps * np.eye(4), G, p)
        W = W - 0.2 * np.linalg.norm(M) / np.linalg.norm(P) * P
        assert _relf(s['W'], W) < 1e-10, t


# ------------------------------------------------------------------ bf16 inputs
def pin_bf16_decode(o):
    """bfloat16 is the top half of an IEEE binary32: sign, 8 exponent bits
    (bias 127), 7 fraction bits.  Every one of the 65536 patterns against
    that definition evaluated with exact integer scaling (math.ldexp), plus
    fixed values: 0x3F80 = 1, 0xC000 = -2, 0x4049 = 3.140625, 0x0001 =
    2^-133 (smallest subnormal), 0x7F7F = (2 - 2^-7) 2^127 (largest finite),
    0x7F80 / 0xFF80 = +-inf, 0x8000 = -0."""
    import math
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):      # NaN patterns
        got = o.bf16_bits_to_f64(bits)
    assert got.dtype == np.float64
    for b in range(65536):
        sgn = -1.0 if b >> 15 else 1.0
        e, f = (b >> 7) & 0xFF, b & 0x7F
        v = got[b]
        if e == 0xFF:
            assert (np.isinf(v) and np.sign(v) == sgn) if f == 0 else np.isnan(v), hex(b)
            continue
        want = sgn * (math.ldexp(f, -133) if e == 0 else math.ldexp(128 + f, e - 134))
        assert v == want and math.copysign(1.0, v) == sgn, hex(b)
    fixed = {0x3F80: 1.0, 0xC000: -2.0, 0x4049: 3.140625, 0x0001: 2.0 ** -133,
             0x7F7F: (2.0 - 2.0 ** -7) * 2.0 ** 127, 0x7F80: np.inf, 0xFF80: -np.inf}
    for b, v in fixed.items():
        assert got[b] == v, hex(b)
    assert got[0x8000] == 0.0 and math.copysign(1.0, got[0x8000]) == -1.0


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith('pin_')]
