"""CPU fp64 oracle for the scalable-Shampoo hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) imports, links or calls this module; only the tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` do.
It shares no code with the GPU path.

Everything is computed in float64 with numpy/scipy.  Inputs are the exact
values the GPU sees (fp32 arrays, or bf16 values decoded exactly), up-cast to
float64 before any arithmetic.

Paper: Anil, Gupta, Koren, Regan, Singer, "Scalable Second Order Optimization
for Deep Learning" (arXiv 2002.09018).  Passages are cited by section,
algorithm, equation or table.

Functions and what pins them (tests under ``tests/test_oracle_*.py``):

* ``stats_update``      -- Preliminaries, "The Shampoo algorithm" (definition
  of L_t, R_t) and Algorithm 2 (beta2 EMA branch).  Pinned by the rank-1
  closed form of the K-FAC comparison appendix, the trace identity, integer
  inputs, the one-hot embedding identity (appendix "Shampoo for embedding
  layers") and Lemmas 1 and 2 as PSD checks.
* ``inv_root``          -- matrix power defined through the eigendecomposition
  (Preliminaries, notation paragraph), with damping (Algorithm 1 and the
  "Scaled damping" item of the coupled-Newton appendix).  Pinned by closed
  forms (diagonal, c*I, p=1 inverse, p=2 squares to the inverse), 50-digit
  mpmath brute force on 4x4, scipy's Schur-Pade fractional power, the
  Kronecker identity (A (x) B)^a = A^a (x) B^a and X^p (A+eps I) = I.
* ``max_sv``            -- Algorithm 1, procedure MaxSV.  Pinned by the
  largest eigenvalue from eigh on matrices with a spectral gap.
* ``coupled_newton``    -- Algorithm 1, procedure CoupledIteration, fp64.
  Pinned against ``inv_root`` (<= 1e-9) and against the scalar recurrence
  for iteration counts on diagonal inputs.
* ``coupled_newton_warm`` -- the warm start of the coupled-Newton appendix
  with its commutator monitor (R21).  Pinned by the exact previous root
  (zero iterations), commuting diagonal starts (scalar recurrence, exact
  root), the non-commuting limit X0 (X0^p A)^{-1/p} from scipy's Schur-Pade
  fractional power, and the abort with cold fallback on an ill-conditioned
  drift.  The GPU counterpart is shampoo_inv_root_warm_batched.
* ``tensor_stats``, ``tensor_precondition`` -- tensors of order k
  (Preliminaries: the design holds for any order; the K-FAC comparison
  appendix: exponent -1/(2k)).  Pinned by pure-Python brute force of the
  per-mode statistics, the trace identity, a rank-1 tensor's closed form, the
  Kronecker identity vec(G x_1 H_1 x_2 H_2 x_3 H_3) = (H_1 (x) H_2 (x) H_3)
  vec(G) with non-symmetric H, and the order-2 case L G R^T.
* ``precondition``      -- Preliminaries (Shampoo update) and Lemma 1's
  one-sided forms.  Pinned by brute force with the Kronecker product of the
  full-matrix AdaGrad preconditioner on tiny shapes.
* ``embedding_grad``, ``embedding_rows`` -- appendix "Shampoo for embedding
  layers": the sparse gradient of a lookup and its active rows.  Pinned by
  the dense lookup-matrix route G = S dy (S^T S = I for distinct one-hot
  rows gives G^T G = dy^T dy), a hand-worked 5-row example with repeated
  rows and weights, and the dropping of out-of-range entries.
* ``lamb_graft_update`` -- the LARS/LAMB layer-wise magnitude of the same
  appendix paragraph (R17).  Pinned by the step-norm identity
  ||dW||_F = eta0 ||W||_F, invariance under scaling G and P, and hand-worked
  1 x 2 and 1 x 1 momentum examples.
* ``graft_update``      -- Algorithm 2 (momentum on both directions) and the
  appendix "Further details on experiments", paragraph "Layer wise learning
  rates" (AdaGrad magnitude, Shampoo direction).  Pinned by the step-norm
  identity ||dW||_F = eta0 ||D^{-1/2} o G||_F and the t=1 closed form
  eta0 * sqrt(nnz(G)).
* ``cond_damped``       -- condition number of the damped matrix, which picks
  the tolerance band of a root comparison (Section 3.2: the loss of
  precision grows with the condition number).  Pinned by the closed form
  (max d + eps_eff) / (min d + eps_eff) on rotated diagonal inputs, with
  absolute and relative damping, and infinity for an indefinite input.
* ``shampoo_step``      -- one step of Algorithm 2 for a block.  Pinned as a
  whole, independently of its parts: statistics by loops, the direction from
  one eigendecomposition of the Kronecker product of the damped statistics
  (the full-matrix form of the Preliminaries), the AdaGrad magnitude from the
  explicit sum of squares (t=1: eta0 sqrt(nnz(G))), stale roots between
  refreshes, the one-sided form, the fallback before the first roots and
  momentum unrolled from M_0 = P_0 = 0.
* ``bf16_bits_to_f64``  -- exact decode of bfloat16 inputs.  Pinned on all
  65536 bit patterns against the binary32 layout (sign, 8-bit exponent with
  bias 127, 7 fraction bits) and on fixed values (1, -2, the smallest
  subnormal, the largest finite value, +-inf, -0).

Readings of the paper where it is silent or ambiguous (each is listed in the
design notes of the repository as well):

R1  ||M - I||_inf in Algorithm 1 is the largest absolute entry.
R2  Algorithm 1 uses one symbol for the stopping tolerance and the damping
    scale; the damping is eps_d, the stop tolerance is ``tol``.
R3  Stopping rules: CONVERGED when r <= tol; DIVERGED when r is not finite or
    exceeds 1e6; STAGNATED when the previous residual was already below
    STAG_GATE (quadratic phase) and the new one did not decrease; MAXITER
    after ``max_iters`` iterations.
R4  MaxSV starts from v = ones(n) and stops on a relative change
    |lambda - lambda_old| <= maxsv_tol * lambda.
R5  The Frobenius norm that sets z is taken after damping.
R6  The cold start is X0 = z^{1/p} I, M0 = z (A + eps_eff I) (Algorithm 1).
R7  The ridge epsilon*I is added exactly once, at the root; statistics
    accumulate from zero.
R8  D^{-1/2} o G is 0 where D is 0 (then G is 0 as well).
R9  When ||P||_F = 0 the step size is 0.
R10 The input to a root is symmetrised, A_s = (A + A^T)/2, before use.
R16 Embedding statistics are those of the exact sparse gradient G of the
    lookup: G^T G = dy^T (S^T S) dy with S the lookup matrix.  The appendix's
    simplification S^T S = I (or diagonal for multi-hot) holds when the
    features hit distinct rows; repeated rows are summed first.  Entries
    with a row outside [0, vocab) or a feature outside [0, m) are dropped.
R20 The appendix leaves the start constant free (X0 = I / c); Algorithm 1
    takes z = (1+p) / (2 ||A_d||_F).  The 'power4' option takes the tighter
    upper bound ||A_d^4||_F^(1/4) = (sum lambda^8)^(1/8) >= lambda_max.
R21 The warm start's commutator monitor has no threshold in the paper:
    abort when max|XM - MX| > comm_tol * max|X| * max|M| (1e-3) after an
    iteration, when the residual grew twice in a row, or when the warm
    iteration stops unconverged; the root then comes from the cold start.
R17 The LARS/LAMB layer-wise learning rate ||W||_F / ||G||_F of the appendix,
    grafted like the AdaGrad magnitude, makes the step eta0 ||W||_F long
    along the unit Shampoo direction (along G / ||G||_F before the roots);
    ||W||_F is that of the block before the step.
"""
from __future__ import annotations

import numpy as np

# Per-matrix outcome codes of an inverse-root computation.  The GPU library
# uses the same numbering.
CONVERGED, STAGNATED, MAXITER, DIVERGED, NOT_PD = 0, 1, 2, 3, 4

STAG_GATE = 1e-3      # R3: stagnation is only tested once r fell below this
DIVERGE_AT = 1e6      # R3: a residual above this (or non-finite) diverged


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def bf16_bits_to_f64(bits):
    """Decode raw bfloat16 bit patterns (uint16) exactly into float64."""
    bits = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return bits.view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Statistics (Preliminaries "The Shampoo algorithm"; Algorithm 2)
# --------------------------------------------------------------------------
def stats_update(L, R, G, beta2=1.0):
    """One statistics step for a block with gradient G (m x n).

    beta2 == 1: L + G G^T and R + G^T G (plain sums, as in the definition of
    L_t, R_t in Preliminaries).  beta2 < 1: beta2 L + (1 - beta2) G G^T, and
    the same for R (Algorithm 2).  Either side may be None (not tracked).
    The ridge is not added here (R7).  Returns (L_new, R_new) in float64.
    """
    G = _f64(G)
    c = 1.0 if beta2 == 1.0 else 1.0 - beta2
    Ln = None if L is None else beta2 * _f64(L) + c * (G @ G.T)
    Rn = None if R is None else beta2 * _f64(R) + c * (G.T @ G)
    return Ln, Rn


# --------------------------------------------------------------------------
# Inverse p-th roots
# --------------------------------------------------------------------------
def max_sv(A, n_step=100, tol=1e-6):
    """Largest eigenvalue of a symmetric PSD matrix: Algorithm 1, MaxSV.

    Power iteration with the Rayleigh quotient lambda = v_hat^T A v_hat,
    starting from v = ones (R4) and stopping after n_step steps or once the
    relative change is at most tol.  Returns (lambda, steps_taken).
    """
    A = _f64(A)
    n = A.shape[0]
    v = np.ones(n)
    lam, i = 0.0, 0
    while i < n_step:
        vh = v / np.linalg.norm(v)
        v = A @ vh
        lam_old, lam = lam, float(vh @ v)
        i += 1
        if abs(lam - lam_old) <= tol * abs(lam):
            break
    return lam, i


def damping(A, eps, eps_relative=False, lam_max=None, maxsv_steps=100,
            maxsv_tol=1e-6):
    """Effective damping eps_eff: eps (absolute) or eps * lambda_max(A).

    The scaled variant follows the "Scaled damping" item of the coupled
    Newton appendix and Algorithm 1.  ``lam_max`` may be supplied (e.g. the
    value the GPU reported) to isolate the root error from the estimate.
    Returns (eps_eff, lam_max_used).
    """
    if not eps_relative:
        return float(eps), None
    if lam_max is None:
        lam_max, _ = max_sv(A, maxsv_steps, maxsv_tol)
    return float(eps) * float(lam_max), float(lam_max)


def sym_eig(A):
    """Symmetric part A_s = (A + A^T) / 2 of an input (R10) and its
    eigendecomposition A_s = Q diag(w) Q^T.  Returns (A_s, w, Q).  The root
    and condition-number functions below take it as ``eig`` so that one
    decomposition can serve several root orders and dampings of one input."""
    A = _f64(A)
    As = 0.5 * (A + A.T)
    w, Q = np.linalg.eigh(As)
    return As, w, Q


def inv_root(A, p, eps=0.0, eps_relative=False, lam_max=None, eig=None):
    """(A_s + eps_eff I)^(-1/p) by symmetric eigendecomposition.

    Definition of A^alpha through A = U D U^T (Preliminaries, notation
    paragraph): A^alpha = U D^alpha U^T, defined for alpha < 0 only when
    every eigenvalue is positive.  ``eig``: sym_eig(A), if already computed.
    Returns (X, status, eps_eff) with status CONVERGED (root defined) or
    NOT_PD (X is None).
    """
    As, w, Q = sym_eig(A) if eig is None else eig
    eps_eff, _ = damping(As, eps, eps_relative, lam_max)
    w = w + eps_eff
    if not np.all(w > 0.0):
        return None, NOT_PD, eps_eff
    X = (Q * w ** (-1.0 / p)) @ Q.T
    return 0.5 * (X + X.T), CONVERGED, eps_eff


def cond_damped(A, eps=0.0, eps_relative=False, lam_max=None, eig=None):
    """Condition number of the damped matrix A_s + eps_eff I (eigh);
    ``eig``: sym_eig(A), if already computed."""
    As, w, _ = sym_eig(A) if eig is None else eig
    eps_eff, _ = damping(As, eps, eps_relative, lam_max)
    w = w + eps_eff
    return float(w.max() / w.min()) if w.min() > 0 else np.inf


def coupled_newton(A, p, eps=0.0, tol=1e-10, max_iters=100,
                   eps_relative=False, lam_max=None, X0=None, scaling='frobenius'):
    """Algorithm 1, CoupledIteration, in float64.

    Steps in the paper's order: optional MaxSV and scaled damping; cold start
    z = (1+p) / (2 ||A_d||_F), X = z^{1/p} I, M = z A_d (R5, R6), or the warm
    start M = X^p A_d; then while ||M - I|| > tol:
        M1 = (1 - alpha) I + alpha M   with alpha = -1/p
        X  = X M1
        M  = M1^p M
    with the stopping rules of R1 and R3.  Returns a dict with X, iters,
    resid (last ||M - I||, R1), status, eps_eff and z.
    """
    A = _f64(A)
    n = A.shape[0]
    As = 0.5 * (A + A.T)
    eps_eff, lam = damping(As, eps, eps_relative, lam_max)
    Ad = As + eps_eff * np.eye(n)
    alpha = -1.0 / p
    I = np.eye(n)
    if X0 is not None:
        X = _f64(X0)
        M = np.linalg.matrix_power(X, p) @ Ad
        z = None
    else:
        z = (1.0 + p) / (2.0 * np.linalg.norm(Ad, 'fro'))
        if scaling == 'power4':
            # R20: the tighter bound ||A_d^4||_F^(1/4) >= lambda_max in place
            # of ||A_d||_F, computed on z A_d (eigenvalues <= (p+1)/2)
            rho = np.linalg.norm(np.linalg.matrix_power(z * Ad, 4), 'fro') ** 0.25
            z *= max(1.0, (1.0 + p) / (2.0 * rho))
        X = z ** (1.0 / p) * I
        M = z * Ad
    r = float(np.max(np.abs(M - I)))
    k = 0
    status = CONVERGED
    while not (r <= tol):
        if not np.isfinite(r) or r > DIVERGE_AT:
            status = DIVERGED
            break
        if k >= max_iters:
            status = MAXITER
            break
        M1 = (1.0 - alpha) * I + alpha * M
        X = X @ M1
        M = np.linalg.matrix_power(M1, p) @ M
        k += 1
        r_new = float(np.max(np.abs(M - I)))
        if not np.isfinite(r_new) or r_new > DIVERGE_AT:
            r = r_new
            status = DIVERGED
            break
        if r < STAG_GATE and r_new >= r and r_new > tol:
            r = r_new
            status = STAGNATED
            break
        r = r_new
    return dict(X=X, iters=k, resid=r, status=status, eps_eff=eps_eff, z=z,
                lam_max=lam)


def coupled_newton_warm(A, p, X0, eps=0.0, tol=1e-10, max_iters=100,
                        eps_relative=False, lam_max=None, comm_tol=1e-3,
                        scaling='frobenius'):
    """Warm start of the coupled-Newton appendix, in float64.

    X = X0 (the previous root), M = X0^p A_d, then the iteration of
    ``coupled_newton``.  The commutator [X, M] = XM - MX is monitored after
    every iteration (R21): the warm start is aborted, and the root computed
    from the cold start instead, when max|XM - MX| exceeds
    comm_tol * max|X| * max|M|, when the residual grew in two consecutive
    iterations, or when the warm iteration stops unconverged (divergence or
    the iteration cap).  A residual that stops decreasing below STAG_GATE has
    reached the rounding floor and is accepted as STAGNATED (R3, as in the
    cold iteration).  When X0
    commutes with A_d the limit is A_d^{-1/p}; otherwise it is
    X0 (X0^p A_d)^{-1/p}, which differs from the root by an amount that
    grows with the commutator.

    Returns the dict of ``coupled_newton`` plus ``warm_aborted``,
    ``warm_iters`` (iterations spent before an abort, or all of them) and
    ``comm`` (the relative commutator after each warm iteration).
    """
    A = _f64(A)
    n = A.shape[0]
    As = 0.5 * (A + A.T)
    eps_eff, lam = damping(As, eps, eps_relative, lam_max)
    Ad = As + eps_eff * np.eye(n)
    I = np.eye(n)
    alpha = -1.0 / p
    X = _f64(X0)
    M = np.linalg.matrix_power(X, p) @ Ad
    r = float(np.max(np.abs(M - I)))
    k, grew, comm = 0, 0, []
    aborted = False
    status = CONVERGED
    while not (r <= tol):
        if not np.isfinite(r) or r > DIVERGE_AT or k >= max_iters:
            aborted = True
            break
        M1 = (1.0 - alpha) * I + alpha * M
        X = X @ M1
        M = np.linalg.matrix_power(M1, p) @ M
        k += 1
        r_new = float(np.max(np.abs(M - I)))
        c = float(np.max(np.abs(X @ M - M @ X)))
        scale = float(np.max(np.abs(X))) * float(np.max(np.abs(M)))
        comm.append(c / scale if scale > 0 else np.inf)
        grew = grew + 1 if r_new > r else 0
        if not (c <= comm_tol * scale) or grew >= 2:
            r = r_new
            aborted = True
            break
        if r < STAG_GATE and r_new >= r and r_new > tol:
            # R3's rounding floor, as in the cold iteration: accepted
            r = r_new
            status = STAGNATED
            break
        r = r_new
    if aborted:
        res = coupled_newton(A, p, eps=eps, tol=tol, max_iters=max_iters,
                             eps_relative=eps_relative, lam_max=lam,
                             scaling=scaling)
        res.update(warm_aborted=True, warm_iters=k, comm=comm)
        return res
    return dict(X=X, iters=k, resid=r, status=status, eps_eff=eps_eff, z=None,
                lam_max=lam, warm_aborted=False, warm_iters=k, comm=comm)


def scalar_newton_iters(m0, p, tol, max_iters=1000):
    """Iterations the scalar recurrence m <- ((p+1-m)/p)^p m needs to reach
    |m - 1| <= tol from m0: Algorithm 1 applied to a 1x1 matrix after
    scaling.  Used to pin iteration counts on diagonal inputs."""
    m, k = float(m0), 0
    while abs(m - 1.0) > tol and k < max_iters:
        m = ((p + 1.0 - m) / p) ** p * m
        k += 1
    return k


# --------------------------------------------------------------------------
# Embedding layers (appendix "Shampoo for embedding layers")
# --------------------------------------------------------------------------
def _valid_entries(idx, feat, weight, vocab, m):
    idx = np.asarray(idx, dtype=np.int64)
    nnz = idx.shape[0]
    feat = np.arange(nnz, dtype=np.int64) if feat is None else np.asarray(feat, dtype=np.int64)
    w = np.ones(nnz) if weight is None else _f64(weight)
    ok = (idx >= 0) & (idx < vocab) & (feat >= 0) & (feat < m)
    return idx[ok], feat[ok], w[ok]


def embedding_grad(vocab, idx, feat, weight, dy):
    """Gradient of the table (vocab x d, row-major) of a lookup whose entry e
    reads row idx[e] into output row feat[e] with weight w[e]:
    G = sum_e w[e] e_{idx[e]} dy[feat[e]]^T.  feat None: feat[e] = e (one
    lookup per output row); weight None: w[e] = 1 (R16)."""
    dy = _f64(dy)
    i, f, w = _valid_entries(idx, feat, weight, vocab, dy.shape[0])
    G = np.zeros((vocab, dy.shape[1]))
    for e in range(i.shape[0]):
        G[i[e]] += w[e] * dy[f[e]]
    return G


def embedding_rows(vocab, idx, feat, weight, dy):
    """Active rows of the lookup (ascending) and the matching rows of G,
    accumulated per row in entry order without forming the vocab x d G."""
    dy = _f64(dy)
    i, f, w = _valid_entries(idx, feat, weight, vocab, dy.shape[0])
    acc = {}
    for e in range(i.shape[0]):
        r = int(i[e])
        if r not in acc:
            acc[r] = np.zeros(dy.shape[1])
        acc[r] += w[e] * dy[f[e]]
    rows = np.array(sorted(acc), dtype=np.int64)
    U = np.array([acc[r] for r in rows]).reshape(len(rows), dy.shape[1])
    return rows, U


# --------------------------------------------------------------------------
# Preconditioned gradient (Preliminaries; Lemma 1 one-sided forms)
# --------------------------------------------------------------------------
def precondition(G, Lr=None, Rr=None):
    """P = Lr G Rr; a missing root acts as the identity on its side."""
    P = _f64(G)
    if Lr is not None:
        P = _f64(Lr) @ P
    if Rr is not None:
        P = P @ _f64(Rr)
    return P


# --------------------------------------------------------------------------
# Tensors of any order (Preliminaries: the design holds for tensors of any
# order; K-FAC comparison appendix: the exponent is -1/(2k) for a tensor of
# order k).  Mode i of an order-k tensor G has its own statistic over the
# mode-i unfolding G_(i) (rows indexed by mode i, columns by all the other
# modes in order), and the preconditioned gradient multiplies every mode by
# its root.
# --------------------------------------------------------------------------
def tensor_stats(stats, G, beta2=1.0):
    """H_i = beta2 H_i + c G_(i) G_(i)^T for every mode i (c as in
    stats_update); stats: list of k matrices or None (start from zero)."""
    G = _f64(G)
    k = G.ndim
    c = 1.0 if beta2 == 1.0 else 1.0 - beta2
    out = []
    for i in range(k):
        Gi = np.moveaxis(G, i, 0).reshape(G.shape[i], -1)
        S = c * (Gi @ Gi.T)
        if stats is not None and stats[i] is not None:
            S = beta2 * _f64(stats[i]) + S
        out.append(S)
    return out


def tensor_precondition(G, roots):
    """G x_1 H_1 x_2 H_2 ... x_k H_k: the mode-i product contracts mode i of
    the tensor with the second index of H_i (a None root is the identity)."""
    P = _f64(G)
    for i, H in enumerate(roots):
        if H is not None:
            P = np.moveaxis(np.tensordot(_f64(H), P, axes=(1, i)), 0, i)
    return P


# --------------------------------------------------------------------------
# Grafting and the parameter update (Algorithm 2; "Layer wise learning rates")
# --------------------------------------------------------------------------
def adagrad_direction(D, G):
    """D^{-1/2} o G with the convention 0 where D == 0 (R8)."""
    D = _f64(D)
    G = _f64(G)
    out = np.zeros_like(G)
    nz = D > 0
    out[nz] = G[nz] / np.sqrt(D[nz])
    return out


def graft_update(W, D, G, P=None, eta0=1.0, beta1=0.0, Mg=None, Ps=None,
                 use_shampoo=True):
    """One parameter update of a block, Algorithm 2 with grafting.

        D  <- D + G o G
        Mg <- beta1 Mg + (1 - beta1) D^{-1/2} o G
        if use_shampoo:
            Ps  <- beta1 Ps + (1 - beta1) P
            eta <- eta0 ||Mg||_F / ||Ps||_F      (0 when ||Ps||_F = 0, R9)
            W   <- W - eta Ps
        else:
            eta <- eta0;  W <- W - eta Mg       (before the first roots)

    At beta1 = 0 this is exactly the appendix graft: step magnitude
    eta0 ||D^{-1/2} o G||_F along the unit Shampoo direction.  Mg and Ps may
    be None when beta1 == 0 (they are then not carried).  Returns a dict
    with W, D, Mg, Ps, eta and the two norms.
    """
    W = _f64(W)
    D = _f64(D) + _f64(G) ** 2
    g = adagrad_direction(D, G)
    Mg_new = g if beta1 == 0.0 or Mg is None else beta1 * _f64(Mg) + (1.0 - beta1) * g
    Ps_new = None if Ps is None else _f64(Ps)
    if use_shampoo:
        Pf = _f64(P)
        Ps_new = Pf if beta1 == 0.0 or Ps is None else beta1 * _f64(Ps) + (1.0 - beta1) * Pf
        nm = float(np.linalg.norm(Mg_new))
        nps = float(np.linalg.norm(Ps_new))
        eta = 0.0 if nps == 0.0 else eta0 * nm / nps
        W_new = W - eta * Ps_new
    else:
        nm = float(np.linalg.norm(Mg_new))
        nps = 0.0 if Ps_new is None else float(np.linalg.norm(Ps_new))
        eta = float(eta0)
        W_new = W - eta * Mg_new
    return dict(W=W_new, D=D, Mg=Mg_new, Ps=Ps_new, eta=eta, norm_mg=nm,
                norm_ps=nps)


def lamb_graft_update(W, G, P=None, eta0=1.0, beta1=0.0, Mg=None, Ps=None,
                      use_shampoo=True):
    """Layer-wise (LARS/LAMB) graft, the alternative magnitude of the
    appendix "Further details on experiments", paragraph "Layer wise learning
    rates" (R17): the layer learning rate eta0 ||W||_F / ||G||_F applied to
    the first-order step G gives a step of norm eta0 ||W||_F, kept along the
    unit Shampoo direction.

        Mg <- beta1 Mg + (1 - beta1) G
        if use_shampoo:
            Ps  <- beta1 Ps + (1 - beta1) P
            eta <- eta0 ||W||_F / ||Ps||_F      (0 when ||Ps||_F = 0, R9)
            W   <- W - eta Ps
        else:
            eta <- eta0 ||W||_F / ||Mg||_F      (LARS step before the roots)
            W   <- W - eta Mg

    ||W||_F is taken before the step.  Returns W, Mg, Ps, eta, norm_w and
    norm_dir.
    """
    W = _f64(W)
    Gf = _f64(G)
    Mg_new = Gf if beta1 == 0.0 or Mg is None else beta1 * _f64(Mg) + (1.0 - beta1) * Gf
    Ps_new = None if Ps is None else _f64(Ps)
    nw = float(np.linalg.norm(W))
    if use_shampoo:
        Pf = _f64(P)
        Ps_new = Pf if beta1 == 0.0 or Ps is None else beta1 * _f64(Ps) + (1.0 - beta1) * Pf
        direction = Ps_new
    else:
        direction = Mg_new
    nd = float(np.linalg.norm(direction))
    eta = 0.0 if nd == 0.0 else eta0 * nw / nd
    return dict(W=W - eta * direction, Mg=Mg_new, Ps=Ps_new, eta=eta, norm_w=nw,
                norm_dir=nd)


# --------------------------------------------------------------------------
# Whole step of one block (Algorithm 2 with tau1 = tau2 = 1 unless given)
# --------------------------------------------------------------------------
def shampoo_step(state, G, p=4, eps=1e-6, eta0=1e-2, beta1=0.0, beta2=1.0,
                 refresh_roots=True, use_shampoo=True, left=True, right=True,
                 eps_relative=False):
    """Stats, optional root refresh (eigh definition), precondition, graft.

    ``state`` holds W, D and optionally L, R, Lr, Rr, Mg, Ps (float64).
    Returns the new state dict.
    """
    s = dict(state)
    L, R = stats_update(s.get('L') if left else None,
                        s.get('R') if right else None, G, beta2)
    if left:
        s['L'] = L
    if right:
        s['R'] = R
    if refresh_roots:
        if left:
            s['Lr'], st, _ = inv_root(L, p, eps, eps_relative)
            assert st == CONVERGED
        if right:
            s['Rr'], st, _ = inv_root(R, p, eps, eps_relative)
            assert st == CONVERGED
    P = precondition(G, s.get('Lr') if left else None,
                     s.get('Rr') if right else None) if use_shampoo else None
    out = graft_update(s['W'], s['D'], G, P, eta0, beta1, s.get('Mg'),
                       s.get('Ps'), use_shampoo)
    s.update(W=out['W'], D=out['D'], Mg=out['Mg'], Ps=out['Ps'],
             eta=out['eta'], P=P)
    return s
