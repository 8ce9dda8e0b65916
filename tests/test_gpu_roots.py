"""GPU batched inverse p-th roots (shampoo_inv_root_batched) against the oracle.

Bar (relative Frobenius error per matrix, against the eigendecomposition
definition): <= 1e-3 when the damped condition number is <= 1e6, <= 5e-3 up
to 1e8.  Iteration counts of fp32 runs are compared with the fp64
transcript of Algorithm 1.  Status codes of degenerate inputs are checked,
and neighbours of a failing matrix must be bit-identical to a clean run.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say, spd, to_dev
from tests.parity_util import band, pool_map, root_parity, summarize

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch, B, dev = gpu_env()
    h = B.shampoo_create(0)
    yield torch, B, dev, h
    B.shampoo_destroy(h)


def roots(env, As, **kw):
    torch, B, dev, h = env
    prm = B.shampoo_root_params_default(**kw)
    dA = [to_dev(torch, a, dev) for a in As]
    dX = [torch.full_like(a, float("nan")) for a in dA]
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([a.shape[0] for a in As], prm.precision),
                     dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    B.shampoo_inv_root_batched(h, dA, dX, prm, ws, info)
    torch.cuda.synchronize()
    return [host(x) for x in dX], B.decode_root_info(info)


@pytest.mark.parametrize("p", [1, 2, 3, 4, 5, 6, 7, 8, 12, 16])
def test_against_eigh_mixed_sizes(env, p):
    """Any root order 1 <= p <= 16 (powers of two and the product programs of
    the others); iteration counts of one matrix against the fp64 transcript."""
    say("roots mixed sizes p", p)
    sizes = [1, 5, 127, 128, 129, 300, 513]
    As = [spd(n, 100.0, 10 * n + p) for n in sizes]
    Xs, info = roots(env, As, p=p, eps=1e-6)
    for A, X, inf in zip(As, Xs, info):
        Xo, st, _ = O.inv_root(A, p, 1e-6)
        assert inf["status"] in (0, 1), inf
        assert rel(X, Xo) <= 1e-3, (A.shape, inf, rel(X, Xo))
        assert np.array_equal(X, X.T)
    tr = O.coupled_newton(As[5], p, 1e-6, tol=1e-6, scaling="power4")  # the library default
    assert abs(info[5]["iters"] - tr["iters"]) <= 1, (info[5], tr["iters"])


@pytest.mark.parametrize("scaling", ["frobenius", "power4"])
@pytest.mark.parametrize("p", [3, 4])
def test_scalings_against_transcript(env, scaling, p):
    """Both cold-start scalings: results against eigh, iteration counts
    against the fp64 transcript with the same scaling (C2-like flat spectrum
    and a cond-1e3 spread), in fp32 and fp64."""
    say("roots scaling", scaling, p)
    torch, B, dev, h = env
    code = B.SCALING_POWER4 if scaling == "power4" else B.SCALING_FROBENIUS
    As = [cfg.wishart_bartlett(384, 40 * 384, 1.0 / 384, 99, p).astype(np.float32), spd(257, 1e3, 3 + p)]
    for prec in (0, 2):
        Xs, info = roots(env, As, p=p, eps=1e-6, scaling=code, precision=prec)
        for A, X, inf in zip(As, Xs, info):
            Xo, _, _ = O.inv_root(A, p, 1e-6)
            assert inf["status"] in (0, 1), inf
            assert rel(X, Xo) <= (1e-3 if prec == 0 else 1e-6), (inf, rel(X, Xo))
            tr = O.coupled_newton(A, p, 1e-6, tol=1e-6, scaling=scaling)
            assert abs(inf["iters"] - tr["iters"]) <= 1, (inf, tr["iters"])


@pytest.mark.parametrize("scaling", ["frobenius", "power4"])
def test_iterations_grow_with_condition(env, scaling):
    """Property: with the eigenvectors and the relative spacing of the
    log-eigenvalues held fixed, the fp32 iteration count does not decrease as
    the condition number grows ten-fold at a time (the scaled smallest
    eigenvalue, which the iteration lifts by a bounded factor per step, gets
    smaller), and grows over the whole range; every root stays in its band."""
    say("roots iterations vs condition", scaling)
    torch, B, dev, h = env
    code = B.SCALING_POWER4 if scaling == "power4" else B.SCALING_FROBENIUS
    conds = [1e1, 1e2, 1e3, 1e4]
    As = [spd(200, c, 7) for c in conds]
    Xs, info = roots(env, As, p=4, eps=0.0, scaling=code, precision=0)
    its = [i["iters"] for i in info]
    assert all(i["status"] in (0, 1) for i in info), info
    assert its == sorted(its) and its[-1] > its[0], its
    for A, X in zip(As, Xs):
        Xo, _, _ = O.inv_root(A, 4, 0.0)
        assert rel(X, Xo) <= 1e-3, (its, rel(X, Xo))


def test_closed_forms(env):
    say("roots closed forms")
    d = np.array([0.5, 2.0, 7.0, 30.0, 1.0, 3.0], dtype=np.float32)
    c = 3.7
    As = [np.diag(d), (c * np.eye(40)).astype(np.float32)]
    Xs, info = roots(env, As, p=4, eps=1e-4, precision=0)
    Xd = Xs[0]
    assert np.count_nonzero(Xd - np.diag(np.diag(Xd))) == 0  # off-diagonal zeros stay exact
    assert rel(np.diag(Xd), (d.astype(np.float64) + 1e-4) ** -0.25) <= 1e-6
    assert rel(Xs[1], (c + 1e-4) ** -0.25 * np.eye(40)) <= 1e-6
    # odd and composite orders on the diagonal matrix: X = (d + eps)^(-1/p)
    for p in (3, 6, 7):
        Xs, _ = roots(env, [np.diag(d)], p=p, eps=1e-4, precision=0)
        assert np.count_nonzero(Xs[0] - np.diag(np.diag(Xs[0]))) == 0
        assert rel(np.diag(Xs[0]), (d.astype(np.float64) + 1e-4) ** (-1.0 / p)) <= 1e-6, p
    # p = 1 is the inverse
    A = spd(64, 50.0, 3)
    Xs, _ = roots(env, [A], p=1, eps=0.0)
    assert rel(Xs[0], np.linalg.inv(A.astype(np.float64))) <= 1e-4


def test_c2_full_size_grouped_all(env):
    """C2: 96 Wishart statistics 1024 x 1024, p = 4, eps = 1e-6, one grouped
    call; every matrix against eigh and its iteration count against the fp64
    transcript of Algorithm 1 with the same start; X^4 A_d = I on the GPU
    result of every matrix."""
    say("roots C2 96 x 1024^2")
    As = pool_map(cfg.c2_stats, range(96))
    Xs, info = roots(env, As, p=4, eps=1e-6)
    assert all(i["status"] in (0, 1) and i["precision"] == 32 for i in info), info[:3]
    res = pool_map(lambda i: root_parity(As[i], Xs[i], 4, 1e-6), range(96))
    _, worst, frac = summarize("C2 roots (all 96)", [r[0] for r in res], [r[2] for r in res])
    assert frac == 1.0, worst
    trs = pool_map(lambda i: O.coupled_newton(As[i], 4, 1e-6, tol=1e-6, scaling="power4")["iters"], range(96))
    off = [abs(inf["iters"] - t) for inf, t in zip(info, trs)]
    say(f"C2 iterations: GPU {sorted(set(i['iters'] for i in info))}, transcript {sorted(set(trs))}")
    assert max(off) <= 1, (off, trs)
    torch, B, dev, h = env
    worst_res = 0.0
    for i in range(96):
        X = torch.tensor(Xs[i], device=dev, dtype=torch.float64)
        Ad = torch.tensor(As[i], device=dev, dtype=torch.float64) + 1e-6 * torch.eye(1024, device=dev,
                                                                                    dtype=torch.float64)
        X2 = X @ X
        Rm = X2 @ X2 @ Ad - torch.eye(1024, device=dev, dtype=torch.float64)
        worst_res = max(worst_res, float(torch.linalg.norm(Rm)))
    say(f"C2 true residual ||X^4 A_d - I||_F max over 96: {worst_res:.3e}")
    assert worst_res <= 4e-3
    # the condition estimate of the info record: the kappa whose cold-start
    # eigenvalue (p+1)/(2 kappa) takes exactly the reported iterations in the
    # scalar recurrence (a bisection on the host, with the same 40 steps)
    for inf in info[::7]:
        est = _cond_from_iters(4, max(1e-6, inf["resid"]), inf["iters"])
        assert abs(inf["cond_est"] - est) <= 1e-5 * est, (inf, est)


def _cond_from_iters(p, tol, iters):
    def count(m):
        k = 0
        while abs(m - 1.0) > tol and k <= iters:
            f, fp = (p + 1.0 - m) / p, 1.0
            for _ in range(p):
                fp *= f
            m = fp * m
            k += 1
        return k
    lo, hi = 1e-30, 1.0
    if count(lo) <= iters:
        return 1.0
    for _ in range(40):
        mid = (lo * hi) ** 0.5
        if count(mid) <= iters:
            hi = mid
        else:
            lo = mid
    return (1.0 + p) / (2.0 * hi)


@pytest.mark.skip(reason="stage-chain Newton launches (one persistent launch per iteration with per-matrix "
                         "dependency counters, per-XCD work queues) stalled on C2's 96 matrices twice on MI355X, the "
                         "second time after its counter poll was changed to an atomic compare-and-swap; the path was "
                         "taken out of the library (see the design notes, Newton kernel), so this case has no code "
                         "to run until a design whose cause is understood replaces it")
def test_c2_stage_chain_grouped():
    """C2's 96 roots through the stage-chain launches, against the per-stage
    launches bit for bit (the same products, tiles and epilogues)."""
    torch, B, dev = gpu_env()
    pytest.fail("the stage-chain launches are not built")


@pytest.mark.parametrize("p", [2, 4])
def test_c3_ill_conditioned_reduced(env, p):
    """C3 recipe at n = 256 (spectrum log-uniform in [1e-6, 1e2], relative
    damping 1e-6 and the 1e-8 variant); AUTO escalates to fp64."""
    say("roots C3 n=256 p", p)
    mats = [cfg.c3_matrix(i, n=256) for i in range(4)]
    As = [m[0] for m in mats]
    for eps in (1e-6, 1e-8):
        Xs, info = roots(env, As, p=p, eps=eps, eps_relative=1)
        for A, X, inf in zip(As, Xs, info):
            As64 = 0.5 * (A.astype(np.float64) + A.T)
            lam = float(np.linalg.eigvalsh(As64).max())
            lam_ps, _ = O.max_sv(As64)  # same power iteration and stop rule
            # the GPU MaxSV follows the oracle's (Algorithm 1): within 1e-5 of
            # it, which is also the floor; a Rayleigh quotient is at most the
            # top eigenvalue, so eigh bounds it from above
            assert abs(inf["lambda_max"] - lam_ps) <= 1e-5 * lam_ps, (inf, lam_ps)
            assert inf["lambda_max"] <= lam * (1 + 1e-6), (inf, lam)
            Xo, st, e = O.inv_root(A, p, eps, eps_relative=True)
            kappa = O.cond_damped(A, eps, True)
            assert inf["status"] in (0, 1), inf
            assert rel(X, Xo) <= band(kappa), (kappa, inf, rel(X, Xo))


@pytest.fixture(scope="module")
def c3_full(env):
    """The 32 C3 matrices on the device, their fp32 values on the host, one
    eigendecomposition each (shared by every order and damping) and the
    oracle's MaxSV of each (Algorithm 1's power iteration)."""
    torch, B, dev, h = env
    say("roots C3: generating 32 x 2048^2 on the device")
    dA = [cfg.c3_matrix_device(i, torch, dev)[0] for i in range(32)]
    hA = [host(a) for a in dA]
    say("roots C3: oracle eigendecompositions and MaxSV")
    eigs = pool_map(O.sym_eig, hA)
    lam_ps = pool_map(lambda a: O.max_sv(a)[0], hA)
    return dA, hA, eigs, lam_ps


@pytest.mark.parametrize("p", [2, 4])
def test_c3_full_size_grouped_all(env, c3_full, p):
    """C3 as benchmarked: all 32 matrices of 2048 x 2048 in one grouped call
    (AUTO: fp32 attempt, fp64 tail), with relative damping eps_d = 1e-6
    (damped condition ~1e6, the 1e-3 band) and the C3b variant eps_d = 1e-8
    (~5e7, the 5e-3 band).  Every root against eigh (fed the GPU's
    lambda_max, so that the root error is isolated), and every lambda_max
    against the oracle's MaxSV (same power iteration, start vector and stop
    rule) and against eigh's largest eigenvalue."""
    torch, B, dev, h = env
    dA, hA, eigs, lam_ps = c3_full
    dX = [torch.full_like(a, float("nan")) for a in dA]
    for epsd in (1e-6, 1e-8):
        say("roots C3 32 x 2048^2 p", p, "eps_d", epsd)
        prm = B.shampoo_root_params_default(p=p, eps=epsd, eps_relative=1)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([2048] * 32, prm.precision), dtype=torch.uint8,
                         device=dev)
        info_t = torch.zeros(8 * 32, dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, dA, dX, prm, ws, info_t)
        torch.cuda.synchronize()
        info = B.decode_root_info(info_t)
        del ws
        assert all(i["status"] in (0, 1) and i["precision"] == 64 for i in info), info[:3]
        # lambda_max: a Rayleigh quotient, so at most the top eigenvalue; the
        # same power iteration as the oracle's MaxSV to 1e-5
        top = [float(e[1].max()) for e in eigs]
        gap_ps = max(abs(i["lambda_max"] - l) / l for i, l in zip(info, lam_ps))
        gap_top = max((t - i["lambda_max"]) / t for i, t in zip(info, top))
        say(f"C3 lambda_max: max |GPU - MaxSV| / MaxSV {gap_ps:.2e}, max (eigh - GPU) / eigh {gap_top:.2e}")
        assert gap_ps <= 1e-5
        assert all(i["lambda_max"] <= t * (1 + 1e-6) for i, t in zip(info, top))
        Xh = [host(x) for x in dX]
        res = pool_map(lambda q: root_parity(hA[q], Xh[q], p, epsd, True, info[q]["lambda_max"], eigs[q]),
                       range(32))
        kap = [r[1] for r in res]
        say(f"C3 p={p} eps_d={epsd:g}: damped condition {min(kap):.3g}..{max(kap):.3g}, fp64 iterations "
            f"{min(i['iters'] for i in info)}..{max(i['iters'] for i in info)}, fp32 attempt "
            f"{min(i['iters_fp32'] for i in info)}..{max(i['iters_fp32'] for i in info)} (0: sent to fp64 by "
            f"the Lanczos witness)")
        _, worst, frac = summarize(f"C3 p={p} eps_d={epsd:g} roots (all 32)", [r[0] for r in res],
                                   [r[2] for r in res])
        assert frac == 1.0, worst
        if epsd == 1e-8:
            assert min(kap) > 1e6          # the 5e-3 band is the one exercised


def test_precision_policies_agree(env):
    say("roots policies")
    As = [spd(200, 1e3, 5), spd(256, 30.0, 6)]
    X32, i32 = roots(env, As, p=4, eps=1e-6, precision=0)
    X64, i64 = roots(env, As, p=4, eps=1e-6, precision=2)
    for A, a, b, ia, ib in zip(As, X32, X64, i32, i64):
        Xo, _, _ = O.inv_root(A, 4, 1e-6)
        assert ia["precision"] == 32 and ib["precision"] == 64
        assert rel(a, Xo) <= 1e-3 and rel(b, Xo) <= 1e-6


def test_auto_escalates_early(env):
    """AUTO: a matrix whose condition number is far above kappa32 leaves the
    fp32 phase before the cap (its residual max|M - I| is above what the
    slowest matrix that still converges within the cap can have); one below
    kappa32 stays in fp32.  Both agree with eigh.  The cap is the scalar
    recurrence's count from (p+1) / (2 kappa32), plus one."""
    say("roots AUTO early escalation")
    A_ok, A_bad = spd(200, 1e3, 21), spd(200, 1e7, 22)
    Xs, info = roots(env, [A_ok, A_bad], p=4, eps=0.0)
    cap = O.scalar_newton_iters(5.0 / (2.0 * 1e4), 4, 1e-6) + 1
    assert info[0]["precision"] == 32, info[0]
    assert info[1]["precision"] == 64 and 1 <= info[1]["iters_fp32"] < cap, (info[1], cap)
    for A, X, inf in zip((A_ok, A_bad), Xs, info):
        Xo, _, _ = O.inv_root(A, 4, 0.0)
        assert rel(X, Xo) <= band(O.cond_damped(A, 0.0)), (inf, rel(X, Xo))


def test_auto_lanczos_preescalation(env):
    """AUTO with scaled damping: a Lanczos witness (its smallest Ritz value
    bounds lambda_min from above) sends a matrix straight to fp64 only when
    the fp32 cap would certainly reject it.  Well-conditioned matrices stay
    in fp32; a C3-like spectrum (log-uniform over 8 decades, damped
    condition ~5e7) goes to fp64 with no fp32 iteration; every root matches
    eigh within its band."""
    say("roots Lanczos pre-escalation")
    ok = [spd(300, 30.0, 41), spd(256, 1e3, 42), cfg.wishart_bartlett(384, 40 * 384, 1.0 / 384, 43, 0)
          .astype(np.float32)]
    bad = [cfg.c3_matrix(i, n=256)[0] for i in range(3)]
    for p in (2, 4):
        Xs, info = roots(env, ok + bad, p=p, eps=1e-8, eps_relative=1)
        for A, X, inf in zip(ok + bad, Xs, info):
            Xo, _, _ = O.inv_root(A, p, 1e-8, eps_relative=True, lam_max=inf["lambda_max"])
            kappa = O.cond_damped(A, 1e-8, True, lam_max=inf["lambda_max"])
            assert inf["status"] in (0, 1), inf
            assert rel(X, Xo) <= band(kappa), (p, kappa, inf, rel(X, Xo))
        for inf in info[:len(ok)]:
            assert inf["precision"] == 32 and inf["iters_fp32"] > 0, inf
        for inf in info[len(ok):]:
            assert inf["precision"] == 64 and inf["iters_fp32"] == 0, inf


def test_status_paths_and_isolation(env):
    """MAXITER at a cap of 1, DIVERGED/NOT_PD on an indefinite matrix,
    NOT_PD on a zero matrix without damping, DIVERGED on NaN; the healthy
    neighbours are bit-identical to a clean grouped run."""
    say("roots status paths")
    good = [spd(96, 50.0, 11), spd(160, 10.0, 12)]
    Xc, ic = roots(env, good, p=4, eps=1e-6, precision=0)
    indef = np.diag(np.array([1.0, 2.0, -1.0, 3.0], dtype=np.float32))
    nan = spd(64, 10.0, 13)
    nan[3, 5] = nan[5, 3] = np.nan
    zero = np.zeros((8, 8), np.float32)
    Xs, info = roots(env, [good[0], indef, nan, zero, good[1]], p=4, eps=0.0, precision=0)
    assert info[1]["status"] in (O.DIVERGED, O.NOT_PD)
    assert info[2]["status"] in (O.DIVERGED, O.NOT_PD)
    assert info[3]["status"] == O.NOT_PD
    # eps = 0 vs 1e-6 changes the neighbours, so compare them to a clean
    # eps = 0 run
    Xc0, ic0 = roots(env, good, p=4, eps=0.0, precision=0)
    assert np.array_equal(Xs[0], Xc0[0]) and np.array_equal(Xs[4], Xc0[1])
    assert info[0]["iters"] == ic0[0]["iters"]
    Xs, info = roots(env, [good[0]], p=4, eps=1e-6, precision=0, max_iters=1)
    assert info[0]["status"] == O.MAXITER and info[0]["iters"] == 1
    Xs, info = roots(env, [good[0]], p=4, eps=1e-6, precision=0, tol=0.0)
    assert info[0]["status"] == O.STAGNATED
    Xo, _, _ = O.inv_root(good[0], 4, 1e-6)
    assert rel(Xs[0], Xo) <= 1e-3


def test_grouped_equals_singleton_and_deterministic(env):
    say("roots grouped == singleton")
    As = [spd(n, 100.0, 20 + n) for n in (100, 256, 384)]
    Xg, ig = roots(env, As, p=4, eps=1e-6)
    Xg2, _ = roots(env, As, p=4, eps=1e-6)
    for i, A in enumerate(As):
        Xs, _ = roots(env, [A], p=4, eps=1e-6)
        assert np.array_equal(Xs[0], Xg[i])
        assert np.array_equal(Xg2[i], Xg[i])


@pytest.mark.parametrize("n,count,pool", [(300, 24, 24), (520, 20, 20), (512, 264, 12)])
def test_uniform_grouped_equals_singleton(env, n, count, pool):
    """Uniform calls: up to 128 diagonal tiles per XCD (24 x 300, 20 x 520),
    the product launches run each XCD's diagonal tiles last; past that
    (264 x 512: 1056 diagonal tiles) they keep the row-major order.  Either
    way every matrix's root equals its singleton call's bit for bit, with
    the condition numbers spread so that matrices leave the iteration at
    different times (the compact tile lists shrink between launches)."""
    say("roots uniform grouped == singleton", n, count)
    conds = np.logspace(1, 5, pool)
    base = [spd(n, float(c), 700 + i) for i, c in enumerate(conds)]
    As = [base[i % pool] for i in range(count)]
    Xg, ig = roots(env, As, p=4, eps=1e-6)
    assert len({i["iters"] for i in ig}) > 1
    for i in sorted({0, 1, count // 2, count - 1} | set(range(0, count, max(1, count // 6)))):
        Xs, is_ = roots(env, [As[i]], p=4, eps=1e-6)
        assert np.array_equal(Xs[0], Xg[i]), i
        assert is_[0]["iters"] == ig[i]["iters"] and is_[0]["status"] == ig[i]["status"], i


def test_async_mode_matches_polling(env):
    say("roots poll=0")
    As = [spd(192, 1e3, 31), cfg.c3_matrix(0, n=128)[0]]
    Xa, ia = roots(env, As, p=4, eps=1e-6, eps_relative=1, poll=0, max_iters=60)
    Xb, ib = roots(env, As, p=4, eps=1e-6, eps_relative=1, poll=1, max_iters=60)
    for a, b, x, y in zip(Xa, Xb, ia, ib):
        assert np.array_equal(a, b) and x == y


def test_argument_errors(env):
    torch, B, dev, h = env
    say("roots errors")
    A = torch.eye(4, device=dev)
    X = torch.zeros(4, 4, device=dev)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([4]), dtype=torch.uint8, device=dev)
    info = torch.zeros(8, dtype=torch.int32, device=dev)
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_inv_root_batched(h, [A], [X], B.shampoo_root_params_default(p=17), ws, info)
    assert e.value.code == B.SHAMPOO_EUNSUPPORTED
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_inv_root_batched(h, [A], [X], B.shampoo_root_params_default(p=0), ws, info)
    assert e.value.code == B.SHAMPOO_EUNSUPPORTED
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_inv_root_batched(h, [A], [X], B.shampoo_root_params_default(), ws[:16], info)
    assert e.value.code == B.SHAMPOO_ENOMEM
    with pytest.raises(B.ShampooError):
        B.shampoo_inv_root_batched(h, [A], [X], B.shampoo_root_params_default(eps=-1.0), ws, info)


def test_early_exit_mixed_sizes_and_precisions(env):
    """One grouped AUTO call over matrices of different sizes and condition
    numbers: some stop after a few fp32 iterations, others run on alone (the
    product launches then cover only the active matrices' tiles), two take
    the fp64 tail.  Every result agrees with eigh to its band and is bit for
    bit the result of a call with that matrix alone."""
    say("roots early exit, mixed sizes and precisions")
    spec = [(130, 10.0), (512, 1e3), (256, 1e7), (384, 2.0), (64, 1e5), (200, 50.0), (129, 3e3)]
    As = [spd(n, c, 40 + i) for i, (n, c) in enumerate(spec)]
    Xs, info = roots(env, As, p=4, eps=0.0)
    assert sorted(i["precision"] for i in info).count(64) >= 2, info
    assert len(set(i["iters"] for i in info)) >= 3, info
    for A, X, inf in zip(As, Xs, info):
        Xo, _, _ = O.inv_root(A, 4, 0.0)
        assert inf["status"] in (0, 1), inf
        assert rel(X, Xo) <= band(O.cond_damped(A, 0.0)), (A.shape, inf, rel(X, Xo))
        X1, i1 = roots(env, [A], p=4, eps=0.0)
        assert np.array_equal(X1[0], X) and i1[0] == inf, (A.shape, inf, i1[0])
