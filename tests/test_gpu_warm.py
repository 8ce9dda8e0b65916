"""GPU warm-started inverse roots (shampoo_inv_root_warm_batched) against the
oracle's warm iteration (coupled_newton_warm: the warm start of the
coupled-Newton appendix with the commutator monitor of reading R21).

A kept warm result is compared with the oracle's warm limit
X0 (X0^p A_d)^(-1/p), which differs from the true root by the drift; the
cases are chosen so that this difference is well above the GPU's rounding,
so a cold root in place of the warm one would fail.  A warm start that is
given up is compared with the eigendecomposition root, to the bands of the
cold call.  Cases sit far from the monitor's threshold on both sides
(commutator ratio at most 1e-5 when kept, 5e-2 to 1e-1 when given up), so the
decision does not depend on rounding.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from tests.gpu_util import gpu_env, host, rel, say, spd, to_dev

pytestmark = pytest.mark.gpu

FP32, AUTO, FP64 = 0, 1, 2


@pytest.fixture(scope="module")
def env():
    torch, B, dev = gpu_env()
    h = B.shampoo_create(0)
    yield torch, B, dev, h
    B.shampoo_destroy(h)


def drift_case(n, cond, drift, p, seed):
    """(A1, X0): X0 = the fp32-rounded root of A0, A1 = A0 plus a seeded SPD
    drift of relative size ~drift."""
    A0 = spd(n, cond, seed).astype(np.float64)
    X0, _, _ = O.inv_root(A0, p, eps=1e-6)
    D = spd(n, 10.0, seed + 1).astype(np.float64)
    A1 = (A0 + drift * cond * D / n).astype(np.float32)
    return A1, X0.astype(np.float32)


def warm_roots(env, As, X0s, comm_tol=1e-3, **kw):
    torch, B, dev, h = env
    prm = B.shampoo_root_params_default(**kw)
    dA = [to_dev(torch, a, dev) for a in As]
    dX = [to_dev(torch, x, dev) for x in X0s]
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([a.shape[0] for a in As], prm.precision),
                     dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    wout = torch.full((2 * len(As),), -1, dtype=torch.int32, device=dev)
    B.shampoo_inv_root_warm_batched(h, dA, dX, prm, ws, info, wout, comm_tol)
    torch.cuda.synchronize()
    return [host(x) for x in dX], B.decode_root_info(info), host(wout).reshape(-1, 2)


@pytest.mark.parametrize("prec", [FP32, AUTO, FP64])
@pytest.mark.parametrize("p", [2, 3, 4])
def test_small_drift_keeps_the_warm_limit(env, prec, p):
    """Small drift on ragged sizes (96, 256, 300: one to three tiles with
    tails): the warm result is kept and equals the oracle's warm limit;
    warm iteration counts agree within one."""
    say("warm small drift prec", prec, "p", p)
    tol = 1e-10 if prec == FP64 else 1e-6
    cases = [drift_case(n, 1e2, 3e-3, p, 7 * n + p) for n in (96, 256, 300)]
    Xs, info, wout = warm_roots(env, [a for a, _ in cases], [x for _, x in cases], p=p, eps=1e-6, tol=tol,
                                precision=prec)
    for (A, X0), X, inf, w in zip(cases, Xs, info, wout):
        ref = O.coupled_newton_warm(A, p, X0, eps=1e-6, tol=tol)
        Xt, _, _ = O.inv_root(A, p, eps=1e-6)
        assert not ref["warm_aborted"]
        assert w[0] == 1 and inf["status"] in (0, 1), (w, inf)
        assert abs(int(w[1]) - ref["warm_iters"]) <= 1, (w, ref["warm_iters"])
        assert inf["iters"] == w[1] and inf["precision"] == (64 if prec == FP64 else 32)
        e = rel(X, ref["X"])
        gap = rel(ref["X"], Xt)  # warm limit vs the root: the drift's effect
        assert e <= (1e-6 if prec == FP64 else 1e-3), (A.shape, e)
        assert e < 0.2 * gap, (A.shape, e, gap)


def test_ill_conditioned_tiny_drift_fp64(env):
    """Where the warm start pays: damped condition ~1e6 (the cold fp64
    iteration takes many steps) and a tiny drift.  The warm start is kept
    after at most two iterations and equals the oracle's warm limit from the
    same fp32 X0; the cold call on the same matrices takes at least ten."""
    torch, B, dev, h = env
    say("warm ill-conditioned tiny drift fp64")
    p, tol = 4, 1e-10
    cases = [drift_case(n, 1e6, 1e-9, p, 13 * n) for n in (200, 256)]
    As, X0s = [a for a, _ in cases], [x for _, x in cases]
    Xs, info, wout = warm_roots(env, As, X0s, p=p, eps=1e-6, tol=tol, precision=FP64)
    prm = B.shampoo_root_params_default(p=p, eps=1e-6, tol=tol, precision=FP64)
    dA = [to_dev(torch, a, dev) for a in As]
    dX = [torch.zeros_like(a) for a in dA]
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([a.shape[0] for a in As], FP64), dtype=torch.uint8,
                     device=dev)
    cinfo = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    B.shampoo_inv_root_batched(h, dA, dX, prm, ws, cinfo)
    torch.cuda.synchronize()
    for (A, X0), X, inf, w, ci in zip(cases, Xs, info, wout, B.decode_root_info(cinfo)):
        ref = O.coupled_newton_warm(A, p, X0, eps=1e-6, tol=tol)
        assert not ref["warm_aborted"]
        assert w[0] == 1 and 1 <= w[1] <= 2 and inf["status"] in (0, 1), (w, inf)
        assert rel(X, ref["X"]) <= 1e-6, (A.shape, rel(X, ref["X"]))
        assert ci["iters"] >= 10, ci


@pytest.mark.parametrize("prec", [AUTO, FP64])
def test_mixed_outcomes_in_one_call(env, prec):
    """One grouped call: kept warm starts, warm starts the commutator monitor
    gives up (then the cold root), and an indefinite matrix (NOT_PD, warm
    start not attempted)."""
    say("warm mixed outcomes prec", prec)
    p = 4
    tol = 1e-10 if prec == FP64 else 1e-6
    kept = [drift_case(n, 1e2, 3e-3, p, 5 * n) for n in (130, 256)]
    given_up = [drift_case(n, 1e3, 1e-1, p, 11 * n) for n in (96, 200)]
    bad = np.diag(np.linspace(-1.0, 1.0, 64)).astype(np.float32)
    As = [kept[0][0], given_up[0][0], bad, kept[1][0], given_up[1][0]]
    X0s = [kept[0][1], given_up[0][1], np.eye(64, dtype=np.float32), kept[1][1], given_up[1][1]]
    Xs, info, wout = warm_roots(env, As, X0s, p=p, eps=1e-6, tol=tol, precision=prec)
    for i in (0, 3):
        ref = O.coupled_newton_warm(As[i], p, X0s[i], eps=1e-6, tol=tol)
        assert not ref["warm_aborted"] and wout[i][0] == 1, (i, wout[i])
        assert rel(Xs[i], ref["X"]) <= (1e-6 if prec == FP64 else 1e-3)
    for i in (1, 4):
        ref = O.coupled_newton_warm(As[i], p, X0s[i], eps=1e-6, tol=tol)
        assert ref["warm_aborted"] and ref["warm_iters"] == 1
        assert wout[i][0] == 2 and wout[i][1] == 1, (i, wout[i])
        Xt, _, _ = O.inv_root(As[i], p, eps=1e-6)
        assert info[i]["status"] in (0, 1), info[i]
        assert rel(Xs[i], Xt) <= 1e-3, (i, rel(Xs[i], Xt))
        assert np.array_equal(Xs[i], Xs[i].T)  # the cold iteration's symmetric products
    assert info[2]["status"] == O.NOT_PD and wout[2][0] == 0


@pytest.mark.parametrize("prec", [FP32, FP64])
def test_exact_previous_root_needs_no_iteration(env, prec):
    """X0 already the root (to the tolerance): zero warm iterations and X
    returned bit for bit."""
    say("warm exact root prec", prec)
    A = spd(200, 50.0, 3)
    X0, _, _ = O.inv_root(A, 4, eps=1e-6)
    X0 = X0.astype(np.float32)
    Xs, info, wout = warm_roots(env, [A], [X0], p=4, eps=1e-6, tol=1e-3, precision=prec)
    assert wout[0][0] == 1 and wout[0][1] == 0 and info[0]["status"] == 0, (wout, info)
    assert np.array_equal(Xs[0], X0)


def test_asynchronous_call_matches_polled(env):
    """poll = 0 (every iteration enqueued, finished matrices skip) gives the
    same bits as the polled call."""
    say("warm poll vs async")
    cases = [drift_case(128, 1e2, 1e-4, 4, 1), drift_case(96, 1e3, 1e-1, 4, 2)]
    As, X0s = [a for a, _ in cases], [x for _, x in cases]
    a = warm_roots(env, As, X0s, p=4, eps=1e-6, max_iters=30)
    b = warm_roots(env, As, X0s, p=4, eps=1e-6, max_iters=30, poll=0)
    for xa, xb in zip(a[0], b[0]):
        assert np.array_equal(xa, xb)
    assert np.array_equal(a[2], b[2])
    # warm_out is optional (NULL)
    torch, B, dev, h = env
    prm = B.shampoo_root_params_default(p=4, eps=1e-6, max_iters=30)
    dA = [to_dev(torch, x, dev) for x in As]
    dX = [to_dev(torch, x, dev) for x in X0s]
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([x.shape[0] for x in As], prm.precision),
                     dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    B.shampoo_inv_root_warm_batched(h, dA, dX, prm, ws, info, None)
    torch.cuda.synchronize()
    for xa, xc in zip(a[0], dX):
        assert np.array_equal(xa, host(xc))


def test_rejects_bad_comm_tol(env):
    torch, B, dev, h = env
    A = spd(16, 10.0, 1)
    with pytest.raises(B.ShampooError) as e:
        warm_roots(env, [A], [np.eye(16, dtype=np.float32)], comm_tol=0.0)
    assert e.value.code == B.SHAMPOO_EINVAL


def test_c2_size_warm_sampled(env):
    """The C2 size in the benchmark's launch configuration: 96 statistics
    1024 x 1024 (Wishart, 19 x 4096 degrees of freedom), cold roots, one
    statistics update with a new gradient (1024 x 4096, N(0, 1/4096)), then
    the 96 roots warm-started from the previous ones in one call.  Sampled
    matrices against the oracle's warm iteration on the same fp32 inputs."""
    torch, B, dev, h = env
    say("warm C2 size: 96 x 1024^2")
    from synth import configs as cfg
    nb, n, k = 96, 1024, 4096
    gen = torch.Generator(device=dev).manual_seed(5)
    Ls = [cfg.wishart_bartlett_device(n, 19 * k, 1.0 / k, torch, dev, cfg.C2, b, 9) for b in range(nb)]
    Gs = [torch.randn(n, k, device=dev, generator=gen) / k ** 0.5 for _ in range(nb)]
    Xs = [torch.zeros(n, n, device=dev) for _ in range(nb)]
    prm = B.shampoo_root_params_default(p=4, eps=1e-6)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([n] * nb, prm.precision), dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * nb, dtype=torch.int32, device=dev)
    B.shampoo_inv_root_batched(h, Ls, Xs, prm, ws, info)
    B.shampoo_update_stats(h, [B.Block(G=Gs[b], L=Ls[b]) for b in range(nb)])
    torch.cuda.synchronize()
    samples = (0, 95)
    X0 = {b: host(Xs[b]) for b in samples}
    A1 = {b: host(Ls[b]) for b in samples}
    wout = torch.full((2 * nb,), -1, dtype=torch.int32, device=dev)
    B.shampoo_inv_root_warm_batched(h, Ls, Xs, prm, ws, info, wout)
    torch.cuda.synchronize()
    w = host(wout).reshape(-1, 2)
    assert (w[:, 0] == 1).all(), w[:4]
    infos = B.decode_root_info(info)
    assert all(i["status"] in (0, 1) for i in infos)
    for b in samples:
        ref = O.coupled_newton_warm(A1[b], 4, X0[b], eps=1e-6, tol=1e-6)
        assert not ref["warm_aborted"]
        assert abs(int(w[b, 1]) - ref["warm_iters"]) <= 1, (w[b], ref["warm_iters"])
        assert rel(host(Xs[b]), ref["X"]) <= 1e-3, b
