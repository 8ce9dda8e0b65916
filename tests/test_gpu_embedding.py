"""Embedding layers on the GPU (shampoo_embedding_*) against the oracle.

Bars: active rows and counts bit-exact; compact gradient rows U relative
error <= 1e-5 (fp32 sums in entry order vs fp64); statistics <= 1e-5; the
grafted step's dW <= 2e-3 (as for dense blocks); rows no entry touched keep
their W and D bits exactly.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch, B, dev = gpu_env()
    h = B.shampoo_create(0)
    yield torch, B, dev, h
    B.shampoo_destroy(h)


def _i32(torch, x, dev):
    return None if x is None else torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev)


def run_rows(env, idx, feat, weight, vocab, dy):
    torch, B, dev, h = env
    nnz, dim = len(idx), dy.shape[1]
    rows = torch.full((nnz,), 7, dtype=torch.int32, device=dev)
    U = torch.full((nnz, dim), float("nan"), device=dev)
    count = torch.zeros(2, dtype=torch.int32, device=dev)
    ws = torch.empty(B.shampoo_embedding_workspace_bytes(nnz, dim), dtype=torch.uint8, device=dev)
    wt = None if weight is None else to_dev(torch, np.asarray(weight, dtype=np.float32), dev)
    B.shampoo_embedding_rows(h, _i32(torch, idx, dev), _i32(torch, feat, dev), wt, vocab, to_dev(torch, dy, dev),
                             rows, U, count, ws)
    return rows, U, count, ws


def check_rows(rows, U, count, idx, feat, weight, vocab, dy):
    r_o, U_o = O.embedding_rows(vocab, idx, feat, weight, dy)
    u = len(r_o)
    c = host(count)
    m = dy.shape[0]
    f = np.arange(len(idx)) if feat is None else np.asarray(feat)
    dropped = int(np.sum((np.asarray(idx) < 0) | (np.asarray(idx) >= vocab) | (f < 0) | (f >= m)))
    assert (int(c[0]), int(c[1])) == (u, dropped)
    rh = host(rows)
    assert np.array_equal(rh[:u], r_o) and np.all(rh[u:] == -1)
    Uh = host(U)
    assert rel(Uh[:u], U_o) <= 1e-5
    assert np.all(np.isnan(Uh[u:]))  # rows past the active ones are not written
    return r_o, U_o


@pytest.mark.parametrize("dim,multi,bad", [(256, False, False), (256, True, True), (203, True, False),
                                           (64, False, True)])
def test_rows_against_oracle(env, dim, multi, bad):
    say("embedding rows", dim, multi, bad)
    vocab, nnz = 5000, 3000
    idx, feat, weight, m = cfg.c6_lookup(1, nnz, vocab, multi=multi)
    if bad:  # out-of-range rows and features are dropped and counted
        idx = idx.copy()
        idx[::97] = -1
        idx[5::89] = vocab
        if feat is not None:
            feat = feat.copy()
            feat[3::71] = m
    dy = cfg.c6_dy(1, m, dim)
    rows, U, count, _ = run_rows(env, idx, feat, weight, vocab, dy)
    env[0].cuda.synchronize()
    check_rows(rows, U, count, idx, feat, weight, vocab, dy)


def test_rows_degenerate(env):
    torch, B, dev, h = env
    say("embedding rows degenerate")
    dy = cfg.c6_dy(2, 4, 32)
    # a single entry
    rows, U, count, _ = run_rows(env, np.array([3]), None, None, 10, dy[:1])
    torch.cuda.synchronize()
    check_rows(rows, U, count, np.array([3]), None, None, 10, dy[:1])
    # every entry invalid: nothing active, U not written
    rows, U, count, ws = run_rows(env, np.array([-1, 10, 11, -5]), None, None, 10, dy)
    torch.cuda.synchronize()
    assert host(count).tolist() == [0, 4] and np.all(host(rows) == -1) and np.all(np.isnan(host(U)))
    U.zero_()
    # statistics from no rows leave R unchanged; the graft changes nothing
    R = torch.eye(32, device=dev)
    B.shampoo_embedding_stats(h, U, count, R, 1.0, ws)
    W = torch.ones(10, 32, device=dev)
    D = torch.zeros(10, 32, device=dev)
    P = torch.zeros_like(U)
    B.shampoo_embedding_precondition(h, U, count, R, P)
    B.shampoo_embedding_graft(h, rows, count, U, P, W, D, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(R, torch.eye(32, device=dev)) and torch.all(W == 1) and torch.all(D == 0)
    # argument errors
    with pytest.raises(B.ShampooError):
        B.shampoo_embedding_rows(h, _i32(torch, [1], dev), None, None, 0, to_dev(torch, dy, dev), rows, U, count, ws)
    big = 100000
    rows_b = torch.zeros(big, dtype=torch.int32, device=dev)
    U_b = torch.zeros(big, 32, device=dev)
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_embedding_rows(h, _i32(torch, np.zeros(big), dev), None, None, 10, to_dev(torch, dy, dev),
                                 rows_b, U_b, count, ws[:16])
    assert e.value.code == B.SHAMPOO_ENOMEM


@pytest.mark.parametrize("vocab,nnz,dim,beta2", [(50000, 20000, 256, 1.0), (3000, 700, 96, 0.9),
                                                 (32768, 65536, 1024, 1.0)])
def test_stats_split_k(env, vocab, nnz, dim, beta2):
    """R = beta2 R + c U^T U over the active rows, split over row chunks
    (40 splits at 20000 x 256, 29 at 65536 x 1024)."""
    torch, B, dev, h = env
    say("embedding stats", vocab, nnz, dim, beta2)
    idx, feat, weight, m = cfg.c6_lookup(3, nnz, vocab)
    dy = cfg.c6_dy(3, m, dim)
    rows, U, count, ws = run_rows(env, idx, feat, weight, vocab, dy)
    R0 = cfg.wishart_bartlett(dim, 4 * dim, 1e-3, cfg.C6, 9, dim)
    R = to_dev(torch, R0.astype(np.float32), dev)
    B.shampoo_embedding_stats(h, U, count, R, beta2, ws)
    torch.cuda.synchronize()
    _, U_o = O.embedding_rows(vocab, idx, feat, weight, dy)
    _, Ro = O.stats_update(None, R0.astype(np.float32), U_o, beta2)
    assert rel(host(R), Ro) <= 1e-5
    assert np.array_equal(host(R), host(R).T)


def test_step_against_dense_oracle(env):
    """Three steps on a 20000 x 256 table with multi-hot bags: AdaGrad
    fallback at step 1, then roots R^(-1/2) (one-sided, p = 2) each step,
    preconditioned grafted updates; the oracle runs the dense definition on
    the whole table."""
    torch, B, dev, h = env
    say("embedding step vs dense oracle")
    vocab, nnz, dim, eta0, eps = 20000, 8000, 256, 1e-2, 1e-6
    W0 = cfg.c6_table(vocab, dim)
    W = to_dev(torch, W0, dev)
    D = torch.zeros(vocab, dim, device=dev)
    R = torch.zeros(dim, dim, device=dev)
    Rr = torch.zeros(dim, dim, device=dev)
    st = dict(W=W0.astype(np.float64), D=np.zeros((vocab, dim)), R=np.zeros((dim, dim)))
    prm = B.shampoo_root_params_default(p=2, eps=eps)
    rws = torch.empty(B.shampoo_inv_root_workspace_bytes([dim]), dtype=torch.uint8, device=dev)
    info = torch.zeros(8, dtype=torch.int32, device=dev)
    norms = torch.zeros(3, device=dev)
    for t in range(1, 4):
        idx, feat, weight, m = cfg.c6_lookup(10 + t, nnz, vocab, multi=True)
        dy = cfg.c6_dy(10 + t, m, dim)
        Wprev, Dprev, Wprev_o = host(W).copy(), host(D).copy(), st["W"].copy()
        rows, U, count, ws = run_rows(env, idx, feat, weight, vocab, dy)
        B.shampoo_embedding_stats(h, U, count, R, 1.0, ws)
        use = t > 1
        P = torch.zeros_like(U)
        if use:
            B.shampoo_inv_root_batched(h, [R], [Rr], prm, rws, info)
            B.shampoo_embedding_precondition(h, U, count, Rr, P)
        B.shampoo_embedding_graft(h, rows, count, U, P, W, D, eta0, use_shampoo=use, norms=norms)
        torch.cuda.synchronize()
        G = O.embedding_grad(vocab, idx, feat, weight, dy)
        st = O.shampoo_step(st, G, p=2, eps=eps, eta0=eta0, left=False, right=True, use_shampoo=use,
                            refresh_roots=use)
        assert rel(host(R), st["R"]) <= 1e-5
        # this step's update against the oracle's own (the W trajectories
        # differ by rounding only and W does not enter the update)
        assert rel(host(W).astype(np.float64) - Wprev, st["W"] - Wprev_o) <= 2e-3, t
        active = np.zeros(vocab, dtype=bool)
        active[host(rows)[: int(host(count)[0])]] = True
        assert np.array_equal(host(W)[~active], Wprev[~active])
        assert np.array_equal(host(D)[~active], Dprev[~active])
        assert rel(host(D), st["D"]) <= 1e-6
        assert abs(float(host(norms)[2]) - st["eta"]) <= 1e-4 * st["eta"]
