"""GPU preconditioning and grafted update against the oracle.

Bar: relative Frobenius error <= 2e-3 on P and on the parameter change dW
(per block); norms of the graft to 1e-5.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say, spd, to_dev

pytestmark = pytest.mark.gpu
TOL = 2e-3


@pytest.fixture(scope="module")
def env():
    torch, B, dev = gpu_env()
    h = B.shampoo_create(0)
    yield torch, B, dev, h
    B.shampoo_destroy(h)


def _roots(m, n, seed):
    Lr, _, _ = O.inv_root(spd(m, 50.0, seed), 4, 1e-6)
    Rr, _, _ = O.inv_root(spd(n, 50.0, seed + 1), 4, 1e-6)
    return Lr.astype(np.float32), Rr.astype(np.float32)


@pytest.mark.parametrize("m,n,sides,pad", [(128, 128, "LR", 0), (200, 96, "LR", 0), (1024, 1024, "LR", 0),
                                           (64, 300, "L", 0), (300, 64, "R", 3), (77, 45, "", 1),
                                           (1, 1, "LR", 0), (129, 257, "LR", 2)])
def test_precondition(env, m, n, sides, pad):
    torch, B, dev, h = env
    say("precondition", m, n, sides, pad)
    r = np.random.default_rng(m + 7 * n)
    G = r.standard_normal((m, n)).astype(np.float32)
    Lr, Rr = _roots(m, n, m + n)
    g = to_dev(torch, G, dev)
    big = torch.zeros(m, n + pad, device=dev)
    P = big[:, :n]
    if pad:
        gb = torch.zeros(m, n + pad, device=dev)
        gb[:, :n] = g
        g = gb[:, :n]
    dLr = to_dev(torch, Lr, dev) if "L" in sides else None
    dRr = to_dev(torch, Rr, dev) if "R" in sides else None
    B.shampoo_precondition(h, [B.Block(G=g, P=P, Lr=dLr, Rr=dRr)])
    torch.cuda.synchronize()
    Po = O.precondition(G, Lr if "L" in sides else None, Rr if "R" in sides else None)
    assert rel(host(P), Po) <= TOL


def test_precondition_bf16_grouped(env):
    torch, B, dev, h = env
    say("precondition bf16 grouped")
    blocks, refs, Ps = [], [], []
    for k, (m, n) in enumerate([(128, 256), (512, 512), (256, 128)]):
        bits = cfg.c5_grad_bf16(k, 1, (m, n))
        g = to_dev(torch, bits.view(np.int16), dev).view(torch.bfloat16)
        Lr, Rr = _roots(m, n, 40 + k)
        P = torch.zeros(m, n, device=dev)
        blocks.append(B.Block(G=g, P=P, Lr=to_dev(torch, Lr, dev), Rr=to_dev(torch, Rr, dev)))
        refs.append(O.precondition(O.bf16_bits_to_f64(bits), Lr, Rr))
        Ps.append(P)
    B.shampoo_precondition(h, blocks)
    torch.cuda.synchronize()
    for P, Po in zip(Ps, refs):
        assert rel(host(P), Po) <= TOL


@pytest.mark.parametrize("beta1,use_shampoo", [(0.0, True), (0.0, False), (0.9, True), (0.9, False)])
def test_graft(env, beta1, use_shampoo):
    torch, B, dev, h = env
    say("graft", beta1, use_shampoo)
    shapes = [(128, 128), (300, 70), (1, 5), (1024, 1024)]
    r = np.random.default_rng(5)
    blocks, refs, outs = [], [], []
    for (m, n) in shapes:
        W = r.standard_normal((m, n)).astype(np.float32)
        D = r.random((m, n)).astype(np.float32)
        G = r.standard_normal((m, n)).astype(np.float32)
        G[r.random((m, n)) < 0.1] = 0.0
        D[G == 0] = 0.0                                  # includes entries with D == 0 and G == 0
        P = r.standard_normal((m, n)).astype(np.float32)
        Mg = r.standard_normal((m, n)).astype(np.float32)
        Ps = r.standard_normal((m, n)).astype(np.float32)
        dW, dD, dG, dP = (to_dev(torch, x, dev) for x in (W, D, G, P))
        dMg, dPs = to_dev(torch, Mg, dev), to_dev(torch, Ps, dev)
        blocks.append(B.Block(G=dG, W=dW, D=dD, P=dP, Mg=dMg if beta1 else None, Ps=dPs if beta1 else None))
        refs.append((W, O.graft_update(W, D, G, P, 0.05, beta1, Mg if beta1 else None, Ps if beta1 else None,
                                       use_shampoo)))
        outs.append((dW, dD, dMg, dPs))
    norms = torch.zeros(3 * len(shapes), device=dev)
    B.shampoo_graft(h, blocks, 0.05, beta1=beta1, use_shampoo=use_shampoo, norms=norms)
    torch.cuda.synchronize()
    nh = host(norms).reshape(-1, 3)
    for k, ((W0, ref), (dW, dD, dMg, dPs)) in enumerate(zip(refs, outs)):
        assert rel(host(dW) - W0, ref["W"] - W0) <= TOL
        assert rel(host(dD), ref["D"]) <= 1e-6
        assert abs(nh[k, 0] - ref["norm_mg"]) <= 1e-5 * ref["norm_mg"]
        assert abs(nh[k, 2] - ref["eta"]) <= 1e-5 * max(ref["eta"], 1e-30)
        # property of the graft: the step has the AdaGrad step's length, ||dW||_F = eta0 ||Mg||_F
        dWn = float(np.linalg.norm(host(dW).astype(np.float64) - W0))
        assert abs(dWn - 0.05 * nh[k, 0]) <= 1e-4 * dWn, (k, dWn, nh[k])
        if beta1:
            assert rel(host(dMg), ref["Mg"]) <= 1e-5
            if use_shampoo:
                assert rel(host(dPs), ref["Ps"]) <= 1e-6


def test_graft_zero_gradient(env):
    torch, B, dev, h = env
    say("graft zero gradient")
    W = torch.ones(16, 16, device=dev)
    D = torch.zeros(16, 16, device=dev)
    G = torch.zeros(16, 16, device=dev)
    P = torch.zeros(16, 16, device=dev)
    norms = torch.full((3,), 7.0, device=dev)
    B.shampoo_graft(h, [B.Block(G=G, W=W, D=D, P=P)], 0.1, norms=norms)
    torch.cuda.synchronize()
    assert torch.all(W == 1.0) and torch.all(torch.isfinite(D)) and float(norms[2]) == 0.0


def test_c1_end_to_end(env):
    """C1: one 128 x 128 block, 10 steps, roots every step (AUTO policy),
    one grouped root call for L and R per step; compared with the oracle's
    own fp64 trajectory (its own statistics and eigh roots)."""
    torch, B, dev, h = env
    say("C1 end to end")
    n, p, eps, eta0 = 128, 4, 1e-6, 1e-2
    W0 = cfg.c1_weight()
    W = to_dev(torch, W0, dev)
    D, P, L, R, Lr, Rr = (torch.zeros(n, n, device=dev) for _ in range(6))
    prm = B.shampoo_root_params_default(p=p, eps=eps)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([n, n]), dtype=torch.uint8, device=dev)
    info = torch.zeros(16, dtype=torch.int32, device=dev)
    st = dict(W=W0.astype(np.float64), D=np.zeros((n, n)), L=np.zeros((n, n)), R=np.zeros((n, n)))
    errs = []
    for t in range(1, 11):
        G = cfg.c1_grad(t)
        Wprev = host(W).astype(np.float64)
        Wprev_o = st["W"].copy()
        blk = B.Block(G=to_dev(torch, G, dev), W=W, D=D, P=P, L=L, R=R, Lr=Lr, Rr=Rr)
        B.shampoo_update_stats(h, [blk])
        B.shampoo_inv_root_batched(h, [L, R], [Lr, Rr], prm, ws, info)
        B.shampoo_precondition(h, [blk])
        B.shampoo_graft(h, [blk], eta0)
        torch.cuda.synchronize()
        st = O.shampoo_step(st, G, p=p, eps=eps, eta0=eta0)
        errs.append(rel(host(W) - Wprev, st["W"] - Wprev_o))
        assert rel(host(L), st["L"]) <= 1e-4
    print("C1 per-step update errors", ["%.1e" % e for e in errs])
    assert max(errs) <= TOL, errs


@pytest.mark.parametrize("beta1,use_shampoo", [(0.0, True), (0.0, False), (0.9, True), (0.9, False)])
def test_graft_lamb(env, beta1, use_shampoo):
    """LARS/LAMB magnitude eta0 ||W||_F along the unit direction."""
    torch, B, dev, h = env
    say("graft lamb", beta1, use_shampoo)
    shapes = [(128, 128), (300, 70), (1, 5), (1024, 1024)]
    r = np.random.default_rng(15)
    blocks, refs, outs = [], [], []
    for (m, n) in shapes:
        W = r.standard_normal((m, n)).astype(np.float32)
        G = r.standard_normal((m, n)).astype(np.float32)
        P = r.standard_normal((m, n)).astype(np.float32)
        Mg = r.standard_normal((m, n)).astype(np.float32)
        Ps = r.standard_normal((m, n)).astype(np.float32)
        dW, dG, dP = (to_dev(torch, x, dev) for x in (W, G, P))
        dMg, dPs = to_dev(torch, Mg, dev), to_dev(torch, Ps, dev)
        blocks.append(B.Block(G=dG, W=dW, P=dP, Mg=dMg if beta1 else None, Ps=dPs if beta1 else None))
        refs.append((W, O.lamb_graft_update(W, G, P, 0.05, beta1, Mg if beta1 else None, Ps if beta1 else None,
                                            use_shampoo)))
        outs.append((dW, dMg, dPs))
    norms = torch.zeros(3 * len(shapes), device=dev)
    B.shampoo_graft_lamb(h, blocks, 0.05, beta1=beta1, use_shampoo=use_shampoo, norms=norms)
    torch.cuda.synchronize()
    nh = host(norms).reshape(-1, 3)
    for k, ((W0, ref), (dW, dMg, dPs)) in enumerate(zip(refs, outs)):
        assert rel(host(dW) - W0, ref["W"] - W0) <= TOL
        assert abs(nh[k, 0] - ref["norm_w"]) <= 1e-5 * ref["norm_w"]
        assert abs(nh[k, 1] - ref["norm_dir"]) <= 1e-5 * ref["norm_dir"]
        assert abs(nh[k, 2] - ref["eta"]) <= 1e-5 * ref["eta"]
        if beta1:
            assert rel(host(dMg), ref["Mg"]) <= 1e-6
            if use_shampoo:
                assert rel(host(dPs), ref["Ps"]) <= 1e-6


def test_graft_lamb_bf16_and_c1_steps(env):
    """bf16 gradients, then six C1 steps with roots every step under the
    LAMB graft against the oracle's own trajectory (per-step dW)."""
    torch, B, dev, h = env
    say("graft lamb bf16 + C1 steps")
    bits = cfg.c5_grad_bf16(3, 1, (256, 128))
    g = to_dev(torch, bits.view(np.int16), dev).view(torch.bfloat16)
    W0 = np.random.default_rng(2).standard_normal((256, 128)).astype(np.float32)
    W = to_dev(torch, W0, dev)
    B.shampoo_graft_lamb(h, [B.Block(G=g, W=W)], 0.1, use_shampoo=False)
    torch.cuda.synchronize()
    ref = O.lamb_graft_update(W0, O.bf16_bits_to_f64(bits), None, 0.1, use_shampoo=False)
    assert rel(host(W) - W0, ref["W"] - W0) <= TOL
    n, p, eps, eta0 = 128, 4, 1e-6, 1e-2
    W0 = cfg.c1_weight()
    W = to_dev(torch, W0, dev)
    P, L, R, Lr, Rr = (torch.zeros(n, n, device=dev) for _ in range(5))
    prm = B.shampoo_root_params_default(p=p, eps=eps)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([n, n]), dtype=torch.uint8, device=dev)
    info = torch.zeros(16, dtype=torch.int32, device=dev)
    Lo, Ro, Wo = np.zeros((n, n)), np.zeros((n, n)), W0.astype(np.float64)
    for t in range(1, 7):
        G = cfg.c1_grad(t)
        Wprev = host(W).astype(np.float64)
        blk = B.Block(G=to_dev(torch, G, dev), W=W, P=P, L=L, R=R, Lr=Lr, Rr=Rr)
        B.shampoo_update_stats(h, [blk])
        B.shampoo_inv_root_batched(h, [L, R], [Lr, Rr], prm, ws, info)
        B.shampoo_precondition(h, [blk])
        B.shampoo_graft_lamb(h, [blk], eta0)
        torch.cuda.synchronize()
        Lo, Ro = O.stats_update(Lo, Ro, G)
        Po = O.precondition(G, O.inv_root(Lo, p, eps)[0], O.inv_root(Ro, p, eps)[0])
        out = O.lamb_graft_update(Wo, G, Po, eta0)
        assert rel(host(W) - Wprev, out["W"] - Wo) <= TOL, t
        Wo = out["W"]
