"""shampoo_precondition_graft (preconditioning with graft pass 1 fused into
the GEMM that writes P, then graft pass 2) against the two separate calls
shampoo_precondition + shampoo_graft(beta1 = 0, use_shampoo) and against the
oracle (precondition, graft_update).

P and D are the same arithmetic in both routes and must agree bit for bit
(also where the separate call runs 128 x 256 tiles and the fused one
128 x 128);
the step size sums the same squares in another order, so W agrees to 1e-5
of the step; against the oracle the bars of the update tests (2e-3 on P and
dW, 1e-6 on D, 1e-5 on the norms).  Cases: left, right and two-sided roots,
ragged shapes on padded (strided) views, one launch over mixed sizes, bf16
gradients, a zero gradient block, and calls large and uniform enough to be
split into groups (graft pass 2 of a group on the handle's side stream,
overlapping the next group's GEMMs), which must give every block bit for
bit what a call with that block alone gives.
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


def _case(torch, dev, m, n, sides, pad, seed, bf16=False):
    r = np.random.default_rng(seed)
    if bf16:
        bits = cfg.c5_grad_bf16(seed, 1, (m, n))
        G = O.bf16_bits_to_f64(bits)
    else:
        G = r.standard_normal((m, n)).astype(np.float32)
        G[r.random((m, n)) < 0.05] = 0.0
    W = (0.1 * r.standard_normal((m, n))).astype(np.float32)
    D = r.random((m, n)).astype(np.float32)
    D[G == 0] = 0.0
    Lr = O.inv_root(spd(m, 30.0, seed + 1), 4, 1e-6)[0].astype(np.float32) if "L" in sides else None
    Rr = O.inv_root(spd(n, 30.0, seed + 2), 4, 1e-6)[0].astype(np.float32) if "R" in sides else None

    def view(x, dtype=torch.float32):
        big = torch.zeros(m, n + pad, device=dev, dtype=dtype)
        big[:, :n] = x
        return big[:, :n]

    def make():
        g = view(to_dev(torch, bits.view(np.int16), dev).view(torch.bfloat16), torch.bfloat16) if bf16 else \
            view(to_dev(torch, G, dev))
        return dict(G=g, W=view(to_dev(torch, W, dev)), D=view(to_dev(torch, D, dev)),
                    P=view(torch.zeros(m, n, device=dev)),
                    Lr=None if Lr is None else to_dev(torch, Lr, dev), Rr=None if Rr is None else to_dev(torch, Rr, dev))
    return dict(G=G, W=W, D=D, Lr=Lr, Rr=Rr), make


def _run_both(env, cases, eta0=0.05):
    torch, B, dev, h = env
    fused = [mk() for _, mk in cases]
    split = [mk() for _, mk in cases]
    nf = torch.zeros(3 * len(cases), device=dev)
    ns = torch.zeros(3 * len(cases), device=dev)
    B.shampoo_precondition_graft(h, [B.Block(**t) for t in fused], eta0, norms=nf)
    bs = [B.Block(**t) for t in split]
    B.shampoo_precondition(h, bs)
    B.shampoo_graft(h, bs, eta0, norms=ns)
    torch.cuda.synchronize()
    return fused, split, host(nf).reshape(-1, 3), host(ns).reshape(-1, 3)


def _check(cases, fused, split, nf, ns, eta0=0.05):
    for k, ((ref, _), f, s) in enumerate(zip(cases, fused, split)):
        assert np.array_equal(host(f["P"]), host(s["P"])), k
        assert np.array_equal(host(f["D"]), host(s["D"])), k
        W0 = ref["W"].astype(np.float64)
        assert rel(host(f["W"]) - W0, host(s["W"]) - W0) <= 1e-5, k
        assert np.allclose(nf[k], ns[k], rtol=1e-6, atol=0), (k, nf[k], ns[k])
        Po = O.precondition(ref["G"], ref["Lr"], ref["Rr"])
        out = O.graft_update(ref["W"], ref["D"], ref["G"], Po, eta0)
        assert rel(host(f["P"]), Po) <= TOL, k
        assert rel(host(f["W"]) - W0, out["W"] - W0) <= TOL, k
        assert rel(host(f["D"]), out["D"]) <= 1e-6, k
        assert abs(nf[k, 0] - out["norm_mg"]) <= 1e-5 * out["norm_mg"], k


@pytest.mark.parametrize("m,n,sides,pad", [(1024, 4096, "L", 0), (256, 384, "R", 0), (512, 512, "LR", 0),
                                           (200, 96, "LR", 3), (129, 257, "L", 2), (77, 45, "R", 1),
                                           (1, 1, "LR", 0), (300, 130, "LR", 4),
                                           # widths that are multiples of 256: the separate call takes
                                           # 128 x 256 tiles, on ragged rows and unaligned row strides
                                           (300, 768, "LR", 5), (129, 512, "L", 3)])
def test_fused_matches_two_calls(env, m, n, sides, pad):
    torch, B, dev, h = env
    say("precondition_graft", m, n, sides, pad)
    cases = [_case(torch, dev, m, n, sides, pad, m + 3 * n + len(sides))]
    _check(cases, *_run_both(env, cases))


def test_fused_mixed_sizes_bf16_and_zero_block(env):
    """One call over blocks of mixed sizes and root layouts (the launch deals
    tile chunks over the XCDs), bf16 gradients, and a block whose gradient
    is zero (eta = 0: W unchanged)."""
    torch, B, dev, h = env
    say("precondition_graft mixed")
    for bf16 in (False, True):
        cases = [_case(torch, dev, m, n, s, 0, 11 + i, bf16)
                 for i, (m, n, s) in enumerate([(128, 256, "LR"), (1024, 1024, "L"), (256, 128, "R"),
                                                (640, 200, "LR"), (96, 96, "LR")])]
        _check(cases, *_run_both(env, cases))
    ref, mk = _case(torch, dev, 64, 64, "LR", 0, 5)
    t = mk()
    t["G"].zero_()
    W0 = host(t["W"]).copy()
    norms = torch.zeros(3, device=dev)
    B.shampoo_precondition_graft(h, [B.Block(**t)], 0.05, norms=norms)
    torch.cuda.synchronize()
    assert np.array_equal(host(t["W"]), W0) and host(norms)[2] == 0.0


@pytest.mark.parametrize("nb,m,n,sides,bf16", [(8, 512, 4096, "L", False), (8, 512, 4096, "L", True),
                                                (16, 1024, 1024, "LR", False)])
def test_fused_groups_match_single_block_calls(env, nb, m, n, sides, bf16):
    """Calls of 8+ blocks of one shape and 2^24 elements run in groups; P, D,
    W and the norms of every block equal those of a call with that block
    alone (one group), and agree with the oracle."""
    torch, B, dev, h = env
    say("precondition_graft groups:", nb, m, n, sides, "bf16", bf16)
    cases = [_case(torch, dev, m, n, sides, 0, 101 + i, bf16) for i in range(nb)]
    grouped = [mk() for _, mk in cases]
    single = [mk() for _, mk in cases]
    ng = torch.zeros(3 * nb, device=dev)
    ns = torch.zeros(3 * nb, device=dev)
    B.shampoo_precondition_graft(h, [B.Block(**t) for t in grouped], 0.05, norms=ng)
    for k, t in enumerate(single):
        B.shampoo_precondition_graft(h, [B.Block(**t)], 0.05, norms=ns[3 * k:3 * k + 3])
    torch.cuda.synchronize()
    for k in range(nb):
        for key in ("P", "D", "W"):
            assert np.array_equal(host(grouped[k][key]), host(single[k][key])), (k, key)
    assert np.array_equal(host(ng), host(ns))
    nf = host(ng).reshape(-1, 3)
    for k in (0, nb // 2, nb - 1):
        ref = cases[k][0]
        W0 = ref["W"].astype(np.float64)
        Po = O.precondition(ref["G"], ref["Lr"], ref["Rr"])
        out = O.graft_update(ref["W"], ref["D"], ref["G"], Po, 0.05)
        assert rel(host(grouped[k]["P"]), Po) <= TOL, k
        assert rel(host(grouped[k]["W"]) - W0, out["W"] - W0) <= TOL, k
        assert rel(host(grouped[k]["D"]), out["D"]) <= 1e-6, k
        assert abs(nf[k, 0] - out["norm_mg"]) <= 1e-5 * out["norm_mg"], k


def test_fused_rejects_rootless_block(env):
    torch, B, dev, h = env
    x = torch.zeros(8, 8, device=dev)
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_precondition_graft(h, [B.Block(G=x, W=x.clone(), D=x.clone(), P=x.clone())], 0.05)
    assert e.value.code == B.SHAMPOO_EINVAL


def test_aliasing_is_rejected(env):
    torch, B, dev, h = env
    x = torch.zeros(8, 8, device=dev)
    r = torch.eye(8, device=dev)
    for kw in (dict(G=x, P=x, Lr=r), dict(G=x, P=r, Lr=r)):
        with pytest.raises(B.ShampooError) as e:
            B.shampoo_precondition(h, [B.Block(**kw)])
        assert e.value.code == B.SHAMPOO_EINVAL
    W, D, P = (torch.zeros(8, 8, device=dev) for _ in range(3))
    for kw in (dict(G=x, W=W, D=D, P=x, Lr=r), dict(G=x, W=W, D=W, P=P, Lr=r), dict(G=x, W=W, D=D, P=P, Lr=P)):
        with pytest.raises(B.ShampooError) as e:
            B.shampoo_precondition_graft(h, [B.Block(**kw)], 0.05)
        assert e.value.code == B.SHAMPOO_EINVAL


def test_aliasing_in_stats_and_graft_is_rejected(env):
    torch, B, dev, h = env
    x = torch.zeros(8, 8, device=dev)
    W, D, P = (torch.zeros(8, 8, device=dev) for _ in range(3))
    with pytest.raises(B.ShampooError):
        B.shampoo_update_stats(h, [B.Block(G=x, L=x)])
    for kw in (dict(G=x, W=x, D=D, P=P), dict(G=x, W=W, D=P, P=P), dict(G=x, W=W, D=W, P=P)):
        with pytest.raises(B.ShampooError) as e:
            B.shampoo_graft(h, [B.Block(**kw)], 0.05)
        assert e.value.code == B.SHAMPOO_EINVAL
