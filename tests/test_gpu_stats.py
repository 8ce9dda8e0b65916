"""GPU statistics update (shampoo_update_stats) against the fp64 oracle.

Bar: relative Frobenius error <= 1e-4 per matrix (fp32 accumulation); exact
equality for integer-valued gradients, whose sums are exact in fp32 in any
order; L and R bitwise symmetric.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say, to_dev

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.fixture(scope="module")
def env():
    torch, B, dev = gpu_env()
    h = B.shampoo_create(0)
    yield torch, B, dev, h
    B.shampoo_destroy(h)


def _run(env, Gs, beta2=1.0, left=True, right=True, bf16=False, ld_pad=0):
    torch, B, dev, h = env
    m, n = Gs[0].shape
    L = torch.zeros(m, m, device=dev) if left else None
    R = torch.zeros(n, n, device=dev) if right else None
    for G in Gs:
        if bf16:
            g = to_dev(torch, cfg.f32_to_bf16_bits(G).view(np.int16), dev).view(torch.bfloat16)
        else:
            g = to_dev(torch, G, dev)
        if ld_pad:
            big = torch.zeros(m, n + ld_pad, device=dev, dtype=g.dtype)
            big[:, :n] = g
            g = big[:, :n]
        B.shampoo_update_stats(h, [B.Block(G=g, L=L, R=R)], beta2=beta2)
    torch.cuda.synchronize()
    return (None if L is None else host(L)), (None if R is None else host(R))


def _oracle(Gs, beta2=1.0, bf16=False):
    m, n = Gs[0].shape
    L, R = np.zeros((m, m)), np.zeros((n, n))
    for G in Gs:
        g = O.bf16_bits_to_f64(cfg.f32_to_bf16_bits(G)) if bf16 else G
        L, R = O.stats_update(L, R, g, beta2)
    return L, R


def test_c1_stats_10_steps(env):
    say("stats C1 128x128 x10")
    Gs = [cfg.c1_grad(t) for t in range(1, 11)]
    L, R = _run(env, Gs)
    Lo, Ro = _oracle(Gs)
    assert rel(L, Lo) <= TOL and rel(R, Ro) <= TOL
    assert np.array_equal(L, L.T) and np.array_equal(R, R.T)


@pytest.mark.parametrize("m,n,pad", [(1, 1, 0), (5, 3, 0), (130, 70, 0), (257, 129, 3), (64, 384, 0),
                                     (300, 1030, 2)])
def test_ragged_and_strided(env, m, n, pad):
    say("stats ragged", m, n, pad)
    r = np.random.default_rng(m * 1000 + n)
    Gs = [r.standard_normal((m, n)).astype(np.float32) for _ in range(3)]
    L, R = _run(env, Gs, ld_pad=pad)
    Lo, Ro = _oracle(Gs)
    assert rel(L, Lo) <= TOL and rel(R, Ro) <= TOL
    assert np.array_equal(L, L.T) and np.array_equal(R, R.T)


def test_integer_gradients_exact(env):
    say("stats integer exact")
    r = np.random.default_rng(7)
    Gs = [r.integers(-8, 9, size=(200, 136)).astype(np.float32) for _ in range(4)]
    L, R = _run(env, Gs)
    Lo, Ro = _oracle(Gs)
    assert np.array_equal(L.astype(np.float64), Lo)
    assert np.array_equal(R.astype(np.float64), Ro)


def test_ema_beta2(env):
    say("stats beta2=0.9")
    r = np.random.default_rng(8)
    Gs = [r.standard_normal((96, 160)).astype(np.float32) for _ in range(5)]
    L, R = _run(env, Gs, beta2=0.9)
    Lo, Ro = _oracle(Gs, beta2=0.9)
    assert rel(L, Lo) <= TOL and rel(R, Ro) <= TOL


def test_one_sided_and_bf16(env):
    say("stats bf16 left only")
    Gs = [cfg.gaussian((256, 384), 1e-3, 99, t) for t in range(3)]
    L, R = _run(env, Gs, right=False, bf16=True)
    Lo, _ = _oracle(Gs, bf16=True)
    assert R is None and rel(L, Lo) <= TOL


def test_c4_two_layers_strided_blocks(env):
    """Two BERT-shaped layers (24 blocks of 1024 x 1024, FFN blocks strided
    views of 1024 x 4096 / 4096 x 1024 tensors) in one grouped call."""
    torch, B, dev, h = env
    say("stats C4 2 layers grouped")
    shapes = dict(cfg.c4_layer_tensors())
    names = [nm for nm, _ in cfg.c4_layer_tensors()]
    blocks, refs = [], []
    Ls, Rs = [], []
    for layer in range(2):
        tens = {}
        for t, nm in enumerate(names):
            tens[t] = (cfg.c4_grad(layer, t, 1, shapes[nm]))
        dtens = {t: to_dev(torch, g, dev) for t, g in tens.items()}
        for (t, r0, c0, rr, cc) in cfg.c4_blocks():
            g = dtens[t][r0:r0 + rr, c0:c0 + cc]
            L = torch.zeros(rr, rr, device=dev)
            R = torch.zeros(cc, cc, device=dev)
            blocks.append(B.Block(G=g, L=L, R=R))
            Ls.append(L)
            Rs.append(R)
            refs.append(tens[t][r0:r0 + rr, c0:c0 + cc])
    B.shampoo_update_stats(h, blocks)
    torch.cuda.synchronize()
    for i in (0, 5, 11, 12, 17, 23):   # sampled blocks, incl. column and row sub-blocks
        Lo, Ro = O.stats_update(np.zeros((1024, 1024)), np.zeros((1024, 1024)), refs[i])
        assert rel(host(Ls[i]), Lo) <= TOL and rel(host(Rs[i]), Ro) <= TOL
    # trace identity on every block: tr L = tr R = ||G||_F^2
    for i in range(len(blocks)):
        tl, tr = float(torch.trace(Ls[i].double())), float(torch.trace(Rs[i].double()))
        g2 = float(np.sum(refs[i].astype(np.float64) ** 2))
        assert abs(tl - g2) <= 1e-5 * g2 and abs(tr - g2) <= 1e-5 * g2


@pytest.mark.parametrize("m,n,count", [(300, 2100, 20), (1024, 4096, 12), (256, 1024, 600)])
def test_uniform_grouped_equals_single(env, m, n, count):
    """Uniform grouped calls against one call per block, bit for bit (the
    tiles' arithmetic does not depend on the launch).  The grouped launches
    order their tiles differently: 300 x 2100 and 1024 x 4096 (contractions
    of 2048 or more, or few diagonal tiles) run each XCD's diagonal tiles
    last, 600 blocks of 256 x 1024 (L: 1200 diagonal tiles of a 1024-deep
    contraction) keep the row-major order."""
    torch, B, dev, h = env
    say("stats uniform grouped == single", m, n, count)
    g = torch.Generator(device=dev).manual_seed(41 + m)
    Gs = [torch.randn(m, n, device=dev, generator=g) for _ in range(min(count, 24))]
    Gs = [Gs[i % len(Gs)] for i in range(count)]
    blocks = [B.Block(G=G, L=torch.zeros(m, m, device=dev), R=torch.zeros(n, n, device=dev)) for G in Gs]
    B.shampoo_update_stats(h, blocks, beta2=1.0)
    for i in sorted({0, 1, count // 2, count - 1} | set(range(0, count, max(1, count // 5)))):
        one = B.Block(G=Gs[i], L=torch.zeros(m, m, device=dev), R=torch.zeros(n, n, device=dev))
        B.shampoo_update_stats(h, [one], beta2=1.0)
        torch.cuda.synchronize()
        assert torch.equal(one.L, blocks[i].L) and torch.equal(one.R, blocks[i].R), i
    Lo, Ro = O.stats_update(np.zeros((m, m)), np.zeros((n, n)), host(Gs[count - 1]).astype(np.float64))
    assert rel(host(blocks[count - 1].L), Lo) <= TOL and rel(host(blocks[count - 1].R), Ro) <= TOL


def test_empty_call_and_errors(env):
    torch, B, dev, h = env
    say("stats errors")
    B.shampoo_update_stats(h, [])
    g = torch.zeros(4, 4, device=dev)
    with pytest.raises(B.ShampooError):
        B.shampoo_update_stats(h, [B.Block(G=g, L=torch.zeros(4, 4, device=dev))], beta2=1.5)
    big = torch.zeros(1, 4097, device=dev)
    with pytest.raises(B.ShampooError):
        B.shampoo_update_stats(h, [B.Block(G=big, R=None, L=torch.zeros(1, 1, device=dev))])
