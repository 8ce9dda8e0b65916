"""shampoo_graft_noalloc (no device allocation; fixed scratch) against
shampoo_graft on the same inputs, through the C ABI: two calls in a row, the
second with fewer and smaller blocks, fp32 and bf16 gradients, with and
without momentum, and the AdaGrad fallback.  Both run the same kernels on
the same block table, so the states, W and the norms must agree bit for bit
(and so within every tolerance of the oracle comparisons).  Sizes beyond the
fixed scratch are rejected with ENOMEM before anything is enqueued."""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu


def _case(torch, dev, shapes, seed, bf16, momentum, pad=5):
    """Per block: G, W, D, P (and Mg, Ps) as views with a padded row stride."""
    gen = torch.Generator(device=dev).manual_seed(seed)
    out = []
    for m, n in shapes:
        def view(x):
            big = torch.zeros(m, n + pad, device=dev, dtype=x.dtype)
            big[:, :n] = x
            return big[:, :n]
        g = torch.randn(m, n, device=dev, generator=gen)
        g[torch.rand(m, n, device=dev, generator=gen) < 0.05] = 0.0
        t = dict(G=view(g.to(torch.bfloat16) if bf16 else g),
                 W=view(torch.randn(m, n, device=dev, generator=gen)),
                 D=view(torch.rand(m, n, device=dev, generator=gen)),
                 P=view(torch.randn(m, n, device=dev, generator=gen)))
        if momentum:
            t["Mg"] = view(torch.randn(m, n, device=dev, generator=gen))
            t["Ps"] = view(torch.randn(m, n, device=dev, generator=gen))
        out.append(t)
    return out


def _run(torch, B, h, entry, case, eta0, beta1, use_shampoo):
    """Runs one entry point on a private copy of the case's states."""
    def copy(v):  # same shape and row stride as the view
        c = torch.empty_strided(v.shape, v.stride(), dtype=v.dtype, device=v.device)
        return c.copy_(v)
    blocks, keep = [], []
    for t in case:
        c = {k: (v if k in ("G", "P") else copy(v)) for k, v in t.items()}
        keep.append(c)
        blocks.append(B.Block(**c))
    norms = torch.full((3 * len(case),), float("nan"), device=case[0]["W"].device)
    entry(h, blocks, eta0, beta1=beta1, use_shampoo=use_shampoo, norms=norms)
    torch.cuda.synchronize()
    return keep, norms


@pytest.fixture(scope="module")
def env():
    torch, B, dev = gpu_env()
    h = B.shampoo_create(0)
    yield torch, B, dev, h
    B.shampoo_destroy(h)


CALLS = [
    # (shapes, bf16, beta1, use_shampoo): the second call of each pair is smaller
    ([(300, 500), (1024, 4096), (7, 3), (128, 128), (1, 1000)], False, 0.0, True),
    ([(64, 96), (5, 5)], False, 0.0, True),
    ([(513, 257), (96, 1024), (33, 1)], True, 0.9, True),
    ([(17, 200)], True, 0.9, True),
    ([(256, 4096), (40, 40)], False, 0.0, False),
    ([(3, 4)], False, 0.0, False),
]


def test_noalloc_matches_graft_two_calls(env):
    torch, B, dev, h = env
    for i in range(0, len(CALLS), 2):
        for j, (shapes, bf16, beta1, use) in enumerate(CALLS[i:i + 2]):
            say("graft noalloc call", j + 1, "of 2:", len(shapes), "blocks, bf16", bf16, "beta1", beta1,
                "use_shampoo", use)
            case = _case(torch, dev, shapes, 100 + i + j, bf16, beta1 > 0)
            ref, n_ref = _run(torch, B, h, B.shampoo_graft, case, 0.05, beta1, use)
            got, n_got = _run(torch, B, h, B.shampoo_graft_noalloc, case, 0.05, beta1, use)
            assert torch.equal(n_got, n_ref), (host(n_got), host(n_ref))
            for r, g in zip(ref, got):
                for k in r:
                    assert torch.equal(g[k], r[k]), (k, shapes)
            # and the first block against the oracle's step (Algorithm 2 graft)
            t, g0 = case[0], got[0]
            st = {k: host(v).astype(np.float64) for k, v in t.items() if k != "G"}
            gg = host(t["G"].float()).astype(np.float64)
            o = O.graft_update(st["W"], st["D"], gg, st["P"] if use else None, 0.05, beta1, st.get("Mg"),
                               st.get("Ps"), use)
            assert rel(host(g0["W"]) - st["W"], o["W"] - st["W"]) <= 2e-3
            assert rel(host(g0["D"]), o["D"]) <= 1e-6


def test_noalloc_limits(env):
    torch, B, dev, h = env
    say("graft noalloc limits")
    # the table holds 8192 blocks: 8192 one-row blocks (distinct rows of one
    # tensor) run and match shampoo_graft; 8193 are rejected
    gen = torch.Generator(device=dev).manual_seed(7)
    x = torch.randn(8193, 4, device=dev, generator=gen)
    p = torch.randn(8193, 4, device=dev, generator=gen)
    outs = []
    for entry in (B.shampoo_graft, B.shampoo_graft_noalloc):
        w, d = torch.ones(8193, 4, device=dev), torch.ones(8193, 4, device=dev)
        blocks = [B.Block(G=x[i:i + 1, :3], W=w[i:i + 1, :3], D=d[i:i + 1, :3], P=p[i:i + 1, :3])
                  for i in range(8192)]
        entry(h, blocks, 0.1)
        torch.cuda.synchronize()
        outs.append((w, d))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    assert bool(torch.all(outs[1][0][8192] == 1))
    blocks.append(B.Block(G=x[8192:, :3], W=w[8192:, :3], D=d[8192:, :3], P=p[8192:, :3]))
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_graft_noalloc(h, blocks, 0.1)
    assert e.value.code == B.SHAMPOO_ENOMEM
    # more chunks than the partials hold: 193 views of one 4096 x 4096 block
    # (1024 chunks each); rejected before any launch, so W is untouched
    big = torch.ones(4096, 4096, device=dev)
    W = torch.ones(4096, 4096, device=dev)
    D = torch.ones(4096, 4096, device=dev)
    blocks = [B.Block(G=big, W=W, D=D, P=big) for _ in range(193)]
    with pytest.raises(B.ShampooError) as e:
        B.shampoo_graft_noalloc(h, blocks, 0.1)
    assert e.value.code == B.SHAMPOO_ENOMEM and "chunks" in B._lib.shampoo_last_error(h).decode()
    torch.cuda.synchronize()
    assert bool(torch.all(W == 1)) and bool(torch.all(D == 1))
