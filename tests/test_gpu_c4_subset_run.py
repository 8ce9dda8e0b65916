"""C4's two-layer subset over 103 steps: 24 blocks of 1024 x 1024 (the Q, K,
V, O, FFN-in and FFN-out views of two BERT-Large-shaped layers), two-sided,
G ~ N(0, 1e-3) per step, beta2 = 1, beta1 = 0, eta0 = 6e-3.  Steps 1..99 take
the AdaGrad graft (no roots yet); at step 100 the 48 factors get their
inverse 4th roots in one grouped call, and steps 100..103 take the Shampoo
direction (Algorithm 2 with the graft of the appendix "Layer wise learning
rates").

Two sampled blocks (Q of layer 0, and a column block of layer 1's FFN-in
tensor, a strided view) follow the oracle's fp64 trajectory on the same
gradients: statistics <= 1e-4 after 103 steps, roots <= 1e-3, D <= 1e-5,
the whole-run dW and the dW of the Shampoo steps <= 2e-3.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu

LAYERS, STEPS, ROOTS_AT, ETA0, EPS, P = 2, 103, 100, 6e-3, 1e-6, 4
SAMPLES = (0, 12 + 6)


def test_c4_two_layer_subset_103_steps():
    torch, B, dev = gpu_env()
    say("C4 subset: 24 blocks, 103 steps")
    d = cfg.C4_D
    tensors = cfg.c4_layer_tensors()
    gen = torch.Generator(device=dev).manual_seed(104)
    Gt, Wt, Dt, Pt = {}, {}, {}, {}
    for l in range(LAYERS):
        for t, (_, sh) in enumerate(tensors):
            Gt[l, t] = torch.zeros(sh, device=dev)
            Wt[l, t] = 0.02 * torch.randn(sh, device=dev, generator=gen)
            Dt[l, t] = torch.zeros(sh, device=dev)
            Pt[l, t] = torch.zeros(sh, device=dev)
    blocks, views = [], []
    for l in range(LAYERS):
        for (t, r0, c0, rr, cc) in cfg.c4_blocks(d):
            sl = (slice(r0, r0 + rr), slice(c0, c0 + cc))
            views.append((l, t, sl))
            blocks.append(B.Block(G=Gt[l, t][sl], W=Wt[l, t][sl], D=Dt[l, t][sl], P=Pt[l, t][sl],
                                  L=torch.zeros(rr, rr, device=dev), R=torch.zeros(cc, cc, device=dev),
                                  Lr=torch.zeros(rr, rr, device=dev), Rr=torch.zeros(cc, cc, device=dev)))
    assert len(blocks) == 24
    As = [b.L for b in blocks] + [b.R for b in blocks]
    Xs = [b.Lr for b in blocks] + [b.Rr for b in blocks]
    wview = lambda i: host(blocks[i].W).astype(np.float64)
    ost = {i: dict(W=wview(i), D=np.zeros((d, d)), L=np.zeros((d, d)), R=np.zeros((d, d))) for i in SAMPLES}
    W0 = {i: ost[i]["W"].copy() for i in SAMPLES}
    W99g, W99o = {}, {}
    h = B.shampoo_create(0)
    try:
        prm = B.shampoo_root_params_default(p=P, eps=EPS)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([d] * len(As), prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
        for step in range(1, STEPS + 1):
            for G in Gt.values():
                G.copy_(torch.randn(G.shape, device=dev, generator=gen) * 1e-3 ** 0.5)
            shampoo = step >= ROOTS_AT
            B.shampoo_update_stats(h, blocks)
            if step == ROOTS_AT:
                B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
            if shampoo:
                B.shampoo_precondition(h, blocks)
            B.shampoo_graft(h, blocks, ETA0, use_shampoo=shampoo)
            torch.cuda.synchronize()
            for i in SAMPLES:
                g = host(blocks[i].G).astype(np.float64)
                s = ost[i]
                s["L"], s["R"] = O.stats_update(s["L"], s["R"], g)
                if step == ROOTS_AT:
                    s["Lr"] = O.inv_root(s["L"], P, EPS)[0]
                    s["Rr"] = O.inv_root(s["R"], P, EPS)[0]
                Pd = O.precondition(g, s["Lr"], s["Rr"]) if shampoo else None
                out = O.graft_update(s["W"], s["D"], g, Pd, ETA0, use_shampoo=shampoo)
                s["W"], s["D"] = out["W"], out["D"]
                if step == ROOTS_AT - 1:
                    W99g[i], W99o[i] = wview(i), s["W"].copy()
        infos = B.decode_root_info(info)
    finally:
        B.shampoo_destroy(h)
    assert all(x["status"] in (0, 1) and x["precision"] == 32 for x in infos)
    for i in SAMPLES:
        s, b = ost[i], blocks[i]
        assert rel(host(b.L), s["L"]) <= 1e-4, i
        assert rel(host(b.R), s["R"]) <= 1e-4, i
        assert rel(host(b.Lr), s["Lr"]) <= 1e-3, i
        assert rel(host(b.Rr), s["Rr"]) <= 1e-3, i
        assert rel(host(b.D), s["D"]) <= 1e-5, i
        Wg = wview(i)
        assert rel(Wg - W0[i], s["W"] - W0[i]) <= 2e-3, i
        assert rel(Wg - W99g[i], s["W"] - W99o[i]) <= 2e-3, i
