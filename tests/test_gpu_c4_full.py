"""C4 at full size, in the launch configuration the benchmark times: 24
BERT-Large-shaped layers (288 blocks of 1024 x 1024, strided views of the Q,
K, V, O, FFN-in and FFN-out tensors), one grouped root refresh of all 576
factors (statistics of 100 earlier gradients), then one step: statistics,
two-sided preconditioning and the AdaGrad graft over all 288 blocks.

Sampled blocks from every tensor kind are checked against the fp64 oracle,
which takes the same inputs (the earlier statistics, G, W) and recomputes
each step itself.  Bars: statistics 1e-4, roots 1e-3 (damped condition
number ~1.5), preconditioned gradient 2e-3 both with the GPU's roots
(kernel parity) and with the oracle's roots (end to end), step dW 2e-3.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu

SAMPLES = (0, 4, 7, 11, 130, 209, 287)   # Q of layer 0, FFN-in, FFN-out, ... last block


def test_c4_full_step_sampled():
    torch, B, dev = gpu_env()
    d, nl, eps, eta0 = cfg.C4_D, cfg.C4_LAYERS, 1e-6, 6e-3
    shapes = dict(cfg.c4_layer_tensors())
    names = [nm for nm, _ in cfg.c4_layer_tensors()]
    say("C4 full: generating 24 layers of gradients")
    keys = [(l, t) for l in range(nl) for t in range(len(names))]
    with ThreadPoolExecutor(16) as ex:
        grads = list(ex.map(lambda lt: cfg.c4_grad(lt[0], lt[1], 1, shapes[names[lt[1]]]), keys))
    G = {k: g for k, g in zip(keys, grads)}
    Gt = {k: torch.from_numpy(g).to(dev) for k, g in G.items()}
    W0 = {k: (0.02 * torch.randn(shapes[names[k[1]]], device=dev,
                                 generator=torch.Generator(device=dev).manual_seed(k[0] * 8 + k[1])))
          for k in keys}
    Wt = {k: w.clone() for k, w in W0.items()}
    Dt = {k: torch.zeros_like(w) for k, w in W0.items()}
    Pt = {k: torch.zeros_like(w) for k, w in W0.items()}
    blocks, Ls, Rs, Lrs, Rrs, where = [], [], [], [], [], []
    for l in range(nl):
        for (t, r0, c0, rr, cc) in cfg.c4_blocks(d):
            sl = (slice(r0, r0 + rr), slice(c0, c0 + cc))
            b = len(blocks)
            L = cfg.wishart_bartlett_device(d, 100 * d, 1e-3, torch, dev, cfg.C4, 7, b, 0)
            R = cfg.wishart_bartlett_device(d, 100 * d, 1e-3, torch, dev, cfg.C4, 7, b, 1)
            Lr, Rr = torch.zeros(d, d, device=dev), torch.zeros(d, d, device=dev)
            Ls.append(L); Rs.append(R); Lrs.append(Lr); Rrs.append(Rr)
            blocks.append(B.Block(G=Gt[l, t][sl], W=Wt[l, t][sl], D=Dt[l, t][sl], P=Pt[l, t][sl],
                                  L=L, R=R, Lr=Lr, Rr=Rr))
            where.append(((l, t), sl))
    assert len(blocks) == 288
    inputs = {b: (host(Ls[b]).astype(np.float64), host(Rs[b]).astype(np.float64)) for b in SAMPLES}
    h = B.shampoo_create(0)
    try:
        say("C4 full: 576 roots in one grouped call")
        prm = B.shampoo_root_params_default(p=4, eps=eps)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([d] * 576, prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(8 * 576, dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, Ls + Rs, Lrs + Rrs, prm, ws, info)
        say("C4 full: stats + precondition + graft over 288 blocks")
        B.shampoo_update_stats(h, blocks)
        B.shampoo_precondition(h, blocks)
        B.shampoo_graft(h, blocks, eta0)
        torch.cuda.synchronize()
        infos = B.decode_root_info(info)
        assert all(i["status"] in (0, 1) for i in infos)
        for b in SAMPLES:
            (k, sl) = where[b]
            L0, R0 = inputs[b]
            g = G[k][sl].astype(np.float64)
            Lo, Ro = O.stats_update(L0, R0, g)
            assert rel(host(Ls[b]), Lo) <= 1e-4, b
            assert rel(host(Rs[b]), Ro) <= 1e-4, b
            Lr_o, _, _ = O.inv_root(L0, 4, eps)
            Rr_o, _, _ = O.inv_root(R0, 4, eps)
            Lr_g, Rr_g = host(Lrs[b]).astype(np.float64), host(Rrs[b]).astype(np.float64)
            assert rel(Lr_g, Lr_o) <= 1e-3, (b, infos[b])
            assert rel(Rr_g, Rr_o) <= 1e-3, (b, infos[288 + b])
            P_g = host(Pt[k][sl]).astype(np.float64)
            assert rel(P_g, O.precondition(g, Lr_g, Rr_g)) <= 2e-3, b
            assert rel(P_g, O.precondition(g, Lr_o, Rr_o)) <= 2e-3, b
            w0 = host(W0[k][sl]).astype(np.float64)
            out = O.graft_update(w0, np.zeros((d, d)), g, O.precondition(g, Lr_g, Rr_g), eta0)
            dw_g = host(Wt[k][sl]).astype(np.float64) - w0
            assert rel(dw_g, out["W"] - w0) <= 2e-3, b
    finally:
        B.shampoo_destroy(h)
