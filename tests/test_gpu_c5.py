"""C5 at full size: a 32768 x 1024 embedding (32 row blocks of 1024 x 1024)
and 200 square blocks with sides drawn from {128, ..., 2048}, bf16-stored
gradients, 10 statistics steps, then one grouped inverse-root call over all
464 factors (per-matrix early exit), preconditioning and the graft.

Parity on sampled blocks of every size class against the fp64 oracle, which
rebuilds those blocks' statistics from the same seeded gradients.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu
STEPS = 10


def shapes():
    emb = [(1024, 1024)] * (cfg.C5_EMB_ROWS // cfg.C5_D)
    return emb + [(k, k) for k in cfg.c5_mixed_sizes()]


def test_c5_full_grouped():
    torch, B, dev = gpu_env()
    shp = shapes()
    nb = len(shp)
    assert nb == 232
    say("C5 full: 232 blocks, 10 bf16 stats steps")
    # the embedding is one 32768 x 1024 tensor; its blocks are row slices
    emb = torch.empty(cfg.C5_EMB_ROWS, cfg.C5_D, dtype=torch.bfloat16, device=dev)
    mixed = [torch.empty(s, dtype=torch.bfloat16, device=dev) for s in shp[32:]]
    Gv = [emb[i * 1024:(i + 1) * 1024] for i in range(32)] + mixed
    Ls = [torch.zeros(m, m, device=dev) for m, _ in shp]
    Rs = [torch.zeros(n, n, device=dev) for _, n in shp]
    h = B.shampoo_create(0)
    try:
        with ThreadPoolExecutor(16) as ex:
            for t in range(1, STEPS + 1):
                bits = list(ex.map(lambda b: cfg.c5_grad_bf16(b, t, shp[b]), range(nb)))
                for b in range(nb):
                    Gv[b].copy_(torch.from_numpy(bits[b].view(np.int16)).view(torch.bfloat16))
                B.shampoo_update_stats(h, [B.Block(G=Gv[b], L=Ls[b], R=Rs[b]) for b in range(nb)])
                torch.cuda.synchronize()
        say("C5 grouped roots: 464 factors")
        As = Ls + Rs
        Xs = [torch.zeros_like(a) for a in As]
        prm = B.shampoo_root_params_default(p=4, eps=1e-6)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([a.shape[0] for a in As], prm.precision),
                         dtype=torch.uint8, device=dev)
        info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
        Ps = [torch.zeros(m, n, device=dev) for m, n in shp]
        blocks = [B.Block(G=Gv[b], P=Ps[b], Lr=Xs[b], Rr=Xs[nb + b]) for b in range(nb)]
        B.shampoo_precondition(h, blocks)
        torch.cuda.synchronize()
        infos = B.decode_root_info(info)
        assert all(i["status"] in (0, 1) for i in infos), [i for i in infos if i["status"] > 1][:3]
        # sampled parity: one embedding block and one block of each size class
        picks = [0]
        for k in cfg.C5_SIZES:
            picks.append(32 + [s[0] for s in shp[32:]].index(k))
        for b in picks:
            m, n = shp[b]
            Gs = [O.bf16_bits_to_f64(cfg.c5_grad_bf16(b, t, (m, n))) for t in range(1, STEPS + 1)]
            Lo, Ro = np.zeros((m, m)), np.zeros((n, n))
            for g in Gs:
                Lo, Ro = O.stats_update(Lo, Ro, g)
            assert rel(host(Ls[b]), Lo) <= 1e-4
            Lr, _, _ = O.inv_root(Lo, 4, 1e-6)
            Rr, _, _ = O.inv_root(Ro, 4, 1e-6)
            assert rel(host(Xs[b]), Lr) <= 1e-3, (b, m, infos[b])
            assert rel(host(Xs[nb + b]), Rr) <= 1e-3, (b, n, infos[nb + b])
            assert rel(host(Ps[b]), O.precondition(Gs[-1], Lr, Rr)) <= 2e-3
        # early exit: iteration counts differ per matrix and every matrix stopped on its own
        its = sorted(set(i["iters"] for i in infos))
        print("C5 iteration counts present:", its)
    finally:
        B.shampoo_destroy(h)
