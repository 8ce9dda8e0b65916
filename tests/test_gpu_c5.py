"""C5 at full size: a 32768 x 1024 embedding (32 row blocks of 1024 x 1024)
and 200 square blocks with sides drawn from {128, ..., 2048}, bf16-stored
gradients, 10 statistics steps, then one grouped inverse-root call over all
464 factors (per-matrix early exit), preconditioning and the graft.

Dense variant: every factor's root against eigh of the same fp32 statistics
(1e-3 band); every block's statistics through the trace identity
tr L = tr R = sum_t ||G_t||_F^2 (Preliminaries), and fully against the
oracle's fp64 statistics rebuilt from the seeded gradients on sampled blocks
of every size class; every block's preconditioned gradient with the GPU's
roots (2e-3), and end to end with the oracle's roots on the sampled blocks.

Row-sparse variant (the embedding's gradient nonzero only on the rows read
by 4096 Zipf(1.1) lookups per step, embedding appendix): the 64 embedding
factors are rank-deficient, so the call takes Algorithm 1's scaled damping
eps * lambda_max (MaxSV) and the embedding factors escalate to the fp64
tail while the 400 others stop in fp32.  Every root against eigh (fed the
GPU's lambda_max), every lambda_max against the oracle's MaxSV.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say
from tests.parity_util import pool_map, root_parity, summarize

pytestmark = pytest.mark.gpu
STEPS = 10


def shapes():
    emb = [(1024, 1024)] * (cfg.C5_EMB_ROWS // cfg.C5_D)
    return emb + [(k, k) for k in cfg.c5_mixed_sizes()]


def _grouped_roots(torch, B, dev, h, As, eps_relative):
    Xs = [torch.zeros_like(a) for a in As]
    prm = B.shampoo_root_params_default(p=4, eps=1e-6, eps_relative=eps_relative)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([a.shape[0] for a in As], prm.precision),
                     dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
    torch.cuda.synchronize()
    return Xs, B.decode_root_info(info)


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
    sqsum = np.zeros(nb)                   # sum_t ||G_t||_F^2 per block, exact inputs in fp64
    h = B.shampoo_create(0)
    try:
        with ThreadPoolExecutor(16) as ex:
            for t in range(1, STEPS + 1):
                bits = list(ex.map(lambda b: cfg.c5_grad_bf16(b, t, shp[b]), range(nb)))
                for b in range(nb):
                    Gv[b].copy_(torch.from_numpy(bits[b].view(np.int16)).view(torch.bfloat16))
                B.shampoo_update_stats(h, [B.Block(G=Gv[b], L=Ls[b], R=Rs[b]) for b in range(nb)])
                sqsum += np.array(list(ex.map(lambda x: float(np.sum(O.bf16_bits_to_f64(x) ** 2)), bits)))
                torch.cuda.synchronize()
        last_bits = bits
        say("C5 grouped roots: 464 factors")
        As = Ls + Rs
        Xs, infos = _grouped_roots(torch, B, dev, h, As, 0)
        Ps = [torch.zeros(m, n, device=dev) for m, n in shp]
        blocks = [B.Block(G=Gv[b], P=Ps[b], Lr=Xs[b], Rr=Xs[nb + b]) for b in range(nb)]
        B.shampoo_precondition(h, blocks)
        torch.cuda.synchronize()
    finally:
        B.shampoo_destroy(h)
    assert all(i["status"] in (0, 1) for i in infos), [i for i in infos if i["status"] > 1][:3]
    its = sorted(set(i["iters"] for i in infos))
    say("C5 iteration counts present:", its)
    hA, hX = [host(a) for a in As], [host(x) for x in Xs]
    say("C5: oracle roots of 464 factors")
    res = pool_map(lambda j: root_parity(hA[j], hX[j], 4, 1e-6), range(len(As)))
    _, worst, frac = summarize("C5 roots (all 464)", [r[0] for r in res], [r[2] for r in res])
    assert frac == 1.0, worst
    # statistics of every block: the trace identity
    trL = np.array([float(np.trace(hA[b].astype(np.float64))) for b in range(nb)])
    trR = np.array([float(np.trace(hA[nb + b].astype(np.float64))) for b in range(nb)])
    e_tr = np.maximum(np.abs(trL - sqsum), np.abs(trR - sqsum)) / sqsum
    summarize("C5 stats trace identity (all 232 blocks)", e_tr, [1e-5] * nb)
    assert e_tr.max() <= 1e-5
    # preconditioned gradient of every block with the GPU's roots
    hP = [host(p) for p in Ps]

    def prec(b):
        g = O.bf16_bits_to_f64(last_bits[b])
        return rel(hP[b], O.precondition(g, hX[b].astype(np.float64), hX[nb + b].astype(np.float64)))
    e_p = pool_map(prec, range(nb))
    _, worst, frac = summarize("C5 preconditioned gradient, GPU roots (all 232)", e_p, [2e-3] * nb)
    assert frac == 1.0, worst
    # sampled blocks of every size class: statistics rebuilt in fp64 from the
    # seeded gradients, and the preconditioned gradient end to end
    picks = [0]
    for k in cfg.C5_SIZES:
        picks.append(32 + [s[0] for s in shp[32:]].index(k))
    for b in picks:
        m, n = shp[b]
        Gs = [O.bf16_bits_to_f64(cfg.c5_grad_bf16(b, t, (m, n))) for t in range(1, STEPS + 1)]
        Lo, Ro = np.zeros((m, m)), np.zeros((n, n))
        for g in Gs:
            Lo, Ro = O.stats_update(Lo, Ro, g)
        assert rel(hA[b], Lo) <= 1e-4 and rel(hA[nb + b], Ro) <= 1e-4, (b, m)
        Lr, _, _ = O.inv_root(Lo, 4, 1e-6)
        Rr, _, _ = O.inv_root(Ro, 4, 1e-6)
        assert rel(hP[b], O.precondition(Gs[-1], Lr, Rr)) <= 2e-3, (b, m)


def test_c5_row_sparse_grouped_all():
    torch, B, dev = gpu_env()
    shp = shapes()
    nb, nemb = len(shp), cfg.C5_EMB_ROWS // cfg.C5_D
    lookups = 4096
    say("C5 row-sparse: 232 blocks, 10 stats steps, embedding from 4096 Zipf lookups per step")
    gen = torch.Generator(device=dev).manual_seed(5)
    emb = torch.zeros(cfg.C5_EMB_ROWS, cfg.C5_D, dtype=torch.bfloat16, device=dev)
    emb32 = torch.zeros(emb.shape, device=dev)
    mixed = [torch.empty(s, dtype=torch.bfloat16, device=dev) for s in shp[nemb:]]
    Gv = [emb[i * cfg.C5_D:(i + 1) * cfg.C5_D] for i in range(nemb)] + mixed
    Ls = [torch.zeros(m, m, device=dev) for m, _ in shp]
    Rs = [torch.zeros(n, n, device=dev) for _, n in shp]
    h = B.shampoo_create(0)
    try:
        for t in range(STEPS):
            for x in mixed:
                x.copy_((torch.randn(x.shape, device=dev, generator=gen) * 1e-3 ** 0.5).to(torch.bfloat16))
            idx = torch.from_numpy(cfg.zipf_rows(lookups, emb.shape[0], 1.1, cfg.C5, 3, t)).to(dev)
            dy = torch.randn(lookups, emb.shape[1], device=dev, generator=gen) * 1e-3 ** 0.5
            emb32.zero_()
            emb32.index_add_(0, idx.long(), dy)
            emb.copy_(emb32.to(torch.bfloat16))
            B.shampoo_update_stats(h, [B.Block(G=Gv[b], L=Ls[b], R=Rs[b]) for b in range(nb)])
        torch.cuda.synchronize()
        say("C5 row-sparse grouped roots: 464 factors, scaled damping")
        As = Ls + Rs
        Xs, infos = _grouped_roots(torch, B, dev, h, As, 1)
    finally:
        B.shampoo_destroy(h)
    assert all(i["status"] in (0, 1) for i in infos), [i for i in infos if i["status"] > 1][:3]
    emb_f = [j for j in range(len(As)) if j < nemb or nb <= j < nb + nemb]
    n64 = [j for j, i in enumerate(infos) if i["precision"] == 64]
    say(f"C5 row-sparse: {len(n64)} factors took the fp64 tail ({len(set(n64) & set(emb_f))} of them embedding "
        f"factors); fp32 iterations {sorted(set(i['iters_fp32'] for i in infos))}")
    hA, hX = [host(a) for a in As], [host(x) for x in Xs]
    say("C5 row-sparse: oracle MaxSV and roots of 464 factors")
    lam_ps = pool_map(lambda j: O.max_sv(hA[j])[0], range(len(As)))
    gap = max(abs(i["lambda_max"] - l) / l for i, l in zip(infos, lam_ps))
    say(f"C5 row-sparse lambda_max: max |GPU - MaxSV| / MaxSV {gap:.2e}")
    assert gap <= 1e-5
    res = pool_map(lambda j: root_parity(hA[j], hX[j], 4, 1e-6, True, infos[j]["lambda_max"]), range(len(As)))
    kap = [res[j][1] for j in emb_f]
    say(f"C5 row-sparse embedding factors: damped condition {min(kap):.3g}..{max(kap):.3g}")
    summarize("C5 row-sparse roots (64 embedding factors)", [res[j][0] for j in emb_f], [res[j][2] for j in emb_f])
    _, worst, frac = summarize("C5 row-sparse roots (all 464)", [r[0] for r in res], [r[2] for r in res])
    assert frac == 1.0, worst
