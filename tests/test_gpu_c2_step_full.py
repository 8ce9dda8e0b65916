"""The C2 step in the benchmark's launch configuration: 96 blocks, each with
statistics L of 19 earlier gradients (Wishart, 19 x 4096 degrees of
freedom) and a gradient G (1024 x 4096, N(0, 1/4096)); one grouped
statistics update, 96 inverse 4th roots in one call, then P = L^(-1/4) G and
the AdaGrad graft in one shampoo_precondition_graft call (as the benchmark
times it: the blocks go in groups whose graft pass 2 overlaps the next
group's GEMMs).

Every block against the oracle, which takes the same inputs (L, G, D, W) and
recomputes the step: L <= 1e-4; root <= 1e-3 and the iteration count within
one of the fp64 transcript with the same start; P <= 2e-3 with the GPU's
root (kernel parity) and with the oracle's (end to end); dW <= 2e-3.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from tests.gpu_util import gpu_env, host, rel, say
from tests.parity_util import pool_map, summarize

pytestmark = pytest.mark.gpu

NB, N, K = 96, 1024, 4096


def _oracle_block(inp):
    """The oracle's step for one block from the GPU's inputs, compared with
    the GPU's outputs; returns the relative errors and iteration counts."""
    L0, g, d0, w0, L_g, Lr_g, P_g, W_g, D_g, gpu_iters = inp
    L0, g, d0, w0 = (x.astype(np.float64) for x in (L0, g, d0, w0))
    Lr_g, P_g = Lr_g.astype(np.float64), P_g.astype(np.float64)
    Lo, _ = O.stats_update(L0, None, g)
    Lr_o, _, _ = O.inv_root(Lo, 4, 1e-6)
    tr = O.coupled_newton(L_g, 4, 1e-6, tol=1e-6, scaling="power4")
    P_k = O.precondition(g, Lr_g, None)
    out = O.graft_update(w0, d0, g, P_k, 1e-2)
    return dict(L=rel(L_g, Lo), root=rel(Lr_g, Lr_o), P_kernel=rel(P_g, P_k),
                P_e2e=rel(P_g, O.precondition(g, Lr_o, None)),
                dW=rel(W_g.astype(np.float64) - w0, out["W"] - w0), D=rel(D_g, out["D"]),
                iters=(gpu_iters, tr["iters"]))


def test_c2_step_full_all_blocks():
    torch, B, dev = gpu_env()
    from synth import configs as cfg
    say("C2 full step: 96 blocks")
    gen = torch.Generator(device=dev).manual_seed(2)
    Ls = [cfg.wishart_bartlett_device(N, 19 * K, 1.0 / K, torch, dev, cfg.C2, b, 9) for b in range(NB)]
    Gs = [torch.randn(N, K, device=dev, generator=gen) / K ** 0.5 for _ in range(NB)]
    Ds = [(19.0 / K) * (0.5 + torch.rand(N, K, device=dev, generator=gen)) for _ in range(NB)]
    Ws = [0.02 * torch.randn(N, K, device=dev, generator=gen) for _ in range(NB)]
    Ps = [torch.zeros(N, K, device=dev) for _ in range(NB)]
    Lrs = [torch.zeros(N, N, device=dev) for _ in range(NB)]
    inputs = [(host(Ls[b]), host(Gs[b]), host(Ds[b]), host(Ws[b])) for b in range(NB)]
    blocks = [B.Block(G=Gs[b], W=Ws[b], D=Ds[b], P=Ps[b], L=Ls[b], Lr=Lrs[b]) for b in range(NB)]
    h = B.shampoo_create(0)
    try:
        prm = B.shampoo_root_params_default(p=4, eps=1e-6)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([N] * NB, prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(8 * NB, dtype=torch.int32, device=dev)
        B.shampoo_update_stats(h, blocks)
        B.shampoo_inv_root_batched(h, Ls, Lrs, prm, ws, info)
        B.shampoo_precondition_graft(h, blocks, 1e-2)
        torch.cuda.synchronize()
    finally:
        B.shampoo_destroy(h)
    infos = B.decode_root_info(info)
    assert all(i["status"] in (0, 1) and i["precision"] == 32 for i in infos), infos[:3]
    say("C2 full step: oracle over 96 blocks")
    res = pool_map(lambda b: _oracle_block(inputs[b] + (host(Ls[b]), host(Lrs[b]), host(Ps[b]), host(Ws[b]),
                                                        host(Ds[b]), infos[b]["iters"])), range(NB))
    for key, bar in (("L", 1e-4), ("root", 1e-3), ("P_kernel", 2e-3), ("P_e2e", 2e-3), ("dW", 2e-3),
                     ("D", 1e-6)):
        _, worst, frac = summarize(f"C2 step {key} (all 96)", [r[key] for r in res], [bar] * NB)
        assert frac == 1.0, (key, worst)
    off = [abs(a - b) for a, b in (r["iters"] for r in res)]
    assert max(off) <= 1, [r["iters"] for r in res]
