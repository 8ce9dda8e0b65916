"""The C2 step in the benchmark's launch configuration: 96 blocks, each with
statistics L of 19 earlier gradients (Wishart, 19 x 4096 degrees of
freedom) and a gradient G (1024 x 4096, N(0, 1/4096)); one grouped
statistics update, 96 inverse 4th roots in one call, P = L^(-1/4) G and the
AdaGrad graft.

Sampled blocks against the oracle, which takes the same inputs (L, G, D, W)
and recomputes the step: L <= 1e-4; root <= 1e-3 and the iteration count
within one of the fp64 transcript with the same start; P <= 2e-3 with the
GPU's root (kernel parity) and with the oracle's (end to end); dW <= 2e-3.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu

NB, N, K = 96, 1024, 4096
SAMPLES = (0, 47, 95)


def test_c2_step_full_sampled():
    torch, B, dev = gpu_env()
    say("C2 full step: 96 blocks")
    gen = torch.Generator(device=dev).manual_seed(2)
    Ls = [cfg.wishart_bartlett_device(N, 19 * K, 1.0 / K, torch, dev, cfg.C2, b, 9) for b in range(NB)]
    Gs = [torch.randn(N, K, device=dev, generator=gen) / K ** 0.5 for _ in range(NB)]
    Ds = [(19.0 / K) * (0.5 + torch.rand(N, K, device=dev, generator=gen)) for _ in range(NB)]
    Ws = [0.02 * torch.randn(N, K, device=dev, generator=gen) for _ in range(NB)]
    Ps = [torch.zeros(N, K, device=dev) for _ in range(NB)]
    Lrs = [torch.zeros(N, N, device=dev) for _ in range(NB)]
    inputs = {b: (host(Ls[b]).astype(np.float64), host(Gs[b]).astype(np.float64), host(Ds[b]).astype(np.float64),
                  host(Ws[b]).astype(np.float64)) for b in SAMPLES}
    blocks = [B.Block(G=Gs[b], W=Ws[b], D=Ds[b], P=Ps[b], L=Ls[b], Lr=Lrs[b]) for b in range(NB)]
    h = B.shampoo_create(0)
    try:
        prm = B.shampoo_root_params_default(p=4, eps=1e-6)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([N] * NB, prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(8 * NB, dtype=torch.int32, device=dev)
        B.shampoo_update_stats(h, blocks)
        B.shampoo_inv_root_batched(h, Ls, Lrs, prm, ws, info)
        B.shampoo_precondition(h, blocks)
        B.shampoo_graft(h, blocks, 1e-2)
        torch.cuda.synchronize()
        infos = B.decode_root_info(info)
        assert all(i["status"] in (0, 1) and i["precision"] == 32 for i in infos), infos[:3]
        for b in SAMPLES:
            L0, g, d0, w0 = inputs[b]
            Lo, _ = O.stats_update(L0, None, g)
            assert rel(host(Ls[b]), Lo) <= 1e-4, b
            Lr_o, _, _ = O.inv_root(Lo, 4, 1e-6)
            Lr_g = host(Lrs[b]).astype(np.float64)
            assert rel(Lr_g, Lr_o) <= 1e-3, (b, infos[b])
            tr = O.coupled_newton(host(Ls[b]), 4, 1e-6, tol=1e-6, scaling="power4")
            assert abs(infos[b]["iters"] - tr["iters"]) <= 1, (infos[b], tr["iters"])
            P_g = host(Ps[b]).astype(np.float64)
            assert rel(P_g, O.precondition(g, Lr_g, None)) <= 2e-3, b
            assert rel(P_g, O.precondition(g, Lr_o, None)) <= 2e-3, b
            out = O.graft_update(w0, d0, g, O.precondition(g, Lr_g, None), 1e-2)
            assert rel(host(Ws[b]).astype(np.float64) - w0, out["W"] - w0) <= 2e-3, b
            assert rel(host(Ds[b]), out["D"]) <= 1e-6, b
    finally:
        B.shampoo_destroy(h)
