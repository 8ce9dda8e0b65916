"""A long Algorithm 2 run against the oracle's fp64 trajectory.

Eight blocks of assorted (some ragged) shapes, 100 steps: EMA statistics
(beta2 = 0.999), momentum beta1 = 0.9 on both graft directions, the AdaGrad
fallback before the first roots, inverse 4th roots refreshed every 10
steps (one grouped call for all 16 factors) and reused in between.  Each
step's dW must match the oracle's within 2e-3; statistics within 1e-4 at
every refresh; the momentum states and W within 2e-3 / 1e-4 at the end, so
errors do not accumulate over the run.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from tests.gpu_util import gpu_env, host, rel, say, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(256, 256), (256, 192), (200, 130), (128, 128), (256, 64), (96, 256), (130, 257), (64, 64)]
STEPS, TAU, P, EPS, ETA0, B1, B2 = 100, 10, 4, 1e-6, 1e-2, 0.9, 0.999


def test_algorithm2_hundred_steps():
    torch, B, dev = gpu_env()
    say("long run: 8 blocks, 100 steps")
    rng = np.random.default_rng(100)
    W0 = [rng.standard_normal(s).astype(np.float32) * 0.1 for s in SHAPES]
    dv = dict(W=[to_dev(torch, w, dev) for w in W0])
    for k in ("D", "P", "Mg", "Ps"):
        dv[k] = [torch.zeros(s, device=dev) for s in SHAPES]
    dv["L"] = [torch.zeros(m, m, device=dev) for m, _ in SHAPES]
    dv["R"] = [torch.zeros(n, n, device=dev) for _, n in SHAPES]
    dv["Lr"] = [torch.zeros(m, m, device=dev) for m, _ in SHAPES]
    dv["Rr"] = [torch.zeros(n, n, device=dev) for _, n in SHAPES]
    Gd = [torch.zeros(s, device=dev) for s in SHAPES]
    blocks = [B.Block(G=Gd[i], **{k: dv[k][i] for k in ("W", "D", "P", "Mg", "Ps", "L", "R", "Lr", "Rr")})
              for i in range(len(SHAPES))]
    ost = [dict(W=w.astype(np.float64), D=np.zeros(s), L=np.zeros((s[0], s[0])), R=np.zeros((s[1], s[1])),
                Mg=np.zeros(s), Ps=np.zeros(s)) for w, s in zip(W0, SHAPES)]
    ns = [m for m, _ in SHAPES] + [n for _, n in SHAPES]
    h = B.shampoo_create(0)
    try:
        prm = B.shampoo_root_params_default(p=P, eps=EPS)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes(ns, prm.precision), dtype=torch.uint8, device=dev)
        info = torch.zeros(8 * len(ns), dtype=torch.int32, device=dev)
        for t in range(1, STEPS + 1):
            grads = [(rng.standard_normal(s) / np.sqrt(s[1])).astype(np.float32) for s in SHAPES]
            for g, gd in zip(grads, Gd):
                gd.copy_(torch.from_numpy(g))
            Wprev = [host(w).astype(np.float64) for w in dv["W"]]
            Wprev_o = [s["W"].copy() for s in ost]
            refresh = t % TAU == 0
            use = t >= TAU
            B.shampoo_update_stats(h, blocks, beta2=B2)
            if refresh:
                B.shampoo_inv_root_batched(h, dv["L"] + dv["R"], dv["Lr"] + dv["Rr"], prm, ws, info)
            if use:
                B.shampoo_precondition(h, blocks)
            B.shampoo_graft(h, blocks, ETA0, beta1=B1, use_shampoo=use)
            torch.cuda.synchronize()
            for i, g in enumerate(grads):
                ost[i] = O.shampoo_step(ost[i], g, p=P, eps=EPS, eta0=ETA0, beta1=B1, beta2=B2,
                                        refresh_roots=refresh, use_shampoo=use)
                e = rel(host(dv["W"][i]).astype(np.float64) - Wprev[i], ost[i]["W"] - Wprev_o[i])
                assert e <= 2e-3, (t, i, e)
            if refresh:
                assert all(r["status"] in (0, 1) for r in B.decode_root_info(info))
                for i in range(len(SHAPES)):
                    assert rel(host(dv["L"][i]), ost[i]["L"]) <= 1e-4, (t, i)
                    assert rel(host(dv["R"][i]), ost[i]["R"]) <= 1e-4, (t, i)
        for i in range(len(SHAPES)):
            assert rel(host(dv["W"][i]), ost[i]["W"]) <= 1e-4, i
            assert rel(host(dv["Mg"][i]), ost[i]["Mg"]) <= 2e-3, i
            assert rel(host(dv["Ps"][i]), ost[i]["Ps"]) <= 2e-3, i
    finally:
        B.shampoo_destroy(h)
