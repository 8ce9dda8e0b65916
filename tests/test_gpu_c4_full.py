"""C4 at full size, in the launch configuration the benchmark times: 24
BERT-Large-shaped layers (288 blocks of 1024 x 1024, strided views of the Q,
K, V, O, FFN-in and FFN-out tensors), one grouped root refresh of all 576
factors (statistics of 100 earlier gradients), then one step: statistics,
then two-sided preconditioning and the AdaGrad graft over all 288 blocks in
one shampoo_precondition_graft call (grouped, graft pass 2 of a group
overlapping the next group's GEMMs).

Every factor's root against eigh (damped condition number ~1.5: the 1e-3
band), and every block's step against the fp64 oracle, which takes the same
inputs (the earlier statistics, G, W) and the GPU's roots: statistics 1e-4,
preconditioned gradient 2e-3, step dW 2e-3.  On sampled blocks of every
tensor kind the preconditioned gradient is also checked end to end, with the
oracle's own roots (2e-3).
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say
from tests.parity_util import pool_map, root_parity, summarize

pytestmark = pytest.mark.gpu

SAMPLES = (0, 4, 7, 11, 130, 209, 287)   # Q of layer 0, FFN-in, FFN-out, ... last block
EPS, ETA0 = 1e-6, 6e-3


@pytest.fixture(scope="module")
def c4_run():
    """Runs the refresh and the step on the GPU once; host copies of every
    input and output the checks need."""
    torch, B, dev = gpu_env()
    d, nl = cfg.C4_D, cfg.C4_LAYERS
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
    A0 = [host(a) for a in Ls + Rs]              # the statistics the refresh roots
    h = B.shampoo_create(0)
    try:
        say("C4 full: 576 roots in one grouped call")
        prm = B.shampoo_root_params_default(p=4, eps=EPS)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([d] * 576, prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(8 * 576, dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, Ls + Rs, Lrs + Rrs, prm, ws, info)
        say("C4 full: stats + precondition + graft over 288 blocks")
        B.shampoo_update_stats(h, blocks)
        B.shampoo_precondition_graft(h, blocks, ETA0)   # as the benchmark times the step
        torch.cuda.synchronize()
        del ws
    finally:
        B.shampoo_destroy(h)
    out = dict(A0=A0, X=[host(x) for x in Lrs + Rrs], info=B.decode_root_info(info),
               L=[host(a) for a in Ls], R=[host(a) for a in Rs], where=where, G=G,
               W0={k: host(w) for k, w in W0.items()}, W={k: host(w) for k, w in Wt.items()},
               P={k: host(p) for k, p in Pt.items()})
    del Gt, W0, Wt, Dt, Pt, Ls, Rs, Lrs, Rrs, blocks
    torch.cuda.empty_cache()
    return out


def test_c4_roots_all_576(c4_run):
    r = c4_run
    assert all(i["status"] in (0, 1) for i in r["info"]), [i for i in r["info"] if i["status"] > 1][:3]
    say("C4 full: oracle roots of 576 factors")
    res = pool_map(lambda j: root_parity(r["A0"][j], r["X"][j], 4, EPS), range(576))
    _, worst, frac = summarize("C4 roots (all 576)", [x[0] for x in res], [x[2] for x in res])
    assert frac == 1.0, worst


def _step_block(r, b, end_to_end):
    (k, sl), d = r["where"][b], cfg.C4_D
    g = r["G"][k][sl].astype(np.float64)
    L0, R0 = r["A0"][b].astype(np.float64), r["A0"][288 + b].astype(np.float64)
    Lo, Ro = O.stats_update(L0, R0, g)
    Lr_g, Rr_g = r["X"][b].astype(np.float64), r["X"][288 + b].astype(np.float64)
    P_g = r["P"][k][sl].astype(np.float64)
    P_k = O.precondition(g, Lr_g, Rr_g)
    w0 = r["W0"][k][sl].astype(np.float64)
    out = O.graft_update(w0, np.zeros((d, d)), g, P_k, ETA0)
    e = dict(L=rel(r["L"][b], Lo), R=rel(r["R"][b], Ro), P_kernel=rel(P_g, P_k),
             dW=rel(r["W"][k][sl].astype(np.float64) - w0, out["W"] - w0))
    if end_to_end:
        Lr_o, _, _ = O.inv_root(L0, 4, EPS)
        Rr_o, _, _ = O.inv_root(R0, 4, EPS)
        e["P_e2e"] = rel(P_g, O.precondition(g, Lr_o, Rr_o))
    return e


def test_c4_step_all_288(c4_run):
    say("C4 full: oracle step of 288 blocks with the GPU's roots")
    res = pool_map(lambda b: _step_block(c4_run, b, b in SAMPLES), range(288))
    for key, bar in (("L", 1e-4), ("R", 1e-4), ("P_kernel", 2e-3), ("dW", 2e-3)):
        _, worst, frac = summarize(f"C4 step {key} (all 288)", [x[key] for x in res], [bar] * 288)
        assert frac == 1.0, (key, worst)
    e2e = [res[b]["P_e2e"] for b in SAMPLES]
    summarize(f"C4 step P end to end ({len(SAMPLES)} sampled blocks)", e2e, [2e-3] * len(e2e))
    assert max(e2e) <= 2e-3
