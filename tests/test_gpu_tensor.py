"""An order-3 tensor through the C ABI (Preliminaries: the design holds for
tensors of any order; the K-FAC comparison appendix: exponent -1/(2k), here
p = 6), against the oracle's tensor_stats / tensor_precondition.

The library's calls take matrices; a tensor G of shape (d1, d2, d3),
row-major, is handled through strided views of its unfoldings:
  mode 1: G_(1) = G viewed d1 x (d2 d3)          -> L side of one block
  mode 3: G viewed (d1 d2) x d3, G_(3) its transpose -> R side of one block
  mode 2: G_(2) G_(2)^T = sum over i1 of G[i1] G[i1]^T (d2 x d3 slices),
          one statistics call per slice accumulating into the same matrix
and the preconditioned gradient G x_1 H_1 x_2 H_2 x_3 H_3 is three
preconditioning calls: H_1 G_(1), then H_2 times every d2 x d3 slice (one
grouped call), then the (d1 d2) x d3 view times H_3.  The AdaGrad graft
works on the flattened tensor.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from tests.gpu_util import gpu_env, host, rel, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [(24, 160, 24), (40, 48, 80)])
def test_order3_tensor_step(shape):
    torch, B, dev = gpu_env()
    say("order-3 tensor step", shape)
    d1, d2, d3 = shape
    k, p, eps, eta0 = 3, 6, 1e-6, 1e-2
    r = np.random.default_rng(sum(shape))
    Gs = [(r.standard_normal(shape) / np.sqrt(d1 * d2 * d3)).astype(np.float32) for _ in range(2)]
    W0 = (0.02 * r.standard_normal(shape)).astype(np.float32)
    h = B.shampoo_create(0)
    try:
        H = [torch.zeros(d, d, device=dev) for d in shape]
        for g in Gs:  # two statistics steps
            G = to_dev(torch, g, dev)
            B.shampoo_update_stats(h, [B.Block(G=G.view(d1, d2 * d3), L=H[0]),
                                       B.Block(G=G.view(d1 * d2, d3), R=H[2])])
            for i1 in range(d1):
                B.shampoo_update_stats(h, [B.Block(G=G[i1], L=H[1])])
        Hr = [torch.zeros(d, d, device=dev) for d in shape]
        prm = B.shampoo_root_params_default(p=p, eps=eps)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes(list(shape), prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(8 * k, dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, H, Hr, prm, ws, info)
        P1, P2, P = (torch.empty(shape, device=dev) for _ in range(3))
        B.shampoo_precondition(h, [B.Block(G=G.view(d1, d2 * d3), Lr=Hr[0], P=P1.view(d1, d2 * d3))])
        B.shampoo_precondition(h, [B.Block(G=P1[i1], Lr=Hr[1], P=P2[i1]) for i1 in range(d1)])
        B.shampoo_precondition(h, [B.Block(G=P2.view(d1 * d2, d3), Rr=Hr[2], P=P.view(d1 * d2, d3))])
        W = to_dev(torch, W0, dev)
        D = torch.zeros(shape, device=dev)
        B.shampoo_graft(h, [B.Block(G=G.view(d1, d2 * d3), W=W.view(d1, d2 * d3), D=D.view(d1, d2 * d3),
                                    P=P.view(d1, d2 * d3))], eta0)
        torch.cuda.synchronize()
    finally:
        B.shampoo_destroy(h)
    assert all(i["status"] in (0, 1) for i in B.decode_root_info(info))
    So = None
    for g in Gs:
        So = O.tensor_stats(So, g)
    Hg = [host(x).astype(np.float64) for x in H]
    for i in range(k):
        assert rel(Hg[i], So[i]) <= 1e-4, (i, rel(Hg[i], So[i]))
    Hr_g = [host(x).astype(np.float64) for x in Hr]
    Hr_o = [O.inv_root(Hg[i], p, eps)[0] for i in range(k)]
    for i in range(k):
        assert rel(Hr_g[i], Hr_o[i]) <= 1e-3, (i, rel(Hr_g[i], Hr_o[i]))
    g = Gs[-1].astype(np.float64)
    P_g = host(P).astype(np.float64)
    assert rel(P_g, O.tensor_precondition(g, Hr_g)) <= 2e-3  # kernel parity (the GPU's roots)
    assert rel(P_g, O.tensor_precondition(g, Hr_o)) <= 2e-3  # end to end
    out = O.graft_update(W0.reshape(d1, -1), np.zeros((d1, d2 * d3)), g.reshape(d1, -1), P_g.reshape(d1, -1), eta0)
    assert rel(host(W).reshape(d1, -1) - W0.reshape(d1, -1), out["W"] - W0.reshape(d1, -1)) <= 2e-3
