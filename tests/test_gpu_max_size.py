"""The largest block the C ABI accepts (4096 rows) with a ragged width (4000
columns, not a multiple of the 128 tile), through every step.

* statistics L = G G^T (4096^2) and R = G^T G (4000^2): sampled entries
  against fp64 dot products of the same rows of G;
* inverse 4th roots of a 4096^2 SPD matrix (condition 1e3) and of R, in one
  grouped call: the property ||X^4 (A + eps I) - I||_F <= 4e-3 sqrt(n) (the
  1e-3 relative band to first order) checked in fp64;
* P = Lr G Rr with the GPU roots: sampled rows against the oracle's
  precondition of those rows;
* the graft: sampled rows of dW against the oracle's graft formula with the
  block norms computed from the same G and P in fp64.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu

M, N = 4096, 4000
ROWS = (0, 1, 2047, 3999, 4095)


def test_max_size_block():
    torch, B, dev = gpu_env()
    say("max size: 4096 x 4000 block")
    gen = torch.Generator(device=dev).manual_seed(4096)
    G = torch.randn(M, N, device=dev, generator=gen) / N ** 0.5
    W = 0.02 * torch.randn(M, N, device=dev, generator=gen)
    W0 = W.clone()
    D = torch.zeros(M, N, device=dev)
    P = torch.zeros(M, N, device=dev)
    L = torch.zeros(M, M, device=dev)
    R = torch.zeros(N, N, device=dev)
    # SPD 4096^2 with condition 1e3 (input; built in fp64 on the device)
    Z = torch.randn(M, M, device=dev, dtype=torch.float64, generator=gen)
    Q, _ = torch.linalg.qr(Z)
    lam = torch.logspace(0, 3, M, device=dev, dtype=torch.float64)
    A1 = ((Q * lam) @ Q.T)
    A1 = (0.5 * (A1 + A1.T)).float()
    del Z, Q
    h = B.shampoo_create(0)
    try:
        blk = B.Block(G=G, W=W, D=D, P=P, L=L, R=R)
        B.shampoo_update_stats(h, [blk])
        torch.cuda.synchronize()
        g = host(G).astype(np.float64)
        Lh, Rh = host(L), host(R)
        for i, j in ((0, 0), (5, 4095), (4095, 17), (2048, 2049)):
            assert abs(Lh[i, j] - g[i] @ g[j]) <= 1e-4 * np.sqrt((g[i] @ g[i]) * (g[j] @ g[j]))
        for i, j in ((0, 0), (3999, 1), (1000, 3000)):
            assert abs(Rh[i, j] - g[:, i] @ g[:, j]) <= 1e-4 * np.sqrt((g[:, i] @ g[:, i]) * (g[:, j] @ g[:, j]))
        assert np.array_equal(Lh, Lh.T) and np.array_equal(Rh, Rh.T)

        say("max size: roots 4096^2 and 4000^2")
        X1 = torch.zeros(M, M, device=dev)
        X2 = torch.zeros(N, N, device=dev)
        prm = B.shampoo_root_params_default(p=4, eps=1e-6)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([M, N], prm.precision), dtype=torch.uint8,
                         device=dev)
        info = torch.zeros(16, dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, [A1, R], [X1, X2], prm, ws, info)
        torch.cuda.synchronize()
        inf = B.decode_root_info(info)
        assert all(i["status"] in (0, 1) for i in inf), inf
        for A, X, n in ((A1, X1, M), (R, X2, N)):
            Xd = X.double()
            Ad = A.double() + 1e-6 * torch.eye(n, device=dev, dtype=torch.float64)
            Rm = Xd @ Xd @ Xd @ Xd @ Ad - torch.eye(n, device=dev, dtype=torch.float64)
            assert float(torch.linalg.norm(Rm)) <= 4e-3 * n ** 0.5, (n, float(torch.linalg.norm(Rm)), inf)

        say("max size: precondition and graft")
        blk = B.Block(G=G, W=W, D=D, P=P, Lr=X1, Rr=X2)
        B.shampoo_precondition(h, [blk])
        B.shampoo_graft(h, [blk], 1e-2)
        torch.cuda.synchronize()
        Lr, Rr = host(X1).astype(np.float64), host(X2).astype(np.float64)
        Ph = host(P).astype(np.float64)
        for i in ROWS:
            want = (Lr[i] @ g) @ Rr
            assert rel(Ph[i], want) <= 2e-3, i
        # graft: dW = -eta0 (||D^-1/2 G|| / ||P||) P with D = G^2 (first step)
        Pref = Lr @ g @ Rr
        out = O.graft_update(host(W0).astype(np.float64), np.zeros((M, N)), g, Pref, 1e-2)
        dW = host(W).astype(np.float64) - host(W0).astype(np.float64)
        dWo = out["W"] - host(W0).astype(np.float64)
        for i in ROWS:
            assert rel(dW[i], dWo[i]) <= 2e-3, i
    finally:
        B.shampoo_destroy(h)
