"""C6 at the benchmarked size: a 32768 x 1024 embedding table, 65536 one-hot
Zipf lookups, one step (compact rows, R += U^T U, U R^(-1/2), row-indexed
graft) with R holding the statistics of 100 earlier steps and its root
refreshed first, all in the benchmark's launch configuration.

Against the oracle's dense definition on the whole table: R <= 1e-5; the
root of the earlier statistics <= 1e-3; the step's dW over every row with
the GPU's root (kernel parity) <= 2e-3; rows no lookup touched keep their W
and D bits.
"""
import numpy as np
import pytest

import oracle.shampoo_oracle as O
from synth import configs as cfg
from tests.gpu_util import gpu_env, host, rel, say

pytestmark = pytest.mark.gpu


def test_c6_full_step():
    torch, B, dev = gpu_env()
    vocab, nnz, dim, eta0, eps = 32768, 65536, 1024, 1e-2, 1e-6
    say("C6 full: 32768 x 1024 table, 65536 lookups")
    idx, _, _, m = cfg.c6_lookup(1, nnz, vocab)
    dy = cfg.c6_dy(1, m, dim)
    W0 = cfg.c6_table(vocab, dim)
    W = torch.from_numpy(W0).to(dev)
    D = torch.zeros(vocab, dim, device=dev)
    R = cfg.wishart_bartlett_device(dim, 100 * nnz, 1e-3, torch, dev, cfg.C6, 8, 0)
    R0 = host(R).astype(np.float64)
    Rr = torch.zeros(dim, dim, device=dev)
    rows = torch.zeros(nnz, dtype=torch.int32, device=dev)
    U = torch.zeros(nnz, dim, device=dev)
    P = torch.zeros(nnz, dim, device=dev)
    count = torch.zeros(2, dtype=torch.int32, device=dev)
    h = B.shampoo_create(0)
    try:
        ws = torch.empty(B.shampoo_embedding_workspace_bytes(nnz, dim), dtype=torch.uint8, device=dev)
        prm = B.shampoo_root_params_default(p=2, eps=eps)
        rws = torch.empty(B.shampoo_inv_root_workspace_bytes([dim], prm.precision), dtype=torch.uint8, device=dev)
        info = torch.zeros(8, dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, [R], [Rr], prm, rws, info)
        idx_d = torch.from_numpy(idx).to(dev)
        B.shampoo_embedding_rows(h, idx_d, None, None, vocab, torch.from_numpy(dy).to(dev), rows, U, count, ws)
        B.shampoo_embedding_stats(h, U, count, R, 1.0, ws)
        B.shampoo_embedding_precondition(h, U, count, Rr, P)
        B.shampoo_embedding_graft(h, rows, count, U, P, W, D, eta0)
        torch.cuda.synchronize()
        assert B.decode_root_info(info)[0]["status"] in (0, 1)
        G = O.embedding_grad(vocab, idx, None, None, dy)
        _, Ro = O.stats_update(None, R0, G)
        assert rel(host(R), Ro) <= 1e-5
        Rr_g = host(Rr).astype(np.float64)
        Rr_o, _, _ = O.inv_root(R0, 2, eps)
        assert rel(Rr_g, Rr_o) <= 1e-3
        out = O.graft_update(W0.astype(np.float64), np.zeros((vocab, dim)), G, O.precondition(G, None, Rr_g), eta0)
        Wh = host(W).astype(np.float64)
        assert rel(Wh - W0, out["W"] - W0) <= 2e-3
        u = int(host(count)[0])
        active = np.zeros(vocab, dtype=bool)
        active[host(rows)[:u]] = True
        assert u == int(np.count_nonzero(np.any(G != 0, axis=1)))
        assert np.array_equal(host(W)[~active], W0[~active])
        assert not np.any(host(D)[~active])
    finally:
        B.shampoo_destroy(h)
