"""Packed block and job lists (PackedBlocks, PackedJobs) against the same
calls made with plain lists: every output bit for bit, over a few steps of
statistics, roots, fused preconditioning and graft, on ragged blocks of two
gradient types; and a packed list made for one handle is refused by
another."""
import numpy as np
import pytest

from tests.gpu_util import gpu_env, say

pytestmark = pytest.mark.gpu


def _state(torch, dev, shapes, dtype, seed):
    g = torch.Generator(device=dev).manual_seed(seed)
    blocks, Gs = [], []
    for (m, n) in shapes:
        G = (torch.randn(m, n, device=dev, generator=g) * 0.1).to(dtype)
        Gs.append(G)
        blocks.append(dict(G=G, W=torch.randn(m, n, device=dev, generator=g), D=torch.zeros(m, n, device=dev),
                           P=torch.zeros(m, n, device=dev), L=torch.eye(m, device=dev) * 1e-3,
                           R=torch.eye(n, device=dev) * 1e-3, Lr=torch.zeros(m, m, device=dev),
                           Rr=torch.zeros(n, n, device=dev)))
    return blocks


def _run(torch, B, h, dev, state, packed, steps=3):
    blocks = [B.Block(**b) for b in state]
    ns = [n for b in state for n in (b["L"].shape[0], b["R"].shape[0])]
    As = [t for b in state for t in (b["L"], b["R"])]
    Xs = [t for b in state for t in (b["Lr"], b["Rr"])]
    prm = B.shampoo_root_params_default(p=4, eps=1e-6)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes(ns, prm.precision), dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    if packed:
        blocks, jobs, outs = B.PackedBlocks(h, blocks), B.PackedJobs(h, As, Xs), None
    else:
        jobs, outs = As, Xs
    for _ in range(steps):
        B.shampoo_update_stats(h, blocks, beta2=0.99)
        B.shampoo_inv_root_batched(h, jobs, outs, prm, ws, info)
        B.shampoo_precondition_graft(h, blocks, 1e-2)
    torch.cuda.synchronize()
    return info


@pytest.mark.parametrize("dtype", ["float32", "bfloat16"])
def test_packed_equals_lists(dtype):
    torch, B, dev = gpu_env()
    say("packed == lists", dtype)
    dt = getattr(torch, dtype)
    shapes = [(300, 200), (128, 520), (256, 256), (77, 130)]
    h = B.shampoo_create(0)
    try:
        s1 = _state(torch, dev, shapes, dt, 5)
        s2 = [{k: v.clone() for k, v in b.items()} for b in s1]
        i1 = _run(torch, B, h, dev, s1, packed=False)
        i2 = _run(torch, B, h, dev, s2, packed=True)
        assert torch.equal(i1, i2)
        for b1, b2 in zip(s1, s2):
            for k in ("W", "D", "P", "L", "R", "Lr", "Rr"):
                assert torch.equal(b1[k], b2[k]), k
    finally:
        B.shampoo_destroy(h)


def test_packed_jobs_warm_equals_lists():
    """The warm-started call with PackedJobs (Xs None) against the same call
    with lists, bit for bit, outputs and warm outcomes."""
    torch, B, dev = gpu_env()
    say("packed jobs warm == lists")
    h = B.shampoo_create(0)
    try:
        g = torch.Generator(device=dev).manual_seed(9)
        ns = [200, 256, 77]
        As = []
        for n in ns:
            a = torch.randn(n, n + 16, device=dev, generator=g)
            As.append((a @ a.T / (n + 16)).contiguous())
        prm = B.shampoo_root_params_default(p=4, eps=1e-6)
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes(ns, prm.precision), dtype=torch.uint8, device=dev)
        info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
        X0 = [torch.zeros_like(a) for a in As]
        B.shampoo_inv_root_batched(h, As, X0, prm, ws, info)
        A2 = [(a + 1e-3 * torch.eye(a.shape[0], device=dev)).contiguous() for a in As]
        X1, X2 = [x.clone() for x in X0], [x.clone() for x in X0]
        w1 = torch.zeros(2 * len(As), dtype=torch.int32, device=dev)
        w2 = torch.zeros_like(w1)
        i1, i2 = torch.zeros_like(info), torch.zeros_like(info)
        B.shampoo_inv_root_warm_batched(h, A2, X1, prm, ws, i1, w1)
        B.shampoo_inv_root_warm_batched(h, B.PackedJobs(h, A2, X2), None, prm, ws, i2, w2)
        torch.cuda.synchronize()
        assert torch.equal(w1, w2) and torch.equal(i1, i2)
        for a, b in zip(X1, X2):
            assert torch.equal(a, b)
    finally:
        B.shampoo_destroy(h)


def test_packed_other_handle_refused():
    torch, B, dev = gpu_env()
    say("packed other handle")
    h1, h2 = B.shampoo_create(0), B.shampoo_create(0)
    try:
        st = _state(torch, dev, [(64, 32)], torch.float32, 1)
        pb = B.PackedBlocks(h1, [B.Block(**st[0])])
        with pytest.raises(ValueError, match="another handle"):
            B.shampoo_update_stats(h2, pb)
        pj = B.PackedJobs(h1, [st[0]["L"]], [st[0]["Lr"]])
        ws = torch.empty(B.shampoo_inv_root_workspace_bytes([64]), dtype=torch.uint8, device=dev)
        info = torch.zeros(8, dtype=torch.int32, device=dev)
        with pytest.raises(ValueError, match="another handle"):
            B.shampoo_inv_root_batched(h2, pj, None, B.shampoo_root_params_default(), ws, info)
        with pytest.raises(ValueError, match="Xs must be None"):
            B.shampoo_inv_root_batched(h1, pj, [st[0]["Lr"]], B.shampoo_root_params_default(), ws, info)
    finally:
        B.shampoo_destroy(h1)
        B.shampoo_destroy(h2)
