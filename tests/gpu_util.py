"""Helpers shared by the GPU parity tests (no oracle arithmetic here)."""
import sys

import numpy as np
import pytest


def say(*a):
    """Names the case before a GPU step (flushed, so a fault still shows it)."""
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def gpu_env():
    """(torch, binding, device) or skip when no GPU is present."""
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2002_09018_amd import binding as B
    return torch, B, torch.device("cuda:0")


def to_dev(torch, x, dev):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def host(t):
    return t.detach().cpu().numpy()


def spd(n, cond, seed, dtype=np.float32):
    """Seeded SPD test matrix Q diag(logspace) Q^T (input generator)."""
    r = np.random.default_rng(seed)
    Q, _ = np.linalg.qr(r.standard_normal((n, n)))
    lam = np.logspace(0, np.log10(cond), n) if n > 1 else np.array([1.0])
    A = (Q * lam) @ Q.T
    return (0.5 * (A + A.T)).astype(dtype)
