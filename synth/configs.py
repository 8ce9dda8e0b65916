"""Seeded synthetic inputs for the five Shampoo workloads.

This module only draws random numbers and lays them out; it contains none of
Shampoo's arithmetic, so both the oracle and the GPU path may consume its
output.  Every stream is ``numpy.random.default_rng(SeedSequence([cfg, ...]))``
(PCG64), so any single block can be regenerated on its own.  "N(0, v)" means
variance v throughout.

Workloads (shapes follow the paper's experiments; no dataset is used):

* C1  one 128 x 128 block, 10 steps of fp32 gradients N(0, 1/128).
* C2  96 SPD 1024 x 1024 statistics, each the sum of 20 outer products
      G_t G_t^T with G_t 1024 x 4096 ~ N(0, 1/4096): a Wishart matrix with
      20 * 4096 degrees of freedom, drawn by the Bartlett decomposition.
* C3  32 SPD 2048 x 2048 matrices Q diag(lam) Q^T, Q from the QR of a
      Gaussian (signs fixed by diag(R)), lam log-uniform in [1e-6, 1e2].
* C4  BERT-Large-shaped layer stack: 24 layers x 12 blocks of 1024 x 1024
      (Q, K, V, O, 4 column blocks of FFN-in 1024 x 4096 and 4 row blocks of
      FFN-out 4096 x 1024), fp32 gradients N(0, 1e-3).
* C5  a 32768 x 1024 embedding (32 row blocks of 1024 x 1024) plus 200
      square blocks, side drawn uniformly from {128, 256, 512, 1024, 2048};
      gradients N(0, 1e-3) stored as bfloat16.
* C6  embedding lookups: a vocab x dim table read by token lookups whose
      rows follow a Zipf law (P(rank k) ~ (k + 1)^-s, s = 1.07, ranks mapped
      to rows by a keyed permutation); one-hot (one row per output row) or
      multi-hot bags of 1..8 rows averaged (weights 1/bag size); output
      gradients dy ~ N(0, 1e-3).
"""
from __future__ import annotations

import math

import numpy as np

C1, C2, C3, C4, C5 = 1, 2, 3, 4, 5


def rng(*key):
    """PCG64 generator keyed by a tuple of non-negative ints."""
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


def gaussian(shape, var, *key):
    """fp32 array of N(0, var) samples (standard_normal in fp32, scaled)."""
    g = rng(*key).standard_normal(shape, dtype=np.float32)
    return (g * np.float32(math.sqrt(var))).astype(np.float32)


def f32_to_bf16_bits(x):
    """Round fp32 values to bfloat16 (round to nearest even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


# ---------------------------------------------------------------- C1
def c1_weight(seed=0, n=128):
    return gaussian((n, n), 1.0, C1, seed, 0, 0)


def c1_grad(step, seed=0, n=128):
    """Gradient of step ``step`` (1-based) of config C1."""
    return gaussian((n, n), 1.0 / n, C1, seed, 1, step)


# ---------------------------------------------------------------- C2
def wishart_bartlett(n, dof, var, *key):
    """Sum of ``dof`` outer products g g^T with g ~ N(0, var I_n), drawn in
    O(n^3) by the Bartlett decomposition A = var * T T^T, T lower triangular
    with T_ii = sqrt(chi2(dof - i)) (i = 0..n-1) and N(0,1) below the
    diagonal.  Returned in float64."""
    r = rng(*key)
    T = np.tril(r.standard_normal((n, n)), -1)
    T[np.diag_indices(n)] = np.sqrt(r.chisquare(dof - np.arange(n)))
    return var * (T @ T.T)


def wishart_bartlett_device(n, dof, var, torch, device, *key):
    """Same distribution as ``wishart_bartlett``, with the O(n^3) product on
    the device: chi-square diagonal from the keyed PCG64 stream, standard
    normals below the diagonal from a torch generator seeded by the key, and
    var * T T^T formed in fp64 there.  Returned as an fp32 device tensor."""
    r = rng(*key)
    diag = np.sqrt(r.chisquare(dof - np.arange(n)))
    seed = int(r.integers(0, 2 ** 62))
    g = torch.Generator(device=device).manual_seed(seed)
    T = torch.randn(n, n, generator=g, device=device, dtype=torch.float64).tril(-1)
    T += torch.diag(torch.from_numpy(diag).to(device))
    return (var * (T @ T.T)).float()


def c2_stats(i, n=1024, steps=20, k=4096):
    """C2 statistics matrix i: sum over ``steps`` gradients of shape n x k,
    N(0, 1/k), rounded to fp32 (the GPU input)."""
    A = wishart_bartlett(n, steps * k, 1.0 / k, C2, i, 0)
    return A.astype(np.float32)


def c2_grad(i, n=1024, k=4096, step=20):
    """The gradient G_step (n x k) of C2 block i for a whole-step run."""
    return gaussian((n, k), 1.0 / k, C2, i, 1, step)


def c2_adagrad_state(i, n=1024, k=4096, steps=19):
    """Diagonal AdaGrad accumulator after ``steps`` gradients N(0, 1/k):
    each entry is chi2(steps) / k."""
    return (rng(C2, i, 2).chisquare(steps, size=(n, k)) / k).astype(np.float32)


def c2_weight(i, n=1024, k=4096):
    return gaussian((n, k), 0.02 ** 2, C2, i, 3)


# ---------------------------------------------------------------- C3
def c3_matrix(i, n=2048, lo=-6.0, hi=2.0):
    """C3 matrix i: Q diag(lam) Q^T in float64, then rounded to fp32.
    Returns (A_fp32, lam sorted ascending, Q)."""
    r = rng(C3, i, n)
    Z = r.standard_normal((n, n))
    Q, Rm = np.linalg.qr(Z)
    Q = Q * np.sign(np.diag(Rm))
    lam = np.sort(10.0 ** r.uniform(lo, hi, size=n))
    A = (Q * lam) @ Q.T
    A = 0.5 * (A + A.T)
    return A.astype(np.float32), lam, Q


def c3_matrix_device(i, torch, device, n=2048, lo=-6.0, hi=2.0):
    """C3 matrix i with the same recipe as ``c3_matrix``, the O(n^3) work on
    the device: Gaussian Z from a torch generator seeded by the key, Q from
    its QR (signs fixed by diag R), lambda = 10^U(lo, hi) from the keyed PCG64
    stream, Q diag(lambda) Q^T in fp64, symmetrised and rounded to fp32.
    Returns (A_fp32 device tensor, lambda sorted ascending as numpy)."""
    r = rng(C3, i, n, 1)
    seed = int(r.integers(0, 2 ** 62))
    lam = np.sort(10.0 ** r.uniform(lo, hi, size=n))
    g = torch.Generator(device=device).manual_seed(seed)
    Z = torch.randn(n, n, generator=g, device=device, dtype=torch.float64)
    Q, Rm = torch.linalg.qr(Z)
    Q = Q * torch.sign(torch.diagonal(Rm))
    A = (Q * torch.from_numpy(lam).to(device)) @ Q.T
    return (0.5 * (A + A.T)).float(), lam


# ---------------------------------------------------------------- C4
C4_LAYERS, C4_BLOCKS, C4_D, C4_FF = 24, 12, 1024, 4096


def c4_layer_tensors():
    """Names and shapes of the six matrices of one transformer layer."""
    d, f = C4_D, C4_FF
    return [("q", (d, d)), ("k", (d, d)), ("v", (d, d)), ("o", (d, d)),
            ("ffn_in", (d, f)), ("ffn_out", (f, d))]


def c4_blocks(d=C4_D):
    """Block partition of one layer: (tensor index, row0, col0, rows, cols),
    12 blocks of d x d (Q, K, V, O whole; FFN-in in 4 column blocks; FFN-out
    in 4 row blocks)."""
    out = []
    for t, (_, (m, n)) in enumerate(c4_layer_tensors()):
        for r0 in range(0, m, d):
            for c0 in range(0, n, d):
                out.append((t, r0, c0, d, d))
    return out


def c4_grad(layer, tensor, step, shape):
    return gaussian(shape, 1e-3, C4, layer, tensor, step)


def c4_weight(layer, tensor, shape):
    return gaussian(shape, 0.02 ** 2, C4, layer, tensor, 10 ** 6)


# ---------------------------------------------------------------- C5
C5_EMB_ROWS, C5_D, C5_NMIXED = 32768, 1024, 200
C5_SIZES = (128, 256, 512, 1024, 2048)


def c5_mixed_sizes(count=C5_NMIXED):
    return [int(s) for s in rng(C5, 0).choice(C5_SIZES, size=count)]


def c5_grad_bf16(block, step, shape):
    """bf16 bit patterns of an N(0, 1e-3) gradient (RNE from fp32)."""
    return f32_to_bf16_bits(gaussian(shape, 1e-3, C5, 1, block, step))


def c5_weight(block, shape):
    return gaussian(shape, 0.02 ** 2, C5, 2, block)


# ---------------------------------------------------------------- C6
C6 = 6
C6_S = 1.07


def zipf_rows(n, vocab, s, *key):
    """n int32 row ids in [0, vocab), P(rank k) proportional to (k+1)^-s, rank
    k stored at row perm[k] of a keyed permutation."""
    r = rng(*key)
    w = 1.0 / np.arange(1, vocab + 1, dtype=np.float64) ** s
    ranks = r.choice(vocab, size=n, p=w / w.sum())
    perm = r.permutation(vocab)
    return perm[ranks].astype(np.int32)


def c6_lookup(step, nnz, vocab, multi=False, seed=0):
    """(idx, feat, weight, m) of one step's lookups.  One-hot: m = nnz,
    feat = weight = None.  Multi-hot: bags of 1..8 entries, each bag one
    output row, weights 1 / bag size; nnz entries in total."""
    idx = zipf_rows(nnz, vocab, C6_S, C6, seed, 0, step)
    if not multi:
        return idx, None, None, nnz
    r = rng(C6, seed, 1, step)
    sizes = []
    left = nnz
    while left > 0:
        b = int(min(left, r.integers(1, 9)))
        sizes.append(b)
        left -= b
    feat = np.repeat(np.arange(len(sizes), dtype=np.int32), sizes)
    weight = np.repeat(1.0 / np.array(sizes, dtype=np.float32), sizes).astype(np.float32)
    return idx, feat, weight, len(sizes)


def c6_dy(step, m, dim, seed=0):
    return gaussian((m, dim), 1e-3, C6, seed, 2, step)


def c6_table(vocab, dim, seed=0):
    return gaussian((vocab, dim), 0.02 ** 2, C6, seed, 3)
