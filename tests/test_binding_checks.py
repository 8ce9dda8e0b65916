"""The Python binding rejects tensors that break the layout include/shampoo.h
states, before any C call: a wrong element type, shape, row stride or
contiguity, a mixed gradient type, an undersized info/warm_out/norms array,
and finally a tensor that is not on the GPU.  Everything here uses CPU
tensors and no handle, so nothing reaches a device."""
import pytest
import torch

from paper_2002_09018_amd import binding as B


def _block(m=6, n=5, pad=3, dtype=torch.float32, **over):
    def view(dt=torch.float32):
        return torch.zeros(m, n + pad, dtype=dt)[:, :n]
    b = dict(G=view(dtype), W=view(), D=view(), P=view(), L=torch.zeros(m, m), R=torch.zeros(n, n),
             Lr=torch.zeros(m, m), Rr=torch.zeros(n, n))
    b.update(over)
    return B.Block(**b)


def _raises(fn, match):
    with pytest.raises(ValueError, match=match):
        fn()


BLOCK_CALLS = [
    lambda blocks: B.shampoo_update_stats(None, blocks),
    lambda blocks: B.shampoo_precondition(None, blocks),
    lambda blocks: B.shampoo_graft(None, blocks, 0.1),
    lambda blocks: B.shampoo_graft_lamb(None, blocks, 0.1),
    lambda blocks: B.shampoo_precondition_graft(None, blocks, 0.1),
    lambda blocks: B.PackedBlocks(None, blocks),
]


@pytest.mark.parametrize("call", BLOCK_CALLS,
                         ids=["stats", "precondition", "graft", "graft_lamb", "precond_graft", "packed"])
def test_block_checks(call):
    m, n = 6, 5
    # a well-formed block passes every layout check and fails only on the device
    _raises(lambda: call([_block()]), "expected a GPU tensor")
    # state views must share G's row stride
    _raises(lambda: call([_block(W=torch.zeros(m, n))]), "row stride")
    _raises(lambda: call([_block(D=torch.zeros(m, n + 7)[:, :n])]), "row stride")
    _raises(lambda: call([_block(P=torch.zeros(n, m + 3)[:, :m].t())]), "shape|row stride")
    # element types
    _raises(lambda: call([_block(W=torch.zeros(m, n + 3, dtype=torch.float64)[:, :n])]), "float32")
    _raises(lambda: call([_block(dtype=torch.float16)]), "float32 or bfloat16")
    _raises(lambda: call([_block(), _block(dtype=torch.bfloat16)]), "one gradient type")
    _raises(lambda: call([_block(L=torch.zeros(m, m, dtype=torch.float64))]), "float32")
    # statistics and roots: square, contiguous, the block's sizes
    _raises(lambda: call([_block(L=torch.zeros(m + 1, m + 1))]), r"expected \(6, 6\)")
    _raises(lambda: call([_block(R=torch.zeros(m, m))]), r"expected \(5, 5\)")
    _raises(lambda: call([_block(Lr=torch.zeros(m, 2 * m)[:, ::2])]), "contiguous")
    _raises(lambda: call([_block(Rr=torch.zeros(n, n).t())]), "contiguous")
    # G itself
    _raises(lambda: call([_block(G=torch.zeros(m, 2 * n)[:, ::2])]), "stride")
    _raises(lambda: call([_block(G=torch.zeros(m * n))]), "dimensions")
    # mixed shapes across views
    _raises(lambda: call([_block(W=torch.zeros(m, n + 4)[:, :n + 1])]), "shape")


def test_norms_checks():
    _raises(lambda: B.shampoo_graft(None, [_block(), _block()], 0.1, norms=torch.zeros(5)), "at least 6")
    _raises(lambda: B.shampoo_graft(None, [_block()], 0.1, norms=torch.zeros(3, dtype=torch.float64)), "float32")
    _raises(lambda: B.shampoo_precondition_graft(None, [_block()], 0.1, norms=torch.zeros(6)[::2]), "contiguous")
    _raises(lambda: B.shampoo_graft(None, [_block()], 0.1, norms=torch.zeros(3)), "expected a GPU tensor")


@pytest.mark.parametrize("warm", [False, True])
def test_root_job_checks(warm):
    def call(As, Xs, ws=torch.zeros(64, dtype=torch.uint8), info=None, warm_out=None):
        info = torch.zeros(8 * len(As), dtype=torch.int32) if info is None else info
        prm = B.shampoo_root_params_default()
        if warm:
            return lambda: B.shampoo_inv_root_warm_batched(None, As, Xs, prm, ws, info, warm_out=warm_out)
        return lambda: B.shampoo_inv_root_batched(None, As, Xs, prm, ws, info)
    A, X = torch.zeros(8, 8), torch.zeros(8, 8)
    _raises(call([A], [X]), "expected a GPU tensor")
    _raises(call([A, A.clone()], [X]), "2 statistics but 1 outputs")
    _raises(call([torch.zeros(8, 9)], [X]), r"expected \(8, 8\)")
    _raises(call([A], [torch.zeros(7, 7)]), r"expected \(8, 8\)")
    _raises(call([A.double()], [X]), "float32")
    _raises(call([A], [X.double()]), "float32")
    _raises(call([torch.zeros(8, 16)[:, ::2]], [X]), "contiguous")
    _raises(call([A], [torch.zeros(16, 8)[::2]]), "contiguous")
    _raises(call([A], [A]), "distinct")
    _raises(call([A], [X], info=torch.zeros(7, dtype=torch.int32)), "at least 8")
    _raises(call([A], [X], info=torch.zeros(8, dtype=torch.int64)), "int32")
    _raises(call([A], [X], ws=None), "workspace")
    if warm:
        _raises(call([A], [X], warm_out=torch.zeros(1, dtype=torch.int32)), "at least 2")
        _raises(call([A], [X], warm_out=torch.zeros(2, dtype=torch.float32)), "int32")


def test_packed_job_checks():
    """PackedJobs runs the job checks when it is made; a packed call passes
    Xs as None."""
    A, X = torch.zeros(8, 8), torch.zeros(8, 8)
    _raises(lambda: B.PackedJobs(None, [A], [X]), "expected a GPU tensor")
    _raises(lambda: B.PackedJobs(None, [A], [A]), "distinct")
    _raises(lambda: B.PackedJobs(None, [torch.zeros(8, 9)], [X]), r"expected \(8, 8\)")
    _raises(lambda: B.PackedJobs(None, [A], [X.double()]), "float32")
    _raises(lambda: B.PackedJobs(None, [], []), "no jobs")


def test_embedding_checks():
    nnz, dim, vocab, m = 10, 4, 50, 10
    i32 = dict(dtype=torch.int32)
    idx, feat, w = torch.zeros(nnz, **i32), torch.zeros(nnz, **i32), torch.ones(nnz)
    dy, rows, U = torch.zeros(m, dim), torch.zeros(nnz, **i32), torch.zeros(nnz, dim)
    count, ws = torch.zeros(2, **i32), torch.zeros(64, dtype=torch.uint8)

    def rows_call(**o):
        a = dict(idx=idx, feat=feat, weight=w, vocab=vocab, dy=dy, rows=rows, U=U, count=count, workspace=ws)
        a.update(o)
        return lambda: B.shampoo_embedding_rows(None, **a)
    _raises(rows_call(), "expected a GPU tensor")
    _raises(rows_call(idx=idx.long()), "int32")
    _raises(rows_call(feat=feat[:5]), "entries")
    _raises(rows_call(weight=w.double()), "float32")
    _raises(rows_call(dy=torch.zeros(m, 2 * dim)[:, ::2]), "stride")
    _raises(rows_call(U=torch.zeros(nnz, dim + 1)), "expected")
    _raises(rows_call(U=torch.zeros(nnz - 1, dim)), "at least")
    _raises(rows_call(U=torch.zeros(nnz + 5, dim)), "expected a GPU tensor")   # a larger buffer is fine
    _raises(rows_call(U=torch.zeros(nnz, dim + 2)[:, :dim]), "contiguous")
    _raises(rows_call(count=torch.zeros(1, **i32)), "at least 2")
    _raises(rows_call(rows=torch.zeros(nnz - 1, **i32)), "at least")
    R = torch.zeros(dim, dim)
    _raises(lambda: B.shampoo_embedding_stats(None, U, count, R, workspace=ws), "expected a GPU tensor")
    _raises(lambda: B.shampoo_embedding_stats(None, U, count, torch.zeros(dim + 1, dim + 1), workspace=ws),
            "expected")
    _raises(lambda: B.shampoo_embedding_stats(None, U, count, R, workspace=None), "workspace")
    P = torch.zeros(nnz, dim)
    _raises(lambda: B.shampoo_embedding_precondition(None, U, count, R, P), "expected a GPU tensor")
    _raises(lambda: B.shampoo_embedding_precondition(None, U, count, R, torch.zeros(nnz, dim + 1)), "expected U's")
    _raises(lambda: B.shampoo_embedding_precondition(None, U, count, R.t().contiguous()[:, :dim - 1], P),
            r"expected \(4, 4\)")
    W, D = torch.zeros(vocab, dim), torch.zeros(vocab, dim)
    _raises(lambda: B.shampoo_embedding_graft(None, rows, count, U, P, W, D, 0.1), "expected a GPU tensor")
    _raises(lambda: B.shampoo_embedding_graft(None, rows, count, U, P, W, torch.zeros(vocab, dim + 2)[:, :dim],
                                              0.1), "row stride")
    _raises(lambda: B.shampoo_embedding_graft(None, rows, count, U, P, W, D.double(), 0.1), "float32")
    _raises(lambda: B.shampoo_embedding_graft(None, rows, count, U, P, W, D, 0.1, norms=torch.zeros(2)),
            "at least 3")
