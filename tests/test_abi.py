"""The C-ABI library loads and exports every function include/shampoo.h
declares; host-only entry points behave (no GPU compute is called here)."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "shampoo.h")
LIB = os.path.join(ROOT, "paper_2002_09018_amd", "libshampoo.so")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(shampoo_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libshampoo.so is not built (run __graft_entry__.build())")
    from paper_2002_09018_amd import binding
    return binding


def test_header_declares_the_boundary():
    names = declared()
    for n in ("shampoo_update_stats", "shampoo_inv_root_batched", "shampoo_precondition", "shampoo_graft",
              "shampoo_create", "shampoo_destroy", "shampoo_last_error", "shampoo_inv_root_workspace_bytes",
              "shampoo_embedding_rows", "shampoo_embedding_stats", "shampoo_embedding_precondition",
              "shampoo_embedding_graft", "shampoo_embedding_workspace_bytes"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    missing = [n for n in declared() if n not in exported]
    assert not missing, missing
    # and the binding binds exactly the declared set
    assert sorted(lib.EXPORTED) == declared()


def test_host_only_entry_points(lib):
    assert "gfx950" in lib.shampoo_version()
    p = lib.shampoo_root_params_default()
    assert (p.p, p.max_iters, p.precision, p.poll) == (4, 100, lib.PRECISION_AUTO, 1)
    assert p.scaling == lib.SCALING_POWER4
    assert abs(p.eps - 1e-6) < 1e-12 and abs(p.kappa32 - 1e4) < 1e-3
    assert lib.shampoo_inv_root_workspace_bytes([0]) == 0
    assert lib.shampoo_inv_root_workspace_bytes([4097]) == 0
    assert lib.shampoo_inv_root_workspace_bytes([128], precision=7) == 0
    w32 = lib.shampoo_inv_root_workspace_bytes([1024], lib.PRECISION_FP32)
    w64 = lib.shampoo_inv_root_workspace_bytes([1024], lib.PRECISION_FP64)
    wa = lib.shampoo_inv_root_workspace_bytes([1024], lib.PRECISION_AUTO)
    # fp32: five n^2 fp32 iterates; fp64: six n^2 fp64 iterates; AUTO both
    assert 5 * 4 * 1024 ** 2 <= w32 < 5 * 4 * 1024 ** 2 + 10 ** 6
    assert 6 * 8 * 1024 ** 2 <= w64 < 6 * 8 * 1024 ** 2 + 10 ** 6
    assert wa >= w32 + w64 - 10 ** 6
    # embedding workspace: 7 int32 arrays of nnz plus split-K partials of dim^2
    assert lib.shampoo_embedding_workspace_bytes(0, 64) == 0
    assert lib.shampoo_embedding_workspace_bytes(10, 0) == 0
    assert lib.shampoo_embedding_workspace_bytes(10, 4097) == 0
    assert lib.shampoo_embedding_workspace_bytes((1 << 26) + 1, 64) == 0
    small = lib.shampoo_embedding_workspace_bytes(100, 64)      # one split: no partials
    assert 7 * 4 * 100 <= small < 7 * 4 * 100 + 4096
    big = lib.shampoo_embedding_workspace_bytes(65536, 1024)    # split-K over 36 upper tiles
    assert big >= 7 * 4 * 65536 + 2 * 4 * 1024 ** 2


def test_struct_layouts_match_header(lib):
    import ctypes as C
    assert C.sizeof(lib.shampoo_block) == 96
    assert C.sizeof(lib.shampoo_root_job) == 24
    assert C.sizeof(lib.shampoo_root_params) == 44
    assert C.sizeof(lib.shampoo_root_info) == 32
