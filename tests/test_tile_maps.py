"""Host check of the workgroup -> tile maps that the product launches use
(xcd_remap, xcd_split_remap, deal_chunks and the upper-tile unranking): the
library's own header is compiled for the host into a small program that
checks every map exhaustively over a range of sizes (bijection, the grid
bound of the two-part map, contiguous per-XCD ranges, the order of the
parts).  No GPU is used."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not (os.path.exists(HIPCC) or shutil.which("hipcc")), reason="hipcc not found")
def test_tile_maps(tmp_path):
    exe = str(tmp_path / "tile_maps_check")
    cmd = [HIPCC, "-O1", "-std=c++17", "-I", os.path.join(ROOT, "paper_2002_09018_amd", "csrc"),
           os.path.join(HERE, "tile_maps_check.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
