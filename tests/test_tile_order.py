"""The grouped GEMMs' tile scheduler on the host (no GPU).

csrc/tiles.h maps each workgroup id to a logical tile and each logical tile
to (expert, row range, column block): dealt to the XCDs in groups of 32 for
the 256-row tiles (GEMM1 in super-rows of one grid round), in contiguous
ranges with the rows shared evenly for the 160-row tiles, striped over the
XCDs for the decode tiles.  tests/native/tile_order_check.cpp compiles that
header for the host and checks, over the library's launch shapes and a
range of row counts (skewed, ragged, empty experts, exact multiples of the
tile height), that every tile is taken by exactly one workgroup and that
every expert's rows are covered exactly once for every column block.  A
mistake there would leave rows of h or y unwritten or written twice, which
the GPU parity tests see only on the shapes they run."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_00993_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_tile_order_is_a_cover(tmp_path):
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    if not os.path.exists(hipcc):
        hipcc = shutil.which("hipcc")
        if hipcc is None:
            pytest.skip("hipcc not found")
    exe = str(tmp_path / "tile_order_check")
    cmd = [hipcc, "-x", "hip", "--offload-host-only", "-O1", "-std=c++17", f"-I{os.path.join(ROOT, 'include')}",
           f"-I{CSRC}", os.path.join(ROOT, "tests", "native", "tile_order_check.cpp"), "-o", exe]
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert p.returncode == 0, f"build failed:\n{' '.join(cmd)}\n{p.stdout}"
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=120)
    assert r.returncode == 0, r.stdout[-3000:]
    assert r.stdout.strip().endswith("ok"), r.stdout[-2000:]
