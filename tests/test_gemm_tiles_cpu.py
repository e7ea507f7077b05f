"""CPU check of the tiled GEMM's launch geometry and block -> tile map.

`tests/gemm_tiles_check.cpp` builds the library's own planning functions
(`csrc/gemm_plan.h`: plan_for_role, tile_geometry, tile_job) for the host
and runs them over the projections of every workload shape (tiny, OPT-1.3B,
6.7B, 13B, 66B) and other prompt lengths, ragged ones included, with and
without LoRA K tiles: each output tile is produced exactly once (whole, or
by `splits` blocks whose K ranges partition its K tiles), LoRA K tiles go
only to the last split of an active output group, and every partial tile
lands where its reduce kernel reads it, inside the workspace.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def test_gemm_tile_map_covers_every_tile_once(tmp_path):
    hipcc = shutil.which("hipcc")
    if not hipcc:
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "gemm_tiles_check")
    cmd = [hipcc, "-x", "hip", "--cuda-host-only", "-O1", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(ROOT, "paper_2503_17707_amd", "csrc"),
           os.path.join(HERE, "gemm_tiles_check.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout[-4000:]
    assert " 0 failures" in r.stdout
