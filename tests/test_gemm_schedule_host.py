"""Host check of the persistent bf16 GEMM's work decomposition.

tests/native/gemm_schedule_check.cpp includes the GEMM source and walks its
scheduler (work items, K-part splits of the last round, the odd workgroups'
reordering, the per-XCD remap) over the window projections of the 1.5B and
7B shapes, ragged shapes and 200 seeded random ones, at several compute-unit
counts and partial-buffer capacities: every (tile, K slice) pair must be
computed by exactly one item.  Compiled with hipcc; no GPU is used.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "native", "gemm_schedule_check.cpp")


def test_gemm_schedule_computes_every_tile_slice_once(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "gemm_schedule_check")
    cmd = [hipcc, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-o", exe, SRC]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok "), out.stdout
    assert int(out.stdout.split()[1]) > 5000
