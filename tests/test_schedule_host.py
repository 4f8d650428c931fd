"""Host checks of the window kernels' work decompositions (no GPU).

tests/native/gemm_schedule_check.cpp includes the GEMM source and walks its
scheduler (work items, K-part splits of the last round, the odd workgroups'
reordering, the per-XCD remap) over the window projections of the 1.5B and
7B shapes, ragged shapes and 200 seeded random ones, at several compute-unit
counts and partial-buffer capacities: every (tile, K slice) pair must be
computed by exactly one item.  tests/native/attn_schedule_check.cpp does the
same for attention's workgroup -> (query head, query block) map.  Both are
compiled with hipcc against the kernel sources and run on the host.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_and_run(tmp_path, name):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / name)
    cmd = [hipcc, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-o", exe,
           os.path.join(ROOT, "tests", "native", name + ".cpp")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok "), out.stdout
    return int(out.stdout.split()[1])


def test_gemm_schedule_computes_every_tile_slice_once(tmp_path):
    assert _build_and_run(tmp_path, "gemm_schedule_check") > 5000


def test_attention_serves_every_head_and_query_block_once(tmp_path):
    assert _build_and_run(tmp_path, "attn_schedule_check") > 2600
