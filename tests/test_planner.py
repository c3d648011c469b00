"""The attention launch's work list, checked on the host: `planner_check.cpp`
includes the planner's source, plans launches of every kind (the 32K shard's
four ranks, a prefix hit, pass-KV partials at 8B and 70B shapes, few rows over
a long prefix, ragged GQA and MHA shapes, a mix of requests) in each
workgroup shape and in the per-launch choice, and checks that every work item
is scheduled exactly once -- whole, or as pieces that tile its key walk with
one workspace slot each -- and that pieces keep their policies' minimum
sizes.  Built with hipcc for the host only; no GPU is touched."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_work_list_invariants(tmp_path):
    exe = tmp_path / "planner_check"
    src = os.path.join(ROOT, "paper_2609_04774_amd", "csrc")
    build = subprocess.run(
        [HIPCC, "-O1", "-std=c++17", "--offload-arch=gfx950", "-I", os.path.join(ROOT, "include"), "-I", src,
         "-x", "hip", os.path.join(ROOT, "tests", "planner_check.cpp"), os.path.join(src, "plan.cpp"),
         "-o", str(exe)],
        capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-3000:]
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0 and run.stdout.startswith("ok"), run.stdout + run.stderr
