"""bench.py's command-line contract that can be checked without a GPU: more
than one GPU is refused with a message (the library runs every rank's shard
on one GPU), and the measured-traffic lookup only returns figures recorded
for the kernel and planner sources as they are now."""

import hashlib
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", "--steps", "1"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_figures_follow_the_kernel_and_planner_sources(tmp_path, monkeypatch):
    csrc = os.path.join(ROOT, "paper_2609_04774_amd", "csrc")
    src = open(os.path.join(csrc, "attn_partial.hip"), "rb").read()
    planner = open(os.path.join(csrc, "cp_attn.cpp"), "rb").read()
    sha = hashlib.sha256(src).hexdigest()
    psha = hashlib.sha256(planner).hexdigest()
    keys = f"kernel_source_sha256={sha}\nplanner_source_sha256={psha}\n"
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_w_allgather.txt").write_text(
        f"# c\n{keys}workload=w\nmode=allgather\nfetch_bytes=10\nwrite_bytes=5\n")
    (prof / "traffic_w_passkv.txt").write_text(f"{keys}workload=w\nmode=passkv\nfetch_bytes=20\nwrite_bytes=5\n")
    (prof / "traffic_stale_allgather.txt").write_text(
        f"kernel_source_sha256=0\nplanner_source_sha256={psha}\nworkload=stale\nmode=allgather\n"
        "fetch_bytes=10\nwrite_bytes=5\n")
    # Counters taken under another plan (or before the planner was recorded)
    # are not used either: the plan decides which pieces are written.
    (prof / "traffic_replanned_allgather.txt").write_text(
        f"kernel_source_sha256={sha}\nplanner_source_sha256=0\nworkload=replanned\nmode=allgather\n"
        "fetch_bytes=10\nwrite_bytes=5\n")
    (prof / "traffic_unkeyed_allgather.txt").write_text(
        f"kernel_source_sha256={sha}\nworkload=unkeyed\nmode=allgather\nfetch_bytes=10\nwrite_bytes=5\n")
    # A file whose recorded mode is not the one its name says is not used.
    (prof / "traffic_odd_passkv.txt").write_text(f"{keys}workload=odd\nmode=allgather\nfetch_bytes=10\nwrite_bytes=5\n")
    (tmp_path / "paper_2609_04774_amd" / "csrc").mkdir(parents=True)
    (tmp_path / "paper_2609_04774_amd" / "csrc" / "attn_partial.hip").write_bytes(src)
    (tmp_path / "paper_2609_04774_amd" / "csrc" / "cp_attn.cpp").write_bytes(planner)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w") == 15
    assert bench.measured_traffic("w", "allgather") == 15
    assert bench.measured_traffic("w", "passkv") == 25
    assert bench.measured_traffic("stale") is None
    assert bench.measured_traffic("replanned") is None
    assert bench.measured_traffic("unkeyed") is None
    assert bench.measured_traffic("odd", "passkv") is None
    assert bench.measured_traffic("missing") is None

