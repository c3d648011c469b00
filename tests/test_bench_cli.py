"""bench.py's command-line contract that can be checked without a GPU: more
than one GPU is refused with a message (this build runs every rank's shard
on one GPU), and the measured-traffic lookup only returns figures recorded
for the kernel source as it is now."""

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


def test_traffic_figures_follow_the_kernel_source(tmp_path, monkeypatch):
    src = os.path.join(ROOT, "paper_2609_04774_amd", "csrc", "attn_partial.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_w_allgather.txt").write_text(
        f"# c\nkernel_source_sha256={sha}\nworkload=w\nmode=allgather\nfetch_bytes=10\nwrite_bytes=5\n")
    (prof / "traffic_w_passkv.txt").write_text(
        f"kernel_source_sha256={sha}\nworkload=w\nmode=passkv\nfetch_bytes=20\nwrite_bytes=5\n")
    (prof / "traffic_stale_allgather.txt").write_text(
        "kernel_source_sha256=0\nworkload=stale\nmode=allgather\nfetch_bytes=10\nwrite_bytes=5\n")
    # A file whose recorded mode is not the one its name says is not used.
    (prof / "traffic_odd_passkv.txt").write_text(
        f"kernel_source_sha256={sha}\nworkload=odd\nmode=allgather\nfetch_bytes=10\nwrite_bytes=5\n")
    (tmp_path / "paper_2609_04774_amd" / "csrc").mkdir(parents=True)
    (tmp_path / "paper_2609_04774_amd" / "csrc" / "attn_partial.hip").write_bytes(open(src, "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w") == 15
    assert bench.measured_traffic("w", "allgather") == 15
    assert bench.measured_traffic("w", "passkv") == 25
    assert bench.measured_traffic("stale") is None
    assert bench.measured_traffic("odd", "passkv") is None
    assert bench.measured_traffic("missing") is None
