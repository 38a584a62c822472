"""Host-side logic of bench.py, on the CPU: the one-GPU refusal, and the rule
that ties the reported HBM traffic to the kernel source the counters were
taken on (a summary from another source reads as no measurement)."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_follows_the_kernel_source(tmp_path, monkeypatch):
    good = bench.kernel_source_hash("partition_kernel")
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.measured_traffic("partition_kernel", "w") is None  # no summary
    f = tmp_path / "traffic_partition_kernel_w.md"
    f.write_text(f"kernel_source_sha256_16: {good}\nhbm_bytes_per_launch: 2554605000\n")
    assert bench.measured_traffic("partition_kernel", "w") == 2554605000.0
    f.write_text("kernel_source_sha256_16: 0123456789abcdef\nhbm_bytes_per_launch: 2554605000\n")
    assert bench.measured_traffic("partition_kernel", "w") is None  # taken on another source
    f.write_text(f"kernel_source_sha256_16: {good}\n")
    assert bench.measured_traffic("partition_kernel", "w") is None  # no figure

