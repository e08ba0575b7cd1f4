"""Host-side pieces of bench.py: the one-GPU guard, the algorithmic operation
count behind the roofline, and the gating of the recorded HBM traffic on the
kernel sources."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_ops_closed_form():
    """n = 2,000 jobs: NP = 2,048, L = 11, 2 lane-ops per compare-exchange of the
    bitonic network (NP/2 * L(L+1)/2 of them), and n (3 min(B, n) + L + 1)."""
    per = 2 * (1024 * 11 * 12 // 2) + 2000 * (3 * 512 + 12)
    assert bench.algorithmic_ops(1, 2000, 512, "isjl", True) == per
    assert bench.algorithmic_ops(65536, 2000, 512, "isjl", True) == 65536.0 * per
    # FCFS over sorted arrivals needs no sort
    assert bench.algorithmic_ops(1, 2000, 512, "fcfs", True) == 2000 * (3 * 512 + 12)
    assert bench.algorithmic_ops(1, 2000, 512, "fcfs", False) == per


def test_traffic_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    summary = tmp_path / "hbm.md"
    summary.write_text("traffic_bytes_per_launch: 1234\n"
                       f"kernel_sources_sha256: {bench.kernel_sources_sha256()}\n")
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", str(summary))
    assert bench.measured_traffic() == 1234
    summary.write_text("traffic_bytes_per_launch: 1234\nkernel_sources_sha256: 0000\n")
    assert bench.measured_traffic() is None
