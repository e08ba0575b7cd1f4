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


def test_algorithmic_ops_terms():
    """n = 2,000 jobs: NP = 2,048, L = 11, 2 lane-ops per compare-exchange of the
    bitonic network (NP/2 L(L+1)/2 of them), 64 per wave operation of the events
    and ceil(B / 64) wave operations per Phase ONE candidate."""
    c = bench.unit_counts("pareto_65536x2000", "isjl", 128)
    per = 2 * (1024 * 11 * 12 // 2) + 64 * c["event_wave_ops_per_instance"] + \
        64 * 8 * c["pack_candidates_per_instance"]
    assert bench.sort_compare_exchanges(2000) == 1024 * 11 * 12 // 2
    assert bench.algorithmic_ops("pareto_65536x2000", 1, 2000, 512, "isjl", 128, True) == per
    assert bench.algorithmic_ops("pareto_65536x2000", 65536, 2000, 512, "isjl", 128,
                                 True) == 65536.0 * per
    for al in (0, 16, 64, 256, 1024, "inf"):
        assert bench.algorithmic_ops("bimodal_sweep_4096x2000", 1, 2000, 128, "isjl", al,
                                     True) > 0


def test_unit_counts_are_the_oracles():
    """The recorded event and Phase ONE counts equal a fresh measurement with
    the oracle (on a smaller leading sample, whose per-instance values are the
    record's first ones: compared through their sum over the record's sample)."""
    sys.path.insert(0, os.path.join(ROOT, "tests", "golden"))
    import make_roofline_counts as mk
    for name, pol, al in (("pareto_65536x2000", "isjl", 128),
                          ("bimodal_sweep_4096x2000", "isjl", 1024)):
        want = bench.unit_counts(name, pol, al)
        got = mk.measure(name, pol, al, sample=want["sample"])
        assert got == want


def test_traffic_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    summary = tmp_path / "hbm.md"
    summary.write_text("traffic_bytes_per_launch: 1234\n"
                       f"kernel_sources_sha256: {bench.kernel_sources_sha256()}\n")
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", str(summary))
    assert bench.measured_traffic() == 1234
    summary.write_text("traffic_bytes_per_launch: 1234\nkernel_sources_sha256: 0000\n")
    assert bench.measured_traffic() is None


def test_valu_busy_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    summary = tmp_path / "hbm.md"
    summary.write_text("valu_busy_fraction: 0.5\n"
                       f"kernel_sources_sha256: {bench.kernel_sources_sha256()}\n")
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", str(summary))
    assert bench.profiled_valu_busy() == 0.5
    summary.write_text("valu_busy_fraction: 0.5\nkernel_sources_sha256: 0000\n")
    assert bench.profiled_valu_busy() is None
