"""Host logic of bench.py (no GPU): the one-GPU contract and the counter
summary it reads the sampler's traffic from."""
import hashlib
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_is_read_only_for_the_profiled_kernel_source(tmp_path, monkeypatch):
    src = tmp_path / "kernels.hip"
    src.write_bytes(b"// some kernel source\n")
    summary = tmp_path / "summary.md"
    sha = hashlib.sha256(src.read_bytes()).hexdigest()
    summary.write_text("kernel_source_sha256: %s\n\ncounter_window_iterations: 5-24\n\n"
                       "k_sampler_fabric_bytes_per_launch: 1.5e+11\n" % sha)
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(src))
    monkeypatch.setattr(bench, "PMC_SUMMARY", str(summary))
    assert bench.traffic_from_profile("c3", 5, 24) == 1.5e11
    # the counters cover the c3 workload only
    assert bench.traffic_from_profile("c5", 5, 24) is None
    # and only the iterations they were taken over
    assert bench.traffic_from_profile("c3", 1, 100) is None
    # the kernel changed since the counters were taken: no traffic figure
    src.write_bytes(b"// some other kernel source\n")
    assert bench.traffic_from_profile("c3", 5, 24) is None
    # no summary at all
    monkeypatch.setattr(bench, "PMC_SUMMARY", str(tmp_path / "missing.md"))
    assert bench.traffic_from_profile("c3", 5, 24) is None


def test_committed_counter_summary_names_a_source_hash_and_a_byte_count():
    txt = open(bench.PMC_SUMMARY).read()
    assert "kernel_source_sha256:" in txt and "k_sampler_fabric_bytes_per_launch:" in txt
    assert "counter_window_iterations:" in txt
