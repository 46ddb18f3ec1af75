"""Host-side checks of bench.py that need no GPU: the one-GPU refusal, the kernel-source hash that
decides whether a committed traffic summary applies, and the reading of the summaries."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_summary_applies_only_to_its_sources(tmp_path):
    text = open(bench.TRAFFIC_SUMMARY).read()
    # the committed summary was taken on the current GEMM sources
    assert bench.measured_traffic() is not None
    assert f"kernel_source_hash: {bench.kernel_source_hash()}" in text
    # a summary recorded for other sources is not used
    stale = tmp_path / "stale.md"
    stale.write_text(text.replace(bench.kernel_source_hash(), "0" * 16))
    assert bench.measured_traffic(str(stale)) is None
    # nor is one without the byte count
    partial = tmp_path / "partial.md"
    partial.write_text(f"kernel_source_hash: {bench.kernel_source_hash()}\n")
    assert bench.measured_traffic(str(partial)) is None
    assert bench.measured_traffic(str(tmp_path / "missing.md")) is None


def test_stream_ceiling_is_read():
    c = bench.stream_ceiling()
    assert c is not None and 1000.0 < c < bench.HBM_PEAK_GBPS
