"""Host-side logic of bench.py that runs without a GPU: the one-GPU guard,
the committed traffic figure keyed on the GEMM source, and the clock-table
parser."""

import hashlib
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_traffic_follows_the_gemm_source(tmp_path, monkeypatch):
    src = tmp_path / "gemm.hip"
    src.write_bytes(b"kernel source v1")
    prof = tmp_path / "traffic.md"
    digest = hashlib.sha256(b"kernel source v1").hexdigest()[:16]
    prof.write_text(f"# t\n\ngemm_source_sha256_16: {digest}   (note)\ntraffic_bytes_per_launch: 1234\n")
    monkeypatch.setattr(bench, "GEMM_SOURCE", str(src))
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(prof))
    assert bench.measured_traffic() == 1234
    src.write_bytes(b"kernel source v2")                      # the kernel changed since the counters
    assert bench.measured_traffic() is None
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(tmp_path / "missing.md"))
    assert bench.measured_traffic() is None


def test_committed_traffic_profile_is_readable():
    """The committed summary parses; its figure is reported only while it
    matches the GEMM source."""
    text = open(bench.TRAFFIC_PROFILE).read()
    assert "gemm_source_sha256_16:" in text and "traffic_bytes_per_launch:" in text
    v = bench.measured_traffic()
    assert v is None or 130e6 < v < 400e6


def test_dpm_table_parser():
    busy = "0: 500Mhz\n1: 2095Mhz *\n2: 2400Mhz\n"
    assert bench.parse_dpm(busy) == {"levels_mhz": [500, 2095, 2400], "current_mhz": 2095}
    idle = "S: 102Mhz *\n0: 500Mhz\n1: 2400Mhz\n"
    assert bench.parse_dpm(idle) == {"levels_mhz": [500, 2400], "current_mhz": 102}
    assert bench.parse_dpm("") == {"levels_mhz": [], "current_mhz": None}
