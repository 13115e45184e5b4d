"""Host logic of bench.py (no GPU): the one-GPU contract and the rule that
the committed HBM-traffic figure is reported only for the fill source it was
measured on."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_fill_source_hash_covers_the_fill_sources():
    for kernel, sources in bench.FILL_SOURCES.items():
        h = bench.fill_source_hash(kernel)
        assert len(h) == 16 and int(h, 16) >= 0
        assert all(os.path.exists(os.path.join(ROOT, p)) for p in sources)
    assert any(p.endswith("wide.hip") for p in bench.FILL_SOURCES["k_fill_wide"])
    assert any(p.endswith("blocked.hip") for p in bench.FILL_SOURCES["k_fill_blocked"])
    # the kernels the binding can name are the ones a traffic figure can cover
    from paper_1905_11722_amd import rcdp
    assert set(rcdp.Solution.FILL_KERNELS) == set(bench.FILL_SOURCES)


def test_traffic_only_for_the_measured_source(monkeypatch, tmp_path):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "k_fill_blocked_demo_traffic.txt").write_text(
        "# demo\n\nfill_source_sha256_16 = 0123456789abcdef\nhbm_bytes_per_launch = 4242\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "fill_source_hash", lambda k: "0123456789abcdef")
    assert bench.read_traffic("k_fill_blocked", "demo") == 4242
    assert bench.read_traffic("k_fill_wide", "demo") is None      # another kernel's profile
    monkeypatch.setattr(bench, "fill_source_hash", lambda k: "fedcba9876543210")
    assert bench.read_traffic("k_fill_blocked", "demo") is None   # the kernel changed since
    assert bench.read_traffic("k_fill_blocked", "other") is None  # no profile at all

