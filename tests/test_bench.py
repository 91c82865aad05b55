"""Host logic of bench.py (CPU): the algorithmic bytes of a row launch, the
counter-derived traffic and its source gate, and the one-GPU refusal."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_row_bytes_per_launch_match_the_workload_sizes():
    # per row: 4d features, 4 norm, 16 F read and written, 1 state byte
    # (eps-SVR: 2 state bytes and the 4-byte target)
    assert bench.row_bytes_per_launch(100000, 128, False) == 53_300_000
    assert bench.row_bytes_per_launch(20000, 50, True) == 4_520_000
    assert bench.row_bytes_per_launch(500000, 784, False) == 1_578_500_000
    assert bench.row_bytes_per_launch(0, 128, False) == 0


@pytest.mark.parametrize("name,alg", [("C3", 53.3e6), ("C4", 1.5785e9)])
def test_committed_counters_match_the_row_kernel_sources(name, alg):
    # the FETCH_SIZE / WRITE_SIZE summary was taken on the current sources
    # (else the bench reports no traffic) and reads about the algorithmic
    # bytes: X once, plus the rows written to the cache
    t = bench.measured_traffic(name)
    assert t is not None, "counters taken on other sources than these"
    assert alg <= t <= 1.1 * alg


def test_traffic_is_withheld_when_the_sources_differ(tmp_path, monkeypatch):
    src = os.path.join(ROOT, "profiles", "k_rows_C3_hbm_counters.md")
    text = open(src).read()
    h = bench.kernel_source_hash()
    assert h in text
    fake_root = tmp_path
    (fake_root / "profiles").mkdir()
    (fake_root / "profiles" / "k_rows_C3_hbm_counters.md").write_text(
        text.replace(h, "0" * 64))
    monkeypatch.setattr(bench, "ROOT", str(fake_root))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: h)
    assert bench.measured_traffic("C3") is None
    assert bench.measured_traffic("C9") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
