"""Host-side parts of bench.py (no GPU): the one-GPU refusal, the algorithmic bytes of the
benchmark's launch, and the counter summary that is used only while it matches the kernel sources."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from workloads import CONFIGS  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes_of_the_benchmark_launch():
    # hidden states 32768 x 7168 and router 256 x 7168 in bf16, then the selection bias, the
    # expert-to-rank table and the counts (E words each), the rank loads and max/mean
    wl = CONFIGS["dsv3"]
    assert bench.algorithmic_bytes(wl) == (32768 * 7168 + 256 * 7168) * 2 + 256 * 4 * 3 + 32 * 4 + 8
    assert bench.algorithmic_bytes(wl) == 473435272


def test_counter_traffic_is_used_only_for_the_current_sources(tmp_path, monkeypatch):
    prof = tmp_path / "counters.txt"
    monkeypatch.setattr(bench, "PROFILE_COUNTERS", str(prof))
    assert bench.traffic_from_profile() is None                      # no summary
    prof.write_text(f"# a comment: 1\nkernel_source_sha256_16: {bench.kernel_source_hash()}\n"
                    "hbm_bytes_per_launch: 499928858\n")
    assert bench.traffic_from_profile() == 499928858
    prof.write_text("kernel_source_sha256_16: 0000000000000000\nhbm_bytes_per_launch: 499928858\n")
    assert bench.traffic_from_profile() is None                      # taken on other sources


def test_the_committed_counter_summary_names_a_source_hash_and_its_traffic():
    with open(bench.PROFILE_COUNTERS) as f:
        rec = dict(l.split(":", 1) for l in f if ":" in l and not l.startswith("#"))
    assert len(rec["kernel_source_sha256_16"].strip()) == 16
    assert int(rec["hbm_bytes_per_launch"].strip()) > bench.algorithmic_bytes(CONFIGS["dsv3"])
