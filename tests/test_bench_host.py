"""Host logic of bench.py (no GPU): the one-GPU guard, the roofline arithmetic, the
algorithmic byte counts of the HBM-bound entry points, and the gating of the
committed byte-counter summaries on the kernel sources they were taken from."""
import os
import subprocess
import sys

import bench
from paper_2609_36314_amd.workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_roofline_arithmetic():
    r = bench.roofline("hbm", 8e9, 2.0, bench.PEAK_HBM_BYTES, "GB/s")
    assert abs(r["achieved"] - 4000.0) < 1e-9 and abs(r["frac"] - 0.5) < 1e-12 and r["peak"] == 8000.0


def test_compulsory_bytes_of_the_paper_shape():
    w = WORKLOADS["paper-nfree-train-b8-l2048"]
    n = 8 * 2048 * 16
    assert bench.nfree_fwd_bytes(w) == n * (2 * 256 * 2 + 4)
    assert bench.nfree_bwd_bytes(w) == n * (3 * 256 * 2 + 8)
    d = WORKLOADS["paper-nfree-decode-b2048-128steps"]
    state = 2048 * 16 * 16 * 256 * 4
    assert bench.decode_bytes_per_step(d) == 2 * state + 2048 * 16 * 256 * 2 * 2 + 2048 * 16 * 4


def test_traffic_is_reported_only_for_the_sources_it_was_measured_on(monkeypatch):
    got = bench.measured_traffic("frac_scan_bwd", "train-b4-l4096-m8")
    assert got is None or got > 1e8
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.measured_traffic("frac_scan_bwd", "train-b4-l4096-m8") is None
    assert bench.measured_traffic("frac_scan_bwd", "no-such-workload") is None


def test_mfma_busy_is_reported_only_for_the_sources_it_was_measured_on(monkeypatch):
    got = bench.measured_mfma_busy("frac_scan_bwd", "train-b4-l4096-m8")
    if got is not None:  # the backward's sweeps, each a share of the SIMD cycles
        assert any(k.startswith("frac_bwd_state_kernel") for k in got)
        assert all(0.0 <= v <= 1.0 for v in got.values())
        assert not any(k.startswith("frac_fwd_kernel") for k in got)
    assert bench.measured_mfma_busy("frac_decode_step", "decode-b256-128steps") is None
    assert bench.measured_mfma_busy("frac_scan_bwd", "no-such-workload") is None
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.measured_mfma_busy("frac_scan_bwd", "train-b4-l4096-m8") is None
