"""Host-side logic of bench.py (no GPU): the one-GPU guard, and the rule that
the measured HBM traffic is reported only for the kernel sources it was
measured on."""

from __future__ import annotations

import ctypes
import os
import subprocess
import sys

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _summary(tmp_path, digest, bwd=207427397, fwd=138284931):
    p = tmp_path / "traffic.md"
    p.write_text("# traffic\n\nsome text: not a field\n\n"
                 "- source_sha256: `%s`\n"
                 "- traffic_bytes_per_launch.iabn_backward: %d\n"
                 "- traffic_bytes_per_launch.iabn_forward_train: %d\n" % (digest, bwd, fwd))
    return str(p)


def test_traffic_reported_for_matching_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARIES", {5: _summary(tmp_path, bench.kernel_source_digest())})
    assert bench.measured_traffic("iabn_backward", 5) == 207427397
    assert bench.measured_traffic("iabn_forward_train", 5) == 138284931
    assert bench.measured_traffic("iabn_forward_eval", 5) is None
    # Only the workloads the counters were taken on.
    assert bench.measured_traffic("iabn_backward", 2) is None
    assert bench.measured_traffic("iabn_backward", 0) is None


def test_traffic_withheld_for_other_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARIES", {5: _summary(tmp_path, "0" * 64)})
    assert bench.measured_traffic("iabn_backward", 5) is None
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARIES", {5: str(tmp_path / "missing.md")})
    assert bench.measured_traffic("iabn_backward", 5) is None


def test_traffic_summaries_cover_the_single_gpu_workloads():
    for c in (2, 3, 4, 5):
        assert c in bench.TRAFFIC_SUMMARIES
        assert bench.TRAFFIC_SUMMARIES[c].endswith("_hbm_traffic.md")


def test_source_digest_covers_kernels_and_header():
    d = bench.kernel_source_digest()
    assert len(d) == 64 and d == bench.kernel_source_digest()


def test_probe_library_validates_before_launching():
    """The bandwidth probes' C entry point rejects bad arguments on the host
    (no launch, so this runs without a GPU)."""
    probe = bench.load_probe()
    a = ctypes.c_void_p(1 << 20)
    assert probe.iabn_probe_launch(0, a, a, 0, 1024, 0, a, None) == 1      # no bytes
    assert probe.iabn_probe_launch(2, a, a, 24, 1024, 0, a, None) == 1     # not a multiple of 16
    assert probe.iabn_probe_launch(9, a, a, 4096, 1024, 0, a, None) == 1   # unknown mix
    assert probe.iabn_probe_launch(2, a, None, 4096, 1024, 0, a, None) == 1  # the mix needs b
    assert probe.iabn_probe_launch(1, ctypes.c_void_p((1 << 20) + 8), None, 4096, 1024, 0, None,
                                   None) == 1                              # misaligned
    assert probe.iabn_probe_launch(1, a, None, 4096, 0, 0, None, None) == 1  # no blocks


def test_timing_event_flag_matches_the_hip_header():
    """TimingEvent's flag is the HIP runtime's hipEventDisableSystemFence (read
    from the installed header where there is one)."""
    import re
    header = "/opt/rocm/include/hip/hip_runtime_api.h"
    if not os.path.exists(header):
        pytest.skip("no HIP header")
    m = re.search(r"#define\s+hipEventDisableSystemFence\s+(0x[0-9a-fA-F]+)", open(header).read())
    assert m, "hipEventDisableSystemFence not in the header"
    assert bench.TimingEvent.DISABLE_SYSTEM_FENCE == int(m.group(1), 16)
