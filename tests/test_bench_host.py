"""Host-side logic of bench.py (no GPU): the one-GPU refusal, the FLOP
accounting behind `value` and `roofline.achieved`, and the rule that the
reported HBM traffic is dropped once the profiled kernel's source changes."""
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2504_06949_amd import workloads  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("d", [64, 128])
def test_flop_accounting(d):
    w = workloads.custom("acct", 2, 3, 256, d, "bf16", 1)
    kept = 17
    f = bench._flops(w, kept)
    tile = 64 * 64 * d
    # dense causal fwd + bwd: 2 B H L^2 d forward (two products over half the
    # square) and 5 B H L^2 d backward (five)
    assert f["effective"] == 7 * 2 * 3 * 256 * 256 * d
    assert f["executed"] == kept * 14 * tile
    # the per-kernel algorithmic shares add up to the executed total
    assert f["fwd"] + f["dq"] + f["dkdv"] == f["executed"]
    # with every causal block kept, the executed count covers the dense causal
    # count plus the diagonal blocks' upper halves
    M = 256 // 64
    full = bench._flops(w, 2 * 3 * M * (M + 1) // 2)["executed"]
    assert full == pytest.approx(f["effective"] + 7 * 2 * 3 * M * 64 * 64 * d)


def test_traffic_follows_the_kernel_source(tmp_path, monkeypatch):
    src_dir = tmp_path / "paper_2504_06949_amd" / "csrc"
    src_dir.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    src = src_dir / "kern.hip"
    src.write_bytes(b"// kernel v1\n")
    hdr = src_dir / "acp_device.h"
    hdr.write_bytes(b"// device header v1\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    digest = bench.source_digest("kern.hip")
    assert digest == hashlib.sha1(src.read_bytes() + hdr.read_bytes()).hexdigest()[:12]
    (tmp_path / "profiles" / "k.md").write_text(
        "# summary\n\n    traffic kern 125m 123456 kern.hip:%s\n" % digest)
    assert bench.measured_traffic("kern", "125m") == 123456
    assert bench.measured_traffic("kern", "360m") is None      # no line for this workload
    assert bench.measured_traffic("other", "125m") is None
    hdr.write_bytes(b"// device header v2\n")                  # a shared header changed
    assert bench.measured_traffic("kern", "125m") is None
    hdr.write_bytes(b"// device header v1\n")
    assert bench.measured_traffic("kern", "125m") == 123456
    src.write_bytes(b"// kernel v2\n")                          # the kernel changed since
    assert bench.measured_traffic("kern", "125m") is None


def test_roofline_takes_the_longest_attention_kernel():
    w = workloads.custom("acct", 2, 3, 256, 64, "bf16", 1)
    kept = 17
    r = {"kept": kept, "per_kernel_ms": {"fwd": 1e-5, "dq": 2e-5, "dkdv": 3e-5, "rownorm": 0.5}}
    got = bench.roofline(w, r)
    assert got["kernel"] == "dkdv"          # stage-1 kernels are not candidates
    want = kept * 8 * 64 * 64 * 64 / 3e-8 / 1e12
    assert got["achieved"] == pytest.approx(want, rel=1e-3)
    assert got["frac"] == pytest.approx(want / bench.PEAK_BF16_TFLOPS, rel=1e-3)


def test_roofline_against_the_measured_clock(tmp_path, monkeypatch):
    """With a clock line for the dominant kernel, the same rate is also reported
    against the peak scaled to that clock; without one (or after the kernel's
    source changed) both fields are None."""
    src_dir = tmp_path / "paper_2504_06949_amd" / "csrc"
    src_dir.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    src = src_dir / "fox_bwd_mfma.hip"
    src.write_bytes(b"// kernel v1\n")
    digest = hashlib.sha1(src.read_bytes()).hexdigest()[:12]
    (tmp_path / "profiles" / "c.md").write_text(
        "    clock dkdv acct 1.800 fox_bwd_mfma.hip:%s\n" % digest)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    w = workloads.custom("acct", 2, 3, 256, 64, "bf16", 1)
    r = {"kept": 17, "per_kernel_ms": {"fwd": 1e-5, "dq": 2e-5, "dkdv": 3e-5}}
    got = bench.roofline(w, r)
    assert got["clock_ghz"] == pytest.approx(1.8)
    assert got["frac_at_clock"] == pytest.approx(got["frac"] * 2.4 / 1.8, rel=1e-3)
    src.write_bytes(b"// kernel v2\n")
    got = bench.roofline(w, r)
    assert got["clock_ghz"] is None and got["frac_at_clock"] is None


def test_step_fraction_at_the_kernels_clock(tmp_path, monkeypatch):
    """The step's executed rate is scaled by the attention kernels' clocks weighted
    by their times; a missing clock line gives None."""
    src_dir = tmp_path / "paper_2504_06949_amd" / "csrc"
    src_dir.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    lines = []
    for name in ("fox_fwd.hip", "fox_bwd_mfma.hip"):
        (src_dir / name).write_bytes(b"// " + name.encode() + b"\n")
    dg = {n: hashlib.sha1((src_dir / n).read_bytes()).hexdigest()[:12]
          for n in ("fox_fwd.hip", "fox_bwd_mfma.hip")}
    lines.append("    clock fwd acct 2.000 fox_fwd.hip:%s" % dg["fox_fwd.hip"])
    lines.append("    clock dq acct 1.800 fox_bwd_mfma.hip:%s" % dg["fox_bwd_mfma.hip"])
    (tmp_path / "profiles" / "c.md").write_text("\n".join(lines) + "\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    w = workloads.custom("acct", 2, 3, 256, 64, "bf16", 1)
    pk = {"fwd": 1.0, "dq": 1.0, "dkdv": 2.0}
    assert bench.frac_at_step_clock(w, pk, 1000.0) is None          # no dK/dV clock yet
    with open(tmp_path / "profiles" / "c.md", "a") as f:
        f.write("    clock dkdv acct 1.600 fox_bwd_mfma.hip:%s\n" % dg["fox_bwd_mfma.hip"])
    clk = (1.0 * 2.0 + 1.0 * 1.8 + 2.0 * 1.6) / 4.0
    assert bench.frac_at_step_clock(w, pk, 1000.0) == pytest.approx(
        1000.0 / (bench.PEAK_BF16_TFLOPS * clk / 2.4), rel=1e-3)
