"""Host-side logic around the library (CPU only): the benchmark's contract
checks, its counter-summary guard, and the build/smoke entry module."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_bench_refuses_more_than_one_gpu():
    # One GPU only: the request for more exits with status 2 and says why,
    # before anything touches a device.
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_bench_traffic_is_tied_to_the_kernel_source(tmp_path, monkeypatch):
    import bench
    # The committed summary names the digest of the kernel source it was
    # measured on; a summary for any other source is not used.
    got = bench.measured_traffic()
    assert got is None or got > 0
    fake = tmp_path / "traffic.txt"
    fake.write_text("source_sha256_16: 0000000000000000\nhbm_bytes_per_launch: 123\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(fake))
    assert bench.measured_traffic() is None
    fake.write_text(f"source_sha256_16: {bench.source_digest(bench.TRAFFIC_SOURCE)}\n"
                    "hbm_bytes_per_launch: 123\n")
    assert bench.measured_traffic() == 123
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.txt"))
    assert bench.measured_traffic() is None
    # the decode GEMM's summary is tied to the decode kernel's source the same way
    dec = bench.measured_traffic(bench.DECODE_TRAFFIC_FILE, bench.DECODE_TRAFFIC_SOURCE,
                                 "traffic_over_algorithmic")
    assert dec is None or 0.9 < dec < 3.0
    assert bench.measured_traffic(str(fake), bench.DECODE_TRAFFIC_SOURCE,
                                  "traffic_over_algorithmic") is None


def test_entry_module_has_build_and_smoke():
    import __graft_entry__ as g
    assert callable(g.build) and callable(g.smoke)


def test_h28_shared_partial_sums_match_in_order_sums(tmp_path):
    # The kernels' 28-point stage shares partial sums between columns; a host
    # build of that routine must give the in-order sums bit for bit.
    import shutil
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = tmp_path / "h28_check"
    src = os.path.join(ROOT, "tests", "h28_prefix_check.cpp")
    csrc = os.path.join(ROOT, "paper_2606_12487_amd", "csrc")
    r = subprocess.run([hipcc, "-O2", "-std=c++20", "-ffp-contract=off", f"-I{csrc}", "-x", "hip",
                        "--offload-arch=gfx950", src, "-o", str(exe)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "28 columns 0," in run.stdout
