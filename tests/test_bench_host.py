"""bench.py's host logic on the CPU: the one-GPU rule, the algorithmic byte counts
the roofline divides by, the iteration form it names, and the traffic record it
reads only while the kernel sources are those it was measured on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "exactly one GPU" in res.stderr
    assert res.stdout == ""


def test_algorithmic_bytes_per_point():
    n, d, r = 10_000_000, 128, 64
    # the one-pass kernel moves X, U in, W out and ytilde: 4 (nd + 2nr + n) = 10.28 GB
    assert bench.algorithmic_bytes("pass_bf", n, d, r) == 4.0 * (n * d + 2 * n * r + n) == 1.028e10
    # the fixed numerator of the effective rate: two passes, 4 (2d + 3r + 2) = 1,800 B per point
    assert bench.algorithmic_bytes("step", n, d, r) / n == 1800.0
    assert bench.algorithmic_bytes("pass_u", n, d, r, dual_frac=1.0) == 4.0 * (n * r + 2 * n)
    with pytest.raises(ValueError):
        bench.algorithmic_bytes("nonsense", n, d, r)


@pytest.mark.parametrize("name,n,d,r,split,two_pass,form", [
    ("tiny", 2_000, 16, 4, True, False, "one-pass"),
    ("tiny fp32", 2_000, 16, 4, False, False, "single-Xhat-pass"),
    ("gmm1m", 1_000_000, 64, 16, True, False, "one-pass"),
    ("d=64 r=20", 100_000, 64, 20, True, False, "single-Xhat-pass"),
    ("gmm10m", 10_000_000, 128, 64, True, False, "one-pass"),
    ("gmm10m fp32", 10_000_000, 128, 64, False, False, "single-Xhat-pass"),
    ("gmm10m two-pass", 10_000_000, 128, 64, True, True, "two-pass"),
    ("gmm50m", 50_000_000, 32, 10, True, False, "one-pass"),
    ("d=32 r=18", 100_000, 32, 18, True, False, "single-Xhat-pass"),
    ("embed2m", 2_000_000, 768, 256, True, False, "two-pass-panel"),
    ("embed2m fp32", 2_000_000, 768, 256, False, False, "two-pass"),
    ("d=100 r=36", 100_000, 100, 36, True, False, "one-pass"),
    ("d=96", 100_000, 96, 64, True, False, "single-Xhat-pass"),
    ("r=32", 100_000, 128, 32, True, False, "single-Xhat-pass"),
    ("Table 2 d=50 fp32", 100_000, 50, 30, False, False, "single-Xhat-pass"),
    ("d=110 fp32", 100_000, 110, 32, False, False, "single-Xhat-pass"),
    ("d=51 fp32", 100_000, 51, 30, False, False, "two-pass"),
    ("Table 2 d=200 r=300 fp32", 100_000, 200, 300, False, False, "two-pass"),
])
def test_iteration_form_comes_from_the_library(name, n, d, r, split, two_pass, form):
    assert bench.iteration_form(n, d, r, r, split, two_pass) == form


def test_iteration_form_rejects_unsupported_shapes():
    with pytest.raises(ValueError):
        bench.iteration_form(100_000, 50, 30, 20, True, False)  # split needs d % 4 == 0 (panel: d % 8)
    with pytest.raises(ValueError):
        bench.iteration_form(100_000, 128, 512, 64, False, False)  # r above the compiled family (448)


def test_physical_rate_counts_the_launched_kernels():
    """achieved_hbm_gbs divides the bytes of the launched row and pass kernels, not the fixed
    two-pass numerator (which the one-pass form does not move)."""
    n, d, r = 10_000_000, 128, 64
    kinfo = {"pass_bf": {"launches": 50}, "pass_u": {"launches": 1}, "finish": {"launches": 1},
             "ctl_b": {"launches": 100}}
    moved = bench.iteration_bytes(kinfo, n, d, r)
    assert moved == 50 * 4.0 * (n * d + 2 * n * r + n) + 4.0 * (n * r + n) + 4.0 * (2 * n * r + n)
    assert moved < 0.6 * 50 * bench.algorithmic_bytes("step", n, d, r)
    two = {"pass_a": {"launches": 50}, "pass_b": {"launches": 50}, "finish": {"launches": 1}}
    assert bench.iteration_bytes(two, n, d, r) == pytest.approx(
        50 * bench.algorithmic_bytes("step", n, d, r) + 4.0 * (2 * n * r + n))


def test_traffic_record_follows_the_sources():
    """A traffic record is read only while the kernel sources hash to what it was measured on."""
    path = os.path.join(ROOT, "profiles", "traffic_pass_bf_split16_gmm10m.json")
    rec = json.load(open(path))
    assert 0.99 < rec["bytes_per_launch"] / rec["algorithmic_bytes_per_launch"] < 1.05
    t = bench.load_traffic("pass_bf_split16", "gmm10m")
    if rec["kernel_source_hash"] == bench.kernel_source_hash("pass_bf_split16"):
        assert t == rec["bytes_per_launch"]
    else:
        assert t is None
    assert bench.load_traffic("pass_bf_split16", "no-such-workload") is None
