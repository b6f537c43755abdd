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


@pytest.mark.parametrize("d,r,split,two_pass,form", [
    (128, 64, True, False, "one-pass"), (97 + 3, 36, True, False, "one-pass"),
    (128, 64, False, False, "single-Xhat-pass"), (64, 16, True, False, "single-Xhat-pass"),
    (96, 64, True, False, "single-Xhat-pass"), (128, 32, True, False, "single-Xhat-pass"),
    (128, 64, True, True, "two-pass")])
def test_iteration_form(d, r, split, two_pass, form):
    assert bench.iteration_form(d, r, split, two_pass) == form


def test_traffic_record_matches_the_sources():
    t = bench.load_traffic("pass_bf_split16", "gmm10m")
    assert t is not None, "the committed traffic record no longer matches the kernel sources"
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic_pass_bf_split16_gmm10m.json")))
    assert rec["kernel_source_hash"] == bench.kernel_source_hash("pass_bf_split16")
    assert 0.99 < rec["bytes_per_launch"] / rec["algorithmic_bytes_per_launch"] < 1.05
    assert bench.load_traffic("pass_bf_split16", "no-such-workload") is None
