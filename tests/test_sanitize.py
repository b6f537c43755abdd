"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

nlr_api.cpp (argument checks, geometry, workspace layout, error paths) is compiled
for the host only with both sanitizers (halting on the first finding) and linked
with the library's regular kernel objects; tests/sanitize_driver.c then drives every
entry point along the paths that return before a HIP call, over extreme and invalid
sizes (n up to 2^63 - 1, d and r up to 2^31 - 1, negative values), with leak
detection on.  No GPU is used.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36074_amd", "csrc")
OBJDIR = os.path.join(ROOT, "paper_2609_36074_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"


def _tools():
    hipcc = "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else shutil.which("hipcc")
    clang = os.path.join(LLVM, "clang")
    clangxx = os.path.join(LLVM, "clang++")
    if not hipcc or not os.path.exists(clang) or not os.path.exists(clangxx):
        pytest.skip("ROCm toolchain not found")
    return hipcc, clang, clangxx


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr}"
    return res


def test_host_code_under_sanitizers(tmp_path):
    hipcc, clang, clangxx = _tools()
    kernels = ["k_iter", "k_init", "k_split", "k_fused", "k_start", "k_labels", "k_panel"]
    if not all(os.path.exists(os.path.join(OBJDIR, k + ".o")) for k in kernels):
        from paper_2609_36074_amd import _build
        _build.build()
    api_o = str(tmp_path / "nlr_api.o")
    # host-side instrumentation only: each sanitizer flag applies to the host pass (the device
    # pass compiles the file's device array without any)
    _run([hipcc, "-xhip", "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
          "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-Xarch_host", "-fno-sanitize-recover=all",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c", os.path.join(CSRC, "nlr_api.cpp"), "-o", api_o])
    lib = str(tmp_path / "libnlr_san.so")
    san = "-fsanitize=" + ",".join(["address", "undefined"])
    _run([clangxx, "-shared", "-fPIC", san, "-o", lib, api_o,
          *[os.path.join(OBJDIR, k + ".o") for k in kernels],
          "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    drv = str(tmp_path / "driver")
    _run([clang, "-g", "-O1", san, "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
          "-o", drv, os.path.join(ROOT, "tests", "sanitize_driver.c"),
          "-L", str(tmp_path), "-lnlr_san", f"-Wl,-rpath,{tmp_path}", "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([drv], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all checks passed" in res.stdout
