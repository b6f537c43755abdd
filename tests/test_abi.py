"""The C ABI on the CPU: the library loads, exports every symbol include/nlr.h
declares, and rejects bad arguments before any HIP call."""
import ctypes
import os
import re

import pytest

from paper_2609_36074_amd import nlr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "nlr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\**\s*(nlr_[a-z_]+)\s*\(", src, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    return nlr.load_library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 14, names
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(nlr.EXPORTED) == names


def test_version_and_status_strings(lib):
    assert lib.nlr_version().decode().startswith("nlr-gfx950")
    for s in range(9):
        assert lib.nlr_status_string(s).decode() != "unknown status"
    assert lib.nlr_status_string(99).decode() == "unknown status"


def test_workspace_holds_no_factor_copy(lib):
    """Section 4.4 (eq. gpu-storage): besides Xhat, one n x r factor and the stored dual, the
    workspace holds partial sums and init temporaries only -- far below one n x r fp32 factor
    (a second factor buffer would make it exceed 1.0)."""
    for n, d, r in [(1_000_000, 64, 16), (10_000_000, 128, 64), (50_000_000, 32, 10),
                    (2_000_000, 768, 256)]:
        assert nlr.nlr_workspace_bytes(n, d, r) < 0.5 * n * r * 4, (n, d, r)
    assert nlr.nlr_workspace_bytes(10_000_000, 128, 64) < 64 << 20


def test_workspace_bytes(lib):
    a = nlr.nlr_workspace_bytes(10_000_000, 128, 64)
    assert a > 0 and a == nlr.nlr_workspace_bytes(10_000_000, 128, 64)
    assert nlr.nlr_workspace_bytes(2000, 16, 4) > 0
    assert nlr.nlr_workspace_bytes(0, 16, 4) == 0       # n < 1
    assert nlr.nlr_workspace_bytes(100, 0, 4) == 0      # d < 1
    assert nlr.nlr_workspace_bytes(100, 16, 0) == 0     # r < 1
    assert nlr.nlr_workspace_bytes(3, 16, 4) == 0       # r > n
    assert nlr.nlr_workspace_bytes(1000, 16, 449) == 0  # r above the kernel family
    assert nlr.nlr_workspace_bytes(1000, 16, 448) > 0 and nlr.nlr_workspace_bytes(1000, 200, 300) > 0
    assert nlr.nlr_workspace_bytes(1000, 4097, 4) == 0  # d above the limit


FAKE = 1 << 20  # a 256-aligned address that is never dereferenced: every call below fails validation first


def _init(lib, X=FAKE, n=1000, d=16, K=4, r=4, U=FAKE, y=FAKE, params=None, flags=0, ws=FAKE, ws_bytes=None):
    if params is None:
        params = nlr.NlrParams(0.01, 1.0, 1e-4, 1e-4, 0, 0)
    if ws_bytes is None:
        ws_bytes = nlr.nlr_workspace_bytes(n, d, r) if r <= 448 else 1 << 30
    ctx = ctypes.c_void_p(123)
    st = lib.nlr_init(ctypes.byref(ctx), X, n, d, K, r, U, y, ctypes.byref(params), flags, ws, ws_bytes, None)
    return st, ctx


def test_init_argument_errors(lib):
    P = nlr.NlrParams
    assert _init(lib, X=None)[0] == nlr.NLR_EINVAL
    assert _init(lib, U=None)[0] == nlr.NLR_EINVAL
    assert _init(lib, y=None)[0] == nlr.NLR_EINVAL
    assert _init(lib, K=0)[0] == nlr.NLR_EINVAL
    assert _init(lib, K=5, r=4)[0] == nlr.NLR_EINVAL            # K > r
    assert _init(lib, n=3, r=4, K=2)[0] == nlr.NLR_EINVAL       # r > n
    assert _init(lib, d=0)[0] == nlr.NLR_EINVAL
    assert _init(lib, r=449, K=4, n=3000)[0] == nlr.NLR_EUNSUPPORTED
    assert _init(lib, params=P(0.0, 1.0, 1e-4, 1e-4, 0, 0))[0] == nlr.NLR_EINVAL      # alpha <= 0
    assert _init(lib, params=P(float("inf"), 1.0, 1e-4, 1e-4, 0, 0))[0] == nlr.NLR_EINVAL
    assert _init(lib, params=P(0.1, -1.0, 1e-4, 1e-4, 0, 0))[0] == nlr.NLR_EINVAL     # beta <= 0
    assert _init(lib, params=P(0.1, 1.0, -1.0, 1e-4, 0, 0))[0] == nlr.NLR_EINVAL      # eps_d < 0
    assert _init(lib, params=P(0.1, 1.0, 1e-4, float("nan"), 0, 0))[0] == nlr.NLR_EINVAL
    assert _init(lib, params=P(0.1, 1.0, 1e-4, 1e-4, -1, 0))[0] == nlr.NLR_EINVAL     # T_min < 0
    assert _init(lib, flags=1 << 7)[0] == nlr.NLR_EINVAL
    assert _init(lib, X=FAKE + 2)[0] == nlr.NLR_EINVAL                                  # misaligned
    assert _init(lib, ws=None)[0] == nlr.NLR_EWORKSPACE
    assert _init(lib, ws=FAKE + 64)[0] == nlr.NLR_EWORKSPACE                           # not 256-aligned
    st, ctx = _init(lib, ws_bytes=1024)
    assert st == nlr.NLR_EWORKSPACE and ctx.value is None
    # split-fp16 products: shapes and alignments outside the supported set
    S = nlr.NLR_INIT_SPLIT_F16
    assert _init(lib, flags=S, d=13)[0] == nlr.NLR_EUNSUPPORTED                      # d % 4 != 0
    assert _init(lib, flags=S, d=132)[0] == nlr.NLR_EUNSUPPORTED                     # d > 128, d % 8 != 0
    assert _init(lib, flags=S, d=136, r=10, K=4)[0] == nlr.NLR_EUNSUPPORTED          # d > 128, r % 4 != 0
    assert _init(lib, flags=S, r=66, K=4)[0] == nlr.NLR_EUNSUPPORTED                 # r > 64, r % 4 != 0
    assert _init(lib, flags=S | nlr.NLR_INIT_TWO_PASS, r=10, K=4)[0] == nlr.NLR_EUNSUPPORTED  # r % 4 != 0
    # panel form (d > 128 or r > 64 with d % 8 == 0, r % 4 == 0): supported, reaches the workspace check
    for kw in (dict(d=136), dict(r=68, K=4), dict(d=768, r=256, K=256, n=3000)):
        st, ctx = _init(lib, flags=S, ws_bytes=1024, **kw)
        assert st == nlr.NLR_EWORKSPACE and ctx.value is None, kw
    st, _ = _init(lib, flags=S, r=10, K=4, ws_bytes=1024)                            # single pass: fine
    assert st == nlr.NLR_EWORKSPACE
    assert _init(lib, flags=S, X=FAKE + 4)[0] == nlr.NLR_EUNSUPPORTED                # X not 16-byte aligned
    assert _init(lib, flags=S, U=FAKE + 8)[0] == nlr.NLR_EUNSUPPORTED                # U not 16-byte aligned
    assert _init(lib, flags=nlr.NLR_INIT_DATA_START | nlr.NLR_INIT_U_IN_OMEGA)[0] == nlr.NLR_EINVAL
    st, ctx = _init(lib, flags=S, ws_bytes=1024)                                      # supported: reaches the
    assert st == nlr.NLR_EWORKSPACE and ctx.value is None                            # workspace check


def test_null_context_calls(lib):
    assert lib.nlr_step(None, None) == nlr.NLR_EINVAL
    assert lib.nlr_run(None, 5, None, None) == nlr.NLR_EINVAL
    assert lib.nlr_labels(None, FAKE) == nlr.NLR_EINVAL
    assert lib.nlr_set_params(None, None) == nlr.NLR_EINVAL
    assert lib.nlr_set_profiling(None, 1) == nlr.NLR_EINVAL
    lib.nlr_destroy(None)  # no-op


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="missing"):
        # a fresh loader pointed at a path with no library
        saved = nlr._lib
        nlr._lib = None
        try:
            nlr.load_library(str(tmp_path / "libnlr.so"))
        finally:
            nlr._lib = saved


def test_solve_static_rejects_before_any_hip_call(lib):
    """The allocation-free entry point checks its arguments as nlr_init does, and rejects shapes
    whose workspace exceeds its fixed device scratch with NLR_EWORKSPACE (no GPU needed)."""
    p = nlr.NlrParams(0.01, 1.0, 1e-4, 1e-4, 0, 0)
    assert nlr.nlr_workspace_bytes(10_000_000, 128, 64) <= nlr.NLR_STATIC_SCRATCH_BYTES
    assert nlr.nlr_workspace_bytes(2_000_000, 768, 256) > nlr.NLR_STATIC_SCRATCH_BYTES
    st, done, _ = nlr.nlr_solve_static(FAKE, 2_000_000, 768, 256, 256, FAKE, FAKE, p, 0, 5)
    assert st == nlr.NLR_EWORKSPACE and done == 0
    assert nlr.nlr_solve_static(FAKE, 1000, 16, 4, 4, FAKE, FAKE, p, 0, -1)[0] == nlr.NLR_EINVAL
    assert nlr.nlr_solve_static(0, 1000, 16, 4, 4, FAKE, FAKE, p, 0, 5)[0] == nlr.NLR_EINVAL
    assert nlr.nlr_solve_static(FAKE, 1000, 16, 4, 449, FAKE, FAKE, p, 0, 5)[0] == nlr.NLR_EUNSUPPORTED
    assert nlr.nlr_solve_static(FAKE, 1000, 16, 8, 16, FAKE + 4, FAKE, p, nlr.NLR_INIT_SPLIT_F16, 5)[0] == \
        nlr.NLR_EUNSUPPORTED
