"""Thin ctypes binding of libnlr.so (include/nlr.h).

Argument marshalling only: every step of the iteration runs in the library's
HIP kernels.  PyTorch provides device memory and the stream.  The library
must be built first (``__graft_entry__.build()``); importing this module on a
machine without it raises immediately — there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libnlr.so")

NLR_OK = 0
NLR_EINVAL = 1
NLR_EWORKSPACE = 2
NLR_EBREAKDOWN = 3
NLR_EDEGENERATE = 4
NLR_EHIP = 5
NLR_ESTATE = 6
NLR_EUNSUPPORTED = 7
NLR_ERANGE = 8

NLR_INIT_U_IN_OMEGA = 1
NLR_INIT_KEEP_Y = 2
NLR_INIT_X_NORMALISED = 4
NLR_INIT_SPLIT_F16 = 8
NLR_INIT_TWO_PASS = 16
NLR_INIT_DATA_START = 32

NLR_MAX_KERNEL_KINDS = 16

NLR_FORM_TWO_PASS = 0
NLR_FORM_PANEL = 1
NLR_FORM_SINGLE_PASS = 2
NLR_FORM_ONE_PASS = 3
FORM_NAMES = {NLR_FORM_TWO_PASS: "two-pass", NLR_FORM_PANEL: "two-pass-panel",
              NLR_FORM_SINGLE_PASS: "single-Xhat-pass", NLR_FORM_ONE_PASS: "one-pass"}

EXPORTED = ["nlr_workspace_bytes", "nlr_iteration_form", "nlr_init", "nlr_set_params", "nlr_step", "nlr_run", "nlr_labels",
            "nlr_labels_spectral",
            "nlr_history", "nlr_normaliser", "nlr_inspect", "nlr_set_profiling", "nlr_kernel_times",
            "nlr_destroy", "nlr_status_string", "nlr_version", "nlr_solve_static"]

NLR_STATIC_SCRATCH_BYTES = 64 << 20


class NlrParams(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_double), ("beta", ctypes.c_double), ("eps_d", ctypes.c_double),
                ("eps_c", ctypes.c_double), ("T_min", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class NlrIterStats(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int64), ("objective", ctypes.c_double), ("theta_fro2", ctypes.c_double),
                ("a", ctypes.c_double), ("b", ctypes.c_double), ("h", ctypes.c_double),
                ("delta", ctypes.c_double), ("rho", ctypes.c_double), ("c", ctypes.c_float),
                ("dual_step", ctypes.c_int32), ("stop", ctypes.c_int32), ("breakdown", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


class NlrError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libnlr.so.  torch is imported first so that the library binds to
    the HIP runtime torch already loaded (they share its SONAME)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build()")
    try:
        import torch  # noqa: F401  (binds the process to torch's HIP runtime)
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    P, i32, i64, u32, sz, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t, ctypes.c_double
    lib.nlr_workspace_bytes.argtypes = [i64, i32, i32]
    lib.nlr_workspace_bytes.restype = sz
    lib.nlr_iteration_form.argtypes = [i64, i32, i32, i32, u32]
    lib.nlr_iteration_form.restype = i32
    lib.nlr_solve_static.argtypes = [P, i64, i32, i32, i32, P, P, ctypes.POINTER(NlrParams), u32, i32,
                                     ctypes.POINTER(i32), ctypes.POINTER(NlrIterStats), P]
    lib.nlr_solve_static.restype = ctypes.c_int
    lib.nlr_init.argtypes = [ctypes.POINTER(P), P, i64, i32, i32, i32, P, P, ctypes.POINTER(NlrParams), u32, P, sz, P]
    lib.nlr_init.restype = ctypes.c_int
    lib.nlr_set_params.argtypes = [P, ctypes.POINTER(NlrParams)]
    lib.nlr_set_params.restype = ctypes.c_int
    lib.nlr_step.argtypes = [P, ctypes.POINTER(NlrIterStats)]
    lib.nlr_step.restype = ctypes.c_int
    lib.nlr_run.argtypes = [P, i32, ctypes.POINTER(i32), ctypes.POINTER(NlrIterStats)]
    lib.nlr_run.restype = ctypes.c_int
    lib.nlr_labels.argtypes = [P, P]
    lib.nlr_labels.restype = ctypes.c_int
    lib.nlr_labels_spectral.argtypes = [P, i32, ctypes.POINTER(i64), i32, P, ctypes.POINTER(i32)]
    lib.nlr_labels_spectral.restype = ctypes.c_int
    lib.nlr_history.argtypes = [P, ctypes.POINTER(NlrIterStats), i32, ctypes.POINTER(i32)]
    lib.nlr_history.restype = ctypes.c_int
    lib.nlr_normaliser.argtypes = [P, ctypes.POINTER(dbl), P]
    lib.nlr_normaliser.restype = ctypes.c_int
    lib.nlr_inspect.argtypes = [P, i32, P, sz]
    lib.nlr_inspect.restype = ctypes.c_int
    lib.nlr_set_profiling.argtypes = [P, i32]
    lib.nlr_set_profiling.restype = ctypes.c_int
    lib.nlr_kernel_times.argtypes = [P, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(dbl),
                                     ctypes.POINTER(i64), ctypes.POINTER(i32)]
    lib.nlr_kernel_times.restype = ctypes.c_int
    lib.nlr_destroy.argtypes = [P]
    lib.nlr_destroy.restype = None
    lib.nlr_status_string.argtypes = [ctypes.c_int]
    lib.nlr_status_string.restype = ctypes.c_char_p
    lib.nlr_version.argtypes = []
    lib.nlr_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().nlr_status_string(int(status)).decode()


def _check(status: int, where: str) -> int:
    if status != NLR_OK:
        raise NlrError(status, where)
    return status


# ---------------------------------------------------------------------------
# Functions with the C ABI's names (raw pointers / integers in, status out)
# ---------------------------------------------------------------------------
def nlr_workspace_bytes(n: int, d: int, r: int) -> int:
    return int(load_library().nlr_workspace_bytes(n, d, r))


def nlr_iteration_form(n: int, d: int, r: int, K: int, flags: int) -> int:
    return int(load_library().nlr_iteration_form(n, d, r, K, flags))


def nlr_solve_static(X_ptr: int, n: int, d: int, K: int, r: int, U_ptr: int, y_ptr: int, params: NlrParams,
                     flags: int, T: int, stream_ptr: int = 0):
    """(status, iterations done, record of the last one): the allocation-free init + run."""
    done = ctypes.c_int32(0)
    last = NlrIterStats()
    st = load_library().nlr_solve_static(X_ptr, n, d, K, r, U_ptr, y_ptr, ctypes.byref(params), flags, T,
                                         ctypes.byref(done), ctypes.byref(last), stream_ptr)
    return int(st), int(done.value), last.as_dict()


def nlr_init(X_ptr: int, n: int, d: int, K: int, r: int, U_ptr: int, y_ptr: int, params: NlrParams,
             flags: int, ws_ptr: int, ws_bytes: int, stream: int):
    """Returns (status, ctx handle)."""
    ctx = ctypes.c_void_p()
    st = load_library().nlr_init(ctypes.byref(ctx), X_ptr, n, d, K, r, U_ptr, y_ptr, ctypes.byref(params),
                                 flags, ws_ptr, ws_bytes, stream)
    return st, ctx


def nlr_step(ctx, stats: NlrIterStats | None = None) -> int:
    return load_library().nlr_step(ctx, ctypes.byref(stats) if stats is not None else None)


def nlr_run(ctx, T: int, last: NlrIterStats | None = None):
    done = ctypes.c_int32(0)
    st = load_library().nlr_run(ctx, T, ctypes.byref(done), ctypes.byref(last) if last is not None else None)
    return st, done.value


def nlr_labels(ctx, labels_ptr: int) -> int:
    return load_library().nlr_labels(ctx, labels_ptr)


def nlr_destroy(ctx) -> None:
    load_library().nlr_destroy(ctx)


# ---------------------------------------------------------------------------
# Convenience wrapper over torch tensors (still marshalling only)
# ---------------------------------------------------------------------------
class Context:
    """Owns an nlr_ctx plus the torch workspace tensor it borrows.

    X (n x d float32, contiguous, on the GPU) is normalised IN PLACE; U (n x r)
    is projected in place; y (n) is the stored dual.  All three stay the
    caller's tensors and are updated by step()/run().
    """

    def __init__(self, X, K: int, U, y=None, *, alpha: float, beta: float = 1.0, eps_d: float = 1e-4,
                 eps_c: float = 1e-4, T_min: int = 0, flags: int = 0, stream=None):
        import torch
        lib = load_library()
        for name, t in (("X", X), ("U", U)):
            if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous() and t.dim() == 2):
                raise ValueError(f"{name} must be a contiguous 2-D float32 GPU tensor")
        n, d = X.shape
        n2, r = U.shape
        if n2 != n:
            raise ValueError("X and U must have the same number of rows")
        if y is None:
            y = torch.zeros(n, dtype=torch.float32, device=X.device)
        if not (y.is_cuda and y.dtype == torch.float32 and y.is_contiguous() and y.numel() == n):
            raise ValueError("y must be a contiguous float32 GPU vector of length n")
        self.X, self.U, self.y = X, U, y
        self.n, self.d, self.r, self.K = int(n), int(d), int(r), int(K)
        ws = int(lib.nlr_workspace_bytes(n, d, r))
        if ws == 0:
            raise NlrError(NLR_EUNSUPPORTED if r > 448 else NLR_EINVAL, "nlr_workspace_bytes")
        self.workspace = torch.empty(ws + 256, dtype=torch.uint8, device=X.device)
        base = self.workspace.data_ptr()
        self._ws_ptr = (base + 255) & ~255
        self._ws_bytes = ws
        self.stream = torch.cuda.current_stream(X.device) if stream is None else stream
        self.params = NlrParams(alpha, beta, eps_d, eps_c, T_min, 0)
        st, ctx = nlr_init(X.data_ptr(), n, d, K, r, U.data_ptr(), y.data_ptr(), self.params, flags,
                           self._ws_ptr, ws, self.stream.cuda_stream)
        _check(st, "nlr_init")
        self._ctx = ctx

    # -- iteration --
    def step(self, with_stats: bool = True):
        st = NlrIterStats() if with_stats else None
        _check(nlr_step(self._ctx, st), "nlr_step")
        return st.as_dict() if st is not None else None

    def run(self, T: int):
        last = NlrIterStats()
        status, done = nlr_run(self._ctx, T, last)
        _check(status, "nlr_run")
        return done, last.as_dict()

    def set_params(self, **kw):
        for k, v in kw.items():
            setattr(self.params, k, v)
        _check(load_library().nlr_set_params(self._ctx, ctypes.byref(self.params)), "nlr_set_params")

    def labels(self, out=None):
        import torch
        if out is None:
            out = torch.empty(self.n, dtype=torch.int32, device=self.X.device)
        _check(nlr_labels(self._ctx, out.data_ptr()), "nlr_labels")
        return out

    def labels_spectral(self, K: int, seed_rows, max_iter: int = 100, out=None):
        """(labels tensor, assignment passes): spectral embedding + K-means (Appendix D)."""
        import torch
        if out is None:
            out = torch.empty(self.n, dtype=torch.int32, device=self.X.device)
        seeds = (ctypes.c_int64 * len(seed_rows))(*[int(s) for s in seed_rows])
        passes = ctypes.c_int32(0)
        _check(load_library().nlr_labels_spectral(self._ctx, int(K), seeds, int(max_iter), out.data_ptr(),
                                                  ctypes.byref(passes)), "nlr_labels_spectral")
        return out, passes.value

    # -- read-back --
    def history(self, max_records: int = 4096):
        buf = (NlrIterStats * max_records)()
        cnt = ctypes.c_int32(0)
        _check(load_library().nlr_history(self._ctx, buf, max_records, ctypes.byref(cnt)), "nlr_history")
        return [buf[i].as_dict() for i in range(cnt.value)]

    def normaliser(self):
        import numpy as np
        a = ctypes.c_double(0.0)
        xbar = np.zeros(self.d, dtype=np.float64)
        _check(load_library().nlr_normaliser(self._ctx, ctypes.byref(a), xbar.ctypes.data), "nlr_normaliser")
        return a.value, xbar

    def inspect(self, what: str):
        import numpy as np
        if what == "rows_run":
            v = ctypes.c_int64(0)
            _check(load_library().nlr_inspect(self._ctx, 3, ctypes.byref(v), 8), "nlr_inspect")
            return int(v.value)
        if what == "theta":
            out = np.zeros((self.d, self.r), dtype=np.float32)
            code = 0
        elif what in ("p", "s"):
            out = np.zeros(self.r, dtype=np.float32)
            code = 1 if what == "p" else 2
        else:
            raise ValueError(what)
        _check(load_library().nlr_inspect(self._ctx, code, out.ctypes.data, out.nbytes), "nlr_inspect")
        return out

    def set_profiling(self, enable):
        """False/0 off, True/1 every launch, 2 the row and pass kernels only."""
        level = int(enable) if not isinstance(enable, bool) else (1 if enable else 0)
        _check(load_library().nlr_set_profiling(self._ctx, level), "nlr_set_profiling")

    def kernel_times(self):
        names = (ctypes.c_char_p * NLR_MAX_KERNEL_KINDS)()
        ms = (ctypes.c_double * NLR_MAX_KERNEL_KINDS)()
        cnt = (ctypes.c_int64 * NLR_MAX_KERNEL_KINDS)()
        nk = ctypes.c_int32(0)
        _check(load_library().nlr_kernel_times(self._ctx, names, ms, cnt, ctypes.byref(nk)), "nlr_kernel_times")
        return {names[k].decode(): (ms[k], cnt[k]) for k in range(nk.value)}

    def close(self):
        if getattr(self, "_ctx", None):
            nlr_destroy(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
