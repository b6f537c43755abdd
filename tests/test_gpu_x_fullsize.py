"""Parity at the benchmark's full sizes, in the configuration bench.py times.

The GPU runs the first iterations of each large workload as bench.py does (same data,
start, step size, tolerances and product form: split products in the form the library
picks, one-pass at 1e7 x 128 x 64, single-Xhat-pass with whole-slab U moves at
5e7 x 32 x 10, the panel form at 2e6 x 768 x 256): ten iterations with split products
and, from the same start, two with fp32 products (bench.py's "alt"), one host call per
iteration so that every iterate is read back.  The fp64 oracle then runs the same
iterations on the full arrays (the GPU's dual-gate decisions replayed) and one
iteration from each of the GPU's own iterates, in worker processes.  Every entry of U
is compared, not a sample: max_ij |U_gpu - U_ref| / max|U_ref|.  Labels must agree on
every row whose reference top-2 gap is not within rounding.  One case forces dual
steps at the headline shape (eps_d above the movement) so that the stored-dual path
runs at full size.  Each case needs about 60-100 GB of host memory.
"""
import gc

import numpy as np
import pytest

from gpu_util import OBJ_TOL, U_TOL, lockstep_parallel, log, make_ctx
from oracle import nlr as onlr
from synth import make_workload

pytestmark = pytest.mark.gpu

SPLIT = 8  # NLR_INIT_SPLIT_F16


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _run(workload, plan, eps_d):
    """plan: {name: (flags, T)}; returns the harness results per name."""
    import torch
    X, Z, _, wl = make_workload(workload)
    K = wl.K
    alpha = onlr.default_step_size(K)
    log(f"full size {workload} n={wl.n} d={wl.d} r={wl.r} eps_d={eps_d}: {plan}")
    ctxs = {s: make_ctx(X, Z, K, alpha, 1.0, eps_d=eps_d, eps_c=1e-4, T_min=T, flags=f)
            for s, (f, T) in plan.items()}
    Xh, _, a_ref = onlr.centre_and_normalise(X)
    del X
    gc.collect()
    for s, c in ctxs.items():
        a_gpu, _ = c.normaliser()
        assert abs(a_gpu / a_ref - 1.0) < 1e-9, (s, a_gpu, a_ref)
    U0 = onlr.project_omega(Z.astype(np.float64), K)
    del Z
    res = lockstep_parallel({s: (ctxs[s], T) for s, (_, T) in plan.items()}, Xh, U0, K, alpha, 1.0, eps_d)
    for c in ctxs.values():
        c.close()
    del ctxs, Xh, U0
    gc.collect()
    torch.cuda.empty_cache()
    for s, r in res.items():
        bad, amb = r["labels"]
        log(f"  {s} max: traj {max(r['traj']):.2e} one-step {max(r['one']):.2e} obj {max(r['obj']):.2e} "
            f"y {max(r['yerr']):.2e} dual steps {sum(r['gates'])}; labels {bad} bad / {amb} ambiguous")
    return res


def _check(r):
    assert max(r["traj"]) < U_TOL
    assert max(r["one"]) < U_TOL / 10
    assert max(r["obj"]) < OBJ_TOL
    assert max(r["yerr"]) <= 1e-5
    assert not r["bad_gates"], r["bad_gates"]
    assert r["labels"][0] == 0


@pytest.mark.parametrize("workload", ["gmm10m", "gmm50m", "embed2m"])
def test_full_size_parity(workload):
    res = _run(workload, {"split16": (SPLIT, 10), "fp32": (0, 2)}, 1e-4)
    for r in res.values():
        _check(r)


def test_full_size_dual_steps():
    """1e7 x 128 x 64 (one-pass form) with eps_d above the movement: dual steps from the
    second iteration on."""
    res = _run("gmm10m", {"split16": (SPLIT, 3)}, 5e-2)
    r = res["split16"]
    _check(r)
    assert sum(r["gates"]) >= 2
