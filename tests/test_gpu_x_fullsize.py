"""Parity at the benchmark's full sizes, in the configuration bench.py times.

The GPU runs the first iterations of each large workload exactly as bench.py
does (same data, start, step size and product form); the fp64 oracle runs the
same iterations on the full arrays (with the GPU's dual-gate decisions
replayed) and, in one-step mode, one iteration from the GPU's own iterate.
Every entry of U is compared, not a sample: max_ij |U_gpu - U_ref| / max|U_ref|.
Labels must agree on every row whose reference top-2 gap is not within
rounding.  Each case needs about 20-40 GB of host memory and a minute of CPU.
"""
import gc

import numpy as np
import pytest

from gpu_util import OBJ_TOL, U_TOL, host, label_agreement, log, make_ctx, obj_rel_err, rel_max_err
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


# (workload, flags): the bench's product form for each shape (split where supported)
CASES = [("gmm10m", SPLIT), ("gmm10m", 0), ("gmm50m", 0), ("embed2m", SPLIT), ("embed2m", 0)]


@pytest.mark.parametrize("workload,flags", CASES)
def test_full_size_parity(workload, flags):
    import torch
    T = 2
    X, Z, _, wl = make_workload(workload)
    K = wl.K
    alpha = onlr.default_step_size(K)
    log(f"full size {workload} n={wl.n} d={wl.d} r={wl.r} flags={flags}: GPU")
    ctx = make_ctx(X, Z, K, alpha, 1.0, T_min=T, flags=flags)
    a_gpu, _ = ctx.normaliser()
    stats = []
    for t in range(T - 1):
        stats.append(ctx.step())
    U_prev = host(ctx.U)
    y_prev = host(ctx.y)
    stats.append(ctx.step())
    U_gpu = host(ctx.U)
    y_gpu = host(ctx.y)
    labels = ctx.labels().cpu().numpy()
    ctx.close()
    del ctx
    torch.cuda.empty_cache()
    gates = [bool(s["dual_step"]) for s in stats]

    log("  oracle: normalisation")
    Xh, _, a_ref = onlr.centre_and_normalise(X)
    del X
    gc.collect()
    assert abs(a_gpu / a_ref - 1.0) < 1e-9, (a_gpu, a_ref)
    log("  oracle: trajectory")
    ref = onlr.run(Xh, Z.astype(np.float64), K, alpha, 1.0, T=T, T_min=T, gates=gates)
    traj = rel_max_err(U_gpu, ref.U)
    objs = [obj_rel_err(stats[t]["objective"], ref.records[t].objective, 1.0) for t in range(T)]
    log("  oracle: one step from the GPU iterate")
    one = onlr.run(Xh, U_prev, K, alpha, 1.0, T=1, T_min=1, project_init=False,
                   y0=onlr.dual_from_stored(y_prev), gates=[gates[-1]])
    one_err = rel_max_err(U_gpu, one.U)
    y_ref = onlr.stored_dual(one.y)
    y_err = float(np.abs(y_gpu - y_ref).max()) if y_ref.size else 0.0
    bad, amb = label_agreement(labels, ref.U)
    log(f"  traj {traj:.2e} one-step {one_err:.2e} obj {max(objs):.2e} y {y_err:.2e} "
        f"labels {bad} bad / {amb} ambiguous")
    assert traj < U_TOL
    assert one_err < U_TOL / 10
    assert max(objs) < OBJ_TOL
    assert y_err <= 1e-5 * max(1e-12, float(np.abs(y_ref).max())) + 1e-12
    assert bad == 0
