"""The two smallest simulation settings of Table 2 (balanced mixture, closest centres
at CNRbar): n = 1e6 with (d, K, r) = (50, 20, 30) and (200, 100, 300).  Neither has the
split products' shapes (d % 4 != 0; r > 256), so both run fp32 products: the first in
the single-Xhat-pass form with 8-byte Xhat rows, the second in the two-pass form with the
pass B that takes the columns two blocks at a time.  Checked against
the fp64 oracle: trajectories with one-step checks on leading-row samples of the draw
(several tiles and a ragged tail) and the label recovery of Appendix D (r > K) on the
GPU's factor there, dual steps at the larger shape, and the full 1e6 rows in lockstep.
"""
import gc

import numpy as np
import pytest

from gpu_util import OBJ_TOL, U_TOL, host, label_agreement, lockstep, log, make_ctx, trajectory
from oracle import labels as olab
from oracle import nlr as onlr
from synth import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def test_table2_forms():
    from paper_2609_36074_amd import nlr
    for name, form in (("t2k20", "single-Xhat-pass"), ("t2k100", "two-pass")):
        _, _, _, wl = make_workload(name, rows=64)
        assert nlr.FORM_NAMES[nlr.nlr_iteration_form(wl.n, wl.d, wl.r, wl.K, 0)] == form
        assert nlr.nlr_iteration_form(wl.n, wl.d, wl.r, wl.K, nlr.NLR_INIT_SPLIT_F16) == -1


# (workload, leading rows, iterations)
@pytest.mark.parametrize("name,rows,T", [("t2k20", 4099, 60), ("t2k100", 3001, 30)])
def test_table2_trajectory(name, rows, T):
    X, Z, _, wl = make_workload(name, rows=rows)
    K = wl.K
    alpha = onlr.default_step_size(K)
    log(f"{name}: first {rows} rows, d={wl.d} K={K} r={wl.r}, T={T}")
    ctx, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z.astype(np.float64), K, alpha, 1.0, T,
                                                         one_step_tol=True)
    log(f"  traj {max(traj):.2e} one-step {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates
    # Appendix D label recovery (r > K) on the GPU's factor, seeded from the first K rows
    seeds = list(range(K))
    lab_gpu, passes = ctx.labels_spectral(K, seeds, 50)
    lab_ref, passes_ref = olab.spectral_labels(host(ctx.U), K, seeds, 50)
    mism = int((lab_gpu.cpu().numpy() != lab_ref).sum())
    log(f"  spectral labels: passes {passes}/{passes_ref}, {mism} mismatches")
    assert passes == passes_ref and mism == 0


def test_table2_dual_steps_wide():
    """r = 300 with eps_d above the movement after the first iterations: dual steps in
    most iterations, each gate decision the oracle's."""
    X, Z, _, wl = make_workload("t2k100", rows=3001)
    K, T, eps_d = wl.K, 12, 5e-2
    alpha = onlr.default_step_size(K)
    _, _, traj, obj, bad_gates, one, _, stats = trajectory(X, Z.astype(np.float64), K, alpha, 1.0, T,
                                                           eps_d=eps_d, one_step_tol=True)
    ngates = sum(s["dual_step"] for s in stats)
    log(f"  dual steps {ngates}; traj {max(traj):.2e} one-step {max(one):.2e}")
    assert ngates >= T - 3
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


@pytest.mark.parametrize("name,T", [("t2k20", 4), ("t2k100", 2)])
def test_table2_full_rows(name, T):
    import torch
    X, Z, truth, wl = make_workload(name)
    K = wl.K
    alpha = onlr.default_step_size(K)
    log(f"{name}: n={wl.n} d={wl.d} K={K} r={wl.r}, lockstep T={T}")
    ctx = make_ctx(X, Z, K, alpha, 1.0, T_min=T)
    Xh, _, _ = onlr.centre_and_normalise(X)
    del X
    gc.collect()
    U0 = onlr.project_omega(Z.astype(np.float64), K)
    del Z
    res = lockstep(ctx, Xh, U0, K, alpha, 1.0, T, 1e-4)
    labels = ctx.labels().cpu().numpy()
    bad, amb = label_agreement(labels, res["U_ref"])
    passes = passes_ref = mism = 0
    if K <= 20:
        # Appendix D label recovery on the GPU's factor, seeded from one row of each cluster
        # (the oracle's K-means over 1e6 rows is too slow for K = 100; that case runs above)
        seeds = [int(np.flatnonzero(truth == k)[0]) for k in range(K)]
        lab_gpu, passes = ctx.labels_spectral(K, seeds, 20)
        lab_ref, passes_ref = olab.spectral_labels(host(ctx.U), K, seeds, 20)
        mism = int((lab_gpu.cpu().numpy() != lab_ref).sum())
    ctx.close()
    del ctx
    torch.cuda.empty_cache()
    log(f"  max: traj {max(res['traj']):.2e} one-step {max(res['one']):.2e} obj {max(res['obj']):.2e}; "
        f"labels {bad} bad / {amb} ambiguous; spectral passes {passes}/{passes_ref}, {mism} mismatches")
    assert max(res["traj"]) < U_TOL and max(res["one"]) < U_TOL / 10 and max(res["obj"]) < OBJ_TOL
    assert not res["bad_gates"]
    assert bad == 0
    assert passes == passes_ref and mism == 0
