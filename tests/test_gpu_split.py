"""Parity of the split-fp16 products (NLR_INIT_SPLIT_F16) with the fp64 oracle.

Same bars as the fp32 path: per-iteration U within 1e-4 max relative error,
objective within 1e-5, labels exact on unambiguous rows, every dual-gate
decision consistent with the oracle's own movement.
"""
import numpy as np
import pytest

from gpu_util import OBJ_TOL, U_TOL, host, label_agreement, log, make_ctx, trajectory
from oracle import nlr as onlr
from synth import gaussian_mixture, make_workload, standard_normal_factor

pytestmark = pytest.mark.gpu
SPLIT = 8  # NLR_INIT_SPLIT_F16


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _gated():
    X, _, _ = gaussian_mixture(2000, 16, 4, 25.0, seed=1)
    Z = standard_normal_factor(2000, 4, seed=2).astype(np.float64)
    K, beta = 4, 2.0
    return X, Z, K, beta, 1.8 * onlr.default_step_size(K, beta)


def test_split_tiny_trajectory():
    X, Z, _, wl = make_workload("tiny")
    Z = Z.astype(np.float64)
    K = wl.K
    log("split: tiny trajectory T=200")
    ctx, ref, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, wl.T,
                                                           one_step_tol=True, flags=SPLIT)
    log(f"  traj {max(traj):.3e} one {max(one):.3e} obj {max(obj):.3e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates
    bad, amb = label_agreement(ctx.labels().cpu().numpy(), ref.U)
    assert bad == 0, (bad, amb)


def test_split_dual_steps():
    X, Z, K, beta, alpha = _gated()
    log("split: gated trajectory T=1000")
    _, _, traj, obj, bad_gates, one, _, stats = trajectory(X, Z, K, alpha, beta, 1000, eps_d=3e-3, eps_c=1e-7,
                                                           one_step_tol=True, flags=SPLIT)
    ngates = sum(s["dual_step"] for s in stats)
    log(f"  dual steps {ngates}; traj {max(traj):.3e} one {max(one):.3e} obj {max(obj):.3e}")
    assert ngates > 200
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates


@pytest.mark.parametrize("n,d,r,K", [(777, 64, 16, 16), (4099, 128, 64, 64), (1000, 36, 12, 3),
                                     (2001, 128, 60, 50), (33, 4, 4, 4), (5000, 100, 36, 9),
                                     (1037, 16, 10, 7), (999, 32, 10, 10), (4001, 64, 30, 12), (70, 8, 1, 1)])
def test_split_ragged(n, d, r, K):
    log(f"split: ragged n={n} d={d} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n * 7 + d)
    Z = standard_normal_factor(n, r, seed=n + r).astype(np.float64)
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, 8,
                                                       one_step_tol=True, flags=SPLIT)
    log(f"  traj {max(traj):.2e} one {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


# The eight-wave fused pass B (d in 97..128, r in 33..64, r % 4 == 0): one tile per
# workgroup (tail only), 2-3 and 3-4 tiles per workgroup (loop and tail), padded
# features (d < 128) and masked columns (r < 64), and fewer rows than one tile.
@pytest.mark.parametrize("n,d,r,K", [(130, 128, 64, 64), (70001, 104, 40, 20), (98381, 128, 64, 30),
                                     (5000, 100, 44, 11), (131072, 128, 64, 64), (100, 128, 64, 8),
                                     (64, 104, 36, 36)])
def test_split_fused8(n, d, r, K):
    log(f"split fused8: n={n} d={d} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n * 5 + d)
    Z = standard_normal_factor(n, r, seed=n + 3 * r).astype(np.float64)
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, 6,
                                                       one_step_tol=True, flags=SPLIT)
    log(f"  traj {max(traj):.2e} one {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


def test_split_fused8_run_equals_steps_and_deterministic():
    X, _, _ = gaussian_mixture(70001, 104, 20, 16.0, seed=11)
    Z = standard_normal_factor(70001, 40, seed=12).astype(np.float64)
    K = 20
    kw = dict(eps_d=1e-9, eps_c=1e-12, T_min=0, flags=SPLIT)
    alpha = onlr.default_step_size(K)
    a = make_ctx(X, Z, K, alpha, 1.0, **kw)
    b = make_ctx(X, Z, K, alpha, 1.0, **kw)
    c = make_ctx(X, Z, K, alpha, 1.0, **kw)
    T = 25
    done, _ = a.run(T)
    assert done == T
    for _ in range(T):
        b.step(with_stats=False)
    c.run(T)
    Ua, Ub, Uc = host(a.U), host(b.U), host(c.U)
    assert np.array_equal(Ua, Ub) and np.array_equal(host(a.y), host(b.y))
    assert np.array_equal(Ua, Uc) and np.array_equal(host(a.y), host(c.y))


@pytest.mark.parametrize("flags", [SPLIT, 0])
def test_tiny_dual_steps_at_config_tolerance(flags):
    """tiny with the configurations' eps_d = 1e-4 and default step: the movement falls below
    eps_d near iteration 800, so 1500 iterations take dual steps under the paper's gate."""
    X, Z, _, wl = make_workload("tiny")
    Z = Z.astype(np.float64)
    K = wl.K
    _, _, traj, obj, bad_gates, one, _, stats = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, 1500,
                                                           eps_d=1e-4, eps_c=1e-4, one_step_tol=True,
                                                           flags=flags)
    ngates = sum(s["dual_step"] for s in stats)
    log(f"  tiny eps_d=1e-4 flags={flags}: {ngates} dual steps; traj {max(traj):.2e} one {max(one):.2e}")
    assert ngates >= 1
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates


def test_split_run_equals_steps_and_deterministic():
    X, Z, K, beta, alpha = _gated()
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0, flags=SPLIT)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    c = make_ctx(X, Z, K, alpha, beta, **kw)
    T = 900
    done, _ = a.run(T)
    assert done == T
    for _ in range(T):
        b.step(with_stats=False)
    c.run(T)
    Ua, Ub, Uc = host(a.U), host(b.U), host(c.U)
    assert np.array_equal(Ua, Ub) and np.array_equal(host(a.y), host(b.y))
    assert np.array_equal(Ua, Uc) and np.array_equal(host(a.y), host(c.y))
    assert sum(h["dual_step"] for h in a.history(T)) > 50


def test_split_two_pass_trajectory():
    """Split products in the two-pass iteration (pass B split, pass A fp32)."""
    X, Z, _, wl = make_workload("tiny")
    Z = Z.astype(np.float64)
    K = wl.K
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, 100,
                                                       one_step_tol=True, flags=SPLIT | 16)
    log(f"  split two-pass: traj {max(traj):.3e} one {max(one):.3e} obj {max(obj):.3e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


def test_split_matches_fp32_path_closely():
    """Both product forms step the same iterate; their difference is far inside the parity bar."""
    X, Z, _, wl = make_workload("tiny")
    K = wl.K
    alpha = onlr.default_step_size(K)
    a = make_ctx(X, Z, K, alpha, T_min=40)
    b = make_ctx(X, Z, K, alpha, T_min=40, flags=SPLIT)
    a.run(40)
    b.run(40)
    Ua, Ub = host(a.U), host(b.U)
    d = np.abs(Ua - Ub).max() / np.abs(Ua).max()
    log(f"  split vs fp32 after 40 steps: {d:.2e}")
    assert d < U_TOL / 10


# ---- panel form: the split products for d > 128 or r > 64 (d % 8 == 0, r % 4 == 0) ----
@pytest.mark.parametrize("n,d,r,K", [(3001, 136, 8, 4), (2049, 256, 68, 10), (4000, 64, 128, 32),
                                     (1500, 768, 256, 256), (777, 200, 100, 20), (5000, 520, 36, 9),
                                     (70, 136, 8, 2), (1200, 8, 96, 5)])
def test_split_panel_ragged(n, d, r, K):
    log(f"split panel: n={n} d={d} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n * 5 + d)
    Z = standard_normal_factor(n, r, seed=n + 3 * r).astype(np.float64)
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, 6,
                                                       one_step_tol=True, flags=SPLIT)
    log(f"  traj {max(traj):.2e} one {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


def _gated_wide():
    X, _, _ = gaussian_mixture(2000, 136, 4, 25.0, seed=21)
    Z = standard_normal_factor(2000, 4, seed=22).astype(np.float64)
    K, beta = 4, 2.0
    return X, Z, K, beta, 1.8 * onlr.default_step_size(K, beta)


def test_split_panel_dual_steps():
    X, Z, K, beta, alpha = _gated_wide()
    log("split panel: gated trajectory T=1000 (d = 136)")
    _, _, traj, obj, bad_gates, one, _, stats = trajectory(X, Z, K, alpha, beta, 1000, eps_d=3e-3, eps_c=1e-7,
                                                           one_step_tol=True, flags=SPLIT)
    ngates = sum(s["dual_step"] for s in stats)
    log(f"  dual steps {ngates}; traj {max(traj):.3e} one {max(one):.3e} obj {max(obj):.3e}")
    assert ngates > 200
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates


def test_split_panel_run_equals_steps_and_deterministic():
    X, Z, K, beta, alpha = _gated_wide()
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0, flags=SPLIT)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    c = make_ctx(X, Z, K, alpha, beta, **kw)
    T = 600
    done, _ = a.run(T)
    assert done == T
    for _ in range(T):
        b.step(with_stats=False)
    c.run(T)
    Ua, Ub, Uc = host(a.U), host(b.U), host(c.U)
    assert np.array_equal(Ua, Ub) and np.array_equal(host(a.y), host(b.y))
    assert np.array_equal(Ua, Uc) and np.array_equal(host(a.y), host(c.y))
    assert sum(h["dual_step"] for h in a.history(T)) > 50
