"""Parity of the HIP path (through the C ABI) with the fp64 oracle on seeded inputs.

Bars (from the target of the build): per-iteration U within max relative error
1e-4 (max_ij |U_gpu - U_ref| / max_ij |U_ref|), objective within 1e-5
relative, labels bit-exact on rows whose top-2 gap is not within rounding.
The dual gate is a discrete decision taken on the GPU's rounded movement
estimate; the oracle replays the GPU's gate sequence, and every gate decision
is checked against the oracle's own movement (disagreement allowed only
within 1e-3 relative of eps_d).
"""
import numpy as np
import pytest

from gpu_util import (OBJ_TOL, U_TOL, host, label_agreement, lockstep_parallel, log, make_ctx, obj_rel_err,
                      rel_max_err, trajectory)
from oracle import nlr as onlr
from synth import gaussian_mixture, make_workload, standard_normal_factor

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _tiny():
    X, Z, lab, wl = make_workload("tiny")
    return X, Z.astype(np.float64), lab, wl


def _gated():
    """A tiny mixture (seed 1) on which, with alpha = 1.8/(2 L0), beta = 2, eps_d = 3e-3, the oracle
    takes 4 dual steps in the first 600 iterations and 358 in the first 1000, and eps_c = 1e-3 stops
    it near iteration 1030."""
    X, lab, _ = gaussian_mixture(2000, 16, 4, 25.0, seed=1)
    Z = standard_normal_factor(2000, 4, seed=2).astype(np.float64)
    K, beta = 4, 2.0
    return X, Z, lab, K, beta, 1.8 * onlr.default_step_size(K, beta)


# ---------------------------------------------------------------- initialisation
# d = 1, 65 and 130 also cover the Gram kernel's ragged 64-feature blocks and the mirrored
# blocks below its diagonal (one, two and three blocks per side); d = 300 the power method's
# matrix-vector products spread over workgroups (above 256 features) with a ragged last one
@pytest.mark.parametrize("n,d", [(2000, 16), (1037, 13), (5000, 128), (300, 768), (500, 1), (777, 65),
                                 (3001, 130), (1501, 300)])
def test_normaliser(n, d):
    log(f"normaliser n={n} d={d}")
    X, _, _ = gaussian_mixture(n, d, 3, 9.0, seed=n + d)
    Z = standard_normal_factor(n, 4, seed=1)
    ctx = make_ctx(X, Z, 4, 0.01)
    a, xbar = ctx.normaliser()
    Xh_ref, xbar_ref, a_ref = onlr.centre_and_normalise(X)
    assert abs(a / a_ref - 1.0) < 1e-9, (a, a_ref)
    assert np.abs(xbar - xbar_ref).max() <= 1e-12 * max(1.0, np.abs(X).max())
    Xh = host(ctx.X)
    # X is stored as fp32(Xhat)
    assert np.abs(Xh - Xh_ref).max() <= 2.0 ** -23 * np.abs(Xh_ref).max()


@pytest.mark.parametrize("n,r,K", [(2000, 4, 4), (1037, 10, 7), (999, 33, 5)])
def test_init_projection(n, r, K):
    log(f"projection n={n} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, 8, 3, 9.0, seed=3)
    Z = standard_normal_factor(n, r, seed=4)
    ctx = make_ctx(X, Z, K, 0.01)
    U = host(ctx.U)
    ref = onlr.project_omega(Z.astype(np.float64), K)
    assert rel_max_err(U, ref) < 1e-6
    p = ctx.inspect("p").astype(np.float64)
    assert np.abs(p - U.sum(axis=0)).max() <= 1e-6 * np.abs(p).max()
    assert np.all(host(ctx.y) == 0.0)


# ---------------------------------------------------------------- one step
TWO_PASS = 16  # NLR_INIT_TWO_PASS


@pytest.mark.parametrize("flags", [0, TWO_PASS])
def test_one_step_tiny(flags):
    X, Z, _, wl = _tiny()
    K = wl.K
    alpha, beta = onlr.default_step_size(K), 1.0
    ctx = make_ctx(X, Z, K, alpha, beta, flags=flags)
    U0 = host(ctx.U)
    st = ctx.step()
    Xh, _, _ = onlr.centre_and_normalise(X)
    theta = ctx.inspect("theta").astype(np.float64)
    # two passes: Theta of the step's starting factor; single Xhat pass: Theta of the new factor,
    # formed as c Xhat^T W inside pass B
    th_ref = Xh.T @ (U0 if flags & TWO_PASS else host(ctx.U))
    assert rel_max_err(theta, th_ref) < 1e-5
    res = onlr.run(Xh, U0, K, alpha, beta, T=1, T_min=1, project_init=False, gates=[bool(st["dual_step"])])
    rec = res.records[0]
    for k in ("a", "b", "h"):
        assert abs(st[k] - getattr(rec, k)) <= 1e-6 * abs(getattr(rec, k)), k
    assert abs(st["c"] - rec.c) <= 2e-7 * rec.c
    assert abs(st["delta"] - rec.delta) <= 1e-4 * rec.delta + 1e-9
    assert obj_rel_err(st["objective"], rec.objective, 1.0) < OBJ_TOL
    assert rel_max_err(host(ctx.U), res.U) < U_TOL / 10
    s_ref = U0.T @ onlr.effective_multiplier(U0, np.zeros(U0.shape[0]), beta)
    assert np.abs(ctx.inspect("s") - s_ref).max() <= 1e-5 * max(1e-12, np.abs(s_ref).max()) + 1e-9


# ---------------------------------------------------------------- trajectories
def test_trajectory_tiny_200():
    X, Z, lab, wl = _tiny()
    K = wl.K
    alpha, beta = onlr.default_step_size(K), 1.0
    log("tiny trajectory T=200")
    ctx, ref, traj, obj, bad_gates, one, U_gpu, stats = trajectory(X, Z, K, alpha, beta, wl.T,
                                                                    one_step_tol=True)
    log(f"max traj err {max(traj):.3e}  max one-step err {max(one):.3e}  max obj err {max(obj):.3e}")
    assert max(traj) < U_TOL, (int(np.argmax(traj)), max(traj))
    assert max(one) < U_TOL / 10
    assert max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates
    labels = ctx.labels().cpu().numpy()
    bad, amb = label_agreement(labels, ref.U)
    log(f"labels: {bad} mismatches, {amb} ambiguous rows")
    assert bad == 0


def test_trajectory_tiny_two_pass():
    """The two-pass iteration (pass A with Theta) on the same trajectory."""
    X, Z, lab, wl = _tiny()
    K = wl.K
    ctx, ref, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, onlr.default_step_size(K), 1.0, wl.T,
                                                           one_step_tol=True, flags=TWO_PASS)
    log(f"two-pass: max traj err {max(traj):.3e}  one-step {max(one):.3e}  obj {max(obj):.3e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates


def test_fused_and_two_pass_agree():
    """Both iteration structures step the same iterate; they differ by rounding only."""
    X, Z, _, K, beta, alpha = _gated()
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, flags=TWO_PASS, **kw)
    a.run(300)
    b.run(300)
    d = np.abs(host(a.U) - host(b.U)).max() / np.abs(host(b.U)).max()
    log(f"fused vs two-pass after 300 steps: {d:.2e}")
    assert d < U_TOL / 10


def test_trajectory_with_dual_steps():
    """Gated dual steps along a 1000-iteration trajectory."""
    X, Z, lab, K, beta, alpha = _gated()
    ctx, ref, traj, obj, bad_gates, one, _, stats = trajectory(X, Z, K, alpha, beta, 1000, eps_d=3e-3,
                                                              eps_c=1e-7, one_step_tol=True)
    ngates = sum(s["dual_step"] for s in stats)
    log(f"dual steps {ngates}; max traj err {max(traj):.3e} one-step {max(one):.3e} obj {max(obj):.3e}")
    assert ngates > 200
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates


@pytest.mark.parametrize("n,d,r,K", [(1037, 13, 10, 7), (777, 64, 16, 16), (4099, 128, 64, 64),
                                     (300, 33, 33, 5), (513, 200, 100, 20), (64, 3, 1, 1),
                                     (1500, 768, 256, 256), (1037, 16, 10, 7), (999, 32, 10, 10),
                                     (4001, 64, 30, 12), (70, 8, 1, 1), (2050, 128, 50, 20),
                                     # even d, d % 4 == 2: the single-Xhat-pass form with 8-byte X rows
                                     (4099, 50, 30, 20), (3001, 110, 32, 10), (1037, 18, 4, 4),
                                     (2001, 46, 12, 6), (999, 126, 60, 12), (513, 2, 2, 2),
                                     # above 256 columns (pass B in pairs of column blocks): Theta in
                                     # LDS, rows not 16-byte aligned, the largest rank
                                     (2001, 16, 300, 8), (1501, 24, 301, 5), (999, 40, 448, 4)])
def test_ragged_shapes(n, d, r, K):
    log(f"ragged n={n} d={d} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n * 7 + d)
    Z = standard_normal_factor(n, r, seed=n + r).astype(np.float64)
    alpha = onlr.default_step_size(K)
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, alpha, 1.0, 8, one_step_tol=True)
    log(f"  traj {max(traj):.2e} one {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


# Two-pass fp32 form with a Theta that does not fit pass B's 64 KiB of LDS (beside p, s and
# the reductions) and 16-byte rows: pass B streams Theta through LDS in chunks, with the
# columns in groups of up to four blocks (1, 2 and 4 blocks; 8, 12 and 14 blocks in groups of
# four, a short last group at 14; 10 blocks in five groups of two); the wide pass A (above
# 128 columns) as a streaming row pass and the register-prefetched product
@pytest.mark.parametrize("n,d,r,K", [(1037, 520, 32, 8), (1501, 300, 64, 16), (1037, 132, 128, 16),
                                     (2001, 96, 256, 32),
                                     (999, 200, 300, 20), (1201, 44, 384, 12), (777, 40, 448, 4),
                                     (3001, 252, 200, 16)])
def test_two_pass_streamed_theta(n, d, r, K):
    log(f"streamed theta n={n} d={d} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n * 3 + d)
    Z = standard_normal_factor(n, r, seed=n + 2 * r).astype(np.float64)
    alpha = onlr.default_step_size(K)
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, alpha, 1.0, 6, one_step_tol=True,
                                                       flags=TWO_PASS)
    log(f"  traj {max(traj):.2e} one {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


# Two-pass fp32 form above 128 columns at its edges: about one tile per workgroup (n = 301
# just above r, a ragged last tile and super-tile), rows not 16-byte aligned (d % 4 == 2: the
# LDS-staged Theta product; r % 4 != 0: the pair-wise pass B), the smallest split width
# (r = 129: three columns per lane in the row launch; its 64 x 256 Theta fills 64 KiB
# exactly, so pass B takes it from L2)
@pytest.mark.parametrize("n,d,r,K", [(301, 40, 300, 6), (777, 130, 160, 8), (1500, 64, 129, 9),
                                     (2049, 132, 260, 10)])
def test_two_pass_wide_edges(n, d, r, K):
    log(f"two-pass wide edge n={n} d={d} r={r} K={K}")
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n * 5 + d)
    Z = standard_normal_factor(n, r, seed=n + 3 * r).astype(np.float64)
    alpha = onlr.default_step_size(K)
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, Z, K, alpha, 1.0, 6, one_step_tol=True,
                                                       flags=TWO_PASS)
    log(f"  traj {max(traj):.2e} one {max(one):.2e} obj {max(obj):.2e}")
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates


def test_gmm1m_parity():
    """gmm1m over its configuration's 100 iterations with split products (the bench's
    single-Xhat-pass form) and with fp32 products, from the same start: each iterate against
    the oracle's trajectory and one oracle step from the GPU's own iterate."""
    X, Z, lab, wl = make_workload("gmm1m")
    K, alpha = wl.K, onlr.default_step_size(wl.K)
    log(f"gmm1m lockstep T={wl.T}, split and fp32 products")
    runs = {"split16": (make_ctx(X, Z, K, alpha, 1.0, T_min=wl.T, flags=8), wl.T),
            "fp32": (make_ctx(X, Z, K, alpha, 1.0, T_min=wl.T), wl.T)}
    Xh, _, _ = onlr.centre_and_normalise(X)
    res = lockstep_parallel(runs, Xh, onlr.project_omega(Z.astype(np.float64), K), K, alpha, 1.0, 1e-4)
    for s, r in res.items():
        bad, amb = r["labels"]
        log(f"  {s}: traj {max(r['traj']):.2e} one {max(r['one']):.2e} obj {max(r['obj']):.2e} "
            f"y {max(r['yerr']):.2e} dual steps {sum(r['gates'])}; labels {bad} bad / {amb} ambiguous")
        assert max(r["traj"]) < U_TOL and max(r["one"]) < U_TOL / 10 and max(r["obj"]) < OBJ_TOL
        assert max(r["yerr"]) <= 1e-5
        assert not r["bad_gates"]
        assert bad == 0


# ---------------------------------------------------------------- API semantics
def test_run_equals_steps_bitwise_and_deterministic():
    X, Z, _, K, beta, alpha = _gated()
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    c = make_ctx(X, Z, K, alpha, beta, **kw)
    T = 900
    done, _ = a.run(T)
    assert done == T
    done_c, _ = c.run(T)
    for _ in range(T):
        b.step(with_stats=False)
    for name in ("U", "y"):
        ua, ub, uc = host(getattr(a, name)), host(getattr(b, name)), host(getattr(c, name))
        assert np.array_equal(ua, ub), name
        assert np.array_equal(ua, uc), name
    assert sum(h["dual_step"] for h in a.history()) > 50


def test_nondefault_stream():
    import torch
    X, Z, _, wl = _tiny()
    K = wl.K
    alpha = onlr.default_step_size(K)
    a = make_ctx(X, Z, K, alpha)
    a.run(25)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = make_ctx(X, Z, K, alpha, stream=s)
        b.run(25)
    s.synchronize()
    assert np.array_equal(host(a.U), host(b.U))


def test_stop_rule():
    X, Z, _, K, beta, alpha = _gated()
    eps_d, eps_c = 3e-3, 1e-3
    ctx = make_ctx(X, Z, K, alpha, beta, eps_d=eps_d, eps_c=eps_c, T_min=5)
    done, last = ctx.run(3000)
    log(f"stopped after {done} iterations: {last}")
    assert done < 3000 and last["stop"] == 1
    assert last["delta"] < min(eps_d, eps_c) and last["rho"] < eps_c and done >= 5
    hist = ctx.history(4096)
    assert len(hist) == done
    for h in hist[:-1]:
        assert not (h["delta"] < min(eps_d, eps_c) and h["rho"] < eps_c and h["t"] + 1 >= 5), h
    # the oracle, replaying the gates, meets its own stopping rule at the same iteration
    gates = [bool(h["dual_step"]) for h in hist]
    Xh, _, _ = onlr.centre_and_normalise(X)
    ref = onlr.run(Xh, Z, K, alpha, beta, T=done, T_min=5, eps_d=eps_d, eps_c=eps_c, gates=gates)
    rec = ref.records[-1]
    band = 1e-3
    assert rec.delta < min(eps_d, eps_c) * (1 + band) and rec.rho < eps_c * (1 + band)
    assert rel_max_err(host(ctx.U), ref.U) < U_TOL
    # the stored dual after the final (gated) step agrees too
    ys = onlr.stored_dual(ref.y)
    assert np.abs(host(ctx.y) - ys).max() <= 1e-4 * np.abs(ys).max()


def test_k1_fixed_point():
    n = 256
    X, _, _ = gaussian_mixture(n, 5, 2, 9.0, seed=9)
    Z = np.full((n, 1), 1.0 / np.sqrt(n))
    ctx = make_ctx(X, Z, 1, 0.3, 2.0)
    for _ in range(3):
        st = ctx.step()
        assert st["delta"] < 1e-6 and abs(st["c"] - 1.0) < 1e-6 and st["rho"] < 1e-6
    assert np.abs(host(ctx.U) - 1.0 / np.sqrt(n)).max() < 1e-6


def test_breakdown_and_sticky_state():
    from paper_2609_36074_amd import nlr
    n, K = 200, 3
    X, _, _ = gaussian_mixture(n, 4, 2, 9.0, seed=10)
    Z = np.ones((n, 3))
    ctx = make_ctx(X, Z, K, 1.0 / (2 * 1.0 * (K - 1)) * 1.5, 1.0)
    with pytest.raises(nlr.NlrError) as e:
        ctx.step()
    assert e.value.status == nlr.NLR_EBREAKDOWN
    assert np.all(host(ctx.U) == 0.0)  # the unnormalised update replaced the factor
    with pytest.raises(nlr.NlrError) as e:
        ctx.run(3)
    assert e.value.status == nlr.NLR_ESTATE


def test_degenerate_and_nonpositive_start():
    from paper_2609_36074_amd import nlr
    X = np.ones((100, 6), dtype=np.float32) * 3.0
    with pytest.raises(nlr.NlrError) as e:
        make_ctx(X, np.abs(standard_normal_factor(100, 2, 1)), 2, 0.01)
    assert e.value.status == nlr.NLR_EDEGENERATE
    X2, _, _ = gaussian_mixture(100, 6, 2, 9.0, seed=1)
    with pytest.raises(nlr.NlrError) as e:
        make_ctx(X2, -np.abs(standard_normal_factor(100, 2, 1)), 2, 0.01)
    assert e.value.status == nlr.NLR_EBREAKDOWN


def test_resume_flags():
    """Resuming from (U, y) with U_IN_OMEGA | KEEP_Y | X_NORMALISED continues the iteration."""
    from paper_2609_36074_amd import nlr
    X, Z, _, wl = _tiny()
    K, beta = wl.K, 2.0
    alpha = 1.8 * onlr.default_step_size(K, beta)
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    a.run(120)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    b.run(60)
    flags = nlr.NLR_INIT_U_IN_OMEGA | nlr.NLR_INIT_KEEP_Y | nlr.NLR_INIT_X_NORMALISED
    c = nlr.Context(b.X, K, b.U, b.y, alpha=alpha, beta=beta, flags=flags, **kw)
    c.run(60)
    # p is recomputed from the stored factor on resume, so agreement is to tolerance, not bitwise
    assert rel_max_err(host(c.U), host(a.U)) < U_TOL


# ---------------------------------------------------------------- data-informed start (Appendix D)
DATA_START = 32  # NLR_INIT_DATA_START


@pytest.mark.parametrize("n,d,r,K,flags", [(2000, 16, 4, 4, 0), (1037, 16, 10, 7, 0), (777, 64, 16, 16, 0),
                                           (4099, 128, 64, 64, 0), (4099, 128, 64, 64, 8),
                                           (1500, 768, 256, 256, 0), (3000, 32, 10, 10, 16),
                                           (1500, 768, 256, 256, 8), (2049, 256, 68, 10, 8)])
def test_data_start(n, d, r, K, flags):
    X, _, _ = gaussian_mixture(n, d, max(K, 2), 16.0, seed=n + 3 * d)
    Z = standard_normal_factor(n, r, seed=n + r + 1).astype(np.float64)
    log(f"data start n={n} d={d} r={r} K={K} flags={flags}")
    ctx = make_ctx(X, Z, K, onlr.default_step_size(K), flags=flags | DATA_START)
    Xh, _, _ = onlr.centre_and_normalise(X)
    U0_ref, Q = onlr.data_informed_start(Xh, Z, K)
    err = rel_max_err(host(ctx.U), U0_ref)
    log(f"  U0 err {err:.2e}")
    assert err < U_TOL / 10
    # and the iteration from there
    _, _, traj, obj, bad_gates, one, _, _ = trajectory(X, U0_ref, K, onlr.default_step_size(K), 1.0, 6,
                                                       one_step_tol=True, flags=flags | 1)  # U0 in Omega
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL


def test_data_start_rank_deficient_is_degenerate():
    """r above the rank of Xhat: V = Xhat Xhat^T Z has dependent columns and Cholesky QR fails."""
    from paper_2609_36074_amd import nlr
    X, _, _ = gaussian_mixture(500, 8, 3, 16.0, seed=11)
    Z = standard_normal_factor(500, 12, seed=12).astype(np.float64)
    with pytest.raises(nlr.NlrError) as e:
        make_ctx(X, Z, 3, 0.01, flags=DATA_START)
    assert e.value.status == nlr.NLR_EDEGENERATE


def test_profiling_levels():
    """nlr_set_profiling: 1 times every launch, 2 only the row and pass kernels, others are rejected."""
    from paper_2609_36074_amd import nlr
    X, Z, _, wl = make_workload("tiny")
    ctx = make_ctx(X, Z.astype(np.float64), wl.K, onlr.default_step_size(wl.K), T_min=10)
    lib = nlr.load_library()
    assert lib.nlr_set_profiling(ctx._ctx, 3) == nlr.NLR_EINVAL
    assert lib.nlr_set_profiling(ctx._ctx, -1) == nlr.NLR_EINVAL
    ctx.set_profiling(1)
    ctx.run(4)
    every = {k: v for k, v in ctx.kernel_times().items() if v[1]}
    ctx.set_profiling(2)
    ctx.run(4)
    passes = {k: v for k, v in ctx.kernel_times().items() if v[1]}
    ctx.set_profiling(0)
    log(f"  level 1: {sorted(every)}; level 2: {sorted(passes)}")
    assert {"ctl_a", "ctl_b", "reduce_theta"} <= set(every)
    assert set(passes) <= {"pass_a", "pass_b", "pass_u", "pass_bf", "finish"} and passes
    assert all(v[0] > 0 for v in passes.values())


def test_history_ring_wraps_in_order():
    """Beyond 4096 iterations the history holds the latest 4096 records, oldest first, and
    their iteration numbers and statistics match the record of the last iteration."""
    X, Z, _, wl = _tiny()
    K = wl.K
    T = 4096 + 700
    ctx = make_ctx(X, Z, K, onlr.default_step_size(K), eps_d=0.0, eps_c=0.0, T_min=T)
    done, last = ctx.run(T)
    assert done == T
    hist = ctx.history(8192)
    assert len(hist) == 4096
    assert [h["t"] for h in hist] == list(range(T - 4096, T))
    assert hist[-1]["t"] == last["t"] and hist[-1]["objective"] == last["objective"]
    assert hist[-1]["delta"] == last["delta"] and hist[-1]["c"] == last["c"]
    assert len(ctx.history(10)) == 10 and ctx.history(10)[-1]["t"] == T - 1


def test_two_contexts_interleaved_on_two_streams():
    """Two contexts on two streams, their runs interleaved call by call, give the same
    iterates bitwise as each run alone (contexts share no state)."""
    import torch
    X1, Z1, _, wl = _tiny()
    X2, _, _ = gaussian_mixture(3000, 16, 4, 16.0, seed=77)
    Z2 = standard_normal_factor(3000, 4, seed=78).astype(np.float64)
    K = wl.K
    alpha = onlr.default_step_size(K)
    ref1 = make_ctx(X1, Z1, K, alpha)
    ref1.run(60)
    ref2 = make_ctx(X2, Z2, K, alpha)
    ref2.run(60)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    a = make_ctx(X1, Z1, K, alpha, stream=s1)
    b = make_ctx(X2, Z2, K, alpha, stream=s2)
    for _ in range(6):
        a.step(with_stats=False)
        b.run(10)
        a.run(9)
    torch.cuda.synchronize()
    assert np.array_equal(host(a.U), host(ref1.U)) and np.array_equal(host(a.y), host(ref1.y))
    assert np.array_equal(host(b.U), host(ref2.U)) and np.array_equal(host(b.y), host(ref2.y))


@pytest.mark.parametrize("r", [1, 4, 10, 64, 128, 188, 256, 300, 384, 448])
def test_labels_argmax_ties_and_layouts(r):
    """nlr_labels on factors written directly into the context's U: exact ties (lowest
    column wins, as numpy's argmax), all-equal rows, the maximum in every column position,
    16-byte rows (r % 4 == 0: one to seven 256-byte pieces per row, one to four rows per
    16-lane group and step) and others; the oracle's labels are the plain argmax."""
    import torch
    n = 4099
    K = min(r, 4)
    X, _, _ = gaussian_mixture(n, 8, 2, 9.0, seed=5)
    Z = standard_normal_factor(n, r, seed=6)
    ctx = make_ctx(X, Z, K, 0.01)
    rng = np.random.default_rng(r)
    U = rng.integers(0, 4, size=(n, r)).astype(np.float32)  # small integers: many exact ties
    U[::7] = 1.0                                             # all-equal rows
    for c in range(r):                                       # a unique maximum in each column
        U[11 * c % n, :] = 0.0
        U[11 * c % n, c] = 5.0
    ctx.U.copy_(torch.from_numpy(U))
    lab = ctx.labels().cpu().numpy()
    assert np.array_equal(lab, onlr.labels(U.astype(np.float64)))
    assert np.array_equal(lab, np.argmax(U, axis=1).astype(np.int32))
