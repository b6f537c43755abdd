"""The one-pass iteration (split products; 97..128 features with 33..64 columns, or
at most 64 features with at most 16 columns, r even -- r % 4 == 2 moves U in column
pairs): one
pass over the rows per iteration does the row work of the iteration (the end of
the previous one) and the primal step, writing W over the factor it reads; s
comes from the Gram terms of the previous pass.  Where the previous iteration's
stopping rule can fire (movement below min(eps_d, eps_c), t >= T_min), the row
work runs in a pass of its own first and settles it.  Checked against the fp64
oracle as the other forms: trajectories with gated dual steps, bitwise equality
of nlr_run and nlr_step (also across iterations whose row pass runs first), the
stopping rule, and breakdown (the unnormalised update replaces the factor).
"""
import numpy as np
import pytest

from gpu_util import OBJ_TOL, U_TOL, host, log, make_ctx, rel_max_err, to_dev, trajectory
from oracle import nlr as onlr
from synth import gaussian_mixture, standard_normal_factor

pytestmark = pytest.mark.gpu

SPLIT = 8  # NLR_INIT_SPLIT_F16


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _gated(d, r):
    """A 3000-row mixture (seed 1) on which, with alpha = 1.8/(2 L0), beta = 2, eps_d = 3e-3 and
    eps_c = 1e-3, the oracle stops after 432 iterations with 144 dual steps at d = 100, r = 36, and
    after 564 with 244 at d = 128, r = 64 (first dual steps near iteration 25); after 769 at
    d = 64, r = 16, 545 at d = 32, r = 12, 834 at d = 16, r = 4, 538 at d = 48, r = 8, 596 at
    d = 32, r = 10 and 625 at d = 64, r = 14."""
    K, beta = 4, 2.0
    X, lab, _ = gaussian_mixture(3000, d, K, 25.0, seed=1)
    Z = standard_normal_factor(3000, r, seed=2).astype(np.float64)
    return X, Z, K, beta, 1.8 * onlr.default_step_size(K, beta)


# with eps_c = 1e-7 (no stop) the oracle takes 162 dual steps in 450 iterations (d = 100),
# 280 in 600 (d = 128), 260 in 700 (d = 64, r = 16), 97 in 450 (d = 32, r = 12) and 258 in
# 800 (d = 16, r = 4)
@pytest.mark.parametrize("d,r,T,gates", [(100, 36, 450, 100), (128, 64, 600, 100), (64, 16, 700, 100),
                                         (32, 12, 450, 50), (16, 4, 800, 100), (32, 10, 600, 100),
                                         (64, 14, 600, 100)])
def test_onepass_gated_trajectory(d, r, T, gates):
    from paper_2609_36074_amd import nlr
    assert nlr.FORM_NAMES[nlr.nlr_iteration_form(3000, d, r, 4, SPLIT)] == "one-pass"
    X, Z, K, beta, alpha = _gated(d, r)
    log(f"one-pass gated trajectory d={d} r={r} T={T}")
    _, _, traj, obj, bad_gates, one, _, stats = trajectory(X, Z, K, alpha, beta, T, eps_d=3e-3, eps_c=1e-7,
                                                           one_step_tol=True, flags=SPLIT)
    ngates = sum(s["dual_step"] for s in stats)
    log(f"  dual steps {ngates}; traj {max(traj):.3e} one {max(one):.3e} obj {max(obj):.3e}")
    assert ngates > gates
    assert max(traj) < U_TOL and max(one) < U_TOL / 10 and max(obj) < OBJ_TOL
    assert not bad_gates, bad_gates


# dual steps in the first 451 iterations: 162 (d = 100), 13 (d = 64), 2 (d = 16), 83 (d = 32,
# r = 10: column pairs), 5 (d = 16, r = 6)
@pytest.mark.parametrize("d,r,gates", [(100, 36, 50), (64, 16, 5), (16, 4, 1), (32, 10, 50), (16, 6, 2)])
def test_onepass_run_equals_steps_bitwise(d, r, gates):
    X, Z, K, beta, alpha = _gated(d, r)
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0, flags=SPLIT)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    c = make_ctx(X, Z, K, alpha, beta, **kw)
    T = 451
    done, _ = a.run(T)
    assert done == T
    done_c, _ = c.run(T)
    for _ in range(T):
        b.step(with_stats=False)
    for name in ("U", "y"):
        ua, ub, uc = host(getattr(a, name)), host(getattr(b, name)), host(getattr(c, name))
        assert np.array_equal(ua, ub), name
        assert np.array_equal(ua, uc), name
    assert sum(h["dual_step"] for h in a.history(T)) >= gates
    # two runs continue as one
    d = make_ctx(X, Z, K, alpha, beta, **kw)
    d.run(200)
    d.run(251)
    assert np.array_equal(host(d.U), host(a.U)) and np.array_equal(host(d.y), host(a.y))


@pytest.mark.parametrize("d,r,expect", [(100, 36, 432), (128, 64, 564), (64, 16, 769), (32, 12, 545),
                                        (32, 10, 596), (64, 14, 625)])
def test_onepass_stop_rule(d, r, expect):
    X, Z, K, beta, alpha = _gated(d, r)
    eps_d, eps_c = 3e-3, 1e-3
    ctx = make_ctx(X, Z, K, alpha, beta, eps_d=eps_d, eps_c=eps_c, T_min=5, flags=SPLIT)
    done, last = ctx.run(3000)
    log(f"one-pass d={d} r={r}: stopped after {done} iterations (oracle {expect}): {last}")
    assert done < 3000 and last["stop"] == 1
    assert last["delta"] < min(eps_d, eps_c) and last["rho"] < eps_c and done >= 5
    hist = ctx.history(4096)
    assert len(hist) == done
    for h in hist[:-1]:
        assert not (h["delta"] < min(eps_d, eps_c) and h["rho"] < eps_c and h["t"] + 1 >= 5), h
    gates = [bool(h["dual_step"]) for h in hist]
    Xh, _, _ = onlr.centre_and_normalise(X)
    ref = onlr.run(Xh, Z, K, alpha, beta, T=done, T_min=5, eps_d=eps_d, eps_c=eps_c, gates=gates)
    rec = ref.records[-1]
    band = 1e-3
    assert rec.delta < min(eps_d, eps_c) * (1 + band) and rec.rho < eps_c * (1 + band)
    assert rel_max_err(host(ctx.U), ref.U) < U_TOL
    ys = onlr.stored_dual(ref.y)
    assert np.abs(host(ctx.y) - ys).max() <= 1e-4 * np.abs(ys).max()
    # a second run continues from the stopped iterate
    more, _ = ctx.run(5)
    assert more >= 1


@pytest.mark.parametrize("d,r", [(100, 36), (128, 64), (48, 8)])
def test_onepass_rows_first_iterations(d, r):
    """eps_c = 1e-3, T_min = 0: from the first iteration whose movement falls below 1e-3 until
    the stop (432 / 564 / 538), nlr_run runs each iteration's row pass first (it settles the stopping
    rule) and then the pass in place; nlr_step settles the rule in the finish pass of each call
    instead.  The two stay bitwise equal (s comes from the Gram terms either way), follow the
    oracle, and the counter of row-first iterations is as expected."""
    X, Z, K, beta, alpha = _gated(d, r)
    kw = dict(eps_d=3e-3, eps_c=1e-3, T_min=0, flags=SPLIT)
    T = 420
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    done, last = a.run(T)
    assert done == T and last["stop"] == 0
    for _ in range(T):
        b.step(with_stats=False)
    assert np.array_equal(host(a.U), host(b.U)) and np.array_equal(host(a.y), host(b.y))
    hist = a.history(T)
    # the row pass runs first at t where delta_{t-1} < min(eps_d, eps_c) (and once after init)
    expect = 1 + sum(1 for h in hist[:-1] if h["delta"] < 1e-3)
    ra, rb = a.inspect("rows_run"), b.inspect("rows_run")
    log(f"one-pass rows-first d={d} r={r}: {ra} of {T} iterations (expected {expect}); steps: {rb}")
    assert ra == expect and ra > 20 and rb == 1
    gates = [bool(h["dual_step"]) for h in hist]
    Xh, _, _ = onlr.centre_and_normalise(X)
    ref = onlr.run(Xh, Z, K, alpha, beta, T=T, T_min=T, eps_d=3e-3, eps_c=1e-3, gates=gates)
    assert rel_max_err(host(a.U), ref.U) < U_TOL
    ys = onlr.stored_dual(ref.y)
    assert np.abs(host(a.y) - ys).max() <= 1e-4 * np.abs(ys).max()
    # one more iteration from the GPU's own iterate, taken by the oracle
    U_t, y_t = host(a.U), host(a.y)
    st = a.step()
    one = onlr.run(Xh, U_t, K, alpha, beta, T=1, T_min=1, project_init=False,
                   y0=onlr.dual_from_stored(y_t), gates=[bool(st["dual_step"])])
    assert rel_max_err(host(a.U), one.U) < U_TOL / 10


@pytest.mark.parametrize("steps_first", [0, 1])
def test_onepass_breakdown(steps_first):
    """A step that leaves no positive entry: the unnormalised update (zero) replaces the factor,
    on the first iteration after init (s from the row pass) and after a run (s from the Gram terms)."""
    from paper_2609_36074_amd import nlr
    n, K = 200, 3
    X, _, _ = gaussian_mixture(n, 100, 2, 9.0, seed=10)
    Z = np.ones((n, 36))
    alpha_bad = 1.0 / (2 * 1.0 * (K - 1)) * 1.5
    if steps_first:
        # one good iteration first, then a step size that leaves every entry below -0.4
        ctx = make_ctx(X, np.abs(standard_normal_factor(n, 36, seed=3)), K, 1e-3, 1.0, flags=SPLIT)
        ctx.run(1)
        ctx.set_params(alpha=100.0 / (2 * 1.0 * (K - 1)))
    else:
        ctx = make_ctx(X, Z, K, alpha_bad, 1.0, flags=SPLIT)
    with pytest.raises(nlr.NlrError) as e:
        ctx.run(1)
    assert e.value.status == nlr.NLR_EBREAKDOWN
    assert np.all(host(ctx.U) == 0.0)
    with pytest.raises(nlr.NlrError) as e:
        ctx.run(3)
    assert e.value.status == nlr.NLR_ESTATE


def test_onepass_beta_change_between_runs():
    """s of the first iteration after nlr_set_params comes from the stored Gram terms with the
    new beta; the trajectory still follows the oracle across the change."""
    X, Z, K, beta, alpha = _gated(100, 36)
    ctx = make_ctx(X, Z, K, alpha, beta, eps_d=3e-3, eps_c=1e-7, T_min=0, flags=SPLIT)
    T1, T2, beta2 = 150, 150, 0.5
    done1, _ = ctx.run(T1)
    ctx.set_params(beta=beta2)
    done2, _ = ctx.run(T2)
    assert done1 == T1 and done2 == T2
    hist = ctx.history(4096)
    gates = [bool(h["dual_step"]) for h in hist]
    Xh, _, _ = onlr.centre_and_normalise(X)
    r1 = onlr.run(Xh, Z, K, alpha, beta, T=T1, T_min=T1, eps_d=3e-3, eps_c=1e-7, gates=gates[:T1])
    r2 = onlr.run(Xh, r1.U, K, alpha, beta2, T=T2, T_min=T2, eps_d=3e-3, eps_c=1e-7, gates=gates[T1:],
                  project_init=False, y0=r1.y, t0=T1)
    err = rel_max_err(host(ctx.U), r2.U)
    log(f"one-pass beta change: {sum(gates)} dual steps, U err {err:.2e}")
    assert sum(gates) > 20
    assert err < U_TOL
    ys = onlr.stored_dual(r2.y)
    assert np.abs(host(ctx.y) - ys).max() <= 1e-4 * np.abs(ys).max()


def test_onepass_resume_flags():
    """Resuming from (U, y) with U_IN_OMEGA | KEEP_Y | X_NORMALISED continues the iteration."""
    from paper_2609_36074_amd import nlr
    X, Z, K, beta, alpha = _gated(128, 64)
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0)
    a = make_ctx(X, Z, K, alpha, beta, flags=SPLIT, **kw)
    a.run(120)
    b = make_ctx(X, Z, K, alpha, beta, flags=SPLIT, **kw)
    b.run(61)
    # X holds the split Xhat after a split init, so the resumed context gets Xhat (fp32) anew
    Xh, _, _ = onlr.centre_and_normalise(X)
    flags = nlr.NLR_INIT_U_IN_OMEGA | nlr.NLR_INIT_KEEP_Y | nlr.NLR_INIT_X_NORMALISED | SPLIT
    c = nlr.Context(to_dev(Xh.astype(np.float32)), K, b.U, b.y, alpha=alpha, beta=beta, flags=flags, **kw)
    c.run(59)
    assert rel_max_err(host(c.U), host(a.U)) < U_TOL


def test_onepass_nondefault_stream_and_profiling():
    """The one-pass form on a non-default stream gives the same iterate bitwise; with
    profiling on, its launches are timed under the pass and control kinds."""
    import torch
    X, Z, K, beta, alpha = _gated(128, 64)
    kw = dict(eps_d=3e-3, eps_c=1e-7, T_min=0, flags=SPLIT)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    a.run(40)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = make_ctx(X, Z, K, alpha, beta, stream=s, **kw)
        b.set_profiling(1)
        b.run(20)
        b.run(20)
    s.synchronize()
    assert np.array_equal(host(a.U), host(b.U)) and np.array_equal(host(a.y), host(b.y))
    times = {k: v for k, v in b.kernel_times().items() if v[1]}
    log(f"  one-pass launches timed: { {k: v[1] for k, v in times.items()} }")
    assert times["pass_bf"][1] == 40 and times["reduce_theta"][1] == 40
    assert all(v[0] > 0 for v in times.values())
