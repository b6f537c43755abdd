"""nlr_run replays the iterations after a call's first one as captured graphs (one
and eight iterations) while profiling is off.  Checked here for every product form:
a context driven by nlr_run, with single steps, a change of the step arguments
(which drops the graphs), profiling switched on and off, and the stop flag in
between, holds the same factor and dual, bit for bit, after every segment as a
context driven by nlr_step alone.  Each nlr_run replays the graphs several times
with the program's own work (reads, single steps) between the calls.
"""
import numpy as np
import pytest

from gpu_util import host, log, make_ctx
from oracle import nlr as onlr
from synth import gaussian_mixture, standard_normal_factor

pytestmark = pytest.mark.gpu

SPLIT, TWO_PASS = 8, 16


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


# (n, d, r, flags, form, T_min): one shape per iteration form; with T_min above every
# iteration of the plan the one-pass form's replays leave out the row pass
FORMS = [(2000, 16, 4, 0, "single-Xhat-pass", 0), (2000, 16, 4, TWO_PASS, "two-pass", 0),
         (3000, 32, 18, SPLIT, "single-Xhat-pass", 0), (3000, 100, 36, SPLIT, "one-pass", 0),
         (3000, 32, 10, SPLIT, "one-pass", 10**6),
         (3000, 100, 36, SPLIT, "one-pass", 10**6), (2000, 16, 4, SPLIT, "one-pass", 10**6),
         (3000, 256, 40, SPLIT, "two-pass-panel", 0), (1000, 13, 5, 0, "two-pass", 0)]


@pytest.mark.parametrize("n,d,r,flags,form,T_min", FORMS)
def test_graph_replay_equals_steps(n, d, r, flags, form, T_min):
    from paper_2609_36074_amd import nlr
    K, beta = 4, 2.0
    assert nlr.FORM_NAMES[nlr.nlr_iteration_form(n, d, r, K, flags)] == form
    X, _, _ = gaussian_mixture(n, d, K, 25.0, seed=1)
    Z = standard_normal_factor(n, r, seed=2).astype(np.float64)
    alpha = 1.8 * onlr.default_step_size(K, beta)
    kw = dict(eps_d=3e-3, eps_c=1e-9, T_min=T_min, flags=flags)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    log(f"graph replay {form} n={n} d={d} r={r} flags={flags} T_min={T_min}")

    def same(tag):
        for name in ("U", "y"):
            assert np.array_equal(host(getattr(a, name)), host(getattr(b, name))), (tag, name)

    def steps(k):
        for _ in range(k):
            b.step(with_stats=False)

    # (action on a, matching action on b)
    plan = [("run", 37), ("step", 1), ("run", 9), ("run", 8), ("run", 1), ("params", 1.5),
            ("run", 41), ("prof", True), ("run", 10), ("prof", False), ("run", 70)]
    t = 0
    for op, v in plan:
        if op == "run":
            done, _ = a.run(v)
            assert done == v
            steps(v)
            t += v
        elif op == "step":
            a.step(with_stats=False)
            steps(1)
            t += 1
        elif op == "params":
            a.set_params(beta=v)
            b.set_params(beta=v)
        else:
            a.set_profiling(v)
        same(f"{op} {v} at t={t}")
    gates = sum(h["dual_step"] for h in a.history(t))
    log(f"  {t} iterations, {gates} dual steps: bitwise equal after every segment")


def test_graph_replay_stop_between_polls():
    """The stopping rule fires inside a replayed graph: the kernels after it return at
    entry, nlr_run reports the iteration it stopped at, and a further nlr_run continues
    from there as nlr_step does."""
    K, beta = 4, 2.0
    X, _, _ = gaussian_mixture(2000, 16, K, 25.0, seed=1)
    Z = standard_normal_factor(2000, 4, seed=2).astype(np.float64)
    alpha = 1.8 * onlr.default_step_size(K, beta)
    kw = dict(eps_d=3e-3, eps_c=1e-3, T_min=5)
    a = make_ctx(X, Z, K, alpha, beta, **kw)
    b = make_ctx(X, Z, K, alpha, beta, **kw)
    done, last = a.run(3000)
    assert done < 3000 and last["stop"] == 1
    k = 0
    while True:
        st = b.step()
        k += 1
        if st["stop"]:
            break
        assert k < 3000
    assert k == done
    for name in ("U", "y"):
        assert np.array_equal(host(getattr(a, name)), host(getattr(b, name))), name
    a.set_params(eps_c=1e-9)
    b.set_params(eps_c=1e-9)
    a.run(19)
    for _ in range(19):
        b.step(with_stats=False)
    for name in ("U", "y"):
        assert np.array_equal(host(getattr(a, name)), host(getattr(b, name))), name
