"""The allocation-free entry point nlr_solve_static (init + run in one call, its scratch a
device array inside the library) against the existing entry points nlr_init + nlr_run on
fresh copies of the same seeded inputs, through the C ABI: U and the stored dual to the
parity bar, the same iteration count and last record.  Three calls in a row, each on a
smaller problem than the one before (one-pass split, single-Xhat-pass split, two-pass
fp32), so that every later call runs on the array the previous call left behind."""
import numpy as np
import pytest

from gpu_util import U_TOL, host, log, make_ctx, rel_max_err, to_dev
from oracle import nlr as onlr
from synth import gaussian_mixture, make_workload, standard_normal_factor

pytestmark = pytest.mark.gpu

SPLIT, TWO_PASS = 8, 16


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _case(name):
    if name == "one-pass":
        X, _, _ = gaussian_mixture(3000, 128, 4, 25.0, seed=1)
        Z = standard_normal_factor(3000, 64, seed=2)
        K, beta = 4, 2.0
        return X, Z, K, beta, 1.8 * onlr.default_step_size(K, beta), SPLIT, 300, 3e-3, 1e-3
    if name == "single-pass":
        X, _, _ = gaussian_mixture(1500, 64, 16, 9.0, seed=4)
        Z = standard_normal_factor(1500, 16, seed=5)
        return X, Z, 16, 1.0, onlr.default_step_size(16), SPLIT, 200, 1e-4, 1e-4
    X, Z, _, wl = make_workload("tiny")
    X, Z = X[:700], Z[:700]
    return X, Z, wl.K, 1.0, onlr.default_step_size(wl.K), TWO_PASS, 50, 1e-4, 1e-4


def test_solve_static_matches_init_and_run():
    import torch
    from paper_2609_36074_amd import nlr
    for name in ("one-pass", "single-pass", "two-pass"):
        X, Z, K, beta, alpha, flags, T, eps_d, eps_c = _case(name)
        n, d = X.shape
        r = Z.shape[1]
        log(f"no-alloc {name}: n={n} d={d} r={r} K={K} flags={flags} T={T}")
        ref = make_ctx(X, Z, K, alpha, beta, eps_d=eps_d, eps_c=eps_c, T_min=0, flags=flags)
        done_ref, last_ref = ref.run(T)
        U_ref, y_ref = host(ref.U), host(ref.y)
        ref.close()
        Xt, Ut = to_dev(X), to_dev(Z)
        yt = torch.full((n,), 7.0, dtype=torch.float32, device=Xt.device)  # zeroed by the call
        p = nlr.NlrParams(alpha, beta, eps_d, eps_c, 0, 0)
        stream = torch.cuda.current_stream().cuda_stream
        st, done, last = nlr.nlr_solve_static(Xt.data_ptr(), n, d, K, r, Ut.data_ptr(), yt.data_ptr(), p, flags,
                                              T, stream)
        torch.cuda.synchronize()
        assert st == nlr.NLR_OK, nlr.status_string(st)
        U, y = host(Ut), host(yt)
        err = rel_max_err(U, U_ref)
        ymax = np.abs(y_ref).max()
        yerr = float(np.abs(y - y_ref).max()) / ymax if ymax > 0 else float(np.abs(y).max())
        log(f"  done {done} (ref {done_ref}); U err {err:.2e} (bitwise {np.array_equal(U, U_ref)}); "
            f"y err {yerr:.2e}; dual steps in the last record {last['dual_step']}")
        assert done == done_ref == T
        assert err < U_TOL and yerr < U_TOL
        assert last["t"] == last_ref["t"] == T - 1
        assert abs(last["objective"] - last_ref["objective"]) <= 1e-5 * max(1.0, abs(last_ref["objective"]))
        assert last["dual_step"] == last_ref["dual_step"]
