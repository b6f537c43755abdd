"""Checks that pin the fp64 oracle to the paper and to mathematics, not to itself.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with
something the paper or the mathematics fixes: closed forms, a hand-worked
iteration, a library routine, invariants of the method, brute force on tiny
inputs.  ``test_oracle.py`` runs them all; ``test_oracle_mutations.py`` plants
plausible mistakes in the oracle (on the CPU) and checks that some pin fails.

Functions look up oracle routines through the module objects at call time, so
a monkeypatched oracle is what they exercise.
"""
from __future__ import annotations

import json
import os

import numpy as np

from oracle import dense, kmeans, labels, nlr
from synth import gaussian_mixture, standard_normal_factor

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- Section 3
def pin_spectral_norm_library():
    """a = sigma_max(X_c) equals LAPACK's 2-norm (SVD)."""
    for seed, (n, d) in enumerate([(300, 7), (50, 20), (1000, 3)]):
        X = _rng(seed).standard_normal((n, d)) * _rng(seed + 9).uniform(0.1, 5.0, d)
        Xh, xbar, a = nlr.centre_and_normalise(X)
        Xc = X - X.mean(axis=0)
        ref = np.linalg.norm(Xc, 2)
        assert abs(a - ref) <= 1e-12 * ref, (a, ref)
        assert np.allclose(xbar, X.mean(axis=0), rtol=0, atol=1e-14 * np.abs(X).max())


def pin_spectral_norm_rank_one():
    """X = u v^T + 1 w^T  =>  X_c = (u - mean(u)) v^T, ||X_c||_2 = ||u - mean u|| ||v||."""
    g = _rng(3)
    u, v, w = g.standard_normal(40), g.standard_normal(6), g.standard_normal(6)
    X = np.outer(u, v) + np.outer(np.ones(40), w)
    _, _, a = nlr.centre_and_normalise(X)
    ref = np.linalg.norm(u - u.mean()) * np.linalg.norm(v)
    assert abs(a - ref) <= 1e-12 * ref, (a, ref)


def pin_normalised_invariants():
    """Xhat^T 1 = 0 and ||Xhat||_2 = 1 (Section 3); all-equal rows are rejected (a > 0)."""
    X = _rng(4).standard_normal((500, 9)) * 3.0 + 7.0
    Xh, _, _ = nlr.centre_and_normalise(X)
    assert np.abs(Xh.sum(axis=0)).max() < 1e-12
    assert abs(np.linalg.norm(Xh, 2) - 1.0) < 1e-12
    try:
        nlr.centre_and_normalise(np.ones((5, 3)))
    except ValueError:
        pass
    else:
        raise AssertionError("degenerate data accepted")


# ---------------------------------------------------------------- projection
def pin_projection_invariants():
    """Pi(V) >= 0, ||Pi(V)||_F^2 = K, idempotent on Omega (eq. projected-primal-step)."""
    g = _rng(5)
    for K in (1, 3, 7):
        V = g.standard_normal((30, 8))
        P = nlr.project_omega(V, K)
        assert P.min() >= 0.0
        assert abs(np.sum(P * P) - K) < 1e-12 * K
        assert np.allclose(nlr.project_omega(P, K), P, rtol=0, atol=1e-14)
        # zero pattern = non-positive entries of V
        assert np.array_equal(P > 0, V > 0)


def pin_projection_closed_form():
    """One positive entry v > 0 maps to sqrt(K) at that entry, zero elsewhere."""
    V = -np.ones((4, 3))
    V[2, 1] = 0.37
    P = nlr.project_omega(V, 5.0)
    ref = np.zeros((4, 3))
    ref[2, 1] = np.sqrt(5.0)
    assert np.allclose(P, ref, rtol=0, atol=1e-15)
    try:
        nlr.project_omega(-np.ones((3, 2)), 2.0)
    except FloatingPointError:
        pass
    else:
        raise AssertionError("projection of a non-positive matrix accepted")


def pin_projection_optimal_bruteforce():
    """Pi(V) is the closest point of Omega: ||V - Pi(V)|| <= ||V - Z|| for 10^4 random Z in Omega."""
    g = _rng(6)
    K = 2.0
    V = g.standard_normal((3, 2))
    V[0, 0] = abs(V[0, 0]) + 0.1
    P = nlr.project_omega(V, K)
    dP = np.linalg.norm(V - P)
    Z = np.abs(g.standard_normal((10_000, 3, 2))) * (g.uniform(size=(10_000, 3, 2)) < 0.7)
    nz = np.sqrt((Z * Z).sum(axis=(1, 2)))
    Z = Z[nz > 0] * (np.sqrt(K) / nz[nz > 0])[:, None, None]
    dZ = np.sqrt(((V[None] - Z) ** 2).sum(axis=(1, 2)))
    assert dP <= dZ.min() + 1e-12, (dP, dZ.min())


# ---------------------------------------------------------------- gradient
def _random_state(seed, n=12, d=3, r=3, K=2.0):
    g = _rng(seed)
    X = g.standard_normal((n, d))
    Xh, _, _ = nlr.centre_and_normalise(X)
    U = np.abs(g.standard_normal((n, r))) * 0.4
    y = g.standard_normal(n)
    return Xh, U, y, K


def pin_gradient_finite_differences():
    """Central differences of fhat_y (eq. normalized) match eq. (gradient) to 1e-7 relative."""
    for seed in range(3):
        Xh, U, y, _ = _random_state(10 + seed)
        beta = 0.7 + seed
        G = nlr.gradient(Xh, U, y, beta)
        eps = 1e-6
        num = np.zeros_like(U)
        for i in range(U.shape[0]):
            for j in range(U.shape[1]):
                E = np.zeros_like(U)
                E[i, j] = eps
                num[i, j] = (nlr.objective(Xh, U + E, y, beta) - nlr.objective(Xh, U - E, y, beta)) / (2 * eps)
        err = np.abs(num - G).max() / max(1e-12, np.abs(G).max())
        assert err < 1e-7, err


def pin_dense_cross_form():
    """Factored gradient/objective/step equal the explicit n x n form (Appendix A) to 1e-12."""
    for seed in range(3):
        g = _rng(20 + seed)
        n, d, r, K = 60, 4, 3, 3.0
        Xh, _, _ = nlr.centre_and_normalise(g.standard_normal((n, d)) + 2.0 * (np.arange(n) % 3)[:, None])
        U = nlr.project_omega(g.standard_normal((n, r)), K)
        y = g.standard_normal(n) * 0.3
        beta, alpha = 1.3, 0.02
        A = dense.dissimilarity(Xh)
        Gf = nlr.gradient(Xh, U, y, beta)
        Gd = dense.gradient_dense(A, U, y, beta)
        assert np.abs(Gf - Gd).max() <= 1e-12 * np.abs(Gd).max()
        of, od = nlr.objective(Xh, U, y, beta), dense.objective_dense(A, U, y, beta)
        assert abs(of - od) <= 1e-12 * max(1.0, abs(od))
        Up, _, st = nlr.primal_step(Xh, U, y, K, alpha, beta)
        Ud, yd, move = dense.step_dense(A, U, y, K, alpha, beta)
        assert np.abs(Up - Ud).max() <= 1e-12 * np.abs(Ud).max()
        res = nlr.run(Xh, U, K, alpha, beta, T=1, project_init=False, y0=y, gates=[True])
        assert np.abs(res.y - yd).max() <= 1e-12 * max(1.0, np.abs(yd).max())
        assert abs(res.records[0].delta - move) <= 1e-12


def pin_dense_trajectory_tiny():
    """Ten iterations of the factored loop agree with the dense loop on n = 400 to 1e-11."""
    X, lab, _ = gaussian_mixture(400, 5, 3, 25.0, seed=7)
    Xh, _, _ = nlr.centre_and_normalise(X)
    K, beta = 3.0, 1.0
    alpha = nlr.default_step_size(K, beta)
    Z = standard_normal_factor(400, 3, seed=8).astype(np.float64)
    gates = [t % 3 == 2 for t in range(10)]
    res = nlr.run(Xh, Z, K, alpha, beta, T=10, T_min=10, gates=gates, keep_trajectory=True)
    A = dense.dissimilarity(Xh)
    U = nlr.project_omega(Z, K)
    y = np.zeros(400)
    for t in range(10):
        U, yg, _ = dense.step_dense(A, U, y, K, alpha, beta)
        if gates[t]:
            y = yg
        assert np.abs(U - res.trajectory[t]).max() <= 1e-11 * np.abs(U).max(), t
        assert np.abs(y - res.duals[t]).max() <= 1e-11 * max(1.0, np.abs(y).max()), t


def pin_lipschitz_bound_valid():
    """Prop. 1: ||grad f(U) - grad f(V)|| <= L ||U - V|| on the ball ||U||_F <= sqrt(K); the
    constant-factor direction U = V + eps 1 1^T (where the penalty curvature is largest) and
    random pairs are sampled."""
    g = _rng(30)
    n, d, r, K, beta = 30, 3, 2, 2.0, 3.0
    Xh, _, _ = nlr.centre_and_normalise(g.standard_normal((n, d)))
    y = 0.1 * g.standard_normal(n)
    L = nlr.lipschitz_bound(y, beta, K)
    pairs = [(np.full((n, r), np.sqrt(K / (n * r))) * 0.999, np.full((n, r), 1e-5))]
    for _ in range(200):
        U = np.abs(g.standard_normal((n, r)))
        U *= np.sqrt(K) / np.linalg.norm(U) * 0.99
        pairs.append((U, 1e-4 * g.standard_normal((n, r))))
    worst = 0.0
    for U, D in pairs:
        V = U + D
        V *= min(1.0, np.sqrt(K) / np.linalg.norm(V))
        ratio = np.linalg.norm(nlr.gradient(Xh, U, y, beta) - nlr.gradient(Xh, V, y, beta)) / np.linalg.norm(U - V)
        worst = max(worst, ratio)
    assert worst <= L, (worst, L)
    assert worst > 0.5 * L, (worst, L)  # the sampled worst case is within a factor 2 of the bound


# ---------------------------------------------------------------- Alg. 1 pieces
def pin_hand_worked_iteration():
    """One iteration on n=2, d=1, K=r=1 worked by hand (tests/golden/hand_step_n2.json)."""
    g = json.load(open(os.path.join(GOLDEN, "hand_step_n2.json")))
    X = np.array(g["X"])
    Xh, xbar, a = nlr.centre_and_normalise(X)
    assert abs(a - g["a_norm"]) < 1e-14 and np.allclose(Xh, g["Xhat"], rtol=0, atol=1e-15)
    U0 = np.array(g["U0"])
    K, alpha, beta = g["K"], g["alpha"], g["beta"]
    y0 = np.zeros(2)
    G = nlr.gradient(Xh, U0, y0, beta)
    assert np.allclose(G, g["grad"], rtol=0, atol=1e-14), G
    assert abs(nlr.objective(Xh, U0, y0, beta) - g["objective0"]) < 1e-14
    res = nlr.run(Xh, U0, K, alpha, beta, T=1, gates=[True])
    rec = res.records[0]
    for k in ("a", "b", "h", "c"):
        assert abs(getattr(rec, k) - g["stats"][k]) < 1e-14, k
    assert np.allclose(res.U, g["U1"], rtol=0, atol=1e-14)
    assert abs(rec.delta - g["delta"]) < 1e-14
    assert abs(rec.delta_identity ** 2 - g["delta_sq_identity"]) < 1e-13
    assert abs(rec.rho - g["rho1"]) < 1e-14
    assert np.allclose(res.y, g["y1_if_gated"], rtol=0, atol=1e-13)
    assert rec.objective == g["objective0"] or abs(rec.objective - g["objective0"]) < 1e-14


def pin_movement_identity():
    """||cW - U||^2 = c^2 a + b - 2 c h (eq. movement-identity) on every logged step."""
    X, _, _ = gaussian_mixture(300, 4, 3, 16.0, seed=11)
    Xh, _, _ = nlr.centre_and_normalise(X)
    K = 3.0
    res = nlr.run(Xh, standard_normal_factor(300, 3, 12).astype(np.float64), K,
                  nlr.default_step_size(K), 1.0, T=60, T_min=60)
    for rec in res.records:
        assert abs(rec.delta ** 2 - rec.delta_identity ** 2) * K <= 1e-12 * K, rec


def pin_descent_fixed_dual():
    """Cor. 1 (eq. descent) on every step while y is fixed and alpha < 1/L; movement -> 0."""
    X, _, _ = gaussian_mixture(500, 6, 4, 16.0, seed=13)
    Xh, _, _ = nlr.centre_and_normalise(X)
    K, beta = 4.0, 1.0
    y = 0.05 * _rng(14).standard_normal(500)
    L = nlr.lipschitz_bound(y, beta, K)
    alpha = 0.9 / L
    res = nlr.run(Xh, standard_normal_factor(500, 4, 15).astype(np.float64), K, alpha, beta,
                  T=400, T_min=400, eps_d=0.0, y0=y, keep_trajectory=True)
    U_prev = nlr.project_omega(standard_normal_factor(500, 4, 15).astype(np.float64), K)
    f_prev = nlr.objective(Xh, U_prev, y, beta)
    for t, U in enumerate(res.trajectory):
        assert not res.records[t].gate
        f = nlr.objective(Xh, U, y, beta)
        bound = f_prev - (1 - alpha * L) / (2 * alpha) * np.sum((U - U_prev) ** 2)
        assert f <= bound + 1e-12 * max(1.0, abs(f_prev)), (t, f, bound)
        assert abs(res.records[t].objective - f_prev) <= 1e-12 * max(1.0, abs(f_prev))
        U_prev, f_prev = U, f
    d = np.array([r.delta for r in res.records])
    assert d[-50:].max() < 0.05 * d[:10].max(), (d[:10].max(), d[-50:].max())


def pin_dual_ascent_closed_form():
    """The gated dual step raises the Lagrangian by exactly beta ||h(U)||^2 (y+ = y + beta h)."""
    X, _, _ = gaussian_mixture(200, 3, 2, 25.0, seed=16)
    Xh, _, _ = nlr.centre_and_normalise(X)
    K, beta = 2.0, 2.5
    res = nlr.run(Xh, standard_normal_factor(200, 2, 17).astype(np.float64), K, 0.02, beta,
                  T=5, T_min=5, gates=[False, True, False, True, True], keep_trajectory=True)
    y_prev = np.zeros(200)
    for t in range(5):
        U, y = res.trajectory[t], res.duals[t]
        hU = nlr.constraint_h(U)
        gain = nlr.objective(Xh, U, y, beta) - nlr.objective(Xh, U, y_prev, beta)
        expect = beta * (hU @ hU) if res.records[t].gate else 0.0
        assert abs(gain - expect) <= 1e-12 * max(1.0, abs(expect)), (t, gain, expect)
        y_prev = y


def pin_breakdown():
    """Constant U0, K >= 2, alpha > 1/(2 beta (K-1)): Theta = 0, grad > 0 everywhere, W = 0."""
    X = _rng(18).standard_normal((50, 3))
    Xh, _, _ = nlr.centre_and_normalise(X)
    K, beta = 3.0, 1.0
    U0 = np.ones((50, 3))
    res = nlr.run(Xh, U0, K, 1.0 / (2 * beta * (K - 1)) * 1.5, beta, T=3)
    assert res.breakdown and res.iters == 0
    assert np.all(res.U == 0.0)


def pin_k1_fixed_point():
    """K = r = 1, y = 0: U = 1/sqrt(n) gives Theta = 0, q = 0, W = U, c = 1, delta = 0."""
    X = _rng(19).standard_normal((64, 5))
    Xh, _, _ = nlr.centre_and_normalise(X)
    U = np.full((64, 1), 1.0 / 8.0)
    res = nlr.run(Xh, U, 1.0, 0.3, 2.0, T=5, T_min=5, keep_trajectory=True)
    for rec, Ut in zip(res.records, res.trajectory):
        assert abs(rec.c - 1.0) < 1e-14 and rec.delta < 1e-14 and rec.rho < 1e-14
        assert np.abs(Ut - U).max() < 1e-14


def pin_lemma1_and_recovery():
    """Exact recovery: from a start inside the basin the iterate converges to U = H, the
    membership factor with one entry 1/sqrt(n_k) per row (Appendix D, "Recover cluster
    labels"), which is feasible and has sigma_max(U) = 1 (Lemma 1)."""
    n, d, K = 600, 5, 3
    thr = np.sqrt(kmeans.exact_recovery_threshold_sq(n, K, d))
    g = _rng(21)
    centers = None
    for _ in range(100):
        c = g.standard_normal((K, d)) * 6.0
        sep = min(np.linalg.norm(c[i] - c[j]) for i in range(K) for j in range(i + 1, K))
        if sep >= 2.0 * thr:
            centers = c
            break
    assert centers is not None
    lab = np.repeat(np.arange(K), n // K)
    g.shuffle(lab)
    X = centers[lab] + g.standard_normal((n, d))
    Xh, _, _ = nlr.centre_and_normalise(X)
    H = kmeans.membership(lab, K)
    beta = 2.0
    alpha = 1.8 * nlr.default_step_size(K, beta)
    U0 = H + np.abs(g.standard_normal((n, K))) / np.sqrt(n / K)
    res = nlr.run(Xh, U0, K, alpha, beta, T=20000, T_min=0, eps_d=3e-3, eps_c=1e-7)
    assert not res.breakdown and res.records[-1].stop, res.records[-1]
    U = res.U
    assert res.records[-1].rho < 1e-6
    s = np.linalg.svd(U, compute_uv=False)
    assert abs(s[0] - 1.0) < 1e-4, s
    assert kmeans.adjusted_rand_index(nlr.labels(U), lab) == 1.0
    assert np.abs(U - H).max() < 1e-6


def pin_random_start_recovery():
    """From the paper's random start Pi_Omega(Z) on a well-separated 4-cluster mixture the
    converged labels equal the truth (ARI = 1)."""
    X, lab, _ = gaussian_mixture(2000, 16, 4, 25.0, seed=1)
    Xh, _, _ = nlr.centre_and_normalise(X)
    Z = standard_normal_factor(2000, 4, 2).astype(np.float64)
    res = nlr.run(Xh, Z, 4, 1.8 * nlr.default_step_size(4, 2.0), 2.0, T=20000, T_min=0,
                  eps_d=3e-3, eps_c=1e-7)
    assert res.records[-1].stop and res.records[-1].rho < 1e-6
    assert kmeans.adjusted_rand_index(nlr.labels(res.U), lab) == 1.0


def pin_stored_dual_convention():
    """The dual buffer stores ytilde = y / sqrt(n), and the dual step y += (beta/sqrt(n)) q is
    ytilde += (beta/n) q on it (Section 3, storage and penalty convention): hand values, the
    hand-worked step's gated dual, and the effective multiplier of eq. (dualnormalized)."""
    y = np.array([2.0, -4.0, 6.0, 0.0])           # n = 4, sqrt(n) = 2
    assert np.array_equal(nlr.stored_dual(y), np.array([1.0, -2.0, 3.0, 0.0]))
    assert np.array_equal(nlr.dual_from_stored(np.array([1.0, -2.0, 3.0, 0.0])), y)
    g = json.load(open(os.path.join(GOLDEN, "hand_step_n2.json")))
    yt = nlr.stored_dual(np.array(g["y1_if_gated"]))
    assert np.allclose(yt, g["ytilde1_if_gated"], rtol=0, atol=1e-14), yt
    assert np.allclose(nlr.dual_from_stored(np.array(g["ytilde1_if_gated"])), g["y1_if_gated"],
                       rtol=0, atol=1e-14)
    # ybar_eff = y/sqrt(n) + (beta/n) g(U): the stored dual plus the stored-scale penalty term
    _, U, yr, beta = _random_state(31)
    ybar = nlr.effective_multiplier(U, yr, beta)
    n = U.shape[0]
    assert np.allclose(ybar, nlr.stored_dual(yr) + (beta / n) * (U @ U.sum(axis=0) - 1.0),
                       rtol=0, atol=1e-14)


def pin_adjusted_rand_index():
    """ARI by pair counting: a hand-worked contingency table (8/33), relabelling and
    symmetry, and scikit-learn's adjusted_rand_score on random labelings."""
    # table [[2,1,0],[0,1,2]]: sum C(n_ij,2) = 2, rows 6, cols 3, C(6,2) = 15:
    # (2 - 6*3/15) / ((6+3)/2 - 6*3/15) = 0.8 / 3.3 = 8/33
    a = np.array([0, 0, 0, 1, 1, 1])
    b = np.array([0, 0, 1, 1, 2, 2])
    assert abs(kmeans.adjusted_rand_index(a, b) - 8.0 / 33.0) < 1e-15
    assert abs(kmeans.adjusted_rand_index(b, a) - 8.0 / 33.0) < 1e-15
    assert kmeans.adjusted_rand_index(a, 5 - 3 * a) == 1.0
    # one class against all-distinct labels: every pair split, ARI = 0
    assert abs(kmeans.adjusted_rand_index(np.zeros(5, int), np.arange(5))) < 1e-15
    from sklearn.metrics import adjusted_rand_score
    rng = _rng(32)
    for n, ka, kb in [(40, 3, 4), (200, 5, 5), (17, 2, 6)]:
        x, z = rng.integers(0, ka, n), rng.integers(0, kb, n)
        assert abs(kmeans.adjusted_rand_index(x, z) - adjusted_rand_score(x, z)) < 1e-12


def pin_recovery_threshold():
    """eq. (exact_recovery_threshold) at special cases: with d = 0 it is 8 log n (natural log);
    with K d = 3 n log n the square root is 2, so the threshold is 12 log n; it grows with d."""
    for n in (10, 1000, 123457):
        assert abs(kmeans.exact_recovery_threshold_sq(n, 4, 0) - 8.0 * np.log(n)) < 1e-12 * np.log(n)
        d = 3.0 * n * np.log(n)
        assert abs(kmeans.exact_recovery_threshold_sq(n, 1, d) - 12.0 * np.log(n)) < 1e-12 * np.log(n)
        assert abs(kmeans.exact_recovery_threshold_sq(n, 2, d / 2) - 12.0 * np.log(n)) < 1e-12 * np.log(n)
    v = [kmeans.exact_recovery_threshold_sq(10_000, 8, d) for d in (1, 10, 100, 1000)]
    assert all(x < y for x, y in zip(v, v[1:])), v


# ---------------------------------------------------------------- brute force K-means
def pin_partition_counts():
    """The partition enumerator yields S(n, k) partitions (Stirling numbers, golden table)."""
    tab = json.load(open(os.path.join(GOLDEN, "stirling_second_kind.json")))["values"]
    for n, row in tab.items():
        for k, cnt in row.items():
            if int(n) > 10:
                continue
            got = sum(1 for _ in kmeans.partitions(int(n), int(k)))
            assert got == cnt, (n, k, got, cnt)


def pin_partition_identity():
    """J(G) as within-cluster sums equals ||X||^2 - <X X^T, Z_G> (eq. partition) for every partition."""
    X = _rng(22).standard_normal((7, 2))
    for lab in kmeans.partitions(7, 3):
        a = kmeans.within_ss(X, lab, 3)
        b = kmeans.within_ss_trace(X, lab, 3)
        assert abs(a - b) <= 1e-12 * max(1.0, a)


def pin_nlr_finds_exact_kmeans():
    """On clear 10-point instances the converged NLR labels are the brute-force K-means optimum."""
    g = _rng(23)
    for K, trial in [(2, 0), (3, 1), (3, 2)]:
        centers = np.array([[0.0, 0.0], [12.0, 0.0], [0.0, 12.0]])[:K]
        lab = np.arange(10) % K
        X = centers[lab] + 0.8 * g.standard_normal((10, 2))
        best, args = kmeans.brute_force(X, K)
        assert len(args) == 1
        Xh, _, _ = nlr.centre_and_normalise(X)
        res = nlr.run(Xh, np.abs(g.standard_normal((10, K))) + 0.1, K, 0.02, 1.0, T=50000,
                      T_min=0, eps_d=1e-5, eps_c=1e-7)
        est = nlr.labels(res.U)
        assert kmeans.same_partition(est, args[0]), (trial, est, args[0])
        assert abs(kmeans.within_ss(X, est, K) - best) <= 1e-9 * best


def pin_hand_kmeans():
    """X = [0, 1, 10, 11] (1-D), K = 2: the optimum {0,1},{10,11} with J = 1 (by hand)."""
    X = np.array([[0.0], [1.0], [10.0], [11.0]])
    best, args = kmeans.brute_force(X, 2)
    assert abs(best - 1.0) < 1e-14
    assert len(args) == 1 and kmeans.same_partition(args[0], np.array([0, 0, 1, 1]))


def _data_start_instance(seed=3, n=400, d=12, K=4):
    X, _, _ = gaussian_mixture(n, d, K, 25.0, seed=seed)
    Xh, _, _ = nlr.centre_and_normalise(X)
    Z = standard_normal_factor(n, K, seed=seed + 1).astype(np.float64)
    return Xh, Z, K


def pin_data_start_is_qr_of_range_sample():
    """Appendix D: Q is the orthonormal factor of V = Xhat Xhat^T Z (numpy QR, signs made positive)."""
    Xh, Z, K = _data_start_instance()
    U0, Q = nlr.data_informed_start(Xh, Z, K)
    V = Xh @ (Xh.T @ Z)
    q, r = np.linalg.qr(V)
    q = q * np.sign(np.diag(r))[None, :]
    assert np.abs(Q - q).max() < 1e-10
    assert np.abs(Q.T @ Q - np.eye(K)).max() < 1e-10
    assert U0.min() >= 0.0 and abs(np.sum(U0 * U0) - K) < 1e-10


def pin_data_start_column_scaling_invariance():
    """The orthonormal factor of V D (D positive diagonal) is that of V: Q(Z D) = Q(Z)."""
    Xh, Z, K = _data_start_instance(seed=5)
    D = np.array([0.5, 3.0, 1.7, 11.0])[:K]
    _, Q1 = nlr.data_informed_start(Xh, Z, K)
    _, Q2 = nlr.data_informed_start(Xh, Z * D[None, :], K)
    assert np.abs(Q1 - Q2).max() < 1e-9


def pin_data_start_lowers_objective():
    """Appendix D reports a lower initial augmented Lagrangian than the random start Pi(Z)."""
    Xh, Z, K = _data_start_instance(seed=7)
    U0, _ = nlr.data_informed_start(Xh, Z, K)
    y = np.zeros(Xh.shape[0])
    assert nlr.objective(Xh, U0, y, 1.0) < nlr.objective(Xh, nlr.project_omega(Z, K), y, 1.0)


# ---------------------------------------------------------------- label recovery (Appendix D)
def pin_lloyd_hand():
    """x = 0, 1, 10, 11 from the centroids at rows 0 and 1, by hand: pass 1 labels (0, 1, 1, 1),
    means (0, 22/3); pass 2 labels (0, 0, 1, 1), means (0.5, 10.5); pass 3 changes nothing."""
    E = np.array([[0.0], [1.0], [10.0], [11.0]])
    lab, passes, C = labels.lloyd(E, [0, 1])
    assert lab.tolist() == [0, 0, 1, 1] and passes == 3
    assert np.allclose(C[:, 0], [0.5, 10.5], rtol=0, atol=1e-15)


def pin_lloyd_tie_lowest_index():
    """A row equidistant from two centroids takes the lower index (x = 1 between 0 and 2)."""
    E = np.array([[0.0], [2.0], [1.0]])
    lab, passes, _ = labels.lloyd(E, [0, 1])
    assert lab.tolist() == [0, 1, 0] and passes == 2


def pin_nearest_is_euclidean():
    """nearest() against scipy's Euclidean distances (a library route), with a point that L1 and
    Euclidean distances assign differently: (2.1, 0) is Euclidean-nearest to (2, 2), not (0, 0)."""
    from scipy.spatial.distance import cdist
    C = np.array([[0.0, 0.0], [2.0, 2.0], [-3.0, 1.0]])
    E = np.concatenate([np.array([[2.1, 0.0]]), _rng(25).standard_normal((50, 2)) * 3.0])
    lab = labels.nearest(E, C)
    assert lab[0] == 1
    assert np.array_equal(lab, np.argmin(cdist(E, C), axis=1))


def pin_lloyd_brute_force_optimum():
    """Well-separated points: Lloyd from one seed per group ends at the exact K-means optimum."""
    rng = _rng(21)
    K, per = 3, 3
    centres = np.array([[0.0, 0.0], [20.0, 0.0], [0.0, 20.0]])
    X = np.concatenate([c + rng.standard_normal((per, 2)) for c in centres])
    lab, passes, _ = labels.lloyd(X, [0, per, 2 * per])
    best, args = kmeans.brute_force(X, K)
    assert any(kmeans.same_partition(lab, a) for a in args)
    assert abs(kmeans.within_ss(X, lab, K) - best) <= 1e-12 * best


def pin_lloyd_fixed_point():
    """A converged result is a fixed point: every row is nearest to the mean of its own group."""
    rng = _rng(22)
    E = rng.standard_normal((300, 3))
    lab, passes, C = labels.lloyd(E, [0, 1, 2, 3], max_iter=500)
    assert passes < 500
    means = np.array([E[lab == k].mean(axis=0) for k in range(4)])
    assert np.array_equal(labels.nearest(E, means), lab)


def pin_embedding_spans_leading_singular_space():
    """The embedding spans the leading eigenvectors of U^T U mapped by U: E E^T = P P^T with
    P = U V_K Lambda_K^(-1/2) (eigh of the Gram matrix, a second library route)."""
    rng = _rng(23)
    U = np.abs(rng.standard_normal((60, 6))) * np.array([5.0, 4.0, 3.0, 1.0, 0.5, 0.1])
    E = labels.spectral_embedding(U, 3)
    lam, V = np.linalg.eigh(U.T @ U)
    P = U @ V[:, ::-1][:, :3] / np.sqrt(lam[::-1][:3])[None, :]
    assert np.abs(E @ E.T - P @ P.T).max() < 1e-10
    assert np.abs(E.T @ E - np.eye(3)).max() < 1e-12


def pin_spectral_labels_exact_recovery():
    """Under exact recovery U = H (rows constant within clusters, Appendix D) the labels are the
    partition, also with r > K extra columns carrying a small perturbation."""
    rng = _rng(24)
    truth = np.repeat(np.arange(4), [7, 12, 5, 9])
    rng.shuffle(truth)
    H = kmeans.membership(truth, 4)
    seeds = [int(np.flatnonzero(truth == k)[0]) for k in range(4)]
    lab, _ = labels.spectral_labels(H, 4, seeds)
    assert kmeans.same_partition(lab, truth)
    U = np.concatenate([H, 1e-3 * np.abs(rng.standard_normal((H.shape[0], 2)))], axis=1)
    lab2, _ = labels.spectral_labels(U, 4, seeds)
    assert kmeans.same_partition(lab2, truth)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_") and callable(v)]
