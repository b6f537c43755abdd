"""The seeded input generator: determinism, shapes, cluster-size rules (CPU only)."""
import numpy as np

from synth import WORKLOADS, cluster_sizes, gaussian_mixture, make_workload, standard_normal_factor


def test_deterministic_and_thread_independent():
    a = gaussian_mixture(600_000, 5, 3, 4.0, seed=3, threads=1)
    b = gaussian_mixture(600_000, 5, 3, 4.0, seed=3, threads=7)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    z1 = standard_normal_factor(300_000, 4, seed=2, threads=1)
    z2 = standard_normal_factor(300_000, 4, seed=2, threads=5)
    assert np.array_equal(z1, z2)
    c = gaussian_mixture(600_000, 5, 3, 4.0, seed=4, threads=2)
    assert not np.array_equal(a[0], c[0])


def test_sizes_rules():
    g = np.random.default_rng(0)
    for rule in ("equal", "dirichlet5", "zipf1.1"):
        s = cluster_sizes(100_003, 17, rule, g)
        assert s.sum() == 100_003 and s.min() >= 1
    z = cluster_sizes(10_000, 8, "zipf1.1", g)
    assert np.all(np.diff(z) <= 0)


def test_tiny_workload_shape_and_moments():
    X, Z, lab, wl = make_workload("tiny")
    assert X.shape == (2000, 16) and X.dtype == np.float32
    assert Z.shape == (2000, 4) and Z.dtype == np.float32
    assert np.bincount(lab).tolist() == [500] * 4
    # within-cluster noise is N(0, I)
    for k in range(4):
        R = X[lab == k] - X[lab == k].mean(axis=0)
        assert abs(R.var() - 1.0) < 0.05
    assert abs(Z.mean()) < 0.05 and abs(Z.std() - 1.0) < 0.05


def test_embedding_rows_unit_norm():
    wl = WORKLOADS["embed2m"]
    X, Z, lab, _ = make_workload(wl, n=5000)
    assert X.shape == (5000, 768)
    assert np.allclose(np.linalg.norm(X, axis=1), 1.0, atol=1e-5)
    counts = np.bincount(lab, minlength=256)
    assert counts[0] > counts[-1]


def test_rows_is_a_true_prefix_of_the_full_draw():
    """make_workload(rows=m) returns bitwise the first m rows of the full draw (the CPU
    baseline's sample), across a generator chunk boundary; n=m is a different draw."""
    full = make_workload("gmm1m")
    m = 300_000  # beyond one 2^18-row chunk
    pre = make_workload("gmm1m", rows=m)
    for a, b in zip(full[:3], pre[:3]):
        assert np.array_equal(a[:m], b)
    other = make_workload("gmm1m", n=m)
    assert not np.array_equal(other[0], pre[0])


def test_table2_workloads_separation():
    """The Table 2 stand-ins: balanced mixtures whose closest pair of centres sits at
    gamma * CNRbar (gamma = 1); CNRbar agrees with the oracle's exact-recovery threshold
    (Section 2), written there independently."""
    from oracle import kmeans
    from synth import TABLE2, cnr_bar
    for name, (n, d, K, r) in {"t2k20": (1_000_000, 50, 20, 30), "t2k100": (1_000_000, 200, 100, 300)}.items():
        wl = TABLE2[name]
        assert (wl.n, wl.d, wl.K, wl.r, wl.sizes) == (n, d, K, r, "equal")
        assert abs(cnr_bar(n, K, d) ** 2 / kmeans.exact_recovery_threshold_sq(n, K, d) - 1.0) < 1e-12
        X, lab, C = gaussian_mixture(n, d, K, 1.0, seed=0, rows=20_000, min_separation=cnr_bar(n, K, d))
        dist = np.sqrt(((C[:, None, :] - C[None, :, :]) ** 2).sum(-1)) + np.diag([np.inf] * K)
        assert abs(dist.min() / cnr_bar(n, K, d) - 1.0) < 1e-12
        # unit within-cluster noise; the prefix is a true prefix of the make_workload draw
        k0 = lab[0]
        R = X[lab == k0] - C[k0]
        assert abs(R.var() - 1.0) < 0.05
        Xw, Zw, lw, _ = make_workload(name, rows=2000)
        assert np.array_equal(Xw, X[:2000]) and np.array_equal(lw, lab[:2000]) and Zw.shape == (2000, r)
