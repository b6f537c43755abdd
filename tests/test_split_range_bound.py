"""The range precondition of the split W operand (CPU, on the fp64 oracle).

The fused split forms store 2^10 w in fp16, finite for w <= 65504 / 2^10 ~ 64.  For U in
Omega (|u_ij| <= sqrt(K)) every gradient entry of eq. (gradient) is bounded by
sqrt(K) (2 + 2 ||y|| + 2 beta (K + 1)) (|x_i^T Xhat^T u_j| <= sqrt(K) since ||Xhat||_2 = 1;
|p_j| <= sqrt(K n); |q_i| <= K sqrt(n) + 1), which is at most sqrt(K) L(y) with L of Prop. 1
(eq. L).  So a step alpha <= 1/L(y) keeps |w| <= 2 sqrt(K) <= 16 at K <= 64.  Checked on
random and adversarial factors in Omega with random duals, and the bound is not slack by
orders of magnitude (the worst case here comes within a factor 20 of it)."""
import numpy as np

from oracle import nlr as onlr
from synth import gaussian_mixture


def _cases():
    rng = np.random.default_rng(5)
    for n, d, K, r in [(400, 8, 4, 4), (1000, 32, 16, 16), (600, 64, 64, 64), (300, 12, 10, 30)]:
        X, _, _ = gaussian_mixture(n, d, max(K, 2), 9.0, seed=n)
        Xh, _, _ = onlr.centre_and_normalise(X)
        for kind in ("random", "one-row", "one-column"):
            if kind == "random":
                V = np.abs(rng.standard_normal((n, r)))
            elif kind == "one-row":      # all mass on one row: |u| = sqrt(K / r) per entry there
                V = np.zeros((n, r)); V[0] = 1.0
            else:                        # all mass in one column
                V = np.zeros((n, r)); V[:, 0] = 1.0
            U = onlr.project_omega(V, K)
            for yscale in (0.0, 1.0, 30.0):
                y = yscale * rng.standard_normal(n)
                for beta in (0.5, 1.0, 4.0):
                    yield Xh, U, y, K, beta


def test_gradient_entry_bound_and_w_range():
    worst = 0.0
    for Xh, U, y, K, beta in _cases():
        G = onlr.gradient(Xh, U, y, beta)
        bound = np.sqrt(K) * (2 + 2 * np.linalg.norm(y) + 2 * beta * (K + 1))
        assert np.abs(G).max() <= bound * (1 + 1e-12)
        L = onlr.lipschitz_bound(y, beta, K)
        assert bound <= np.sqrt(K) * L
        W = np.maximum(U - G / L, 0.0)
        assert W.max() <= 2 * np.sqrt(K) * (1 + 1e-12)
        assert W.max() < 65504.0 / 1024.0
        worst = max(worst, np.abs(G).max() / bound)
    assert worst > 0.05, worst
