"""Second, structurally different fp64 oracle: the explicit n x n form.

TEST INFRASTRUCTURE ONLY (see ``oracle.nlr``).  For small n it builds the
dissimilarity matrix Ahat = -Xhat Xhat^T explicitly and writes the gradient in
the form used in the proof of Prop. 1 (Appendix A):

    grad f(U) = 2 Ahat U + e ybar(U)^T U + ybar(U) e^T U,
    e = 1_n / sqrt(n),  ybar(U) = y + beta h(U),  h(U) = U U^T e - e.

It shares no helper with ``oracle.nlr`` so that the two cross-check each other:
the factored oracle never forms Ahat and writes the gradient with the
effective multiplier of eq. (dualnormalized) instead.
"""
from __future__ import annotations

import numpy as np


def dissimilarity(Xhat: np.ndarray) -> np.ndarray:
    """Ahat = -Xhat Xhat^T (Section 3), n x n."""
    Xhat = np.asarray(Xhat, dtype=np.float64)
    return -(Xhat @ Xhat.T)


def objective_dense(A: np.ndarray, U: np.ndarray, y: np.ndarray, beta: float) -> float:
    """<A, U U^T> + y^T h(U) + beta/2 ||h(U)||^2 with h(U) = U U^T e - e."""
    n = U.shape[0]
    e = np.full(n, 1.0 / np.sqrt(n))
    Z = U @ U.T
    hU = Z @ e - e
    return float(np.sum(A * Z) + y @ hU + 0.5 * beta * hU @ hU)


def gradient_dense(A: np.ndarray, U: np.ndarray, y: np.ndarray, beta: float) -> np.ndarray:
    n = U.shape[0]
    e = np.full(n, 1.0 / np.sqrt(n))
    Z = U @ U.T
    ybar = y + beta * (Z @ e - e)
    return 2.0 * (A @ U) + np.outer(e, ybar @ U) + np.outer(ybar, e @ U)


def step_dense(A: np.ndarray, U: np.ndarray, y: np.ndarray, K: float, alpha: float,
               beta: float):
    """One primal step and the gated dual step, written independently.

    Returns (U_plus, y_plus_if_gated, movement) where the projection is
    sqrt(K) V_+ / ||V_+||_F and the dual step is y + beta h(U_plus).
    """
    V = U - alpha * gradient_dense(A, U, y, beta)
    Vp = np.where(V > 0.0, V, 0.0)
    Up = np.sqrt(K) * Vp / np.linalg.norm(Vp.ravel())
    n = U.shape[0]
    e = np.full(n, 1.0 / np.sqrt(n))
    y_gated = y + beta * ((Up @ (Up.T @ e)) - e)
    move = float(np.linalg.norm((Up - U).ravel()) / np.sqrt(K))
    return Up, y_gated, move
