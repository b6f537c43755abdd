"""fp64 CPU oracle of the spectrally normalised NLR iteration (GEM-KMeans).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this
module: only the tests, the smoke check and the CPU-baseline leg of the
benchmark use it.  It shares no code with the HIP library.

It is the plain, unfused iteration in float64, step by step, so that it can be
read against the paper:

* centring and spectral normalisation, Section 3 ("Scaling Issues"):
  X_c = X - 1 xbar^T, a = ||X_c||_2, Xhat = X_c / a, Ahat = -Xhat Xhat^T;
* the normalised augmented Lagrangian, eq. (normalized):
  fhat_y(U) = <Ahat, U U^T> + y^T h(U) + beta/2 ||h(U)||^2, h = g / sqrt(n),
  g(U) = U U^T 1 - 1;
* its gradient, eq. (gradient), with the effective multiplier of
  eq. (dualnormalized): ybar_eff = y/sqrt(n) + (beta/n) g(U);
* the projection onto Omega = {U >= 0, ||U||_F^2 = K}, eq.
  (projected-primal-step): Pi(W) = sqrt(K) W_+ / ||W_+||_F;
* the loop of Algorithm 1 (Section 4.3): primal step, normalisation
  breakdown test, movement, residual, gated dual ascent
  y <- y + (beta/sqrt(n)) q, stopping rule;
* Prop. 1 (eq. L) for the fixed-dual smoothness bound;
* the data-informed starting factor of Appendix D (range finder on the Gram
  matrix, Cholesky QR in feature space, projection onto Omega).

Unlike the GPU path it forms the full n x r gradient, takes the exact fp64
normalising multiplier c = sqrt(K / ||W||_F^2) and measures the movement
directly as ||U_{t+1} - U_t||_F / sqrt(K) (the value of the movement identity,
eq. (movement-identity), is logged beside it).

The multiplier ``y`` here is the paper's mathematical dual for h.  The GPU
stores ytilde = y / sqrt(n); use ``stored_dual`` / ``dual_from_stored``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

BREAKDOWN_NU = 1e-20  # normalisation breakdown threshold on ||W||_F (Alg. 1)


# ----------------------------------------------------------------------------
# Section 3: centring and spectral normalisation
# ----------------------------------------------------------------------------
def spectral_norm(Xc: np.ndarray) -> float:
    """Largest singular value of Xc, from the d x d Gram matrix Xc^T Xc.

    sigma_max(Xc)^2 = lambda_max(Xc^T Xc); for tall data the Gram matrix is
    the cheap route (the paper's initialisation reuses C = X^T X as well,
    Appendix D).
    """
    Xc = np.asarray(Xc, dtype=np.float64)
    C = Xc.T @ Xc
    lam = np.linalg.eigvalsh(C)[-1]
    return float(np.sqrt(max(lam, 0.0)))


def centre_and_normalise(X: np.ndarray):
    """(Xhat, xbar, a) with Xhat = (X - 1 xbar^T) / a and a = ||X - 1 xbar^T||_2.

    Section 3 requires a > 0; a ValueError is raised when every row is equal.
    """
    X = np.asarray(X, dtype=np.float64)
    xbar = X.mean(axis=0)
    Xc = X - xbar[None, :]
    a = spectral_norm(Xc)
    if not a > 0.0:
        raise ValueError("degenerate data: the centred matrix is zero (a = 0)")
    return Xc / a, xbar, a


# ----------------------------------------------------------------------------
# Section 2 / 3: constraint, objective, gradient, projection
# ----------------------------------------------------------------------------
def constraint_g(U: np.ndarray) -> np.ndarray:
    """g(U) = U U^T 1_n - 1_n, evaluated as U (U^T 1) - 1 (eq. Kmeans_NLR)."""
    return U @ U.sum(axis=0) - 1.0


def constraint_h(U: np.ndarray) -> np.ndarray:
    """h(U) = g(U) / sqrt(n) (eq. normalized)."""
    return constraint_g(U) / np.sqrt(U.shape[0])


def objective(Xhat: np.ndarray, U: np.ndarray, y: np.ndarray, beta: float) -> float:
    """fhat_y(U) = <Ahat, U U^T> + y^T h(U) + beta/2 ||h(U)||^2, Ahat = -Xhat Xhat^T.

    <Ahat, U U^T> = -||Xhat^T U||_F^2 is used, so the n x n matrix is not
    formed (the dense form lives in ``oracle.dense``).
    """
    Theta = Xhat.T @ U
    hU = constraint_h(U)
    return float(-np.sum(Theta * Theta) + y @ hU + 0.5 * beta * (hU @ hU))


def effective_multiplier(U: np.ndarray, y: np.ndarray, beta: float) -> np.ndarray:
    """ybar_eff = y / sqrt(n) + (beta / n) g(U) (eq. dualnormalized)."""
    n = U.shape[0]
    return y / np.sqrt(n) + (beta / n) * constraint_g(U)


def gradient(Xhat: np.ndarray, U: np.ndarray, y: np.ndarray, beta: float) -> np.ndarray:
    """grad fhat_y(U) = 2 Ahat U + ybar_eff (U^T 1)^T + 1 (U^T ybar_eff)^T (eq. gradient).

    Ahat U = -Xhat (Xhat^T U).
    """
    ybar = effective_multiplier(U, y, beta)
    AU = -(Xhat @ (Xhat.T @ U))
    colsum = U.sum(axis=0)
    return 2.0 * AU + np.outer(ybar, colsum) + np.outer(np.ones(U.shape[0]), U.T @ ybar)


def project_omega(V: np.ndarray, K: float) -> np.ndarray:
    """Pi_Omega(V) = sqrt(K) V_+ / ||V_+||_F (eq. projected-primal-step).

    Raises FloatingPointError when V_+ = 0 (the projection is not defined).
    """
    Vp = np.maximum(np.asarray(V, dtype=np.float64), 0.0)
    nrm = np.sqrt(np.sum(Vp * Vp))
    if not nrm > 0.0:
        raise FloatingPointError("projection of a matrix with no positive entry")
    return np.sqrt(K) * Vp / nrm


# ----------------------------------------------------------------------------
# Appendix D "Initialization": data-informed starting factor
# ----------------------------------------------------------------------------
def data_informed_start(Xhat: np.ndarray, Z: np.ndarray, K: float):
    """(U0, Q) with V = Xhat Xhat^T Z, V = Q R, U0 = Pi_Omega(Q) (Appendix D).

    The range finder is applied to the Gram matrix of the normalised data (the
    matrix C is the one reused from the normalisation).  The QR factorisation
    is the Cholesky QR of the appendix, taken in feature space:
        M = Xhat^T Z,  C = Xhat^T Xhat,  V^T V = M^T C M = R^T R  (R upper
        triangular with positive diagonal),  Q = Xhat (M R^{-1}).
    Needs V of full column rank (r <= rank Xhat); raises LinAlgError otherwise.
    """
    Xhat = np.asarray(Xhat, dtype=np.float64)
    Z = np.asarray(Z, dtype=np.float64)
    M = Xhat.T @ Z
    C = Xhat.T @ Xhat
    G = M.T @ C @ M
    L = np.linalg.cholesky(G)           # G = L L^T, R = L^T
    # M R^{-1} = M L^{-T}: solve L Y = M^T, then (M R^{-1}) = Y^T
    MRinv = np.linalg.solve(L, M.T).T
    Q = Xhat @ MRinv
    return project_omega(Q, K), Q


def lipschitz_bound(y: np.ndarray, beta: float, K: float) -> float:
    """L = 2 + 2 ||y||_2 + beta (6K + 2) (Prop. 1, eq. L)."""
    return float(2.0 + 2.0 * np.linalg.norm(y) + beta * (6.0 * K + 2.0))


def stored_dual(y: np.ndarray) -> np.ndarray:
    """The implementation's dual buffer ytilde = y / sqrt(n) (Section 3, Appendix C)."""
    return y / np.sqrt(y.shape[0])


def dual_from_stored(ytilde: np.ndarray) -> np.ndarray:
    return np.asarray(ytilde, dtype=np.float64) * np.sqrt(ytilde.shape[0])


def labels(U: np.ndarray) -> np.ndarray:
    """Row argmax of U, lowest column index on ties (int32)."""
    return np.argmax(np.asarray(U), axis=1).astype(np.int32)


# ----------------------------------------------------------------------------
# Algorithm 1: one iteration and the loop
# ----------------------------------------------------------------------------
@dataclass
class StepRecord:
    t: int
    objective: float        # fhat_{y_t}(U_t), before the step
    theta_fro2: float       # ||Xhat^T U_t||_F^2
    a: float                # ||W||_F^2
    b: float                # ||U_t||_F^2
    h: float                # <W, U_t>_F
    c: float                # exact sqrt(K / a)
    delta: float            # ||U_{t+1} - U_t||_F / sqrt(K), measured directly
    delta_identity: float   # sqrt(max(c^2 a + b - 2 c h, 0) / K) (eq. movement-estimate)
    rho: float              # ||q_{t+1}||_2 / sqrt(n)
    gate: bool              # dual step taken at the end of this iteration
    stop: bool
    L: float                # Prop. 1 bound at y_t
    y_norm: float           # ||y_t||_2


@dataclass
class RunResult:
    U: np.ndarray
    y: np.ndarray
    iters: int
    breakdown: bool
    records: list = field(default_factory=list)
    trajectory: list | None = None  # U_{t+1} after every iteration, when requested
    duals: list | None = None       # y_{t+1} after every iteration, when requested

    @property
    def ytilde(self) -> np.ndarray:
        return stored_dual(self.y)


def primal_step(Xhat: np.ndarray, U: np.ndarray, y: np.ndarray, K: float,
                alpha: float, beta: float):
    """Projected gradient step U^+ = Pi_Omega(U - alpha grad fhat_y(U)) (eq. projected-primal-step).

    Returns (U_plus or None on breakdown, W, stats) where W = (U - alpha grad)_+
    is the unnormalised update and stats = dict(a, b, h, c).
    """
    G = gradient(Xhat, U, y, beta)
    W = np.maximum(U - alpha * G, 0.0)
    a = float(np.sum(W * W))
    b = float(np.sum(U * U))
    h = float(np.sum(W * U))
    if np.sqrt(a) <= BREAKDOWN_NU:
        return None, W, dict(a=a, b=b, h=h, c=float("nan"))
    c = float(np.sqrt(K / a))
    return c * W, W, dict(a=a, b=b, h=h, c=c)


def run(Xhat: np.ndarray, U0: np.ndarray, K: float, alpha: float, beta: float, T: int,
        T_min: int = 0, eps_d: float = 1e-4, eps_c: float = 1e-4, *, y0: np.ndarray | None = None,
        project_init: bool = True, gates=None, keep_trajectory: bool = False,
        t0: int = 0) -> RunResult:
    """Algorithm 1 in float64.

    U0 is projected onto Omega first unless ``project_init`` is False (Alg. 1
    requires U in Omega).  ``y0`` defaults to 0.  ``gates`` optionally fixes the
    dual-gate decision of each iteration (a sequence of bools, used to replay
    the GPU's decisions); otherwise the gate is delta < eps_d.  ``t0`` offsets
    the iteration counter used by the T_min test.
    """
    Xhat = np.asarray(Xhat, dtype=np.float64)
    U = np.asarray(U0, dtype=np.float64)
    if project_init:
        U = project_omega(U, K)
    n = U.shape[0]
    y = np.zeros(n) if y0 is None else np.asarray(y0, dtype=np.float64).copy()
    res = RunResult(U=U, y=y, iters=0, breakdown=False,
                    trajectory=[] if keep_trajectory else None,
                    duals=[] if keep_trajectory else None)
    sqrtn = np.sqrt(n)
    for t in range(T):
        f_t = objective(Xhat, U, y, beta)
        Theta = Xhat.T @ U
        L = lipschitz_bound(y, beta, K)
        U_new, W, st = primal_step(Xhat, U, y, K, alpha, beta)
        if U_new is None:
            res.breakdown = True
            res.U = W  # the unnormalised update has replaced the factor
            res.y = y
            return res
        delta = float(np.linalg.norm(U_new - U) / np.sqrt(K))
        c = st["c"]
        delta_id = float(np.sqrt(max(c * c * st["a"] + st["b"] - 2.0 * c * st["h"], 0.0) / K))
        U = U_new
        q = constraint_g(U)  # p = U^T 1, q = U p - 1
        gate = bool(gates[t]) if gates is not None else bool(delta < eps_d)
        y_norm = float(np.linalg.norm(y))
        if gate:
            y = y + (beta / sqrtn) * q
        rho = float(np.linalg.norm(q) / sqrtn)
        stop = bool(delta < min(eps_d, eps_c) and rho < eps_c and t0 + t + 1 >= T_min)
        res.records.append(StepRecord(t=t0 + t, objective=f_t, theta_fro2=float(np.sum(Theta * Theta)),
                                      a=st["a"], b=st["b"], h=st["h"], c=c, delta=delta,
                                      delta_identity=delta_id, rho=rho, gate=gate, stop=stop,
                                      L=L, y_norm=y_norm))
        res.iters = t + 1
        if keep_trajectory:
            res.trajectory.append(U.copy())
            res.duals.append(y.copy())
        if stop:
            break
    res.U = U
    res.y = y
    return res


def default_step_size(K: float, beta: float = 1.0) -> float:
    """alpha = 1 / (2 L_0) with L_0 the Prop. 1 bound at y = 0.

    The paper fixes no value for alpha; this is the reading used by the tests
    and the benchmark (half the largest step Cor. 1 allows at y = 0).
    """
    return 1.0 / (2.0 * (2.0 + beta * (6.0 * K + 2.0)))
