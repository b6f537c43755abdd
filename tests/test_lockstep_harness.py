"""The parallel full-size lockstep harness (tests/gpu_util.py), on the CPU: contexts
that step with the oracle itself in float32 give errors at float32 rounding, a context
with a wrong sign in one iteration's update is caught in that iteration, and runs
whose gate decisions differ get trajectories of their own."""
import numpy as np
import torch

from gpu_util import lockstep_parallel
from oracle import nlr as onlr
from synth import gaussian_mixture, standard_normal_factor


class OracleCtx:
    """Steps with the fp64 oracle and stores float32 iterates, as the GPU context does;
    `flip` (iteration, row) negates one step entry there; `gates` forces decisions."""

    def __init__(self, Xh, U0, K, alpha, beta, gates, flip=None):
        self.Xh, self.K, self.alpha, self.beta = Xh, K, alpha, beta
        self._U, self._y = U0.copy(), np.zeros(U0.shape[0])
        self.gates, self.flip, self.t = gates, flip, 0

    @property
    def U(self):
        return torch.from_numpy(self._U.astype(np.float32))

    @property
    def y(self):
        return torch.from_numpy(onlr.stored_dual(self._y).astype(np.float32))

    def step(self):
        g = self.gates[self.t]
        r = onlr.run(self.Xh, self._U.astype(np.float32).astype(np.float64), self.K, self.alpha, self.beta,
                     T=1, T_min=1, project_init=False,
                     y0=onlr.dual_from_stored(onlr.stored_dual(self._y).astype(np.float32).astype(np.float64)),
                     gates=[g], t0=self.t)
        U = r.U.copy()
        if self.flip is not None and self.flip[0] == self.t:
            U[self.flip[1]] = U[self.flip[1]] * 0.5  # a wrong update of one row
        self._U, self._y = U, r.y
        self.t += 1
        return {"dual_step": int(g), "objective": r.records[0].objective}

    def labels(self):
        return torch.from_numpy(onlr.labels(self._U).astype(np.int32))


def test_lockstep_parallel_catches_a_wrong_row():
    X, _, _ = gaussian_mixture(3000, 8, 3, 16.0, seed=5)
    Z = standard_normal_factor(3000, 4, seed=6).astype(np.float64)
    K, beta = 3, 1.0
    alpha = onlr.default_step_size(K, beta)
    Xh, _, _ = onlr.centre_and_normalise(X)
    U0 = onlr.project_omega(Z, K)
    runs = {"good": (OracleCtx(Xh, U0, K, alpha, beta, [False] * 4), 4),
            "bad": (OracleCtx(Xh, U0, K, alpha, beta, [False] * 3, flip=(1, 17)), 3),
            "gated": (OracleCtx(Xh, U0, K, alpha, beta, [False, True]), 2),
            "short": (OracleCtx(Xh, U0, K, alpha, beta, [False] * 2), 2)}
    res = lockstep_parallel(runs, Xh, U0, K, alpha, beta, eps_d=1e-4, workers=2)
    good, bad, gated, short = res["good"], res["bad"], res["gated"], res["short"]
    assert max(good["traj"]) < 1e-6 and max(good["one"]) < 1e-6 and max(good["obj"]) < 1e-6
    assert good["labels"][0] == 0 and gated["labels"][0] == 0
    # a shorter run shares the trajectory; its labels are compared at its own last iteration
    assert len(short["traj"]) == 2 and max(short["traj"]) < 1e-6 and short["labels"][0] == 0
    assert bad["one"][0] < 1e-6 and bad["one"][1] > 1e-3 and bad["one"][2] < 1e-6
    assert bad["traj"][0] < 1e-6 and min(bad["traj"][1:]) > 1e-4
    # the gated run has its own trajectory: no error from the dual step it takes
    assert max(gated["traj"]) < 1e-6 and max(gated["one"]) < 1e-6 and max(gated["yerr"]) < 1e-6
    assert gated["bad_gates"] == [1]  # the oracle's own movement is not below eps_d there
