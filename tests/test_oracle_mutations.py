"""Plants plausible mistakes in a copy of the oracle (on the CPU) and checks that
at least one pin catches each.  The oracle module on disk is never modified."""
import os
import sys
import types

import pytest

import oracle_pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = open(os.path.join(ROOT, "oracle", "nlr.py")).read()

# (name, original text, mutated text)
MUTATIONS = [
    ("sign of the 2 Ahat U term", "return 2.0 * AU + np.outer", "return -2.0 * AU + np.outer"),
    ("dropped 1 s^T term", " + np.outer(np.ones(U.shape[0]), U.T @ ybar)", ""),
    ("dropped ybar p^T term", "2.0 * AU + np.outer(ybar, colsum) +", "2.0 * AU +"),
    ("p and s swapped", "np.outer(ybar, colsum) + np.outer(np.ones(U.shape[0]), U.T @ ybar)",
     "np.outer(ybar, U.T @ ybar) + np.outer(np.ones(U.shape[0]), colsum)"),
    ("beta/sqrt(n) in ybar", "(beta / n) * constraint_g(U)", "(beta / np.sqrt(n)) * constraint_g(U)"),
    ("y not scaled in ybar", "return y / np.sqrt(n) + (beta / n)", "return y + (beta / n)"),
    ("projection by K not sqrt(K)", "return np.sqrt(K) * Vp / nrm", "return K * Vp / nrm"),
    ("no positive part", "W = np.maximum(U - alpha * G, 0.0)", "W = U - alpha * G"),
    ("ascent instead of descent", "W = np.maximum(U - alpha * G, 0.0)", "W = np.maximum(U + alpha * G, 0.0)"),
    ("c = K/a", "c = float(np.sqrt(K / a))", "c = float(K / a)"),
    ("dual step sign", "y = y + (beta / sqrtn) * q", "y = y - (beta / sqrtn) * q"),
    ("dual step scale", "y = y + (beta / sqrtn) * q", "y = y + beta * q"),
    ("dual step uses stale residual", "q = constraint_g(U)  # p = U^T 1", "q = constraint_g(res.U)  # p = U^T 1"),
    ("movement not divided by sqrt(K)", "np.linalg.norm(U_new - U) / np.sqrt(K)", "np.linalg.norm(U_new - U)"),
    ("no centring", "Xc = X - xbar[None, :]", "Xc = X"),
    ("squared spectral norm", "return float(np.sqrt(max(lam, 0.0)))", "return float(max(lam, 0.0))"),
    ("penalty without 1/2", "0.5 * beta * (hU @ hU)", "beta * (hU @ hU)"),
    ("residual without -1", "return U @ U.sum(axis=0) - 1.0", "return U @ U.sum(axis=0)"),
    ("h not scaled", "return constraint_g(U) / np.sqrt(U.shape[0])", "return constraint_g(U)"),
    ("Lipschitz bound without the beta term", "2.0 * np.linalg.norm(y) + beta * (6.0 * K + 2.0))", "2.0 * np.linalg.norm(y))"),
    ("argmax over columns", "np.argmax(np.asarray(U), axis=1)", "np.argmax(np.asarray(U), axis=0)"),
    ("objective sign", "return float(-np.sum(Theta * Theta) + y @ hU", "return float(np.sum(Theta * Theta) + y @ hU"),
    ("range finder without the Gram matrix", "C = Xhat.T @ Xhat\n", "C = np.eye(Xhat.shape[1])\n"),
    ("range finder without R^-1", "Q = Xhat @ MRinv", "Q = Xhat @ M"),
    ("range finder with the transposed Cholesky factor", "MRinv = np.linalg.solve(L, M.T).T",
     "MRinv = np.linalg.solve(L.T, M.T).T"),
    ("range finder on Z instead of Xhat^T Z", "M = Xhat.T @ Z\n", "M = Z[: Xhat.shape[1]]\n"),
    ("stored dual scaled up by sqrt(n)", "return y / np.sqrt(y.shape[0])", "return y * np.sqrt(y.shape[0])"),
    ("stored dual read back divided by sqrt(n)", "* np.sqrt(ytilde.shape[0])", "/ np.sqrt(ytilde.shape[0])"),
    ("stored dual scaled by n", "return y / np.sqrt(y.shape[0])", "return y / y.shape[0]"),
]


LABEL_SRC = open(os.path.join(ROOT, "oracle", "labels.py")).read()

# (name, original text, mutated text) planted in oracle/labels.py
LABEL_MUTATIONS = [
    ("trailing singular vectors", "return Uq[:, :K]", "return Uq[:, -K:]"),
    ("farthest instead of nearest centroid", "np.argmin(D, axis=1)", "np.argmax(D, axis=1)"),
    ("centroid as a sum", "C[k] = members.mean(axis=0)", "C[k] = members.sum(axis=0)"),
    ("no convergence test", "if lab is not None and np.array_equal(new, lab):", "if False:"),
    ("distance without the square", "np.sum((E - C[k][None, :]) ** 2, axis=1)", "np.sum(np.abs(E - C[k][None, :]) - 1.0, axis=1)"),
    ("right singular vectors", "Uq, _, _ = np.linalg.svd(np.asarray(U, dtype=np.float64), full_matrices=False)\n    return Uq[:, :K]",
     "_, _, Vt = np.linalg.svd(np.asarray(U, dtype=np.float64), full_matrices=False)\n    return Vt.T[:, :K]"),
]


KMEANS_SRC = open(os.path.join(ROOT, "oracle", "kmeans.py")).read()

# (name, original text, mutated text) planted in oracle/kmeans.py
KMEANS_MUTATIONS = [
    ("ARI without the chance adjustment", "return float((s_ij - exp) / (mx - exp))", "return float(s_ij / mx)"),
    ("ARI always one", "if mx == exp:", "if True:"),
    ("ARI with the row pairs twice", "mx = 0.5 * (s_a + s_b)", "mx = s_a"),
    ("recovery threshold in log10", "ln = np.log(n)", "ln = np.log10(n)"),
    ("recovery threshold without the 1 + under the root", "np.sqrt(1.0 + K * d / (n * ln))",
     "np.sqrt(K * d / (n * ln))"),
    ("recovery threshold with K d / n", "K * d / (n * ln)", "K * d / n"),
]


def _load_mutant(monkeypatch, orig, new, src=SRC, name="oracle_nlr_mutant"):
    assert orig in src, f"mutation anchor not found: {orig!r}"
    mod = types.ModuleType(name)
    mod.__file__ = "<mutant>"
    monkeypatch.setitem(sys.modules, mod.__name__, mod)
    exec(compile(src.replace(orig, new), "<mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,orig,new", LABEL_MUTATIONS, ids=[m[0] for m in LABEL_MUTATIONS])
def test_label_mutation_is_caught(monkeypatch, name, orig, new):
    mutant = _load_mutant(monkeypatch, orig, new, LABEL_SRC, "oracle_labels_mutant")
    monkeypatch.setattr(oracle_pins, "labels", mutant)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin()
        except Exception:
            caught.append(pin.__name__)
            break
    assert caught, f"no pin catches the planted mistake: {name}"


@pytest.mark.parametrize("name,orig,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(monkeypatch, name, orig, new):
    mutant = _load_mutant(monkeypatch, orig, new)
    monkeypatch.setattr(oracle_pins, "nlr", mutant)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin()
        except Exception as e:  # any failure (assertion, error) counts as caught
            caught.append(pin.__name__)
            break
    assert caught, f"no pin catches the planted mistake: {name}"


@pytest.mark.parametrize("name,orig,new", KMEANS_MUTATIONS, ids=[m[0] for m in KMEANS_MUTATIONS])
def test_kmeans_mutation_is_caught(monkeypatch, name, orig, new):
    mutant = _load_mutant(monkeypatch, orig, new, KMEANS_SRC, "oracle_kmeans_mutant")
    monkeypatch.setattr(oracle_pins, "kmeans", mutant)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin()
        except Exception:
            caught.append(pin.__name__)
            break
    assert caught, f"no pin catches the planted mistake: {name}"
