"""Cluster labels from a factor U by spectral embedding and K-means (TEST INFRASTRUCTURE ONLY).

Appendix D, "Recover cluster labels from U": take the leading K left singular
vectors of U as an embedding of the n points and run K-means on its rows.
The appendix fixes neither the K-means initialisation nor its stopping rule;
here (the readings the GPU path follows as well):

* the initial centroids are the embedded rows at K given row indices (a random
  choice is the caller's, passed in as input);
* Lloyd's iteration: assign every row to its nearest centroid (squared
  Euclidean distance, lowest centroid index on ties), stop as soon as an
  assignment pass changes no label, otherwise move every centroid to the mean
  of its rows (a centroid with no rows stays where it is); at most max_iter
  assignment passes.

The embedding is determined up to an orthogonal change of basis inside the
span of the leading K left singular vectors (column signs, repeated singular
values); distances between embedded rows, and so the labels, do not depend on
it.
"""
from __future__ import annotations

import numpy as np


def spectral_embedding(U: np.ndarray, K: int) -> np.ndarray:
    """Rows of the leading K left singular vectors of U (n x K)."""
    Uq, _, _ = np.linalg.svd(np.asarray(U, dtype=np.float64), full_matrices=False)
    return Uq[:, :K]


def nearest(E: np.ndarray, C: np.ndarray) -> np.ndarray:
    """Index of the nearest centroid of every row (lowest index on ties)."""
    D = np.empty((E.shape[0], C.shape[0]))
    for k in range(C.shape[0]):
        D[:, k] = np.sum((E - C[k][None, :]) ** 2, axis=1)
    return np.argmin(D, axis=1).astype(np.int32)  # argmin returns the first minimum


def lloyd(E: np.ndarray, init_rows, max_iter: int = 100):
    """(labels, assignment passes, centroids) of Lloyd's iteration from the rows init_rows."""
    E = np.asarray(E, dtype=np.float64)
    C = E[np.asarray(init_rows, dtype=np.int64)].copy()
    lab = None
    passes = 0
    for _ in range(max_iter):
        new = nearest(E, C)
        passes += 1
        if lab is not None and np.array_equal(new, lab):
            break
        lab = new
        for k in range(C.shape[0]):
            members = E[lab == k]
            if members.shape[0] > 0:
                C[k] = members.mean(axis=0)
    return lab, passes, C


def spectral_labels(U: np.ndarray, K: int, init_rows, max_iter: int = 100):
    """(labels, assignment passes) for factor U (Appendix D label recovery)."""
    lab, passes, _ = lloyd(spectral_embedding(U, K), init_rows, max_iter)
    return lab, passes
