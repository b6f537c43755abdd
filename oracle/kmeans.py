"""Exact K-means by partition enumeration, for tiny n (TEST INFRASTRUCTURE ONLY).

Section 2, eq. (partition): for a partition G = (G_1..G_K) of [n],
J(G) = sum_k sum_{i in G_k} ||x_i - xbar_k||^2 = ||X||_F^2 - <X X^T, Z_G>,
Z_G = H H^T, H_ik = 1{i in G_k} / sqrt(|G_k|).  The partition problem
(eq. Kmeans_partition) minimises J over all partitions into K non-empty
blocks; here that is done by brute force over restricted-growth strings.
"""
from __future__ import annotations

import numpy as np


def partitions(n: int, K: int):
    """Yield label vectors (restricted-growth strings) of every partition of [n]
    into exactly K non-empty blocks; each partition appears once."""
    a = [0] * n

    def rec(i: int, m: int):
        # m = number of blocks used by a[0..i-1]
        if i == n:
            if m == K:
                yield np.array(a, dtype=np.int64)
            return
        if K - m > n - i:  # not enough positions left to open the missing blocks
            return
        for v in range(min(m + 1, K)):
            a[i] = v
            yield from rec(i + 1, max(m, v + 1))

    if n == 0:
        return
    a[0] = 0
    yield from rec(1, 1)


def within_ss(X: np.ndarray, lab: np.ndarray, K: int) -> float:
    """J(G) as the sum of squared distances to the block means."""
    X = np.asarray(X, dtype=np.float64)
    J = 0.0
    for k in range(K):
        B = X[lab == k]
        J += float(np.sum((B - B.mean(axis=0)) ** 2))
    return J


def membership(lab: np.ndarray, K: int) -> np.ndarray:
    """H with H_ik = 1{i in G_k} / sqrt(|G_k|)."""
    n = lab.shape[0]
    H = np.zeros((n, K))
    for k in range(K):
        idx = lab == k
        H[idx, k] = 1.0 / np.sqrt(idx.sum())
    return H


def within_ss_trace(X: np.ndarray, lab: np.ndarray, K: int) -> float:
    """J(G) = ||X||_F^2 - <X X^T, Z_G> with Z_G = H H^T."""
    X = np.asarray(X, dtype=np.float64)
    H = membership(lab, K)
    return float(np.sum(X * X) - np.sum((X @ X.T) * (H @ H.T)))


def brute_force(X: np.ndarray, K: int):
    """(best J, list of optimal label vectors) over all partitions into K blocks."""
    best = np.inf
    arg = []
    for lab in partitions(X.shape[0], K):
        J = within_ss(X, lab, K)
        if not arg or J < best - 1e-12 * max(1.0, abs(best)):
            best, arg = J, [lab.copy()]
        elif abs(J - best) <= 1e-12 * max(1.0, abs(best)):
            arg.append(lab.copy())
    return best, arg


def same_partition(a: np.ndarray, b: np.ndarray) -> bool:
    """True when two label vectors describe the same partition (labels up to renaming)."""
    a = np.asarray(a)
    b = np.asarray(b)
    if a.shape != b.shape:
        return False
    fwd: dict = {}
    bwd: dict = {}
    for x, y in zip(a.tolist(), b.tolist()):
        if fwd.setdefault(x, y) != y or bwd.setdefault(y, x) != x:
            return False
    return True


def exact_recovery_threshold_sq(n: int, K: int, d: int) -> float:
    """CNRbar^2 = 4 (1 + sqrt(1 + K d / (n log n))) log n (eq. exact_recovery_threshold)."""
    ln = np.log(n)
    return float(4.0 * (1.0 + np.sqrt(1.0 + K * d / (n * ln))) * ln)


def adjusted_rand_index(a: np.ndarray, b: np.ndarray) -> float:
    """ARI between two labelings (standard pair-counting definition)."""
    a = np.asarray(a)
    b = np.asarray(b)
    ua, ia = np.unique(a, return_inverse=True)
    ub, ib = np.unique(b, return_inverse=True)
    M = np.zeros((ua.size, ub.size), dtype=np.int64)
    np.add.at(M, (ia, ib), 1)

    def c2(x):
        x = np.asarray(x, dtype=np.float64)
        return x * (x - 1) / 2.0

    s_ij = c2(M).sum()
    s_a = c2(M.sum(axis=1)).sum()
    s_b = c2(M.sum(axis=0)).sum()
    tot = c2(a.size)
    exp = s_a * s_b / tot if tot > 0 else 0.0
    mx = 0.5 * (s_a + s_b)
    if mx == exp:
        return 1.0
    return float((s_ij - exp) / (mx - exp))


__all__ = ["partitions", "within_ss", "within_ss_trace", "membership", "brute_force",
           "same_partition", "exact_recovery_threshold_sq", "adjusted_rand_index"]
