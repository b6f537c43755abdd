"""Seeded synthetic Gaussian-mixture inputs for the NLR K-means iteration.

This module only draws random numbers. It holds none of the method's
arithmetic (no centring, no normalisation, no projection), so that the fp64
oracle and the GPU path can both take their inputs from it without sharing
any step of the computation.

Workloads follow the paper's experimental setting (Section 5, "Simulation
benchmarks", and Table 2): a K-component Gaussian mixture x_i = mu_{z_i} +
eps_i in R^d with rows shuffled.  The five named shapes below are the
synthetic stand-ins used for parity and measurement; the paper's real datasets
(CyTOF, Gaia DR3) are not available and are not imitated item by item.

The initial factor is the paper's random initialisation U_0 = Pi_Omega(Z)
with Z having i.i.d. N(0,1) entries (Appendix D, "Initialization"); this module
returns the raw draw Z only.  Both consumers apply the projection themselves.

Generation is chunked over rows with one child generator per chunk
(``numpy.random.SeedSequence.spawn``), so the same seed gives the same bits
whatever the number of worker threads.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

CHUNK_ROWS = 1 << 18  # rows per generator chunk; part of the stream definition


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    d: int
    K: int
    r: int
    T: int
    center_var: float
    sizes: str = "equal"          # "equal" | "dirichlet5" | "zipf1.1"
    noise: str = "iso"            # "iso" (N(0, I)) | "aniso" (per-cluster diag, U[0.2, 2])
    l2_normalise: bool = False    # rows scaled to unit L2 norm after sampling
    seed: int = 0
    extra: dict = field(default_factory=dict)
    gamma: float | None = None    # set: centres scaled to min separation gamma * CNRbar (Table 2)


# The five shapes.  Seeds: data seed 0; the U_0 draw uses seed + 1.
WORKLOADS = {
    "tiny": Workload("tiny", 2_000, 16, 4, 4, 200, 25.0),
    "gmm1m": Workload("gmm1m", 1_000_000, 64, 16, 16, 100, 9.0, sizes="dirichlet5"),
    "gmm10m": Workload("gmm10m", 10_000_000, 128, 64, 64, 50, 4.0),
    "gmm50m": Workload("gmm50m", 50_000_000, 32, 10, 10, 50, 16.0),
    "embed2m": Workload("embed2m", 2_000_000, 768, 256, 256, 30, 1.0,
                        sizes="zipf1.1", noise="aniso", l2_normalise=True),
}
WORKLOAD_ORDER = ["tiny", "gmm1m", "gmm10m", "gmm50m", "embed2m"]

# The two smallest Table 2 settings (balanced mixture, minimum centre separation
# gamma * CNRbar with gamma = 1, unit noise): shapes for parity and timing beside
# the five above.
TABLE2 = {
    "t2k20": Workload("t2k20", 1_000_000, 50, 20, 30, 100, 1.0, gamma=1.0),
    "t2k100": Workload("t2k100", 1_000_000, 200, 100, 300, 100, 1.0, gamma=1.0),
}
WORKLOADS.update(TABLE2)


def cnr_bar(n: int, K: int, d: int) -> float:
    """CNRbar = sqrt(4 (1 + sqrt(1 + K d / (n log n))) log n): the exact-recovery
    threshold on the centroid-to-noise ratio (Section 2), the separation scale of
    the paper's simulated mixtures (Section 5, Table 2).  A generator parameter."""
    ln = np.log(n)
    return float(np.sqrt(4.0 * (1.0 + np.sqrt(1.0 + K * d / (n * ln))) * ln))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cluster_sizes(n: int, K: int, rule: str, rng: np.random.Generator) -> np.ndarray:
    """Cluster sizes summing to n.

    equal: n/K each (remainder spread over the first clusters).
    dirichlet5: pi ~ Dir(5 * 1_K), sizes by largest-remainder rounding of n*pi.
    zipf1.1: pi_k proportional to k^-1.1, largest-remainder rounding.
    Every cluster gets at least one point.
    """
    if rule == "equal":
        base = np.full(K, n // K, dtype=np.int64)
        base[: n - base.sum()] += 1
        return base
    if rule == "dirichlet5":
        pi = rng.dirichlet(np.full(K, 5.0))
    elif rule == "zipf1.1":
        k = np.arange(1, K + 1, dtype=np.float64)
        pi = k ** -1.1
        pi /= pi.sum()
    else:
        raise ValueError(f"unknown size rule {rule!r}")
    raw = n * pi
    sizes = np.floor(raw).astype(np.int64)
    short = n - int(sizes.sum())
    order = np.argsort(-(raw - sizes), kind="stable")
    sizes[order[:short]] += 1
    # guarantee non-empty clusters (moves points from the largest cluster)
    for k in range(K):
        if sizes[k] == 0:
            j = int(np.argmax(sizes))
            sizes[j] -= 1
            sizes[k] += 1
    return sizes


def _fill_chunks(out: np.ndarray, seed_seq: np.random.SeedSequence, fill, threads: int) -> None:
    # Child ci of a fresh SeedSequence is the same whatever the number spawned, so
    # the rows of chunk ci do not depend on how many rows are drawn in all: the
    # first m rows of an n-row draw are an m-row draw's rows (same labels given).
    n = out.shape[0]
    nchunks = (n + CHUNK_ROWS - 1) // CHUNK_ROWS
    children = seed_seq.spawn(nchunks)

    def work(ci: int) -> None:
        lo = ci * CHUNK_ROWS
        hi = min(n, lo + CHUNK_ROWS)
        fill(np.random.Generator(np.random.PCG64(children[ci])), lo, hi)

    if threads <= 1 or nchunks == 1:
        for ci in range(nchunks):
            work(ci)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(work, range(nchunks)))


def gaussian_mixture(n: int, d: int, K: int, center_var: float, *, sizes: str = "equal",
                     noise: str = "iso", l2_normalise: bool = False, seed: int = 0,
                     threads: int | None = None, rows: int | None = None,
                     min_separation: float | None = None):
    """Draw (X float32 [m, d], labels int32 [m], centers float64 [K, d]), m = n or `rows`.

    Centers mu_k ~ N(0, center_var * I_d); with ``min_separation`` = Delta (and
    K >= 2) the same draw is then scaled so that min_{k != l} ||mu_k - mu_l|| =
    Delta.  Noise eps_i ~ N(0, I_d) ("iso") or
    N(0, diag(v_{z_i})) with v_k ~ U[0.2, 2]^d ("aniso").  Labels are a
    shuffled assignment with the requested cluster sizes over all n rows.
    With ``rows = m < n`` only the first m rows of the n-row draw are made:
    bitwise the leading rows of the full draw.
    """
    threads = _threads() if threads is None else threads
    root = np.random.SeedSequence(seed)
    s_meta, s_noise = root.spawn(2)
    meta = np.random.Generator(np.random.PCG64(s_meta))
    centers = meta.standard_normal((K, d)) * np.sqrt(center_var)
    if min_separation is not None and K >= 2:
        diff = centers[:, None, :] - centers[None, :, :]
        dist = np.sqrt(np.einsum("kld,kld->kl", diff, diff))
        dist[np.arange(K), np.arange(K)] = np.inf
        centers = centers * (float(min_separation) / dist.min())
    sz = cluster_sizes(n, K, sizes, meta)
    labels = np.repeat(np.arange(K, dtype=np.int32), sz)
    meta.shuffle(labels)
    if noise == "aniso":
        sd = np.sqrt(meta.uniform(0.2, 2.0, size=(K, d)))
    elif noise == "iso":
        sd = None
    else:
        raise ValueError(f"unknown noise {noise!r}")
    c32 = centers.astype(np.float32)
    sd32 = None if sd is None else sd.astype(np.float32)
    m = n if rows is None else int(rows)
    if not 0 < m <= n:
        raise ValueError(f"rows must be in 1..{n}")
    labels = labels[:m]
    X = np.empty((m, d), dtype=np.float32)

    def fill(g: np.random.Generator, lo: int, hi: int) -> None:
        z = labels[lo:hi]
        e = g.standard_normal((hi - lo, d), dtype=np.float32)
        if sd32 is not None:
            e *= sd32[z]
        e += c32[z]
        if l2_normalise:
            nrm = np.sqrt(np.einsum("ij,ij->i", e, e, dtype=np.float64)).astype(np.float32)
            nrm[nrm == 0] = 1.0
            e /= nrm[:, None]
        X[lo:hi] = e

    _fill_chunks(X, s_noise, fill, threads)
    return X, labels, centers


def standard_normal_factor(n: int, r: int, seed: int, threads: int | None = None) -> np.ndarray:
    """Z with i.i.d. N(0, 1) entries, float32 [n, r] (the raw draw behind U_0).

    Rows do not depend on n: the first m rows of an n-row draw are the m-row draw.
    """
    threads = _threads() if threads is None else threads
    Z = np.empty((n, r), dtype=np.float32)

    def fill(g: np.random.Generator, lo: int, hi: int) -> None:
        Z[lo:hi] = g.standard_normal((hi - lo, r), dtype=np.float32)

    _fill_chunks(Z, np.random.SeedSequence([seed, 0x5A]), fill, threads)
    return Z


def make_workload(name_or_wl, n: int | None = None, threads: int | None = None,
                  rows: int | None = None):
    """Inputs of a named workload: (X, Z, labels, workload).

    ``n`` replaces the number of rows: a new, smaller draw of the same
    distribution (its cluster sizes and label shuffle are drawn for that n, so
    its rows are not those of the full workload).  ``rows`` instead keeps the
    full workload's n and returns only its first ``rows`` rows, bitwise equal to
    the leading rows of the full draw (used for bounded CPU samples).
    """
    wl = WORKLOADS[name_or_wl] if isinstance(name_or_wl, str) else name_or_wl
    nn = wl.n if n is None else int(n)
    sep = None if wl.gamma is None else wl.gamma * cnr_bar(nn, wl.K, wl.d)
    X, labels, _ = gaussian_mixture(nn, wl.d, wl.K, wl.center_var, sizes=wl.sizes,
                                    noise=wl.noise, l2_normalise=wl.l2_normalise,
                                    seed=wl.seed, threads=threads, rows=rows, min_separation=sep)
    Z = standard_normal_factor(X.shape[0], wl.r, wl.seed + 1, threads=threads)
    return X, Z, labels, wl
