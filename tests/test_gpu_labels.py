"""Label recovery by spectral embedding and K-means (Appendix D) against the fp64 oracle.

The oracle runs on the GPU's own factor (downloaded after the iterations) with
the same seed rows, so the comparison isolates the label step: the labels and
the number of Lloyd passes must be identical.
"""
import numpy as np
import pytest

from gpu_util import host, log, make_ctx
from oracle import kmeans
from oracle import labels as olab
from oracle import nlr as onlr
from synth import gaussian_mixture, make_workload, standard_normal_factor

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _check(ctx, K, seeds, truth=None, max_iter=100):
    lab_gpu, passes = ctx.labels_spectral(K, seeds, max_iter)
    lab_gpu = lab_gpu.cpu().numpy()
    lab_ref, passes_ref = olab.spectral_labels(host(ctx.U), K, seeds, max_iter)
    mism = int((lab_gpu != lab_ref).sum())
    log(f"  passes gpu {passes} oracle {passes_ref}; mismatches {mism}")
    assert passes == passes_ref
    assert mism == 0
    if truth is not None:
        ari = kmeans.adjusted_rand_index(lab_gpu, truth)
        log(f"  ARI vs truth {ari:.6f}")
        return ari
    return None


def test_labels_spectral_tiny_converged():
    X, Z, truth, wl = make_workload("tiny")
    ctx = make_ctx(X, Z.astype(np.float64), wl.K, onlr.default_step_size(wl.K), T_min=wl.T)
    ctx.run(wl.T)
    seeds = [int(np.flatnonzero(truth == k)[0]) for k in range(wl.K)]
    _check(ctx, wl.K, seeds, truth)


def test_labels_spectral_exact_recovery_factor():
    """U = H, the normalised membership matrix of the true partition (exact recovery, Appendix D):
    the labels are that partition."""
    X, Z, truth, wl = make_workload("tiny")
    H = kmeans.membership(truth.astype(np.int64), wl.K)  # in Omega: H >= 0, ||H||_F^2 = K
    ctx = make_ctx(X, H, wl.K, onlr.default_step_size(wl.K), flags=1)  # NLR_INIT_U_IN_OMEGA
    seeds = [int(np.flatnonzero(truth == k)[0]) for k in range(wl.K)]
    lab, passes = ctx.labels_spectral(wl.K, seeds)
    assert kmeans.same_partition(lab.cpu().numpy(), truth)


def test_labels_spectral_random_seeds_and_r_above_K():
    """r = 8 > K = 4 (the paper's r > K setting) and seed rows drawn at random."""
    X, truth, _ = gaussian_mixture(3000, 16, 4, 25.0, seed=9)
    Z = standard_normal_factor(3000, 8, seed=10).astype(np.float64)
    ctx = make_ctx(X, Z, 4, onlr.default_step_size(4), T_min=150)
    ctx.run(150)
    rng = np.random.default_rng(11)
    seeds = rng.choice(3000, size=4, replace=False).tolist()
    _check(ctx, 4, seeds)


def test_labels_spectral_gmm1m():
    X, Z, truth, wl = make_workload("gmm1m")
    ctx = make_ctx(X, Z.astype(np.float64), wl.K, onlr.default_step_size(wl.K), T_min=30)
    ctx.run(30)
    rng = np.random.default_rng(12)
    seeds = rng.choice(wl.n, size=wl.K, replace=False).tolist()
    _check(ctx, wl.K, seeds)


def test_labels_spectral_max_iter_and_split_path():
    X, Z, truth, wl = make_workload("tiny")
    ctx = make_ctx(X, Z.astype(np.float64), wl.K, onlr.default_step_size(wl.K), T_min=20, flags=8)
    ctx.run(20)
    seeds = [0, 1, 2, 3]
    _check(ctx, wl.K, seeds, max_iter=2)
    _check(ctx, wl.K, seeds, max_iter=100)


def test_labels_spectral_degenerate_and_errors():
    from paper_2609_36074_amd import nlr
    X, _, _ = gaussian_mixture(500, 8, 4, 16.0, seed=13)
    Z = standard_normal_factor(500, 4, seed=14).astype(np.float64)
    Z[:, 3] = -np.abs(Z[:, 3])  # projected start has a zero column: U^T U is singular
    ctx = make_ctx(X, Z, 4, 0.01)
    with pytest.raises(nlr.NlrError) as e:
        ctx.labels_spectral(4, [0, 1, 2, 3])
    assert e.value.status == nlr.NLR_EDEGENERATE
    with pytest.raises(nlr.NlrError) as e:
        ctx.labels_spectral(3, [0, 1, 500])  # seed row out of range
    assert e.value.status == nlr.NLR_EINVAL
    lab, passes = ctx.labels_spectral(3, [0, 1, 2])  # rank 3 is enough for K = 3
    assert passes >= 1
