"""Sizes beyond 2^31 and 2^32 elements, checked by a property that holds at any size.

Every row of X and of the start U0 appears twice, at rows i and i + m (m not a
multiple of any tile height, so the copies sit at different places in their
tiles).  The method treats rows alike: a row's update depends on its own x_i,
u_i, ytilde_i and on quantities summed over all rows (Theta, p, s, the scalars
of Algorithm 2), and the labels are row-wise.  So after any number of
iterations the two copies of every row of U and of the stored dual must be
bitwise equal, and so must their labels.  An index that wraps at 2^31 or 2^32
elements in any kernel (normalisation, projection, the passes, the finish pass,
labels) sends one copy to another row's data and breaks this equality; the
rescaled factor must also keep ||U||_F^2 = K.  The inputs are generated on the
GPU (Gaussian rows around K centres); each case holds 20-75 GB of device memory
and no large host arrays.
"""
import pytest

from gpu_util import log

pytestmark = pytest.mark.gpu

SPLIT = 8        # NLR_INIT_SPLIT_F16
DATA_START = 32  # NLR_INIT_DATA_START


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_36074_amd import nlr
    nlr.load_library()


def _doubled(m, d, r, K, seed):
    """X (2m x d) and U0 (2m x r) on the GPU, rows i and i + m equal."""
    import torch
    gen = torch.Generator(device="cuda:0")
    gen.manual_seed(seed)
    n = 2 * m
    X = torch.empty(n, d, dtype=torch.float32, device="cuda:0")
    X[:m].normal_(generator=gen)
    centres = 2.0 * torch.randn(K, d, generator=gen, device="cuda:0")
    chunk = 1 << 20
    for i0 in range(0, m, chunk):
        i1 = min(m, i0 + chunk)
        lab = torch.randint(0, K, (i1 - i0,), generator=gen, device="cuda:0")
        X[i0:i1] += centres[lab]
    X[m:].copy_(X[:m])
    U = torch.empty(n, r, dtype=torch.float32, device="cuda:0")
    U[:m].normal_(generator=gen)
    U[m:].copy_(U[:m])
    return X, U


def _frob2(U):
    import torch
    tot = 0.0
    for i0 in range(0, U.shape[0], 1 << 22):
        tot += float(torch.sum(U[i0:i0 + (1 << 22)].double() ** 2))
    return tot


# (what, m, d, r, K, flags): each doubles to n = 2m rows with n d > 2^32
CASES = [
    ("one-pass split, n r > 2^32", 34_000_003, 128, 64, 64, SPLIT),
    ("single pass fp32", 17_000_003, 128, 64, 64, 0),
    ("single pass split, 64 features", 34_000_003, 64, 16, 16, SPLIT),
    ("single pass fp32, 10 columns", 68_000_003, 32, 10, 10, 0),
    ("panel split", 2_900_003, 768, 256, 256, SPLIT),
    ("two-pass fp32, 768 x 256", 2_900_003, 768, 256, 256, 0),
    ("one-pass split, data-informed start, spectral labels", 17_000_003, 128, 64, 32, SPLIT | DATA_START),
]


@pytest.mark.parametrize("what,m,d,r,K,flags", CASES, ids=[c[0] for c in CASES])
def test_doubled_rows_bitwise(what, m, d, r, K, flags):
    import torch
    from paper_2609_36074_amd import nlr
    n = 2 * m
    T = 4
    log(f"max size: {what}: n={n} d={d} r={r} K={K} flags={flags}, n d = {n * d:.3e}, n r = {n * r:.3e}")
    X, U = _doubled(m, d, r, K, seed=m % 1000)
    log("  init")
    # eps_d = 1: every iteration takes the gated dual step, so the stored dual moves too
    ctx = nlr.Context(X, K, U, alpha=1.0 / (2 * (2 + 6 * K + 2)), beta=1.0, eps_d=1.0, eps_c=1e-12,
                      T_min=T, flags=flags)
    log(f"  run {T}")
    done, last = ctx.run(T)
    torch.cuda.synchronize()
    assert done == T
    hist = ctx.history(16)
    assert sum(h["dual_step"] for h in hist) >= 1, hist
    log("  labels")
    lab = ctx.labels()
    torch.cuda.synchronize()
    assert torch.equal(ctx.U[:m], ctx.U[m:]), "U rows i and i + m differ"
    assert torch.equal(ctx.y[:m], ctx.y[m:]), "stored dual entries i and i + m differ"
    assert torch.equal(lab[:m], lab[m:]), "labels i and i + m differ"
    assert bool(torch.isfinite(ctx.U).all()) and float(ctx.U.min()) >= 0.0
    assert float(ctx.y.abs().max()) > 0.0
    f2 = _frob2(ctx.U)
    log(f"  ||U||_F^2 / K = {f2 / K:.9f}, objective {last['objective']:.6e}")
    assert abs(f2 / K - 1.0) < 1e-4
    if flags & DATA_START:
        log("  spectral labels")
        seeds = [int(s) for s in torch.randperm(m, generator=torch.Generator().manual_seed(5))[:K]]
        slab, passes = ctx.labels_spectral(K, seeds, max_iter=20)
        torch.cuda.synchronize()
        assert torch.equal(slab[:m], slab[m:]), "spectral labels i and i + m differ"
        assert int(slab.min()) >= 0 and int(slab.max()) < K and passes >= 1
    ctx.close()
    del ctx, X, U, lab
    torch.cuda.empty_cache()
