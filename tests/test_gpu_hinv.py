"""GPU parity of crvq_hessian_inverse_diagonal, the denominator of the W-A importance of Sec. 4.1 Eq. 7,
against the oracle's diag((H + damp * mean(diag H) * I)^-1): sizes below, at and across the 64-wide
blocks (ragged tails), rank-deficient and full-rank proxies, the not-positive-definite contract,
determinism, and the full 4096- and 8192-channel proxies of the LLaMA-7B attention and 70B MLP
calibration sets.

Tolerance: a backward-stable Cholesky factorization and triangular inverse give each [A^-1]_jj to
about N * eps * kappa(A) relative (kappa from the damped proxy's eigenvalues, computed here); the
oracle carries an error of the same order, so the comparison allows 4 N eps kappa, at least 1e-12."""
import numpy as np
import pytest
import torch

import oracle
from oracle.refine import gram
from paper_2412_09282_amd import crvq as C
from paper_2412_09282_amd import inputs

from gpu_util import say

pytestmark = pytest.mark.gpu
EPS = np.finfo(np.float64).eps


def _gpu(H: np.ndarray, damp: float):
    Hd = torch.from_numpy(np.ascontiguousarray(H)).cuda()
    N = H.shape[0]
    hinv = torch.empty(N, dtype=torch.float64, device="cuda")
    scale = torch.empty(N, dtype=torch.float32, device="cuda")
    C.crvq_hessian_inverse_diagonal(Hd, hinv, scale, damp=damp)
    torch.cuda.synchronize()
    return hinv.cpu().numpy(), scale.cpu().numpy()


def _calib(rng, tokens, N):
    """N(0, 1) activations with per-channel scales log-uniform in [0.1, 10] (the calibration recipe)."""
    s = np.exp(rng.uniform(np.log(0.1), np.log(10.0), N))
    return (rng.standard_normal((tokens, N)) * s).astype(np.float32)


def _check(H, damp, what):
    N = H.shape[0]
    got, sc = _gpu(H, damp)
    exp = oracle.hessian_inverse_diagonal(H, damp)
    lam = np.linalg.eigvalsh(H) + damp * np.mean(np.diag(H)) if N <= 2048 else None
    kappa = lam[-1] / lam[0] if lam is not None else None
    tol = max(1e-12, 4 * N * EPS * kappa) if kappa is not None else 1e-8
    rel = np.abs(got / exp - 1.0)
    say(f"{what}: N {N} kappa {kappa if kappa is None else f'{kappa:.3g}'} max rel err {rel.max():.3g} (tol {tol:.3g})")
    assert np.all(np.isfinite(got)) and rel.max() <= tol, (rel.max(), tol)
    # the float32 factor is Eq. 7's 1 / (2 hinv), rounded once from the device's own fp64 value
    np.testing.assert_array_equal(sc, np.float32(1.0 / (2.0 * got)))
    np.testing.assert_allclose(sc.astype(np.float64), oracle.obs_scale(exp), rtol=max(2 ** -23, 2 * tol))
    return got


@pytest.mark.parametrize("N,tokens", [(1, 4), (5, 3), (63, 200), (64, 64), (65, 40), (130, 500), (257, 100),
                                      (700, 300), (1000, 2000)])
def test_hinv_parity(N, tokens):
    rng = np.random.default_rng([2412, N, tokens])
    H = gram(_calib(rng, tokens, N))
    _check(H, 0.01, f"hinv N={N} tokens={tokens}")


def test_hinv_full_rank_undamped_and_strong_damping():
    rng = np.random.default_rng(77)
    H = gram(_calib(rng, 600, 200))
    _check(H, 0.0, "hinv undamped, full rank")
    _check(H, 1.0, "hinv damp 1.0")


def test_hinv_structured():
    """Identity, diagonal and block-diagonal proxies across block boundaries."""
    rng = np.random.default_rng(78)
    got, _ = _gpu(np.eye(130) * 2.5, 0.0)
    np.testing.assert_allclose(got, 1.0 / 2.5, rtol=1e-15)
    h = rng.uniform(0.1, 50.0, 200)
    got, _ = _gpu(np.diag(h), 0.02)
    np.testing.assert_allclose(got, 1.0 / (h + 0.02 * h.mean()), rtol=1e-14)
    Hb = np.zeros((150, 150))
    for a, b in ((0, 70), (70, 150)):
        Hb[a:b, a:b] = gram(_calib(rng, 200, b - a))
    _check(Hb, 0.01, "hinv block-diagonal")


def test_hinv_reads_only_the_lower_triangle():
    rng = np.random.default_rng(79)
    H = gram(_calib(rng, 100, 90))
    Hg = np.tril(H) + np.triu(np.full_like(H, 1e30), 1)
    got, _ = _gpu(Hg, 0.01)
    ref, _ = _gpu(H, 0.01)
    np.testing.assert_array_equal(got, ref)


def test_hinv_not_positive_definite_gives_nan():
    for H, damp, what in ((np.zeros((70, 70)), 0.01, "zero proxy"), (-np.eye(9), 0.0, "negative definite")):
        got, sc = _gpu(H, damp)
        assert np.all(np.isnan(got)) and np.all(np.isnan(sc)), what
    rng = np.random.default_rng(80)
    X = _calib(rng, 300, 100)
    X[:, 77] = 0.0  # a channel never active: a zero row and column, singular without damping
    got, sc = _gpu(gram(X), 0.0)
    assert np.all(np.isnan(got)) and np.all(np.isnan(sc))
    _check(gram(X), 0.01, "hinv dead channel, damped")


def test_hinv_deterministic():
    rng = np.random.default_rng(81)
    H = gram(_calib(rng, 256, 300))
    a, sa = _gpu(H, 0.01)
    b, sb = _gpu(H, 0.01)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(sa, sb)


@pytest.mark.parametrize("wid", [2, 4])
def test_hinv_full_size(wid):
    """The proxies of the LLaMA-7B attention (2048 tokens x 4096 channels, rank-deficient) and 70B MLP
    (1024 x 8192) calibration sets, damped by 1 %; H formed on the device (crvq_gram)."""
    wl = inputs.workload(wid)
    X = inputs.make_calib(wl, 0)
    N = X.shape[1]
    say(f"hinv full size: workload {wid}, X {X.shape}")
    Xd = torch.from_numpy(X).cuda()
    Hd = torch.empty(N, N, dtype=torch.float64, device="cuda")
    C.crvq_gram(Xd, Hd)
    torch.cuda.synchronize()
    H = Hd.cpu().numpy()
    got, sc = _gpu(H, 0.01)
    exp = oracle.hessian_inverse_diagonal(H, 0.01)
    rel = np.abs(got / exp - 1.0)
    say(f"hinv full size N {N}: max rel err {rel.max():.3g}")
    assert rel.max() <= 1e-8
    np.testing.assert_array_equal(sc, np.float32(1.0 / (2.0 * got)))
