"""Pins of the oracle's Eq. 7 pieces (Sec. 4.1): the diagonal of the damped inverse Hessian proxy and
the W-A importance built on it.  Each pin reaches the value by a route other than the oracle's own
(closed forms, a Schur complement by plain Gaussian elimination, eigenvalues, symmetry), so a dropped
damping term, a transposed or mis-indexed inverse or a lost factor 1/2 fails one of them."""
import numpy as np
import pytest

import oracle
from oracle import F32, colreduce, hessian_inverse_diagonal, obs_scale
from oracle.pipeline import channel_importance, prequantize
from oracle.refine import gram


def _spd(rng, n, tokens):
    X = rng.standard_normal((tokens, n)) * rng.uniform(0.2, 3.0, n)
    return X.T @ X


def test_scaled_identity():
    for c, damp in ((1.0, 0.01), (3.5, 0.0), (0.25, 0.1)):
        got = hessian_inverse_diagonal(c * np.eye(7), damp)
        np.testing.assert_allclose(got, np.full(7, 1.0 / (c * (1.0 + damp))), rtol=1e-15)


def test_diagonal_matrix():
    h = np.array([0.5, 2.0, 7.0, 1e-3, 40.0])
    damp = 0.02
    got = hessian_inverse_diagonal(np.diag(h), damp)
    np.testing.assert_allclose(got, 1.0 / (h + damp * h.mean()), rtol=1e-15)


def test_two_by_two_closed_form():
    a, b, c, damp = 4.0, -1.5, 2.0, 0.01
    dl = damp * (a + c) / 2
    det = (a + dl) * (c + dl) - b * b
    got = hessian_inverse_diagonal(np.array([[a, b], [b, c]]), damp)
    np.testing.assert_allclose(got, [(c + dl) / det, (a + dl) / det], rtol=1e-14)


def _solve_by_elimination(A, y):
    """Plain Gaussian elimination with partial pivoting (pure Python lists)."""
    n = len(y)
    M = [list(map(float, A[i])) + [float(y[i])] for i in range(n)]
    for c in range(n):
        p = max(range(c, n), key=lambda r: abs(M[r][c]))
        M[c], M[p] = M[p], M[c]
        for r in range(c + 1, n):
            f = M[r][c] / M[c][c]
            for k in range(c, n + 1):
                M[r][k] -= f * M[c][k]
    x = [0.0] * n
    for r in range(n - 1, -1, -1):
        x[r] = (M[r][n] - sum(M[r][k] * x[k] for k in range(r + 1, n))) / M[r][r]
    return x


def test_schur_complement_brute_force():
    """[A^-1]_jj = 1 / (A_jj - a_j^T A_{-j,-j}^-1 a_j) for the damped A, every j."""
    rng = np.random.default_rng(7)
    H = _spd(rng, 6, 20)
    damp = 0.01
    A = H + damp * np.mean(np.diag(H)) * np.eye(6)
    got = hessian_inverse_diagonal(H, damp)
    for j in range(6):
        rest = [i for i in range(6) if i != j]
        a = A[rest, j]
        y = _solve_by_elimination(A[np.ix_(rest, rest)], a)
        np.testing.assert_allclose(got[j], 1.0 / (A[j, j] - float(np.dot(a, y))), rtol=1e-11)


def test_trace_is_sum_of_inverse_eigenvalues():
    rng = np.random.default_rng(8)
    H = _spd(rng, 40, 25)  # rank 25 < 40: singular without the damping
    damp = 0.01
    lam = np.linalg.eigvalsh(H) + damp * np.mean(np.diag(H))
    np.testing.assert_allclose(hessian_inverse_diagonal(H, damp).sum(), np.sum(1.0 / lam), rtol=1e-10)


def test_permutation_equivariance():
    rng = np.random.default_rng(9)
    H = _spd(rng, 12, 30)
    p = rng.permutation(12)
    a = hessian_inverse_diagonal(H, 0.01)
    b = hessian_inverse_diagonal(H[np.ix_(p, p)], 0.01)
    np.testing.assert_allclose(b, a[p], rtol=1e-12)


def test_not_positive_definite_gives_nan():
    H = np.zeros((5, 5))
    assert np.all(np.isnan(hessian_inverse_diagonal(H, 0.01)))
    rng = np.random.default_rng(10)
    X = rng.standard_normal((16, 5))
    X[:, 2] = 0.0  # a channel that is never active: H has a zero row and column
    assert np.all(np.isnan(hessian_inverse_diagonal(X.T @ X, 0.0)))
    assert np.all(np.isfinite(hessian_inverse_diagonal(X.T @ X, 0.01)))


def test_obs_scale_rounds_once_to_float32():
    hinv = np.array([0.1, 3.0, 1e-7])
    s = obs_scale(hinv)
    assert s.dtype == np.float64
    np.testing.assert_array_equal(s, np.float32(1.0 / (2.0 * hinv)).astype(np.float64))


def test_eq7_equals_eq10_for_orthogonal_activations():
    """With orthogonal activation channels X X^T is diagonal, [(X X^T)^-1]_jj = 1 / [X X^T]_jj, so
    Eq. 7 (no damping) is the unpacked form of Appendix A.2, max_i (dW_ij)^2 * h_j / 2."""
    rng = np.random.default_rng(11)
    M, N, d, tokens = 16, 32, 8, 64
    Q, _ = np.linalg.qr(rng.standard_normal((tokens, N)))
    s = rng.uniform(0.5, 4.0, N)
    X = (Q * s).astype(np.float32)
    W = (rng.standard_normal((M, N)) * 0.02).astype(np.float32)
    base_idx = rng.choice(M * N // d, 16, replace=False)
    H = gram(X)
    np.testing.assert_allclose(H, np.diag(np.diag(H)), atol=1e-5 * np.max(np.diag(H)))
    got = channel_importance(W, None, F32, "obs", d, base_idx, 1, H, 0.0)
    Wq = prequantize(W, F32, d, base_idx, 1)
    h = np.diag(H)
    want = oracle.round_to(colreduce(W, Wq, scale=h / 2, reduce="max"), F32)
    np.testing.assert_allclose(got, want, rtol=1e-5)


@pytest.mark.parametrize("damp", [0.0, 0.01])
def test_damping_moves_only_toward_smaller_inverse(damp):
    """A larger damping adds a positive multiple of I: every [A^-1]_jj can only shrink."""
    rng = np.random.default_rng(12)
    H = _spd(rng, 10, 40)
    a = hessian_inverse_diagonal(H, damp)
    b = hessian_inverse_diagonal(H, damp + 0.05)
    assert np.all(b < a)
