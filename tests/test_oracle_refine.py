"""Pins of the oracle's loss-driven refinement (Alg. 1 QuantLoss / FineTuneCodebook /
BeamSearchOptimize at width 1) against definitions written out independently, brute force, closed
forms and a special case that reduces to plain nearest-codeword assignment."""
import numpy as np
import pytest

import oracle
from oracle import refine as orf


@pytest.fixture(scope="module")
def oracle_mod():
    oracle.build()
    return oracle


def rv(shape, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(shape) * scale).astype(np.float32)


def tiny_layer(M=5, N=12, d=4, K=6, n_ext=1, n_crit=4, T=9, seed=0):
    W = rv((M, N), seed, 0.5)
    X = rv((T, N), seed + 1)
    books = [rv((K, d), seed + 2, 0.5)] + [rv((K, d), seed + 3 + e, 0.2) for e in range(n_ext)]
    g = np.random.default_rng(seed + 9)
    codes = [g.integers(0, K, M * N // d).astype(np.int32)] + \
            [g.integers(0, K, M * n_crit // d).astype(np.int32) for _ in range(n_ext)]
    return W, X, books, codes


def what_of(W, d, n_crit, books, codes, n_base=1):
    R = orf.residual_f64(W, "f32", d, n_crit, codes, books, ["f32"] * len(books), n_base)
    return W.astype(np.float64) - R


def test_gram_brute_force(oracle_mod):
    X = rv((7, 5), 3)
    H = orf.gram(X)
    for i in range(5):
        for j in range(5):
            assert H[i, j] == pytest.approx(sum(float(X[t, i]) * float(X[t, j]) for t in range(7)), rel=1e-14)
    np.testing.assert_array_equal(H, H.T)


def test_quant_loss_definition_and_gram_form(oracle_mod):
    W, X, books, codes = tiny_layer()
    Wh = what_of(W, 4, 4, books, codes)
    L = orf.quant_loss(W, Wh.astype(np.float32), X)
    # independent form: sum over tokens and rows of the squared output error, in loops
    Wh32 = Wh.astype(np.float32).astype(np.float64)
    brute = 0.0
    for r in range(W.shape[0]):
        for t in range(X.shape[0]):
            brute += float(np.dot(W[r].astype(np.float64) - Wh32[r], X[t].astype(np.float64))) ** 2
    assert L == pytest.approx(brute, rel=1e-12)
    # the gram form the GPU path uses: sum_r R_r H R_r^T
    R = W.astype(np.float64) - Wh32
    assert float(np.sum(R * (R @ orf.gram(X)))) == pytest.approx(L, rel=1e-12)
    assert orf.quant_loss(W, W, X) == 0.0


def test_codebook_gradient_is_exact_central_difference(oracle_mod):
    """QuantLoss is quadratic in every codeword entry, so a central difference is exact up to
    rounding: each analytic gradient entry must match it."""
    M, N, d, K, n_crit = 5, 12, 4, 6, 4
    W, X, books, codes = tiny_layer(M, N, d, K, 1, n_crit)
    H = orf.gram(X)
    R = orf.residual_f64(W, "f32", d, n_crit, codes, books, ["f32", "f32"], 1)
    grads, loss = orf.codebook_grads(R, H, d, n_crit, codes, [K, K], 1)
    assert loss == pytest.approx(orf.quant_loss(W, what_of(W, d, n_crit, books, codes), X), rel=1e-12)
    h = 2.0 ** -6
    for b in range(2):
        for k in range(K):
            for t in range(d):
                Lp, Lm = [], []
                for sgn, out in ((1, Lp), (-1, Lm)):
                    bk = [x.copy() for x in books]
                    bk[b][k, t] = np.float32(bk[b][k, t] + sgn * h)
                    Rb = orf.residual_f64(W, "f32", d, n_crit, codes, bk, ["f32", "f32"], 1)
                    out.append(float(np.sum(Rb * (Rb @ H))))
                # the +-h values are exact in fp32 only when h is above the entry's ulp: use the
                # actual perturbation
                step = (np.float32(books[b][k, t] + h) - np.float32(books[b][k, t] - h))
                fd = (Lp[0] - Lm[0]) / float(step)
                assert grads[b][k, t] == pytest.approx(fd, rel=1e-7, abs=1e-9 * (abs(loss) + 1)), (b, k, t)
    # an unused codeword has zero gradient; the extended book sees only critical vectors
    unused = np.setdiff1d(np.arange(K), codes[1])
    assert np.all(grads[1][unused] == 0.0)


def test_adam_first_step_closed_form(oracle_mod):
    """With bias correction the first Adam step moves every coordinate by lr * g / (|g| + eps)."""
    C = rv((8, 4), 5)
    g = np.random.default_rng(6).standard_normal((8, 4))
    g[0, 0] = 0.0
    st = orf.AdamState(np.zeros_like(g), np.zeros_like(g))
    C1 = orf.adam_step(C, g, st, lr=1e-3, eps=1e-8)
    exp = (C.astype(np.float64) - 1e-3 * g / (np.abs(g) + 1e-8)).astype(np.float32)
    np.testing.assert_array_equal(C1, exp)
    assert C1[0, 0] == C[0, 0] and st.t == 1
    # second step with the same gradient: m_hat = g and v_hat = g^2 again, the same move
    C2 = orf.adam_step(C1, g, st, lr=1e-3, eps=1e-8)
    np.testing.assert_allclose(C2.astype(np.float64) - C1, exp.astype(np.float64) - C, rtol=1e-5, atol=1e-9)


def brute_force_sweep(W, X, d, n_crit, books, codes, b, n_base=1):
    """Greedy width-1 search for book b by the definition: for each group in order and each row,
    try every codeword, evaluate QuantLoss by its X form, keep the smallest (lowest index on ties)."""
    M, N = W.shape
    codes = [c.copy() for c in codes]
    cover = N // d if b < n_base else n_crit // d
    q = codes[b].reshape(M, cover)
    for g in range(cover):
        for r in range(M):
            best, best_k = None, None
            for k in range(books[b].shape[0]):
                q[r, g] = k
                L = orf.quant_loss(W[r:r + 1], what_of(W[r:r + 1], d, n_crit, books,
                                                       [c.reshape(M, -1)[r] for c in codes], n_base), X)
                if best is None or L < best:
                    best, best_k = L, k
            q[r, g] = best_k
    return codes


@pytest.mark.parametrize("b", [0, 1])
def test_refine_book_matches_brute_force_greedy(oracle_mod, b):
    M, N, d, K, n_crit = 4, 12, 4, 6, 8
    W, X, books, codes = tiny_layer(M, N, d, K, 1, n_crit, T=20, seed=11)
    exp = brute_force_sweep(W, X, d, n_crit, books, codes, b)
    H = orf.gram(X)
    R = orf.residual_f64(W, "f32", d, n_crit, codes, books, ["f32", "f32"], 1)
    got = [c.copy() for c in codes]
    L0 = float(np.sum(R * (R @ H)))
    orf.refine_book(R, H, books[b], got[b], d, N if b == 0 else n_crit)
    np.testing.assert_array_equal(got[b], exp[b])
    R2 = orf.residual_f64(W, "f32", d, n_crit, got, books, ["f32", "f32"], 1)
    np.testing.assert_allclose(R, R2, rtol=0, atol=1e-12)   # the running residual stays exact
    assert float(np.sum(R2 * (R2 @ H))) <= L0


def test_refine_with_identity_hessian_is_nearest_codeword(oracle_mod):
    """With X = I (so H = I) and a single book, the width-1 search is the Euclidean nearest codeword
    of every vector: it must agree with the oracle's assignment."""
    M, N, d, K = 16, 32, 8, 20
    W = rv((M, N), 21, 0.5)
    C = rv((K, d), 22, 0.5)
    X = np.eye(N, dtype=np.float32)
    codes = [np.zeros(M * N // d, np.int32)]
    H = orf.gram(X)
    R = orf.residual_f64(W, "f32", d, 0, codes, [C], ["f32"], 1)
    orf.refine_book(R, H, C, codes[0], d, N)
    exp, _ = oracle.assign(oracle.vectors(W, d), C)
    np.testing.assert_array_equal(codes[0], exp)


def test_refine_layer_loss_decreases(oracle_mod):
    M, N, d, K, n_crit = 24, 64, 8, 16, 16
    W = rv((M, N), 31, 0.5)
    X = rv((40, N), 32)
    g = np.random.default_rng(33)
    books = [rv((K, d), 34, 0.5), rv((K, d), 35, 0.1)]
    codes = [g.integers(0, K, M * N // d).astype(np.int32), g.integers(0, K, M * n_crit // d).astype(np.int32)]
    res0 = orf.refine_layer(W, X, d, n_crit, books, codes, 1, lr=0.0, steps=0, max_rounds=3)
    assert all(b <= a for a, b in zip(res0.losses, res0.losses[1:]))
    assert res0.changes[0] > 0
    res = orf.refine_layer(W, X, d, n_crit, books, codes, 1, lr=1e-3, steps=5, max_rounds=3)
    assert res.losses[-1] < res.losses[0]
    assert res.losses[-1] <= res0.losses[-1] * 1.05
    # eps above the starting loss: no round runs
    res_e = orf.refine_layer(W, X, d, n_crit, books, codes, 1, lr=1e-3, steps=5, max_rounds=3,
                             eps=res0.losses[0] * 2)
    assert res_e.rounds == 0


def test_bf16_layer_reduces_to_the_fp32_loop_without_steps(oracle_mod):
    """With bf16-representable values and no codebook steps, the bf16 path (bf16 W and first book) runs
    the same code search as the fp32 path on the widened values: the same codes and losses."""
    M, N, d, K, n_crit = 16, 48, 8, 12, 16
    W = oracle.round_to(rv((M, N), 41, 0.5).astype(np.float64), "bf16")
    X = rv((30, N), 42)
    g = np.random.default_rng(43)
    b0 = oracle.round_to(rv((K, d), 44, 0.5).astype(np.float64), "bf16")
    b1 = rv((K, d), 45, 0.1)
    codes = [g.integers(0, K, M * N // d).astype(np.int32), g.integers(0, K, M * n_crit // d).astype(np.int32)]
    a = orf.refine_layer(W, X, d, n_crit, [b0, b1], codes, 1, lr=1e-3, steps=0, max_rounds=2, w_dtype="bf16")
    f = orf.refine_layer(oracle.widen(W, "bf16"), X, d, n_crit, [oracle.widen(b0, "bf16"), b1], codes, 1, lr=1e-3,
                         steps=0, max_rounds=2)
    assert a.changes[0] > 0
    np.testing.assert_array_equal(a.losses, f.losses)
    for x, y in zip(a.codes, f.codes):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(a.books[0], b0)  # no step: the bf16 book is untouched


def test_bf16_book_is_its_master_rounded(oracle_mod):
    """A bf16 book after Adam steps is the nearest bf16 (ties to even) of an fp32 master that moved by
    the fp32 rule: every entry is within half a bf16 step of a value the fp32 update could reach, and
    the book does move when the steps exceed half an ulp."""
    M, N, d, K, n_crit = 16, 48, 8, 12, 16
    W = oracle.round_to(rv((M, N), 51, 0.5).astype(np.float64), "bf16")
    X = rv((30, N), 52)
    g = np.random.default_rng(53)
    b0 = oracle.round_to(rv((K, d), 54, 0.5).astype(np.float64), "bf16")
    codes = [g.integers(0, K, M * N // d).astype(np.int32)]
    res = orf.refine_layer(W, X, d, 0, [b0], codes, 1, lr=0.05, steps=3, max_rounds=1, w_dtype="bf16")
    book = res.books[0]
    assert book.dtype == np.uint16 and (book != b0).any()
    # brute force nearest-even on the bf16 grid around every entry is what round_to gives
    v = oracle.widen(book, "bf16").astype(np.float64)
    for x in (v * (1 + 2 ** -12)).ravel()[:64]:
        lo = np.float32(x).view(np.uint32) & 0xFFFF0000
        cands = [lo, lo + 0x10000]
        vals = [float(np.uint32(c).view(np.float32)) for c in cands]
        best = min(range(2), key=lambda i: (abs(vals[i] - x), cands[i] & 0x10000))
        assert oracle.round_to(np.array([x]), "bf16")[0] == np.uint16(cands[best] >> 16)
