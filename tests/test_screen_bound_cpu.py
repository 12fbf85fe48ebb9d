"""The fp16 first screen's per-row split bound, checked on the host.

With a = alpha c and y = -2 alpha x (alpha a power of two, so both exact in fp32), a1 = fp16(a) and
y1 = fp16(y), the one-MFMA screen forms sum_t a1_t y1_t where the distance needs sum_t a_t y_t.  The
library certifies each row with

    |sum_t a_t y_t - sum_t a1_t y1_t| <= ||a|| (||y - y1|| + 2^-11 (1 + 2^-11) ||y||)

when every a_t and y_t lies in the fp16 normal range (below it the certificate carries separate
underflow terms), i.e. with ||a|| <= alpha R it adds R (||y2|| + 2^-11 (1 + 2^-11) ||y||) / alpha to the
bound in place of the worst case 2^-9 ||x|| R.  Both sides are evaluated here with exact products and
a correctly rounded sum, on random inputs, on inputs whose rounding remainders all point the same way
(the bound's worst case, to show the test is not vacuous) and at the edges of the fp16 range.
"""
import math

import numpy as np

D = 8


def f16(v):
    return np.asarray(v, dtype=np.float32).astype(np.float16).astype(np.float64)


def scale_for(cb):
    # alpha = 2^(11 - floor(log2 max|c|)): alpha max|c| in [2^11, 2^12)
    return 2.0 ** (11 - math.floor(math.log2(float(np.abs(cb).max()))))


def dropped_and_bound(x, c, alpha):
    y = (-2.0 * alpha * x.astype(np.float64)).astype(np.float32).astype(np.float64)
    a = (alpha * c.astype(np.float64)).astype(np.float32).astype(np.float64)
    assert np.array_equal(y, -2.0 * alpha * x.astype(np.float64)) and np.array_equal(a, alpha * c.astype(np.float64))
    y1, a1 = f16(y), f16(a)
    # products of two fp32 (or fp16) values are exact in fp64; fsum rounds the exact sum once
    exact = math.fsum(float(p) for p in a * y)
    screen = math.fsum(float(p) for p in a1 * y1)
    dropped = abs(exact - screen)
    y2 = y - y1  # exact
    bound = float(np.linalg.norm(a)) * (float(np.linalg.norm(y2)) + 2.0 ** -11 * (1 + 2.0 ** -11) * float(np.linalg.norm(y)))
    return dropped, bound


def in_normal_range(v):
    return bool((np.abs(v) >= 2.0 ** -14).all() and (np.abs(v) < 65504.0).all())


def test_random_rows_and_codewords():
    g = np.random.default_rng(5)
    for trial in range(2000):
        s = 10.0 ** g.uniform(-3, 3)
        cb = (g.standard_normal((16, D)) * s).astype(np.float32)
        cb[np.abs(cb) < s * 1e-2] = np.float32(s * 1e-2)
        alpha = scale_for(cb)
        x = (g.standard_normal(D) * s).astype(np.float32)
        x[np.abs(x) < s * 1e-2] = np.float32(s * 1e-2)
        for c in cb:
            y, a = -2.0 * alpha * x.astype(np.float64), alpha * c.astype(np.float64)
            if not (in_normal_range(y) and in_normal_range(a)):
                continue
            dropped, bound = dropped_and_bound(x, c, alpha)
            assert dropped <= bound * (1 + 1e-12), (trial, dropped, bound)


def test_aligned_remainders_reach_the_bound():
    """Every remainder of y points the same way and every a_t has that sign; the a remainders point
    along y1: the dropped sum is then close to the bound, which must still hold."""
    g = np.random.default_rng(6)
    worst = 0.0
    for trial in range(500):
        # y in [256, 512) where fp16 values are 0.25 apart: 256 + 0.25 j + (0.125 - 2^-13)
        j = g.integers(0, 1024, D).astype(np.float64)
        y = 256.0 + 0.25 * j + (0.125 - 2.0 ** -13)
        x = (-y / (2.0 * 2.0 ** 11)).astype(np.float32)          # alpha = 2^11
        # a in (-4096, -2048] (fp16 spacing 2) just short of a midpoint, so that a_t y2_t and a2_t y1_t
        # all share one sign; c = a / 2^11 then has max|c| in [1, 2), which is what makes alpha 2^11
        k = g.integers(0, 1024, D).astype(np.float64)
        a = -(2048.0 + 2.0 * k + (1.0 - 2.0 ** -11))
        c = (a / 2.0 ** 11).astype(np.float32)
        assert scale_for(c) == 2.0 ** 11
        dropped, bound = dropped_and_bound(x, c, 2.0 ** 11)
        assert dropped <= bound * (1 + 1e-12), (trial, dropped, bound)
        worst = max(worst, dropped / bound)
    assert worst > 0.8, worst   # the bound is nearly attained (about 0.88): the check above is not vacuous


def test_per_row_factor_never_exceeds_the_worst_case():
    """In the fp16 normal range ||y2|| <= 2^-11 ||y||, so the per-row factor is at most the worst-case
    factor 2^-9 (1 + 2^-9) ||x|| the certificate used before (with ||a|| <= alpha R, ||y|| = 2 alpha ||x||)."""
    g = np.random.default_rng(7)
    for _ in range(5000):
        x = (g.standard_normal(D) * 10.0 ** g.uniform(-2, 2)).astype(np.float32)
        alpha = 2.0 ** int(g.integers(-10, 20))
        y = -2.0 * alpha * x.astype(np.float64)
        if not in_normal_range(y):
            continue
        y2 = y - f16(y)
        e = (np.linalg.norm(y2) + 2.0 ** -11 * (1 + 2.0 ** -11) * np.linalg.norm(y)) / alpha
        assert e <= 2.0 ** -9 * (1 + 2.0 ** -9) * np.linalg.norm(x.astype(np.float64)) * (1 + 1e-12)
