"""GPU parity of the nearest-codeword search on the shapes that select each screen variant.

Long top-1 searches (at least 256 16-codeword tiles per codebook split, e.g. 65536 rows x 65536
codewords) run on 32 x 32 tiles under a power-of-two codebook scale: one fp16 MFMA per tile, exact for
bf16 operands, and for fp32 operands a second, split-fp16 screen of the rows the first leaves
uncertain; shorter ones on 16 x 16 tiles with split-bf16 operands.  Whatever the variant, the certified screen plus the
exact rescue must return the oracle's codes (the fp64 definition of Eq. 3, ties to the lower index)
and its distances, including rows the scaled screen cannot represent (forced to the exact rescue),
codebooks of extreme magnitude and ragged tails."""
import numpy as np
import pytest
import torch

import oracle
from paper_2412_09282_amd import crvq as C
from paper_2412_09282_amd import inputs
from paper_2412_09282_amd.crvq import VecSet

from gpu_util import dev, say

pytestmark = pytest.mark.gpu


def rv(n, d, seed, scale=0.02):
    return inputs.random_vectors(n, d, seed, scale)


def assign_both(V, Cb, dtype="f32"):
    Vt = dev(V, dtype)
    Ct = dev(Cb, dtype)
    n = V.shape[0]
    codes = torch.empty(n, dtype=torch.int32, device="cuda")
    dist = torch.empty(n, dtype=torch.float32, device="cuda")
    C.crvq_assign(VecSet.of_vectors(Vt), Ct, codes, dist)
    torch.cuda.synchronize()
    exp, ed = oracle.assign(V, Cb, dtype, dtype)
    return codes.cpu().numpy(), dist.cpu().numpy(), exp, ed


def check(V, Cb, dtype="f32"):
    got, gd, exp, ed = assign_both(V, Cb, dtype)
    bad = np.flatnonzero(got != exp)
    assert len(bad) == 0, f"{len(bad)} codes differ, e.g. rows {bad[:5]} got {got[bad[:5]]} want {exp[bad[:5]]}"
    np.testing.assert_array_equal(gd, ed.astype(np.float32))


@pytest.mark.parametrize("n,K,d", [(65536, 65536, 8), (65536 + 37, 65536 - 5, 8), (70001, 32768 + 17, 5)])
def test_long_search_f32(n, K, d):
    say(f"long top-1 search fp32 n={n} K={K} d={d}")
    check(rv(n, d, 31 + d), rv(K, d, 32 + K))


def test_long_search_bf16():
    say("long top-1 search bf16 n=65536 K=65536")
    V = inputs.f32_to_bf16_bits(rv(65536, 8, 33))
    Cb = inputs.f32_to_bf16_bits(rv(65536, 8, 34))
    check(V, Cb, "bf16")


@pytest.mark.parametrize("case", ["ties", "outliers", "tiny", "huge"])
def test_long_search_bf16_exact_operands(case):
    """bf16 rows against a bf16 codebook take the one-MFMA screen (exact fp16 operands)."""
    say(f"long top-1 search bf16, exact-operand screen: {case}")
    g = np.random.default_rng(44)
    if case == "ties":
        base = rv(16384, 8, 45)
        Cb = np.ascontiguousarray(np.concatenate([base, base, base[::-1], base])[g.permutation(65536)])
        V = np.concatenate([base[g.integers(0, 16384, 40000)], rv(25536 + 11, 8, 46)])
    elif case == "outliers":
        Cb = (g.standard_t(4.0, size=(65536 - 3, 8)) * 0.02).astype(np.float32)
        Cb[:, 5] *= np.float32(10.0)
        V = (g.standard_t(4.0, size=(65536 + 29, 8)) * 0.02).astype(np.float32)
        big = g.choice(len(V), 300, replace=False)
        V[big, g.integers(0, 8, 300)] *= np.float32(1e5)   # beyond the scaled fp16 range
        tiny = g.choice(len(V), 300, replace=False)
        V[tiny] *= np.float32(1e-9)                        # below the fp16 normal range once scaled
    else:
        s = np.float32(1e-30 if case == "tiny" else 1e30)
        V, Cb = rv(65536, 8, 47) * s, rv(65536, 8, 48) * s
    check(inputs.f32_to_bf16_bits(V), inputs.f32_to_bf16_bits(Cb), "bf16")


def test_long_search_outlier_rows_and_heavy_tails():
    say("long top-1 search: t4 codebook with outlier columns, rows far outside the codebook range")
    g = np.random.default_rng(35)
    K, n = 65536, 65536
    Cb = (g.standard_t(4.0, size=(K, 8)) * 0.02).astype(np.float32)
    Cb[:, 3] *= np.float32(10.0)
    V = (g.standard_t(4.0, size=(n, 8)) * 0.02).astype(np.float32)
    big = g.choice(n, 300, replace=False)
    V[big, g.integers(0, 8, 300)] *= np.float32(1e5)   # beyond the scaled fp16 range: exact rescue
    tiny = g.choice(n, 300, replace=False)
    V[tiny] *= np.float32(1e-6)                       # far below the codebook scale
    check(V, Cb)


@pytest.mark.parametrize("scale", [1e-30, 1e30])
def test_long_search_extreme_magnitude(scale):
    say(f"long top-1 search at magnitude {scale:g}")
    s = np.float32(scale)
    check(rv(65536, 8, 36) * s, rv(65536, 8, 37) * s)


def test_long_search_duplicates_and_ties():
    say("long top-1 search with duplicated codewords and rows equal to codewords")
    g = np.random.default_rng(38)
    base = rv(16384, 8, 39)
    Cb = np.ascontiguousarray(np.concatenate([base, base, base[::-1], base])[g.permutation(65536)])
    V = np.concatenate([base[g.integers(0, 16384, 40000)], rv(25536, 8, 40)])
    check(V, Cb)


def test_beam_width_one_long_codebook():
    say("residual beam, width 1, over a K=65536 basic and K=256 extended codebook")
    n = 65536
    V = rv(n, 8, 41)
    books = [rv(65536, 8, 42), rv(256, 8, 43, 0.005)]
    Vt = dev(V)
    bt = [dev(b) for b in books]
    codes = [torch.empty(n, dtype=torch.int32, device="cuda") for _ in books]
    err = torch.empty(n, dtype=torch.float32, device="cuda")
    C.crvq_assign_residual_beam(VecSet.of_vectors(Vt), bt, 1, codes, err)
    torch.cuda.synchronize()
    exp_codes, exp_err = oracle.beam(V, books, 1)
    for t in range(2):
        got = codes[t].cpu().numpy()
        bad = np.flatnonzero(got != exp_codes[t])
        assert len(bad) == 0, f"book {t}: {len(bad)} codes differ, e.g. rows {bad[:5]}"
    np.testing.assert_array_equal(err.cpu().numpy(), np.asarray(exp_err, dtype=np.float64).astype(np.float32))


@pytest.mark.parametrize("n", [65536 + 37, (1 << 20) + 37])
def test_beam_width_one_long_extended_book(n):
    """Width 1 over a K=4096 basic and a K=65536 extended book: the extended step searches the fp64
    residuals on the 32 x 32 fp16 screens (unpruned with codebook splits at 65,573 rows, pruned in key
    order at 1,048,613), whose operands are the residuals rounded to fp32; the certificate adds that
    rounding to each row's own fp16 remainder."""
    say(f"residual beam, width 1, K=4096 basic + K=65536 extended over fp64 residuals, n={n}")
    V = rv(n, 8, 81)
    books = [rv(4096, 8, 82), rv(65536, 8, 83, 0.006)]
    codes = [torch.empty(n, dtype=torch.int32, device="cuda") for _ in books]
    err = torch.empty(n, dtype=torch.float32, device="cuda")
    C.crvq_assign_residual_beam(VecSet.of_vectors(dev(V)), [dev(b) for b in books], 1, codes, err)
    torch.cuda.synchronize()
    exp_codes, exp_err = oracle.beam(V, books, 1)
    for t in range(2):
        got = codes[t].cpu().numpy()
        bad = np.flatnonzero(got != exp_codes[t])
        assert len(bad) == 0, f"book {t}: {len(bad)} codes differ, e.g. rows {bad[:5]}"
    np.testing.assert_array_equal(err.cpu().numpy(), np.asarray(exp_err, dtype=np.float64).astype(np.float32))


# Long searches on fp32 operands (here 262144 rows x 65536 codewords, four codebook splits) get two
# screens: one MFMA per tile on fp16-rounded operands with the wider certificate, then the split form
# on the rows it left uncertain, then the exact rescue of what is left.
@pytest.mark.parametrize("case", ["plain", "ties", "mixed_bf16_book"])
def test_two_pass_screen(case):
    n, K, d = 262144 + 37, 65536, 8
    say(f"two-pass screen fp32 n={n} K={K} ({case})")
    g = np.random.default_rng(44)
    if case == "ties":
        base = rv(16384, 8, 45)
        Cb = np.ascontiguousarray(np.concatenate([base, base, base[::-1], base])[g.permutation(K)])
        V = np.concatenate([base[g.integers(0, 16384, n // 2)], rv(n - n // 2, 8, 46)])
        check(V, Cb)
    elif case == "mixed_bf16_book":
        V = rv(n, d, 47)
        Cb = inputs.f32_to_bf16_bits(rv(K, d, 48))
        Vt, Ct = dev(V), dev(Cb, "bf16")
        codes = torch.empty(n, dtype=torch.int32, device="cuda")
        dist = torch.empty(n, dtype=torch.float32, device="cuda")
        C.crvq_assign(VecSet.of_vectors(Vt), Ct, codes, dist)
        torch.cuda.synchronize()
        exp, ed = oracle.assign(V, Cb, "f32", "bf16")
        np.testing.assert_array_equal(codes.cpu().numpy(), exp)
        np.testing.assert_array_equal(dist.cpu().numpy(), ed.astype(np.float32))
    else:
        # codewords drawn near the rows, as K-means leaves them: many near-ties for the first screen
        V = rv(n, d, 49)
        Cb = np.ascontiguousarray(V[g.choice(n, K, replace=False)] + rv(K, d, 50, 0.002))
        check(V, Cb)


# The first screen on fp16-rounded operands certifies each row with its own fp16 remainder: with
# a = alpha c and y = -2 alpha x = y1 + y2 the dropped terms are sum_t a_t y2_t + sum_t a2_t y1_t, bounded
# by R (||y2|| + 2^-11 (1 + 2^-11) ||y||) / alpha.  Here every row sits just below the midpoint between
# two fp16 values after the power-of-two scale (each y2_t positive and 2^-13 short of half a spacing,
# the largest it can be), and the codewords share the rows' signs, so sum_t a_t y2_t is close to its
# Cauchy-Schwarz bound; the codewords come in near-tied pairs, so many rows stay uncertain.  Codes
# and distances must remain the oracle's (unpruned: 4 codebook splits; pruned: one split, key order).
@pytest.mark.parametrize("n,K", [(262144 + 37, 65536), ((1 << 20) + 37, 16384)])
def test_first_screen_aligned_remainders(n, K):
    d = 8
    say(f"first screen, remainders aligned with the codewords: n={n} K={K}")
    g = np.random.default_rng(71)
    # -2^12 x in [256, 512), where fp16 values are 0.25 apart: 256 + 0.25 j + (0.125 - 2^-13), exact in fp32
    j = g.integers(0, 1024, size=(n, d)).astype(np.float64)
    V = (-(256.0 + 0.25 * j + (0.125 - 2.0 ** -13)) / 4096.0).astype(np.float32)
    base = V[g.choice(n, K // 2, replace=False)]
    e1 = (g.random((K // 2, d)) * 2e-6).astype(np.float32)
    e2 = (g.random((K // 2, d)) * 2e-6).astype(np.float32)
    Cb = np.ascontiguousarray(np.concatenate([base - e1, base - e2])[g.permutation(K)])
    assert (Cb < 0).all() and (V < 0).all()
    check(V, Cb)


def test_second_screen_own_rows_full():
    """From 2^23 rows up the second (split) screen of fp32 rows gives every wave rows of its own
    instead of sharing them across a workgroup.  Every row of a (2^23 + 37)-row search against 4096
    codewords drawn next to the rows (so several percent of the rows reach the second screen) is
    compared with the oracle."""
    n, K, d = (1 << 23) + 37, 4096, 8
    say(f"two-pass screen fp32 n={n} K={K}: second screen with rows per wave, full comparison")
    g = np.random.default_rng(51)
    V = rv(n, d, 52)
    Cb = np.ascontiguousarray(V[g.choice(n, K, replace=False)] + rv(K, d, 53, 0.002))
    check(V, Cb)


# From about a million rows (no codebook splits) the first screen visits the codebook in the order
# of a key (norm, then two coordinates, each binned over a robust range of the codebook) and skips
# pairs of tiles whose norms or coordinates are certified too far from every row of a wave; the
# results must stay the oracle's exactly.  "constant": both key coordinates constant over the codebook
# (no spread to bin); "outlier_cols": heavy tails with 10x outlier coordinates in 8 % of the vectors
# (the bins follow the bulk, the outliers fall into the end bins); "d1": one dimension (both key
# coordinates are the same one).
@pytest.mark.parametrize("case,K", [("near", 65536), ("bf16", 16384), ("outliers", 16384), ("ties", 16384),
                                    ("tiny", 4096), ("constant", 16384), ("outlier_cols", 16384),
                                    ("d1", 4096)])
def test_pruned_first_screen(case, K):
    n, d = (1 << 20) + 4096 + 37, (1 if case == "d1" else 8)
    say(f"pruned first screen n={n} K={K} ({case})")
    g = np.random.default_rng(60)
    if case in ("near", "bf16"):
        V = rv(n, d, 61)
        Cb = np.ascontiguousarray(V[g.choice(n, K, replace=False)] + rv(K, d, 62, 0.002))
        if case == "bf16":
            check(inputs.f32_to_bf16_bits(V), inputs.f32_to_bf16_bits(Cb), "bf16")
            return
    elif case == "outliers":
        Cb = (g.standard_t(4.0, size=(K, d)) * 0.02).astype(np.float32)
        Cb[:, 0] *= np.float32(10.0)                       # the coordinate of the second band
        V = (g.standard_t(4.0, size=(n, d)) * 0.02).astype(np.float32)
        big = g.choice(n, 500, replace=False)
        V[big, g.integers(0, d, 500)] *= np.float32(1e5)   # beyond the scaled fp16 range: rescued exactly
        tiny = g.choice(n, 500, replace=False)
        V[tiny] *= np.float32(1e-6)
    elif case == "ties":
        base = rv(K // 4, d, 63)
        Cb = np.ascontiguousarray(np.concatenate([base, base, base[::-1], base])[g.permutation(K)])
        V = np.concatenate([base[g.integers(0, K // 4, n // 2)], rv(n - n // 2, d, 64)])
    elif case == "constant":
        V = rv(n, d, 67)
        Cb = rv(K, d, 68)
        Cb[:, 0] = np.float32(0.01)
        Cb[:, 1] = np.float32(-0.02)
        V[: n // 2, 0] = np.float32(0.01)
    elif case == "outlier_cols":
        V = (g.standard_t(4.0, size=(n, d)) * 0.02).astype(np.float32)
        hit = g.random(n) < 0.08
        V[hit, g.integers(0, d, int(hit.sum()))] *= np.float32(10.0)
        Cb = np.ascontiguousarray(V[g.choice(n, K, replace=False)])
    elif case == "d1":
        V = rv(n, d, 69)
        Cb = rv(K, d, 70)
    else:  # magnitudes far below one: the bands are kept in units of the codebook scale
        V = rv(n, d, 65) * np.float32(1e-30)
        Cb = rv(K, d, 66) * np.float32(1e-30)
    check(V, Cb)


def test_rescue_of_most_rows():
    """Rows equal to codewords that the book holds four times (exact ties on every row, so nearly every
    row reaches the exact rescue) over 1,048,579 rows: more listed rows than the parted rescue has
    room for, so the rescue scans the whole codebook per row batch; sampled rows against the oracle."""
    say("long top-1 search, 1048579 rows that all tie: whole-codebook rescue")
    g = np.random.default_rng(44)
    base = rv(16384, 8, 45)
    Cb = np.ascontiguousarray(np.concatenate([base, base, base, base])[g.permutation(65536)])
    n = 1048579
    V = np.ascontiguousarray(base[g.integers(0, 16384, n)])
    codes = torch.empty(n, dtype=torch.int32, device="cuda")
    dist = torch.empty(n, dtype=torch.float32, device="cuda")
    C.crvq_assign(VecSet.of_vectors(dev(V)), dev(Cb), codes, dist)
    torch.cuda.synchronize()
    S = np.sort(g.choice(n, 3000, replace=False))
    S[-1] = n - 1
    exp, ed = oracle.assign(V[S], Cb)
    np.testing.assert_array_equal(codes.cpu().numpy()[S], exp)
    np.testing.assert_array_equal(dist.cpu().numpy()[S], ed.astype(np.float32))


# Small codebooks (K <= 256) at row counts that take the wide top-1 kernel (128 rows per wave): fp32 and
# bf16 rows packed at a 16-byte aligned base take its fast forms, any other layout the generic form;
# codes and distances must equal the oracle's, including exact ties (duplicated codewords, rescued)
# and a last tile of padding codewords (K = 37).
@pytest.mark.parametrize("case", ["f32", "f32_k37", "bf16", "unaligned", "ties"])
def test_small_book_wide_forms(case):
    n, d = 600_001, 8
    say(f"small-book top-1, wide form: {case}, n={n}")
    K = 37 if case == "f32_k37" else 256
    V = rv(n, d, 71)
    Cb = rv(K, d, 72)
    if case == "ties":
        Cb[128:] = Cb[:128]
        V[: n // 3] = Cb[np.random.default_rng(73).integers(0, 128, n // 3)]
    if case == "bf16":
        check(inputs.f32_to_bf16_bits(V), inputs.f32_to_bf16_bits(Cb), "bf16")
        return
    if case == "unaligned":
        buf = torch.empty(n * d + 1, dtype=torch.float32, device="cuda")
        buf[1:] = torch.from_numpy(V.reshape(-1)).cuda()
        Vt = buf[1:].view(n, d)  # base 4 bytes past a 16-byte boundary
        codes = torch.empty(n, dtype=torch.int32, device="cuda")
        dist = torch.empty(n, dtype=torch.float32, device="cuda")
        C.crvq_assign(VecSet.of_vectors(Vt), dev(Cb), codes, dist)
        torch.cuda.synchronize()
        exp, ed = oracle.assign(V, Cb)
        np.testing.assert_array_equal(codes.cpu().numpy(), exp)
        np.testing.assert_array_equal(dist.cpu().numpy(), ed.astype(np.float32))
        return
    check(V, Cb)
