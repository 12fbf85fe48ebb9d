"""GPU parity of the matrix-vector product with a CRVQ-quantized layer (crvq_dequant_gemv) against
the oracle's fp64 product of the exact reconstruction (Sec. 4.3, Fig. 3 right).

Tolerance: the kernel forms fp32 products (an 8-term dot product per column group or a table entry
of one), fp32 partial sums over at most 1024 columns and fp64 sums across them, so its error is a
few tens of 2^-24 * a_r with a_r = sum_j |W_hat_rj x_j|; the test asks for 1e-5 * a_r (and reports
the largest ratio seen).  Shapes run from tiny, ragged layers to the LLaMA gate projections the
paper times (11008 x 4096, 13824 x 5120, 17920 x 6656) with 0, 1 and 3 extended books at 2 %
critical channels."""
import numpy as np
import pytest
import torch

import oracle
from paper_2412_09282_amd import crvq as C
from paper_2412_09282_amd import inputs

from gpu_util import dev, say

pytestmark = pytest.mark.gpu

TOL = 1e-5


def make_layer(M, N, n_crit, n_ext, K_base, K_ext, dtype, seed, with_perm=True):
    g = np.random.default_rng(seed)
    d = 8
    books = [inputs.random_vectors(K_base, d, seed + 1, 0.02)] + \
            [inputs.random_vectors(K_ext, d, seed + 2 + e, 0.005) for e in range(n_ext)]
    if dtype == "bf16":
        books[0] = inputs.f32_to_bf16_bits(books[0])
    codes = [g.integers(0, K_base, M * N // d).astype(np.int32)] + \
            [g.integers(0, K_ext, M * n_crit // d).astype(np.int32) for _ in range(n_ext)]
    perm = g.permutation(N).astype(np.int32) if with_perm else None
    x = inputs.random_vectors(1, N, seed + 9, 1.0)[0]
    if dtype == "bf16":
        x = inputs.f32_to_bf16_bits(x)
    return books, codes, perm, x


def run_gemv(M, N, n_crit, books, codes, perm, x, dtype):
    d = 8
    q8 = [torch.empty(c.size, dtype=torch.uint8, device="cuda") for c in codes]
    for c, t in zip(codes, q8):
        C.crvq_pack_codes_u8(dev(c), t)
    y = torch.empty(M, dtype=torch.float32, device="cuda")
    C.crvq_dequant_gemv(M, N, q8[0], N // d, dev(books[0], dtype), dev(x, dtype), y, n_crit=n_crit,
                        q_ext=q8[1:], ldq_ext=max(1, n_crit // d), C_ext=[dev(b) for b in books[1:]],
                        perm=None if perm is None else dev(perm))
    torch.cuda.synchronize()
    return y.cpu().numpy(), [t.cpu().numpy() for t in q8]


def check(M, N, n_crit, n_ext, K_base, K_ext, dtype, seed, with_perm=True):
    books, codes, perm, x = make_layer(M, N, n_crit, n_ext, K_base, K_ext, dtype, seed, with_perm)
    got, packed = run_gemv(M, N, n_crit, books, codes, perm, x, dtype)
    for c, p in zip(codes, packed):
        np.testing.assert_array_equal(p, (c & 255).astype(np.uint8))
    bdt = [dtype] + ["f32"] * n_ext
    exp, a = oracle.gemv(M, N, 8, n_crit, codes, books, perm, x, bdt, dtype)
    err = np.abs(got.astype(np.float64) - exp)
    ratio = float((err / (a + 1e-300)).max()) if M else 0.0
    assert np.isfinite(got).all()
    assert (err <= TOL * a + 1e-30).all(), f"worst |y - W x| / sum|W x| = {ratio:.3g}"
    say(f"gemv {M}x{N} n_crit={n_crit} ext={n_ext} K={K_base} {dtype}: worst error / a = {ratio:.3g}")


@pytest.mark.parametrize("M,N,n_crit,n_ext,K_base,K_ext,dtype,perm", [
    (37, 128, 16, 1, 256, 256, "f32", True),
    (1, 64, 64, 2, 256, 256, "f32", True),       # every group critical
    (64, 1024, 0, 0, 16, 16, "f32", False),      # short basic book, no reorder
    (33, 2048, 40, 3, 100, 7, "bf16", True),     # ragged rows, odd book sizes
    (200, 4096, 88, 3, 256, 256, "f32", True),   # 8+8x3 at 2 % of a 4096-wide layer
    (100, 6656, 136, 1, 256, 256, "bf16", True),
    (513, 1984, 8, 1, 256, 256, "f32", True),    # 248 groups: a short last slice
])
def test_gemv_parity(M, N, n_crit, n_ext, K_base, K_ext, dtype, perm):
    check(M, N, n_crit, n_ext, K_base, K_ext, dtype, 300 + M, perm)


@pytest.mark.parametrize("M,N,n_ext", [(11008, 4096, 1), (13824, 5120, 3), (17920, 6656, 0)])
def test_gemv_parity_llama_gate_shapes(M, N, n_ext):
    n_crit = inputs.n_crit_columns(N, 8, 0.02)
    check(M, N, n_crit, n_ext, 256, 256, "f32", 400 + n_ext)


def test_gemv_empty_and_bad_codes():
    y = torch.zeros(0, dtype=torch.float32, device="cuda")
    q = torch.zeros(8, dtype=torch.uint8, device="cuda")
    Cb = torch.zeros(4, 8, dtype=torch.float32, device="cuda")
    C.crvq_dequant_gemv(0, 64, q, 8, Cb, torch.zeros(64, device="cuda"), y)  # M = 0: nothing to do
    # a code outside a short basic book makes its row NaN, the other rows stay exact
    M, N, K = 40, 256, 200
    books, codes, perm, x = make_layer(M, N, 16, 1, K, 256, "f32", 77)
    codes[0][3 * (N // 8) + 5] = 250
    got, _ = run_gemv(M, N, 16, books, codes, perm, x, "f32")
    assert np.isnan(got[3])
    ok = np.setdiff1d(np.arange(M), [3])
    codes[0][3 * (N // 8) + 5] = 0
    exp, a = oracle.gemv(M, N, 8, 16, codes, books, perm, x)
    assert (np.abs(got[ok] - exp[ok]) <= TOL * a[ok]).all()
