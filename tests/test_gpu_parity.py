"""GPU parity: every library call against the CPU oracle on the same seeded inputs, through the C ABI.

Codes, permutations and counts must match exactly (codes: except within 1e-6 relative distance
ties); floating outputs within 1e-5 relative (fp32) or 1e-2 (bf16 storage).  Sizes span several
tiles with ragged tails and the degenerate cases (K = 1, K < 16, duplicate and near-duplicate
codewords, empty clusters, out-of-range codes)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline as opipe
from paper_2412_09282_amd import crvq as C
from paper_2412_09282_amd import inputs
from paper_2412_09282_amd.crvq import VecSet
from paper_2412_09282_amd.pipeline import LayerConfig, LayerQuantizer

from gpu_util import check_codes, dev, dt, rel_close, say, to_host_bits

pytestmark = pytest.mark.gpu


def rv(n, d, seed, scale=0.02):
    return inputs.random_vectors(n, d, seed, scale)


def run_assign(V, Cb, v_dtype="f32", c_dtype="f32", vs=None):
    Vt = dev(V, v_dtype)
    Ct = dev(Cb, c_dtype)
    n = V.shape[0]
    codes = torch.empty(n, dtype=torch.int32, device="cuda")
    dist = torch.empty(n, dtype=torch.float32, device="cuda")
    C.crvq_assign(vs(Vt) if vs else VecSet.of_vectors(Vt), Ct, codes, dist)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), dist.cpu().numpy()


@pytest.mark.parametrize("n,d,K", [(1000, 8, 256), (777, 8, 37), (513, 1, 16), (1500, 3, 100), (2049, 4, 7),
                                   (900, 16, 300), (3000, 8, 1), (5000, 8, 1000), (300, 5, 2000), (20000, 8, 65536)])
def test_assign_parity(n, d, K):
    say(f"assign n={n} d={d} K={K}")
    V = rv(n, d, 1 + d)
    Cb = rv(K, d, 100 + K)
    got, gd = run_assign(V, Cb)
    exp, ed = oracle.assign(V, Cb)
    check_codes(V, Cb, got, exp)
    assert (got == exp).all(), "exact parity expected (certified screen + exact rescue)"
    np.testing.assert_array_equal(gd, ed.astype(np.float32))


def test_assign_bf16():
    say("assign bf16 n=4000 d=8 K=1024")
    V = inputs.f32_to_bf16_bits(rv(4000, 8, 5))
    Cb = inputs.f32_to_bf16_bits(rv(1024, 8, 6))
    got, gd = run_assign(V, Cb, "bf16", "bf16")
    exp, ed = oracle.assign(V, Cb, "bf16", "bf16")
    assert (got == exp).all()
    np.testing.assert_array_equal(gd, ed.astype(np.float32))


def test_assign_ties_and_near_ties():
    say("assign ties / near-ties n=4096 d=8 K=512")
    g = np.random.default_rng(7)
    base = rv(128, 8, 8)
    eps = (g.standard_normal((128, 8)) * 1e-9).astype(np.float32)
    Cb = np.concatenate([base, base, base + eps, base[::-1]])  # exact duplicates and 1e-7-relative neighbours
    p = g.permutation(512)
    Cb = np.ascontiguousarray(Cb[p])
    V = np.concatenate([base[g.integers(0, 128, 2048)], rv(2048, 8, 9)])
    got, gd = run_assign(V, Cb)
    exp, ed = oracle.assign(V, Cb)
    assert (got == exp).all()
    np.testing.assert_array_equal(gd, ed.astype(np.float32))


def test_assign_exact_reconstruction():
    say("assign codebook = vectors n=K=3000")
    V = rv(3000, 8, 10)
    p = np.random.default_rng(10).permutation(3000)
    got, gd = run_assign(V, V[p])
    np.testing.assert_array_equal(p[got], np.arange(3000))
    assert (gd == 0).all()


def test_assign_strided_slab():
    say("assign over a column slab of a 300x96 matrix, 40 columns")
    W = rv(300, 96, 11)
    Cb = rv(50, 8, 12)
    Wt = dev(W)
    codes = torch.empty(300 * 5, dtype=torch.int32, device="cuda")
    C.crvq_assign(VecSet.of_matrix(Wt, 8, 40), dev(Cb), codes)
    torch.cuda.synchronize()
    exp, _ = oracle.assign(oracle.vectors(np.ascontiguousarray(W[:, :40]), 8), Cb)
    np.testing.assert_array_equal(codes.cpu().numpy(), exp)


@pytest.mark.parametrize("n,K,dtype", [(20000, 256, "f32"), (3000, 4096, "f32"), (70000, 256, "f32"),
                                       (5000, 300, "bf16"), (0, 16, "f32")])
def test_kmeans_update_parity(n, K, dtype):
    say(f"kmeans update n={n} K={K} {dtype}")
    d = 8
    V = rv(max(n, 1), d, 13)[:n]
    g = np.random.default_rng(13)
    codes = g.integers(0, K, n).astype(np.int32)
    codes[codes % 7 == 3] = codes[codes % 7 == 3] // 2  # leave some clusters empty
    if n > 100:
        codes[:5] = [-1, K, K + 7, -100, 2 ** 30]  # out of range: belong to no cluster
    C0 = rv(K, d, 14)
    if dtype == "bf16":
        V = inputs.f32_to_bf16_bits(V)
        C0 = inputs.f32_to_bf16_bits(C0)
    Vt = dev(V, dtype) if n else torch.empty(0, d, dtype=torch.float32 if dtype == "f32" else torch.bfloat16,
                                            device="cuda")
    Ct = dev(C0, dtype)
    counts = torch.empty(K, dtype=torch.int32, device="cuda")
    C.crvq_kmeans_update(VecSet(Vt, n, 1, d, d), dev(codes), Ct, counts)
    torch.cuda.synchronize()
    valid = (codes >= 0) & (codes < K)
    Cexp, cnt, _ = oracle.kmeans_update(V[valid], codes[valid], C0, dtype, dtype)
    np.testing.assert_array_equal(counts.cpu().numpy(), cnt)
    got = to_host_bits(Ct)
    tol = 1e-5 if dtype == "f32" else 1e-2
    rel_close(oracle.widen(got, dtype), oracle.widen(Cexp, dtype), tol, "centroids", axis_vec=True)
    empty = cnt == 0
    np.testing.assert_array_equal(got[empty], C0[empty])  # empty clusters untouched, bitwise


@pytest.mark.parametrize("n,K,d,dtype,layout", [(3_000_017, 256, 8, "f32", "packed"), (200_001, 256, 8, "bf16", "packed"),
                                                 (50_000, 37, 5, "f32", "packed"), (40_000, 256, 8, "f32", "slab"),
                                                 (30_000, 200, 3, "bf16", "slab"), (100_000, 1, 8, "f32", "packed"),
                                                 (70_000, 256, 8, "f32", "skewed"), (63, 256, 8, "f32", "packed")])
def test_kmeans_update_small_k(n, K, d, dtype, layout):
    """K <= 256: per-wave tables over contiguous vector ranges (ragged tails, strided slabs, d < 8,
    one code shared by most vectors)."""
    say(f"kmeans update small K n={n} K={K} d={d} {dtype} {layout}")
    g = np.random.default_rng(17)
    if layout == "slab":  # the first `vpr` vectors of every row of a wider matrix
        vpr, width = 4, 11 * d
        rows = -(-n // vpr)
        Wm = rv(rows, width, 18)
        n = rows * vpr
        V = np.ascontiguousarray(Wm[:, :vpr * d]).reshape(n, d)
    else:
        V = rv(n, d, 18)
    codes = g.integers(0, K, n).astype(np.int32)
    if layout == "skewed":
        codes[g.random(n) < 0.9] = 7
    if n > 100:
        codes[3:8] = [-1, K, K + 7, -100, 2 ** 30]
    C0 = rv(K, d, 19)
    if dtype == "bf16":
        V = inputs.f32_to_bf16_bits(V)
        C0 = inputs.f32_to_bf16_bits(C0)
        if layout == "slab":
            Wm = inputs.f32_to_bf16_bits(Wm)
    if layout == "slab":
        Vs = VecSet(dev(Wm, dtype), rows, vpr, width, d)
    else:
        Vs = VecSet(dev(V, dtype), n, 1, d, d)
    Ct = dev(C0, dtype)
    counts = torch.empty(K, dtype=torch.int32, device="cuda")
    C.crvq_kmeans_update(Vs, dev(codes), Ct, counts)
    torch.cuda.synchronize()
    valid = (codes >= 0) & (codes < K)
    Cexp, cnt, _ = oracle.kmeans_update(V[valid], codes[valid], C0, dtype, dtype)
    np.testing.assert_array_equal(counts.cpu().numpy(), cnt)
    got = to_host_bits(Ct)
    tol = 1e-5 if dtype == "f32" else 1e-2
    rel_close(oracle.widen(got, dtype), oracle.widen(Cexp, dtype), tol, "centroids", axis_vec=True)
    np.testing.assert_array_equal(got[cnt == 0], C0[cnt == 0])


@pytest.mark.parametrize("M,N,dtype,n_ext,n_crit", [(37, 8200, "f32", 1, 200), (29, 13824, "bf16", 1, 344),
                                                     (300, 5120, "bf16", 2, 128), (1, 64, "f32", 0, 0),
                                                     (20, 4096, "f32", 3, 96), (16, 8192, "f32", 1, 2400),
                                                     (9, 2048, "bf16", 2, 2048)])
def test_dequant_reverse_reorder_rows(M, N, dtype, n_ext, n_crit):
    """Reconstruction in original channel order for rows of one or several LDS rounds, 0-3 extended
    books, critical groups beyond the first vector of a lane pair's round."""
    say(f"dequant reverse reorder M={M} N={N} {dtype} ext={n_ext} n_crit={n_crit}")
    d = 8
    ncv = n_crit // d
    g = np.random.default_rng(26)
    Cb = rv(65536, d, 27)
    Ce = [rv(256, d, 28 + e, 0.005) for e in range(n_ext)]
    if dtype == "bf16":
        Cb = inputs.f32_to_bf16_bits(Cb)
    qb = g.integers(0, 65536, (M, N // d)).astype(np.int32)
    qe = [g.integers(0, 256, (M, ncv)).astype(np.int32) for _ in range(n_ext)]
    perm = g.permutation(N).astype(np.int32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = torch.empty(M, N, dtype=tdt, device="cuda")
    C.crvq_dequant(M, N, d, dev(qb.ravel()), N // d, dev(Cb, dtype), out, n_crit=n_crit,
                   q_ext=[dev(q.ravel()) for q in qe], ldq_ext=max(ncv, 1), C_ext=[dev(c) for c in Ce],
                   perm=dev(perm))
    torch.cuda.synchronize()
    crit = opipe.crit_mask(M, N, d, n_crit)
    codes = [qb.ravel()]
    for q in qe:
        z = np.zeros((M, N // d), np.int32)
        z[:, :ncv] = q
        codes.append(z.ravel())
    R = oracle.reconstruct(codes, [Cb] + Ce, crit, [dtype] + ["f32"] * n_ext)
    Rs = oracle.round_to(R, dtype).reshape(M, N)
    np.testing.assert_array_equal(to_host_bits(out), oracle.scatter_columns(Rs, perm))


@pytest.mark.parametrize("M,N,dtype,n_ext,n_crit,K_ext", [(4100, 8192, "f32", 1, 168, 65536),
                                                           (3077, 8192, "f32", 2, 200, 256),
                                                           (2600, 13824, "bf16", 1, 696, 256)])
def test_dequant_reverse_reorder_many_rows(M, N, dtype, n_ext, n_crit, K_ext):
    """Reverse-reorder reconstruction of more rows than the kernel keeps resident workgroups (several
    rows per workgroup), compared in full: the 70B MLP width with a K = 65536 extended book, two
    extended books, and the 13B down-projection width in bf16."""
    say(f"dequant reverse reorder, many rows: M={M} N={N} {dtype} ext={n_ext}x{K_ext} n_crit={n_crit}")
    d = 8
    ncv = n_crit // d
    g = np.random.default_rng(61)
    Cb = rv(65536, d, 62)
    Ce = [rv(K_ext, d, 63 + e, 0.005) for e in range(n_ext)]
    if dtype == "bf16":
        Cb = inputs.f32_to_bf16_bits(Cb)
    qb = g.integers(0, 65536, (M, N // d)).astype(np.int32)
    qe = [g.integers(0, K_ext, (M, ncv)).astype(np.int32) for _ in range(n_ext)]
    perm = g.permutation(N).astype(np.int32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = torch.empty(M, N, dtype=tdt, device="cuda")
    C.crvq_dequant(M, N, d, dev(qb.ravel()), N // d, dev(Cb, dtype), out, n_crit=n_crit,
                   q_ext=[dev(q.ravel()) for q in qe], ldq_ext=ncv, C_ext=[dev(c) for c in Ce], perm=dev(perm))
    torch.cuda.synchronize()
    crit = opipe.crit_mask(M, N, d, n_crit)
    codes = [qb.ravel()]
    for q in qe:
        z = np.zeros((M, N // d), np.int32)
        z[:, :ncv] = q
        codes.append(z.ravel())
    R = oracle.reconstruct(codes, [Cb] + Ce, crit, [dtype] + ["f32"] * n_ext)
    Rs = oracle.round_to(R, dtype).reshape(M, N)
    np.testing.assert_array_equal(to_host_bits(out), oracle.scatter_columns(Rs, perm))


def test_assign_rows_with_nan_elements():
    """Inputs must be finite; a row holding a NaN still gets an in-range code (0) and a NaN distance,
    and every other row the oracle's result, on each search variant (small book, generic screen,
    long-book two-screen path)."""
    for n, K in [(5000, 256), (3000, 1000), (70000, 65536)]:
        say(f"assign with NaN rows n={n} K={K}")
        V = rv(n, 8, 71)
        Cb = rv(K, 8, 72)
        bad = np.array([0, 17, n // 2, n - 1])
        V[bad, 3] = np.nan
        got, gd = run_assign(V, Cb)
        assert (got[bad] == 0).all() and np.isnan(gd[bad]).all()
        ok = np.setdiff1d(np.arange(n), bad)
        exp, ed = oracle.assign(V[ok], Cb)
        np.testing.assert_array_equal(got[ok], exp)
        np.testing.assert_array_equal(gd[ok], ed.astype(np.float32))


@pytest.mark.parametrize("M,N,dtype,mode", [(513, 300, "f32", "sum"), (64, 1000, "f32", "max"),
                                            (1000, 96, "bf16", "sum"), (200, 77, "f32", "maxB"),
                                            (4096, 4096, "f32", "sum")])
def test_importance_parity(M, N, dtype, mode):
    say(f"importance M={M} N={N} {dtype} {mode}")
    A = rv(M, N, 15, 1.0)
    B = rv(M, N, 16, 1.0) if mode == "maxB" else None
    s = np.abs(rv(1, N, 17, 1.0)[0]) + 0.1
    if dtype == "bf16":
        A = inputs.f32_to_bf16_bits(A)
    out = torch.empty(N, dtype=torch.float32, device="cuda")
    C.crvq_channel_importance(dev(A, dtype), out, None if B is None else dev(B), dev(s),
                              C.CRVQ_REDUCE_SUM if mode == "sum" else C.CRVQ_REDUCE_MAX)
    torch.cuda.synchronize()
    exp = oracle.colreduce(A, B, s.astype(np.float64), "sum" if mode == "sum" else "max", dtype)
    got = out.cpu().numpy()
    if mode == "sum":
        rel_close(got, exp, 1e-6, "importance")
    else:
        np.testing.assert_array_equal(got, exp.astype(np.float32))  # max is exact


@pytest.mark.parametrize("N,M,dtype", [(300, 17, "f32"), (4096, 64, "bf16"), (20000, 3, "f32")])
def test_reorder_parity(N, M, dtype):
    say(f"reorder N={N} M={M} {dtype}")
    g = np.random.default_rng(18)
    I = g.integers(0, 50, N).astype(np.float32)  # many ties
    I[g.integers(0, N, 5)] = np.nan
    I[g.integers(0, N, 5)] = -0.0
    W = rv(M, N, 19, 1.0)
    if dtype == "bf16":
        W = inputs.f32_to_bf16_bits(W)
    Wt = dev(W, dtype)
    out = torch.empty_like(Wt)
    perm = torch.empty(N, dtype=torch.int32, device="cuda")
    C.crvq_reorder(Wt, out, perm, importance=dev(I))
    back = torch.empty_like(Wt)
    C.crvq_reorder(out, back, perm, inverse=True)
    torch.cuda.synchronize()
    pexp = oracle.rank_perm(I)
    np.testing.assert_array_equal(perm.cpu().numpy(), pexp)
    np.testing.assert_array_equal(to_host_bits(out), oracle.gather_columns(W, pexp))
    np.testing.assert_array_equal(to_host_bits(back), W)


def test_gather_vectors():
    say("gather vectors")
    W = rv(40, 64, 20)
    idx = np.array([0, 5, 319, 100, 7, 7], np.int64)
    out = torch.empty(6, 8, dtype=torch.float32, device="cuda")
    C.crvq_gather_vectors(VecSet.of_matrix(dev(W), 8), dev(idx), out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), oracle.vectors(W, 8)[idx])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dequant_parity(dtype):
    say(f"dequant {dtype}")
    M, N, d, n_crit = 100, 96, 8, 24
    ncv = n_crit // d
    g = np.random.default_rng(21)
    Cb = rv(64, d, 22)
    Ce = [rv(16, d, 23, 0.005), rv(8, d, 24, 0.001)]
    if dtype == "bf16":
        Cb = inputs.f32_to_bf16_bits(Cb)
    qb = g.integers(0, 64, (M, N // d)).astype(np.int32)
    qe = [g.integers(0, 16, (M, ncv)).astype(np.int32), g.integers(0, 8, (M, ncv)).astype(np.int32)]
    perm = g.permutation(N).astype(np.int32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = torch.empty(M, N, dtype=tdt, device="cuda")
    C.crvq_dequant(M, N, d, dev(qb.ravel()), N // d, dev(Cb, dtype), out, n_crit=n_crit,
                   q_ext=[dev(q.ravel()) for q in qe], ldq_ext=ncv, C_ext=[dev(c) for c in Ce], perm=dev(perm))
    plain = torch.empty(M, N, dtype=tdt, device="cuda")
    C.crvq_dequant(M, N, d, dev(qb.ravel()), N // d, dev(Cb, dtype), plain, n_crit=n_crit,
                   q_ext=[dev(q.ravel()) for q in qe], ldq_ext=ncv, C_ext=[dev(c) for c in Ce])
    # residual mode on the critical slab: E = W[:, :n_crit] - basic codewords
    W = rv(M, N, 25)
    if dtype == "bf16":
        W = inputs.f32_to_bf16_bits(W)
    E = torch.empty(M, n_crit, dtype=torch.float32, device="cuda")
    C.crvq_dequant(M, n_crit, d, dev(qb.ravel()), N // d, dev(Cb, dtype), E, minuend=dev(W, dtype))
    torch.cuda.synchronize()
    crit = opipe.crit_mask(M, N, d, n_crit)
    full_codes = [qb.ravel()]
    for q in qe:
        z = np.zeros((M, N // d), np.int32)
        z[:, :ncv] = q
        full_codes.append(z.ravel())
    R = oracle.reconstruct(full_codes, [Cb] + Ce, crit, [dtype, "f32", "f32"])
    Rs = oracle.round_to(R, dtype).reshape(M, N)
    np.testing.assert_array_equal(to_host_bits(plain), Rs)
    np.testing.assert_array_equal(to_host_bits(out), oracle.scatter_columns(Rs, perm))
    Wv = oracle.vectors(np.ascontiguousarray(W[:, :n_crit]), d)
    Eexp = oracle.residual(Wv, qb[:, :ncv].ravel(), Cb, dtype, dtype).reshape(M, n_crit)
    np.testing.assert_array_equal(E.cpu().numpy(), Eexp)


@pytest.mark.parametrize("beam,Ks,n", [(1, (256, 16, 16), 3000), (2, (64, 16), 2000), (4, (256, 256), 4000),
                                       (8, (256, 256, 256), 2500), (4, (3, 2, 16), 500), (4, (4096, 64), 3000),
                                       (16, (32, 32), 300)])
def test_beam_parity(beam, Ks, n):
    say(f"beam B={beam} Ks={Ks} n={n}")
    d = 8
    V = rv(n, d, 26)
    books = [rv(K, d, 27 + t, 0.02 / (4 ** t)) for t, K in enumerate(Ks)]
    check_beam(V, books, beam)


@pytest.mark.parametrize("beam", [2, 4, 8])
def test_beam_ties(beam):
    """Small-integer vectors against books with every codeword twice: children of different parents
    tie on their error all the time, so the merge's (error, parent rank, codeword) order decides which
    tuples survive each step."""
    say(f"beam ties B={beam} n=3001")
    g = np.random.default_rng(40 + beam)
    n, d = 3001, 8
    V = g.integers(-3, 4, (n, d)).astype(np.float32)
    books = []
    for K, lo in ((64, -3), (16, -1), (16, -1)):
        b = g.integers(lo, -lo + 1, (K, d)).astype(np.float32)
        b[K // 2:] = b[:K // 2]
        books.append(b)
    check_beam(V, books, beam)


@pytest.mark.parametrize("beam", [2, 4, 8])
def test_beam_long_codebook(beam):
    """A first book of 65536 codewords drawn next to the rows (near-ties, as K-means leaves them) over
    30001 rows: the top-B screen tracks chunks of tiles on its long tile ranges, and the finalize
    re-scores whole kept chunks."""
    say(f"beam long codebook B={beam} K=(65536, 64) n=30001")
    g = np.random.default_rng(50 + beam)
    n, d = 30001, 8
    V = rv(n, d, 51)
    b0 = V[g.choice(n, 65536, replace=True)] + (g.standard_normal((65536, d)) * 0.0005).astype(np.float32)
    books = [b0.astype(np.float32), rv(64, d, 52, 0.005)]
    check_beam(V, books, beam)


def check_beam(V, books, beam):
    n = V.shape[0]
    Ks = [b.shape[0] for b in books]
    codes = [torch.empty(n, dtype=torch.int32, device="cuda") for _ in Ks]
    err = torch.empty(n, dtype=torch.float32, device="cuda")
    C.crvq_assign_residual_beam(VecSet.of_vectors(dev(V)), [dev(b) for b in books], beam, codes, err)
    torch.cuda.synchronize()
    exp_codes, exp_err = oracle.beam(V, books, beam)
    got = np.stack([c.cpu().numpy() for c in codes])
    bad = np.flatnonzero((got != exp_codes).any(0))
    if len(bad):  # only tuples whose error ties the oracle's within 1e-6 relative are acceptable
        R = oracle.reconstruct([g for g in got[:, bad]], books, np.ones(len(bad), np.uint8))
        e_got = ((V[bad].astype(np.float64) - R) ** 2).sum(1)
        assert (e_got <= exp_err[bad] * (1 + 1e-6)).all(), f"{len(bad)} tuples differ beyond ties"
    assert len(bad) == 0, f"{len(bad)} tie substitutions (exact parity expected)"
    np.testing.assert_array_equal(err.cpu().numpy(), exp_err.astype(np.float32))


def test_determinism():
    say("determinism: two identical assign + update + beam runs are bitwise equal")
    V = rv(30000, 8, 30)
    outs = []
    for _ in range(2):
        Vt = dev(V)
        Cb = dev(V[:2048].copy())
        q = torch.empty(30000, dtype=torch.int32, device="cuda")
        C.crvq_assign(VecSet.of_vectors(Vt), Cb, q)
        C.crvq_kmeans_update(VecSet.of_vectors(Vt), q, Cb)
        codes = [torch.empty(30000, dtype=torch.int32, device="cuda") for _ in range(2)]
        C.crvq_assign_residual_beam(VecSet.of_vectors(Vt), [Cb, dev(rv(64, 8, 31, 0.005))], 4, codes)
        torch.cuda.synchronize()
        outs.append([q.cpu().numpy(), Cb.cpu().numpy(), codes[0].cpu().numpy(), codes[1].cpu().numpy()])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)
