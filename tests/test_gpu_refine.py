"""GPU parity of the loss-driven refinement calls (Alg. 1 QuantLoss / FineTuneCodebook /
BeamSearchOptimize at width 1) against the oracle in oracle/refine.py.

Tolerances: H, G, the row losses and the per-code sums are fp64 sums of exact products in an order
the oracle does not share, so each entry is compared within 1e-12 of the sum of the absolute values
of its terms.  The residual, the code search (same fp64 decisions on the same inputs) and Adam (the
same rounded operations) are compared bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from oracle import refine as orf
from oracle import pipeline as opipe
from paper_2412_09282_amd import crvq as C
from paper_2412_09282_amd import inputs
from paper_2412_09282_amd.pipeline import LayerConfig, LayerQuantizer

from gpu_util import dev, say

pytestmark = pytest.mark.gpu

TOL = 1e-12


def rv(shape, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(shape) * scale).astype(np.float32)


def host(t):
    return t.detach().cpu().numpy()


@pytest.mark.parametrize("T,N", [(300, 200), (64, 1), (2048, 512), (5, 130)])
def test_gram(T, N):
    say(f"gram {T}x{N}")
    X = rv((T, N), T + N)
    H = torch.empty(N, N, dtype=torch.float64, device="cuda")
    C.crvq_gram(dev(X), H)
    torch.cuda.synchronize()
    X64 = X.astype(np.float64)
    exp = X64.T @ X64
    scale = np.abs(X64).T @ np.abs(X64)
    assert (np.abs(host(H) - exp) <= TOL * scale + 1e-300).all()


@pytest.mark.parametrize("M,N,n_out", [(37, 200, 200), (130, 256, 64), (1, 8, 8), (300, 1000, 1000)])
def test_hessian_product(M, N, n_out):
    say(f"hessian product {M}x{N} -> {n_out}")
    g = np.random.default_rng(M + N)
    R = g.standard_normal((M, N)) * 0.01
    X = g.standard_normal((N + 7, N))
    H = X.T @ X
    Gt = torch.empty(M, n_out, dtype=torch.float64, device="cuda")
    loss = torch.empty(M, dtype=torch.float64, device="cuda") if n_out == N else None
    total = torch.empty(1, dtype=torch.float64, device="cuda") if n_out == N else None
    C.crvq_hessian_product(torch.from_numpy(R).cuda(), torch.from_numpy(H).cuda(), Gt, loss, total)
    torch.cuda.synchronize()
    exp = R @ H[:, :n_out]
    assert (np.abs(host(Gt) - exp) <= TOL * (np.abs(R) @ np.abs(H[:, :n_out])) + 1e-300).all()
    if loss is not None:
        el = np.sum(R * exp, axis=1)
        terms = np.sum(np.abs(R) * (np.abs(R) @ np.abs(H)), axis=1)
        assert (np.abs(host(loss) - el) <= TOL * terms).all()
        assert abs(float(host(total)[0]) - el.sum()) <= TOL * terms.sum()


@pytest.mark.parametrize("M,N,d,cover,K", [(64, 256, 8, 256, 256), (300, 512, 8, 40, 1000), (17, 64, 16, 64, 7),
                                           (5, 24, 3, 24, 1), (1000, 1024, 8, 1024, 256),
                                           # books past 1024 codewords: grouped by a radix pass first
                                           (300, 512, 8, 512, 4096), (40, 96, 16, 96, 1025), (7, 30, 3, 30, 2000),
                                           (2048, 4096, 8, 4096, 65536)])
def test_code_sums(M, N, d, cover, K):
    say(f"code sums {M}x{N} d={d} cover={cover} K={K}")
    g = np.random.default_rng(M * 3 + K)
    G = g.standard_normal((M, N))
    n = M * (cover // d)
    codes = g.integers(0, K, n).astype(np.int32)
    codes[::97] = -1            # outside the book: counted nowhere
    sums = torch.empty(K, d, dtype=torch.float64, device="cuda")
    counts = torch.empty(K, dtype=torch.int32, device="cuda")
    Gt = torch.from_numpy(G).cuda()
    C.crvq_code_sums(C.VecSet.of_matrix(Gt, d, cover), dev(codes), K, sums, counts)
    torch.cuda.synchronize()
    V = G[:, :cover].reshape(-1, d)
    ok = codes >= 0
    exp = np.zeros((K, d))
    np.add.at(exp, codes[ok], V[ok])
    absn = np.zeros((K, d))
    np.add.at(absn, codes[ok], np.abs(V[ok]))
    assert (np.abs(host(sums) - exp) <= TOL * absn + 1e-300).all()
    np.testing.assert_array_equal(host(counts), np.bincount(codes[ok], minlength=K))


def test_adam_steps_bitwise():
    say("adam 3 steps")
    K, d = 300, 8
    Cb = rv((K, d), 1, 0.05)
    Ct = dev(Cb.copy())
    m = torch.zeros(K, d, dtype=torch.float64, device="cuda")
    v = torch.zeros(K, d, dtype=torch.float64, device="cuda")
    st = orf.AdamState(np.zeros((K, d)), np.zeros((K, d)))
    Co = Cb.copy()
    for t in range(1, 4):
        grad = np.random.default_rng(t).standard_normal((K, d)) * 10.0
        grad[0] = 0.0
        C.crvq_adam_step(Ct, torch.from_numpy(grad).cuda(), -2.0, m, v, t, 1e-3)
        Co = orf.adam_step(Co, -2.0 * grad, st, 1e-3)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(Ct), Co)
        np.testing.assert_array_equal(host(m), st.m)
        np.testing.assert_array_equal(host(v), st.v)


def refine_case(M, N, d, K, n_cols, c_dtype, seed):
    g = np.random.default_rng(seed)
    W = rv((M, N), seed, 0.02)
    X = rv((2 * N + 3, N), seed + 1)
    Cb = rv((K, d), seed + 2, 0.02)
    if c_dtype == "bf16":
        Cb = inputs.f32_to_bf16_bits(Cb)
    codes = g.integers(0, K, M * (n_cols // d)).astype(np.int32)
    H = orf.gram(X)
    # residual of W against this one book on its columns (the rest of R as W itself)
    R = W.astype(np.float64)
    Cw = oracle.widen(Cb, c_dtype).astype(np.float64)
    R[:, :n_cols] -= Cw[codes].reshape(M, n_cols)
    return R, H, Cb, codes


@pytest.mark.parametrize("M,N,d,K,n_cols,c_dtype", [(37, 256, 8, 64, 256, "f32"), (64, 256, 8, 256, 32, "f32"),
                                                   (20, 128, 16, 50, 128, "f32"), (33, 96, 8, 16, 96, "bf16"),
                                                   (9, 64, 4, 1024, 64, "f32"),
                                                   # few output tiles, long k: S = R H[:, :n_cols] split over k
                                                   # into parts (ragged last part, M and n_cols not multiples
                                                   # of the 128 x 128 tile)
                                                   (300, 2056, 8, 256, 64, "f32"), (130, 2049, 1, 64, 48, "f32"),
                                                   # books too large for one CU's LDS: searched one group at a
                                                   # time over all rows, in codebook slices
                                                   (40, 256, 8, 4096, 256, "f32"), (65, 128, 8, 65536, 64, "f32"),
                                                   (33, 96, 8, 2048, 96, "bf16"), (9, 64, 16, 600, 64, "f32"),
                                                   (130, 512, 8, 1100, 200, "f32")])
def test_refine_codes(M, N, d, K, n_cols, c_dtype):
    say(f"refine codes {M}x{N} d={d} K={K} cols={n_cols} {c_dtype}")
    R, H, Cb, codes = refine_case(M, N, d, K, n_cols, c_dtype, M + K)
    Rt = torch.from_numpy(R.copy()).cuda()
    qt = dev(codes.copy())
    C.crvq_refine_codes(Rt, torch.from_numpy(H).cuda(), dev(Cb, c_dtype), qt, d, n_cols, n_cols // d)
    torch.cuda.synchronize()
    Ro, qo = R.copy(), codes.copy()
    changes = orf.refine_book(Ro, H, Cb, qo, d, n_cols, c_dtype)
    got = host(qt)
    np.testing.assert_array_equal(got, qo)
    np.testing.assert_array_equal(host(Rt), Ro)
    assert changes > 0
    say(f"refine codes: {changes} of {len(codes)} codes moved, identical to the oracle")


def test_refine_codes_sampled_rows_full_size():
    """The code search on a 4096 x 4096 layer with a K = 256 book: rows are independent given H and
    the book, so sampled rows are re-run on the oracle from the same inputs."""
    M, N, d, K = 4096, 4096, 8, 256
    say(f"refine codes full size {M}x{N} K={K}")
    g = np.random.default_rng(7)
    W = rv((M, N), 8, 0.02)
    X = rv((2048, N), 9)
    Cb = rv((K, d), 10, 0.02)
    codes = g.integers(0, K, M * N // d).astype(np.int32)
    Xt = dev(X)
    Ht = torch.empty(N, N, dtype=torch.float64, device="cuda")
    C.crvq_gram(Xt, Ht)
    R = W.astype(np.float64) - Cb.astype(np.float64)[codes].reshape(M, N)
    Rt = torch.from_numpy(R).cuda()
    qt = dev(codes.copy())
    C.crvq_refine_codes(Rt, Ht, dev(Cb), qt, d, N, N // d)
    torch.cuda.synchronize()
    H = host(Ht)
    rows = np.sort(g.choice(M, 6, replace=False))
    Ro = R[rows].copy()
    qo = codes.reshape(M, -1)[rows].copy().ravel()
    orf.refine_book(Ro, H, Cb, qo, d, N)
    np.testing.assert_array_equal(host(qt).reshape(M, -1)[rows].ravel(), qo)
    np.testing.assert_array_equal(host(Rt)[rows], Ro)


def test_refine_codes_sampled_rows_full_size_k65536():
    """The code search on a 4096 x 4096 layer against a K = 65536 book (searched in slices, one group
    at a time): sampled rows re-run on the oracle from the same inputs."""
    M, N, d, K = 4096, 4096, 8, 65536
    say(f"refine codes full size {M}x{N} K={K}")
    g = np.random.default_rng(17)
    W = rv((M, N), 18, 0.02)
    X = rv((2048, N), 19)
    Cb = rv((K, d), 20, 0.02)
    codes = g.integers(0, K, M * N // d).astype(np.int32)
    Xt = dev(X)
    Ht = torch.empty(N, N, dtype=torch.float64, device="cuda")
    C.crvq_gram(Xt, Ht)
    R = W.astype(np.float64) - Cb.astype(np.float64)[codes].reshape(M, N)
    Rt = torch.from_numpy(R).cuda()
    qt = dev(codes.copy())
    C.crvq_refine_codes(Rt, Ht, dev(Cb), qt, d, N, N // d)
    torch.cuda.synchronize()
    H = host(Ht)
    rows = np.sort(g.choice(M, 3, replace=False))
    Ro = R[rows].copy()
    qo = codes.reshape(M, -1)[rows].copy().ravel()
    moved = orf.refine_book(Ro, H, Cb, qo, d, N)
    np.testing.assert_array_equal(host(qt).reshape(M, -1)[rows].ravel(), qo)
    np.testing.assert_array_equal(host(Rt)[rows], Ro)
    say(f"refine codes K={K}: sampled rows identical ({moved} codes moved in them)")


def test_refine_loop_lockstep():
    """The whole refinement loop after a layer pass: every call re-run on the oracle from the GPU's
    inputs, then the loss trajectory and codes against the oracle's own loop from the same start."""
    M, N, d = 96, 256, 8
    wl = inputs.small_workload(M=M, N=N, tokens=128, d=d, K_base=64, K_ext=(16,), crit_frac=0.1, beam=1, iters=2,
                               dtype="f32", wid=140)
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    n = M * N // d
    n_crit = inputs.n_crit_columns(N, d, wl.crit_frac)
    base_idx = inputs.base_init_indices(wl, 0, n)
    ext_idx = [inputs.ext_init_indices(wl, 0, 1, M * n_crit // d)]
    cfg = LayerConfig(d, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters)
    q = LayerQuantizer(M, N, torch.float32, cfg, tokens=128, device="cuda")
    Xt = torch.from_numpy(X).cuda()
    st = q.run(dev(W), Xt, torch.from_numpy(base_idx).cuda(), [torch.from_numpy(e).cuda() for e in ext_idx])
    torch.cuda.synchronize()
    start_books = [host(b).copy() for b in q.C_basic + q.C_ext]
    start_codes = [host(c).copy() for c in q.codes_basic + q.codes_ext]
    perm = host(st.perm)
    Ws = host(st.Ws)
    trace = []
    losses = q.refine(Xt, rounds=2, steps=3, lr=1e-4, trace=trace)
    torch.cuda.synchronize()
    H = None
    for c in trace:
        name, ci, co = c["name"], c["in"], c["out"]
        if name == "gram":
            Xs = oracle.gather_columns(X, perm)
            np.testing.assert_array_equal(co["Xs"].numpy(), Xs)
            H = co["H"].numpy()
            exp = orf.gram(Xs)
            assert (np.abs(H - exp) <= TOL * (np.abs(Xs).T.astype(np.float64) @ np.abs(Xs)) + 1e-300).all()
        elif name.startswith("residual"):
            books = [b.numpy() for b in ci["books"]]
            codes = [x.numpy() for x in ci["codes"]]
            exp = orf.residual_f64(Ws, "f32", d, n_crit, codes, books, ["f32"] * len(books), 1)
            np.testing.assert_array_equal(co["out"].numpy(), exp)
        elif name.startswith("hessian"):
            R = ci["R"].numpy()
            G = co["G"].numpy()
            assert (np.abs(G - R @ H) <= TOL * (np.abs(R) @ np.abs(H)) + 1e-300).all()
            terms = np.sum(np.abs(R) * (np.abs(R) @ np.abs(H)))
            assert abs(float(co["loss_total"].numpy()[0]) - np.sum(R * (R @ H))) <= TOL * terms
        elif name.startswith("refine"):
            Ro = ci["R"].numpy().copy()
            qo = ci["codes"].numpy().copy()
            orf.refine_book(Ro, H, ci["C"].numpy(), qo, d, ci["n_cols"])
            np.testing.assert_array_equal(co["codes"].numpy(), qo)
            np.testing.assert_array_equal(co["R"].numpy(), Ro)
        elif name.startswith("adam"):
            grad = ci["grad"].numpy()
            stt = orf.AdamState(ci["m"].numpy().copy(), ci["v"].numpy().copy(), ci["step"] - 1)
            Cn = orf.adam_step(ci["C"].numpy(), -2.0 * grad, stt, 1e-4)
            np.testing.assert_array_equal(co["C"].numpy(), Cn)
    ref = orf.refine_layer(Ws, oracle.gather_columns(X, perm), d, n_crit, start_books, start_codes, 1, lr=1e-4,
                           steps=3, max_rounds=2)
    np.testing.assert_allclose(losses, ref.losses, rtol=1e-9)
    assert losses[-1] < losses[0]
    for a, b in zip(q.codes_basic + q.codes_ext, ref.codes):
        np.testing.assert_array_equal(host(a), b)
    Wh = host(st.W_hat)
    assert orf.quant_loss(W, Wh, X) == pytest.approx(losses[-1], rel=1e-5)
    say(f"refine loop: QuantLoss {losses[0]:.6e} -> {losses[-1]:.6e} over {len(losses) - 1} rounds, "
        f"{len(trace)} calls matched")


def test_refine_two_basic_books_d16():
    """The refinement loop on the m = 2, d = 16 layout (two basic books on every vector) against the
    oracle's loop from the same start."""
    M, N, d = 64, 256, 16
    wl = inputs.small_workload(M=M, N=N, tokens=96, d=d, K_base=32, K_ext=(16,), crit_frac=0.1, beam=2, iters=2,
                               dtype="f32", wid=141, m_base=2)
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    n = M * N // d
    n_crit = inputs.n_crit_columns(N, d, wl.crit_frac)
    cfg = LayerConfig(d, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters, m_base=2)
    q = LayerQuantizer(M, N, torch.float32, cfg, tokens=96, device="cuda")
    Xt = torch.from_numpy(X).cuda()
    st = q.run(dev(W), Xt, torch.from_numpy(inputs.base_init_indices(wl, 0, n)).cuda(),
               [torch.from_numpy(inputs.ext_init_indices(wl, 0, 1, M * n_crit // d)).cuda()],
               base_idx_extra=[torch.from_numpy(inputs.extra_base_init_indices(wl, 0, 1, n)).cuda()])
    torch.cuda.synchronize()
    books = [host(b).copy() for b in q.C_basic + q.C_ext]
    codes = [host(c).copy() for c in q.codes_basic + q.codes_ext]
    perm = host(st.perm)
    losses = q.refine(Xt, rounds=2, steps=2, lr=1e-4)
    torch.cuda.synchronize()
    ref = orf.refine_layer(host(st.Ws), oracle.gather_columns(X, perm), d, n_crit, books, codes, 2, lr=1e-4, steps=2,
                           max_rounds=2)
    np.testing.assert_allclose(losses, ref.losses, rtol=1e-9)
    for a, b in zip(q.codes_basic + q.codes_ext, ref.codes):
        np.testing.assert_array_equal(host(a), b)
    assert losses[-1] < losses[0]
    say(f"refine m=2 d=16: QuantLoss {losses[0]:.6e} -> {losses[-1]:.6e}, codes identical to the oracle")


def tbits(t):
    """A trace tensor (CPU) as numpy; bf16 as uint16 bit patterns."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def test_refine_loop_lockstep_bf16():
    """The refinement loop on a bf16 layer: the first basic book is bf16 and tuned through an fp32
    master (set from the book at step 1, re-rounded after every step); every call re-run on the oracle
    from the GPU's inputs, then the whole loop against the oracle's from the same start."""
    M, N, d = 64, 128, 8
    wl = inputs.small_workload(M=M, N=N, tokens=96, d=d, K_base=32, K_ext=(8,), crit_frac=0.25, beam=1, iters=1,
                               dtype="bf16", wid=142)
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    n_crit = inputs.n_crit_columns(N, d, wl.crit_frac)
    cfg = LayerConfig(d, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters)
    q = LayerQuantizer(M, N, torch.bfloat16, cfg, tokens=96, device="cuda")
    Xt = torch.from_numpy(X).cuda()
    st = q.run(dev(W, "bf16"), Xt, torch.from_numpy(inputs.base_init_indices(wl, 0, M * N // d)).cuda(),
               [torch.from_numpy(inputs.ext_init_indices(wl, 0, 1, M * n_crit // d)).cuda()])
    torch.cuda.synchronize()
    books_gpu = q.C_basic + q.C_ext
    start_books = [tbits(b.cpu()).copy() for b in books_gpu]
    start_codes = [host(c).copy() for c in q.codes_basic + q.codes_ext]
    perm = host(st.perm)
    Ws = tbits(st.Ws.cpu())
    lr = 2e-3
    trace = []
    losses = q.refine(Xt, rounds=2, steps=3, lr=lr, trace=trace)
    torch.cuda.synchronize()
    H = None
    dts = ["bf16", "f32"]
    n_adam_bf16 = 0
    for c in trace:
        name, ci, co = c["name"], c["in"], c["out"]
        if name == "gram":
            H = co["H"].numpy()
        elif name.startswith("residual"):
            books = [tbits(b) for b in ci["books"]]
            codes = [x.numpy() for x in ci["codes"]]
            exp = orf.residual_f64(Ws, "bf16", d, n_crit, codes, books, dts, 1)
            np.testing.assert_array_equal(co["out"].numpy(), exp)
        elif name.startswith("refine"):
            Ro = ci["R"].numpy().copy()
            qo = ci["codes"].numpy().copy()
            b = int(name.rsplit("_", 1)[1])
            orf.refine_book(Ro, H, tbits(ci["C"]), qo, d, ci["n_cols"], dts[b])
            np.testing.assert_array_equal(co["codes"].numpy(), qo)
            np.testing.assert_array_equal(co["R"].numpy(), Ro)
        elif name.startswith("adam"):
            grad = ci["grad"].numpy()
            stt = orf.AdamState(ci["m"].numpy().copy(), ci["v"].numpy().copy(), ci["step"] - 1)
            if "master" in ci:
                n_adam_bf16 += 1
                m_in = oracle.widen(tbits(ci["C"]), "bf16").astype(np.float32) if ci["step"] == 1 else ci["master"].numpy()
                m_out = orf.adam_step(m_in, -2.0 * grad, stt, lr)
                np.testing.assert_array_equal(co["master"].numpy(), m_out)
                np.testing.assert_array_equal(tbits(co["C"]), oracle.round_to(m_out.astype(np.float64), "bf16"))
            else:
                np.testing.assert_array_equal(co["C"].numpy(), orf.adam_step(ci["C"].numpy(), -2.0 * grad, stt, lr))
    assert n_adam_bf16 == 6
    ref = orf.refine_layer(Ws, oracle.gather_columns(X, perm), d, n_crit, start_books, start_codes, 1, lr=lr,
                           steps=3, max_rounds=2, w_dtype="bf16")
    np.testing.assert_allclose(losses, ref.losses, rtol=1e-9)
    assert losses[-1] < losses[0]
    for a, b in zip(q.codes_basic + q.codes_ext, ref.codes):
        np.testing.assert_array_equal(host(a), b)
    np.testing.assert_array_equal(tbits(q.C_basic[0].cpu()), ref.books[0])
    assert (tbits(q.C_basic[0].cpu()) != start_books[0]).any()  # the bf16 book did move
    say(f"refine loop bf16: QuantLoss {losses[0]:.6e} -> {losses[-1]:.6e}, {len(trace)} calls matched")
