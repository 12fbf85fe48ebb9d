"""GPU parity of the codebook-layout variants of Sec. 3.2 / Sec. 6.4: several basic codebooks (the
m = 2, d = 16 setting, through crvq_dequant_books and the layer pipeline), d = 16 vectors, and wider
basic books (e = 10 and 12, i.e. K = 1024 and 4096).

Every call the pipeline makes is re-run on the oracle from the GPU's own inputs (lockstep): codes
must match up to exact ties, centroids to 1e-5 (fp32) / one bf16 step, residuals and reconstructions
bit for bit.  Then the whole layer is compared with the oracle's pipeline from the same seeds."""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline as opipe
from paper_2412_09282_amd import crvq as C
from paper_2412_09282_amd import inputs
from paper_2412_09282_amd.pipeline import LayerConfig, LayerQuantizer

from gpu_util import check_codes, dev, rel_close, say, to_host_bits

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------------------------------------
# crvq_dequant_books
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("M,N,d,n_base,n_ext,n_crit,dtype,mode", [
    (37, 128, 16, 2, 0, 0, "f32", "perm"),
    (37, 128, 16, 2, 3, 32, "f32", "perm"),
    (64, 256, 16, 2, 1, 16, "bf16", "perm"),
    (20, 64, 8, 2, 2, 16, "f32", "plain"),
    (20, 64, 8, 3, 1, 8, "bf16", "minuend"),
    (300, 4096, 16, 2, 3, 96, "f32", "perm"),
    (5, 40, 4, 2, 0, 0, "f32", "plain"),
])
def test_dequant_books(M, N, d, n_base, n_ext, n_crit, dtype, mode):
    say(f"dequant_books {M}x{N} d={d} basic={n_base} ext={n_ext} n_crit={n_crit} {dtype} {mode}")
    g = np.random.default_rng(M * 7 + N + n_base)
    K_b, K_e = 256, 64
    books = [inputs.random_vectors(K_b, d, 40 + b, 0.02) for b in range(n_base)] + \
            [inputs.random_vectors(K_e, d, 50 + e, 0.005) for e in range(n_ext)]
    bdt = [dtype] + ["f32"] * (len(books) - 1)
    if dtype == "bf16":
        books[0] = inputs.f32_to_bf16_bits(books[0])
    vpr, ncv = N // d, n_crit // d
    qb = [g.integers(0, K_b, M * vpr).astype(np.int32) for _ in range(n_base)]
    qe = [g.integers(0, K_e, max(1, M * ncv)).astype(np.int32) for _ in range(n_ext)]
    perm = g.permutation(N).astype(np.int32)
    minuend = inputs.random_vectors(M, N, 60, 0.02)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.empty(M, N, dtype=tdt, device="cuda")
    C.crvq_dequant_books(M, N, d, [dev(q) for q in qb], vpr, [dev(b, t) for b, t in zip(books[:n_base], bdt)], out,
                         n_crit=n_crit, q_ext=[dev(q) for q in qe], ldq_ext=max(1, ncv),
                         C_ext=[dev(b) for b in books[n_base:]], perm=dev(perm) if mode == "perm" else None,
                         minuend=dev(minuend) if mode == "minuend" else None)
    torch.cuda.synchronize()
    got = to_host_bits(out)
    # oracle: every book's codes laid out per vector, extended ones on the critical groups only
    full = list(qb)
    for q in qe:
        z = np.zeros((M, vpr), np.int32)
        z[:, :ncv] = q[:M * ncv].reshape(M, ncv)
        full.append(z.ravel())
    R = oracle.reconstruct(full, books, opipe.crit_mask(M, N, d, n_crit), bdt, n_full=n_base)
    if mode == "minuend":
        exp = oracle.round_to(oracle.vectors(minuend, d).astype(np.float64) - R, dtype).reshape(M, N)
    else:
        Rs = oracle.round_to(R, dtype).reshape(M, N)
        exp = oracle.scatter_columns(Rs, perm) if mode == "perm" else Rs
    np.testing.assert_array_equal(got, exp)


# ------------------------------------------------------------------------------------------------
# the layer pipeline with the variants
# ------------------------------------------------------------------------------------------------
def lockstep(trace, dtype, d, beam):
    """Re-runs every traced call on the oracle from the GPU's own inputs."""
    bits = lambda t: to_host_bits(t) if isinstance(t, torch.Tensor) else [to_host_bits(x) for x in t]
    first = lambda name: name.startswith(("assign_base_", "update_base_", "assign_pre", "update_pre"))
    n_checked = 0
    for c in trace:
        name, ci, co = c["name"], c["in"], c["out"]
        if name.startswith("assign"):
            vdt = dtype if first(name) else "f32"
            V = oracle.vectors(np.ascontiguousarray(bits(ci["X"])), d)
            exp, _ = oracle.assign(V, bits(ci["C"]), vdt, vdt)
            check_codes(V, bits(ci["C"]), bits(co["codes"]), exp, vdt, vdt, name)
        elif name.startswith("update"):
            vdt = dtype if first(name) else "f32"
            V = oracle.vectors(np.ascontiguousarray(bits(ci["X"])), d)
            Cexp, _, _ = oracle.kmeans_update(V, bits(ci["codes"]), bits(ci["C"]), vdt, vdt)
            rel_close(oracle.widen(bits(co["C"]), vdt), oracle.widen(Cexp, vdt), 1e-5 if vdt == "f32" else 1e-2, name,
                      axis_vec=True)
        elif name.startswith("residual"):
            mn = np.ascontiguousarray(bits(ci["minuend"]))
            mdt = dtype if name in ("residual_base", "residual_all1") else "f32"
            Mv = oracle.vectors(mn, d)
            if isinstance(ci["codes"], list):
                bdt = [dtype] + ["f32"] * (len(ci["book"]) - 1)
                exp = opipe.residual_books(Mv, [np.ascontiguousarray(q).ravel() for q in bits(ci["codes"])],
                                           bits(ci["book"]), mdt, bdt)
            else:
                exp = oracle.residual(Mv, np.ascontiguousarray(bits(ci["codes"])).ravel(), bits(ci["book"]), mdt, mdt)
            np.testing.assert_array_equal(oracle.vectors(bits(co["out"]), d), exp)
        elif name in ("beam", "beam_basic"):
            X = np.ascontiguousarray(bits(ci["X"]))
            V = oracle.vectors(X, d)
            books = bits(ci["books"])
            bdt = [dtype] + ["f32"] * (len(books) - 1)
            exp, _ = oracle.beam(V, books, beam, dtype, bdt)
            if name == "beam":
                got = [np.ascontiguousarray(q).ravel() for q in bits(co["codes_basic"])] + \
                      [np.ascontiguousarray(q).ravel() for q in bits(co["codes_ext"])]
            else:
                got = [q.ravel() for q in bits(co["codes"])]
            got = np.stack(got)
            bad = np.flatnonzero((got != exp).any(0))
            if len(bad):  # only exact-tie substitutions are allowed
                R = lambda q: oracle.reconstruct([x for x in q[:, bad]], books, np.ones(len(bad), np.uint8), bdt,
                                                 n_full=len(books))
                V64 = oracle.widen(V[bad], dtype).astype(np.float64)
                e_got = ((V64 - R(got)) ** 2).sum(1)
                e_exp = ((V64 - R(exp)) ** 2).sum(1)
                assert (e_got <= e_exp * (1 + 1e-6)).all(), f"{name}: {len(bad)} tuples differ beyond ties"
        elif name == "dequant":
            books = bits(ci["books"])
            mb = len(ci["codes_basic"])
            bdt = [dtype] + ["f32"] * (len(books) - 1)
            out = bits(co["out"])
            M, N = out.shape
            vpr = N // d
            full = [q.ravel() for q in bits(ci["codes_basic"])]
            ext = bits(ci["codes_ext"])
            ncv = len(ext[0]) // M if ext else 0
            for q in ext:
                z = np.zeros((M, vpr), np.int32)
                z[:, :ncv] = q.reshape(M, ncv)
                full.append(z.ravel())
            R = oracle.reconstruct(full, books, opipe.crit_mask(M, N, d, ncv * d), bdt, n_full=mb)
            exp = oracle.scatter_columns(oracle.round_to(R, dtype).reshape(M, N), bits(ci["perm"]))
            np.testing.assert_array_equal(out, exp)
        else:
            continue
        n_checked += 1
    return n_checked


VARIANTS = {
    # name: (M, N, d, m_base, K_base, K_ext, crit_frac, beam, iters, dtype)
    "m2_d16": (96, 256, 16, 2, 64, (16, 16), 0.1, 2, 2, "f32"),
    "m2_d16_bf16": (64, 256, 16, 2, 64, (16,), 0.1, 4, 2, "bf16"),
    "m2_d16_beam1": (64, 128, 16, 2, 32, (16,), 0.2, 1, 3, "f32"),
    "m3_d8": (48, 128, 8, 3, 16, (8,), 0.1, 3, 2, "f32"),
    "d16": (96, 256, 16, 1, 64, (16, 16, 16), 0.1, 2, 2, "f32"),
    "e10": (128, 256, 8, 1, 1024, (64,), 0.05, 2, 2, "f32"),
    "e12": (128, 512, 8, 1, 4096, (64,), 0.05, 1, 1, "bf16"),
}


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_layer_variant(variant):
    M, N, d, mb, K_base, K_ext, lam, width, iters, dtype = VARIANTS[variant]
    say(f"layer variant {variant}: {M}x{N} d={d} basic={mb}x{K_base} ext={K_ext} beam={width} {dtype}")
    wl = inputs.small_workload(M=M, N=N, tokens=64, d=d, K_base=K_base, K_ext=K_ext, crit_frac=lam, beam=width,
                               iters=iters, dtype=dtype, wid=130, m_base=mb)
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    n = M * N // d
    n_crit = inputs.n_crit_columns(N, d, lam)
    base_idx = inputs.base_init_indices(wl, 0, n)
    extra = [inputs.extra_base_init_indices(wl, 0, b, n) for b in range(1, mb)]
    ext_idx = [inputs.ext_init_indices(wl, 0, t + 1, M * n_crit // d) for t in range(len(K_ext))]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    cfg = LayerConfig(d, K_base, list(K_ext), lam, width, iters, m_base=mb)
    q = LayerQuantizer(M, N, tdt, cfg, tokens=64, device="cuda")
    trace = []
    st = q.run(dev(W, dtype), torch.from_numpy(X).cuda(), torch.from_numpy(base_idx).cuda(),
               [torch.from_numpy(e).cuda() for e in ext_idx], trace=trace,
               base_idx_extra=[torch.from_numpy(e).cuda() for e in extra])
    torch.cuda.synchronize()
    checked = lockstep(trace, dtype, d, width)
    ref = opipe.quantize_layer(W, X, dtype, d, K_base, list(K_ext), lam, width, iters, base_idx, ext_idx,
                               m_base=mb, base_idx_extra=extra)
    np.testing.assert_array_equal(st.perm.cpu().numpy(), ref.perm)
    same = np.mean([np.mean(to_host_bits(a) == b) for a, b in zip(st.codes_basic, ref.codes_basic)])
    err = opipe.frob_err(W, to_host_bits(st.W_hat), dtype)
    err_ref = opipe.frob_err(W, ref.W_hat, dtype)
    assert abs(err - err_ref) <= 1e-3 * err_ref, (err, err_ref)
    bpw = C.crvq_bits_per_weight(M, N, d, n_crit, [K_base] * mb, list(K_ext))
    say(f"layer variant {variant}: {checked} calls matched in lockstep, perm identical, {100 * same:.2f}% basic "
        f"codes identical to the oracle pipeline, ||W - W_hat||^2 {err:.6e} (oracle {err_ref:.6e}), "
        f"{bpw:.4f} bits per weight")
