"""CPU-only checks of the C ABI: the library loads, exports every symbol the header declares, and
rejects invalid arguments on the host before anything is enqueued (no GPU is touched).  Also checks
that the oracle and the GPU path share no code."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2412_09282_amd import crvq
    return crvq.lib()


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation first


def test_exports_every_declared_symbol(L):
    from paper_2412_09282_amd import build
    declared = build.exported_symbols()
    assert len(declared) >= 15
    so = os.path.join(ROOT, "paper_2412_09282_amd", "libcrvq.so")
    out = os.popen(f"nm -D --defined-only {so}").read()
    exported = set(re.findall(r" T (crvq_[a-z0-9_]+)", out))
    missing = [s for s in declared if s not in exported]
    assert not missing, missing
    for s in declared:
        assert hasattr(L, s)


def test_version_and_error_text(L):
    assert L.crvq_version() >= 100
    assert isinstance(L.crvq_last_error(), bytes)


def err(L):
    return L.crvq_last_error().decode()


def test_assign_validation(L):
    ws = ctypes.c_void_p(0x100000)
    # bad dtype
    assert L.crvq_assign(FAKE, 7, 4, 2, 16, 8, FAKE, 0, 16, FAKE, None, ws, 1 << 30, None) == 1
    assert "x_dtype" in err(L)
    # unsupported d
    assert L.crvq_assign(FAKE, 0, 4, 2, 64, 32, FAKE, 0, 16, FAKE, None, ws, 1 << 30, None) == 2
    # ld too small
    assert L.crvq_assign(FAKE, 0, 4, 2, 15, 8, FAKE, 0, 16, FAKE, None, ws, 1 << 30, None) == 1
    # K out of range
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, FAKE, 0, 0, FAKE, None, ws, 1 << 30, None) == 1
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, FAKE, 0, 65537, FAKE, None, ws, 1 << 30, None) == 1
    # NULL codebook / codes
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, None, 0, 16, FAKE, None, ws, 1 << 30, None) == 1
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, FAKE, 0, 16, None, None, ws, 1 << 30, None) == 1
    # workspace too small / NULL / misaligned
    need = L.crvq_assign_workspace_size(8, 8, 16)
    assert need > 0
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, FAKE, 0, 16, FAKE, None, ws, need - 1, None) == 3
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, FAKE, 0, 16, FAKE, None, None, need, None) == 3
    assert L.crvq_assign(FAKE, 0, 4, 2, 16, 8, FAKE, 0, 16, FAKE, None, ctypes.c_void_p(0x100010), need, None) == 3
    # empty input is a no-op
    assert L.crvq_assign(None, 0, 0, 2, 16, 8, FAKE, 0, 16, None, None, None, 0, None) == 0


def test_workspace_sizes_are_deterministic_and_monotone(L):
    a = L.crvq_assign_workspace_size(1 << 20, 8, 65536)
    assert a == L.crvq_assign_workspace_size(1 << 20, 8, 65536)
    assert L.crvq_assign_workspace_size(1 << 21, 8, 65536) >= a
    assert L.crvq_assign_workspace_size(10, 8, 0) == 0
    assert L.crvq_kmeans_workspace_size(1000, 8, 256) > 0
    assert L.crvq_importance_workspace_size(4096, 4096) > 0
    Ks = (ctypes.c_int64 * 2)(256, 256)
    assert L.crvq_beam_workspace_size(1000, 8, 2, ctypes.cast(Ks, ctypes.c_void_p), 4) > 0
    assert L.crvq_beam_workspace_size(1000, 8, 2, ctypes.cast(Ks, ctypes.c_void_p), 17) == 0


def test_beam_validation(L):
    Ks = (ctypes.c_int64 * 2)(256, 256)
    dts = (ctypes.c_int32 * 2)(0, 0)
    books = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    codes = (ctypes.c_void_p * 2)(0x3000, 0x4000)
    PP = ctypes.POINTER(ctypes.c_void_p)
    args = lambda nb, beam, ks=Ks: (FAKE, 0, 10, 2, 16, 8, nb, ctypes.cast(books, PP), ctypes.cast(dts, ctypes.c_void_p),
                                    ctypes.cast(ks, ctypes.c_void_p), beam, ctypes.cast(codes, PP), None, None,
                                    FAKE, 1 << 30, None)
    assert L.crvq_assign_residual_beam(*args(0, 4)) == 1
    assert L.crvq_assign_residual_beam(*args(9, 4)) == 1
    assert L.crvq_assign_residual_beam(*args(2, 0)) == 1
    assert L.crvq_assign_residual_beam(*args(2, 17)) == 1
    bad = (ctypes.c_int64 * 2)(256, 70000)
    assert L.crvq_assign_residual_beam(*args(2, 4, bad)) == 1
    ldc = (ctypes.c_int64 * 2)(1, 2)
    a = list(args(2, 4))
    a[12] = ctypes.cast(ldc, ctypes.c_void_p)
    assert L.crvq_assign_residual_beam(*a) == 1 and "ldc" in err(L)


def test_kmeans_importance_reorder_dequant_validation(L):
    ws = ctypes.c_void_p(0x100000)
    assert L.crvq_kmeans_update(FAKE, 0, 4, 2, 16, 8, FAKE, 0, FAKE, 0, None, ws, 1 << 30, None) == 1
    assert L.crvq_kmeans_update(FAKE, 0, 4, 2, 16, 8, None, 16, FAKE, 0, None, ws, 1 << 30, None) == 1
    assert L.crvq_kmeans_update(FAKE, 0, 4, 2, 16, 8, FAKE, 16, FAKE, 0, None, ws, 0, None) == 3
    assert L.crvq_channel_importance(FAKE, 4, None, 0, 0, 0, 4, None, 0, FAKE, ws, 1 << 30, None) == 1
    assert L.crvq_channel_importance(FAKE, 3, None, 0, 0, 4, 4, None, 0, FAKE, ws, 1 << 30, None) == 1
    assert L.crvq_channel_importance(FAKE, 4, None, 0, 0, 4, 4, None, 5, FAKE, ws, 1 << 30, None) == 1
    assert L.crvq_channel_importance(FAKE, 4, None, 0, 0, 4, 4, None, 0, FAKE, None, 0, None) == 3
    # reorder: in == out rejected, perm required
    assert L.crvq_reorder(FAKE, 8, FAKE, 8, 0, 4, 8, None, FAKE, 0, None, 0, None) == 1
    assert "overlap" in err(L)
    assert L.crvq_reorder(FAKE, 8, ctypes.c_void_p(0x9000), 8, 0, 4, 8, None, None, 0, None, 0, None) == 1
    assert L.crvq_reorder(None, 0, None, 0, 0, 0, 0, FAKE, FAKE, 0, None, 0, None) == 1
    # dequant: n_cols % d, n_crit not multiple of d, perm + minuend
    PP = ctypes.POINTER(ctypes.c_void_p)
    assert L.crvq_dequant(4, 12, 8, 0, FAKE, 2, FAKE, 0, 16, 0, None, 0, None, None, None, None, None, 0, 0, FAKE, 0, 12,
                          None, 0, None) == 1
    assert L.crvq_dequant(4, 16, 8, 4, FAKE, 2, FAKE, 0, 16, 0, None, 0, None, None, None, None, None, 0, 0, FAKE, 0, 16,
                          None, 0, None) == 1
    assert L.crvq_dequant(4, 16, 8, 8, FAKE, 2, FAKE, 0, 16, 0, None, 0, None, None, None, FAKE, FAKE, 0, 16, FAKE, 0, 16,
                          ws, 1 << 20, None) == 1
    assert "mutually exclusive" in err(L)
    assert L.crvq_gather_vectors(FAKE, 0, 4, 2, 16, 8, None, 3, FAKE, 0, None) == 1
    assert L.crvq_gather_vectors(FAKE, 0, 4, 2, 16, 8, FAKE, 3, FAKE, 1, None) == 1


def _imports(path):
    src = open(path).read()
    return set(re.findall(r"^\s*(?:from|import)\s+([\w\.]+)", src, re.M))


def test_gemv_validation(L):
    """crvq_dequant_gemv / crvq_pack_codes_u8 reject bad arguments before touching the device."""
    ws = ctypes.c_void_p(0x100000)
    big = 1 << 30
    q8 = ctypes.c_void_p(0x2000)  # 8-byte aligned
    ok = lambda **kw: dict(dict(M=16, N=128, n_crit=16, q=q8, ldq=16, C=FAKE, bdt=0, K=256, ne=0, qe=None, ldqe=0,
                                Ce=None, edt=None, Ke=None, perm=None, x=FAKE, xdt=0, y=FAKE, ws=ws, wsb=big), **kw)
    call = lambda a: L.crvq_dequant_gemv(a["M"], a["N"], a["n_crit"], a["q"], a["ldq"], a["C"], a["bdt"], a["K"],
                                         a["ne"], a["qe"], a["ldqe"], a["Ce"], a["edt"], a["Ke"], a["perm"], a["x"],
                                         a["xdt"], a["y"], a["ws"], a["wsb"], None)
    assert call(ok(N=120)) == 2 and "multiple of 64" in err(L)
    assert call(ok(n_crit=12)) == 1
    assert call(ok(n_crit=136)) == 1
    assert call(ok(K=257)) == 2 and "8-bit" in err(L)
    assert call(ok(K=0)) == 2
    assert call(ok(ldq=15)) == 1
    assert call(ok(ldq=12)) == 1
    assert call(ok(q=ctypes.c_void_p(0x2001))) == 1 and "aligned" in err(L)
    assert call(ok(x=None)) == 1
    assert call(ok(y=None)) == 1
    assert call(ok(bdt=3)) == 1
    assert call(ok(ne=8)) == 1
    assert call(ok(ne=1)) == 1 and "must not be NULL" in err(L)
    PP = ctypes.POINTER(ctypes.c_void_p)
    qe = (ctypes.c_void_p * 1)(0x3000)
    ce = (ctypes.c_void_p * 1)(0x4000)
    edt = (ctypes.c_int32 * 1)(0)
    kbad = (ctypes.c_int64 * 1)(300)
    ext = dict(ne=1, qe=ctypes.cast(qe, PP), ldqe=2, Ce=ctypes.cast(ce, PP), edt=ctypes.cast(edt, ctypes.c_void_p),
               Ke=ctypes.cast(kbad, ctypes.c_void_p))
    assert call(ok(**ext)) == 2 and "K_ext" in err(L)
    kok = (ctypes.c_int64 * 1)(256)
    ext["Ke"] = ctypes.cast(kok, ctypes.c_void_p)
    assert call(ok(**dict(ext, ldqe=1))) == 1 and "ldq_ext" in err(L)
    need = L.crvq_gemv_workspace_size(16, 128, 256)
    assert need > 0 and L.crvq_gemv_workspace_size(16, 128, 300) == 0
    assert call(ok(wsb=need - 1)) == 3
    assert L.crvq_pack_codes_u8(FAKE, -1, FAKE, None) == 1
    assert L.crvq_pack_codes_u8(None, 4, FAKE, None) == 1
    assert L.crvq_pack_codes_u8(None, 0, None, None) == 0


def test_oracle_and_gpu_path_share_no_code():
    odir = os.path.join(ROOT, "oracle")
    pdir = os.path.join(ROOT, "paper_2412_09282_amd")
    for f in os.listdir(odir):
        if f.endswith(".py"):
            assert not any(m.startswith("paper_2412_09282_amd") for m in _imports(os.path.join(odir, f))), f
    for root, _, files in os.walk(pdir):
        for f in files:
            p = os.path.join(root, f)
            if f.endswith(".py"):
                assert not any(m.startswith("oracle") for m in _imports(p)), p
            if f.endswith((".hip", ".h", ".cpp")):
                assert "oracle" not in open(p).read().lower(), p


def test_dequant_books_validation(L):
    """crvq_dequant_books rejects bad book counts and NULL arrays before touching the device."""
    PP = ctypes.POINTER(ctypes.c_void_p)
    q = ctypes.cast((ctypes.c_void_p * 3)(0x1000, 0x2000, 0x3000), PP)
    C = ctypes.cast((ctypes.c_void_p * 3)(0x4000, 0x5000, 0x6000), PP)
    dts = ctypes.cast((ctypes.c_int32 * 3)(0, 0, 0), ctypes.c_void_p)
    Ks = ctypes.cast((ctypes.c_int64 * 3)(256, 256, 16), ctypes.c_void_p)
    call = lambda nb, ne, q=q, C=C, n_crit=16, ldq_ext=1: L.crvq_dequant_books(
        4, 32, 16, n_crit, nb, ne, q, 2, ldq_ext, C, dts, Ks, None, None, 0, 0, FAKE, 0, 32, None, 0, None)
    assert call(0, 1) == 1 and "n_base" in err(L)
    assert call(2, 7) == 1
    assert call(2, 1, q=None) == 1 and "must not be NULL" in err(L)
    assert call(2, 1, C=None) == 1
    assert call(2, 1, n_crit=8) == 1            # not a multiple of d = 16
    assert call(2, 1, ldq_ext=0) == 1 and "ldq_ext" in err(L)
    Kbad = ctypes.cast((ctypes.c_int64 * 3)(256, 0, 16), ctypes.c_void_p)
    assert L.crvq_dequant_books(4, 32, 16, 16, 2, 1, q, 2, 1, C, dts, Kbad, None, None, 0, 0, FAKE, 0, 32, None, 0,
                                None) == 1 and "outside" in err(L)
    assert L.crvq_dequant_books(4, 32, 16, 16, 2, 1, q, 2, 1, C, dts, Ks, FAKE, None, 0, 0, FAKE, 0, 32, None, 0,
                                None) == 3  # perm without the workspace


def test_bits_per_weight_against_eq6_eq8():
    """crvq_bits_per_weight (host-only) against Eq. 6 / Eq. 8 as the oracle states them, the paper's
    printed values (tests/golden/bits_per_weight.json) and the increments each stored object adds."""
    import json
    import oracle
    from paper_2412_09282_amd import crvq as C
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "bits_per_weight.json")))
    g = gold["vq_m1_e8_d8"]
    v = C.crvq_bits_per_weight(4096, 4096, 8, 0, [256], perm_bits=0)
    assert abs(v - g["printed"]) <= g["printed_precision"]
    assert v == oracle.bits_per_weight_vq(1, 8, 8)
    # 8+8x3 at lambda = 0.02: 88 critical columns (8 * ceil(0.02 * 4096 / 8)) stand in for lambda N
    for perm_bits in (0, 16):
        v = C.crvq_bits_per_weight(4096, 4096, 8, 88, [256], [256] * 3, perm_bits=perm_bits)
        e = oracle.bits_per_weight_crvq(4, 8, 8, 88 / 4096, include_perm=perm_bits == 16)
        assert abs(v - e) < 1e-12, (v, e)
    # the m = 2, d = 16 setting, with and without three extended books
    v = C.crvq_bits_per_weight(4096, 4096, 16, 0, [256, 256], perm_bits=0)
    assert v == oracle.bits_per_weight_vq(2, 8, 16)
    v = C.crvq_bits_per_weight(4096, 4096, 16, 96, [256, 256], [256] * 3, perm_bits=0)
    assert abs(v - oracle.bits_per_weight_crvq(5, 8, 16, 96 / 4096, m_base=2)) < 1e-12
    # wider basic books (e = 10, 12) then one extended e = 8 book: Eq. 6 plus one extended book's share
    for e in (10, 12):
        base = C.crvq_bits_per_weight(4096, 4096, 8, 0, [2 ** e], perm_bits=0)
        assert abs(base - oracle.bits_per_weight_vq(1, e, 8)) < 1e-12
        v = C.crvq_bits_per_weight(4096, 4096, 8, 88, [2 ** e], [256], perm_bits=0)
        inc = oracle.bits_per_weight_crvq(2, 8, 8, 88 / 4096) - oracle.bits_per_weight_vq(1, 8, 8)
        assert abs(v - base - inc) < 1e-12
    # a book of K codewords that is not a power of two takes ceil(log2 K)-bit codes and K stored codewords
    v100 = C.crvq_bits_per_weight(64, 64, 8, 0, [100], perm_bits=0)
    v128 = C.crvq_bits_per_weight(64, 64, 8, 0, [128], perm_bits=0)
    assert abs((v128 - v100) - 28 * 8 * 16 / (64 * 64)) < 1e-12
    assert C.crvq_bits_per_weight(64, 64, 8, 0, [1], perm_bits=0, codeword_bits=16) == 8 * 16 / (64 * 64)
    with pytest.raises(C.CrvqError):
        C.crvq_bits_per_weight(64, 60, 8, 0, [256])      # cols not a multiple of d
    with pytest.raises(C.CrvqError):
        C.crvq_bits_per_weight(64, 64, 8, 4, [256], [16])  # n_crit not a multiple of d
    with pytest.raises(C.CrvqError):
        C.crvq_bits_per_weight(64, 64, 8, 0, [0])
    with pytest.raises(C.CrvqError):
        C.crvq_bits_per_weight(64, 64, 8, 0, [256], codeword_bits=0)


def test_refinement_validation(L):
    """The refinement calls reject bad arguments on the host (nothing is enqueued)."""
    ws = ctypes.c_void_p(0x100000)
    assert L.crvq_gram(FAKE, 1, 16, 8, 8, FAKE, 8, None) == 1            # bf16 activations not accepted
    assert L.crvq_gram(FAKE, 0, 16, 8, 4, FAKE, 8, None) == 1            # ld < n_cols
    assert L.crvq_gram(None, 0, 16, 0, 0, None, 0, None) == 0            # nothing to do
    assert L.crvq_hessian_product(4, 8, 4, FAKE, 8, FAKE, 8, FAKE, 4, FAKE, None, None) == 1  # row_loss: n_out == N
    assert L.crvq_hessian_product(4, 8, 9, FAKE, 8, FAKE, 8, FAKE, 9, None, None, None) == 1
    assert L.crvq_hessian_product(4, 8, 8, FAKE, 8, FAKE, 8, FAKE, 8, None, FAKE, None) == 1  # total needs row_loss
    assert "loss_total" in err(L)
    assert L.crvq_code_sums(FAKE, 4, 2, 16, 8, FAKE, 70000, FAKE, None, ws, 1 << 30, None) == 2  # K > 65536
    assert L.crvq_code_sums(FAKE, 4, 2, 8, 8, FAKE, 16, FAKE, None, ws, 1 << 30, None) == 1     # ld < vpr * d
    assert L.crvq_code_sums(FAKE, 4, 2, 16, 8, FAKE, 16, FAKE, None, ws, 0, None) == 3          # no workspace
    assert L.crvq_code_sums_workspace_size(100, 8, 70000) == 0
    assert L.crvq_code_sums_workspace_size(100, 8, 65536) > L.crvq_code_sums_workspace_size(100, 8, 1024) > 0
    dbl = ctypes.c_double
    assert L.crvq_adam_step(FAKE, FAKE, dbl(-2.0), FAKE, FAKE, 8, 0, dbl(1e-3), dbl(0.9), dbl(0.95), dbl(1e-8),
                            None) == 1                                    # step 0
    assert L.crvq_adam_step(FAKE, FAKE, dbl(-2.0), FAKE, FAKE, 8, 1, dbl(1e-3), dbl(1.0), dbl(0.95), dbl(1e-8),
                            None) == 1                                    # beta1 = 1
    need = L.crvq_refine_workspace_size(64, 256, 256)
    assert need > 64 * 256 * 8 and L.crvq_refine_workspace_size(64, 128, 256) == 0
    assert L.crvq_refine_codes(64, 256, 8, 256, FAKE, 256, FAKE, 256, FAKE, 0, 70000, FAKE, 32, ws, need, None) == 2
    assert L.crvq_refine_codes(64, 256, 8, 250, FAKE, 256, FAKE, 256, FAKE, 0, 256, FAKE, 32, ws, need, None) == 1
    assert L.crvq_refine_codes(64, 256, 8, 256, FAKE, 256, FAKE, 256, FAKE, 0, 256, FAKE, 31, ws, need, None) == 1
    assert L.crvq_refine_codes(64, 256, 8, 256, FAKE, 256, FAKE, 256, FAKE, 0, 256, FAKE, 32, ws, need - 1, None) == 3
    assert L.crvq_refine_codes(64, 256, 8, 256, FAKE, 256, FAKE, 256, FAKE, 2, 256, FAKE, 32, ws, need, None) == 1
    dbl = ctypes.c_double
    nh = L.crvq_hessian_inverse_workspace_size(100)
    assert nh >= 16 * 128 * 128 and L.crvq_hessian_inverse_workspace_size(0) == 0
    assert L.crvq_hessian_inverse_diagonal(FAKE, 99, 100, dbl(0.01), FAKE, None, ws, nh, None) == 1   # ldh < N
    assert L.crvq_hessian_inverse_diagonal(FAKE, 100, 100, dbl(-0.5), FAKE, None, ws, nh, None) == 1  # damp < 0
    assert L.crvq_hessian_inverse_diagonal(FAKE, 100, 100, dbl(float("nan")), FAKE, None, ws, nh, None) == 1
    assert L.crvq_hessian_inverse_diagonal(FAKE, 100, 100, dbl(0.01), None, None, ws, nh, None) == 1  # no output
    assert L.crvq_hessian_inverse_diagonal(FAKE, 100, 100, dbl(0.01), FAKE, None, ws, nh - 1, None) == 3
    assert L.crvq_hessian_inverse_diagonal(FAKE, 70000, 70000, dbl(0.01), FAKE, None, ws, nh, None) == 1
    assert L.crvq_hessian_inverse_diagonal(None, 0, 0, dbl(0.01), None, None, None, 0, None) == 0     # N = 0


def test_workspace_size_dispatcher(L):
    """crvq_workspace_size(op, ...) returns what the per-call sizing function returns for the same
    shape, for every op, and 0 for an unknown op or a rejected shape."""
    from paper_2412_09282_amd import crvq as C
    for n, d, K in [(1, 8, 1), (8192, 8, 256), (2097152, 8, 65536), (300, 5, 2000), (70001, 16, 4096)]:
        assert C.crvq_workspace_size("assign", n_vectors=n, d=d, K=K) == L.crvq_assign_workspace_size(n, d, K) > 0
        assert C.crvq_workspace_size("kmeans", n_vectors=n, d=d, K=K) == L.crvq_kmeans_workspace_size(n, d, K)
        if K <= 1024:
            assert C.crvq_workspace_size("code_sums", n_vectors=n, d=d, K=K) == \
                L.crvq_code_sums_workspace_size(n, d, K) > 0
    Ks = [65536, 256, 256]
    arr = (ctypes.c_int64 * 3)(*Ks)
    for beam in (1, 4, 16):
        assert C.crvq_workspace_size("beam", n_vectors=65536, d=8, Ks=Ks, beam=beam) == \
            L.crvq_beam_workspace_size(65536, 8, 3, ctypes.cast(arr, ctypes.c_void_p), beam) > 0
    assert C.crvq_workspace_size("beam", n_vectors=100, d=8, Ks=Ks, beam=17) == 0
    assert C.crvq_workspace_size("importance", M=28672, N=8192) == L.crvq_importance_workspace_size(28672, 8192) > 0
    assert C.crvq_workspace_size("reorder", N=13824) == L.crvq_reorder_workspace_size(13824) > 0
    assert C.crvq_workspace_size("dequant", N=8192) == L.crvq_dequant_workspace_size(8192) > 0
    assert C.crvq_workspace_size("refine", M=300, N=2056, n_cols=64) == L.crvq_refine_workspace_size(300, 2056, 64) > 0
    assert C.crvq_workspace_size("gemv", M=11008, N=4096, K=256) == L.crvq_gemv_workspace_size(11008, 4096, 256) > 0
    assert C.crvq_workspace_size("hinv", N=4097) == L.crvq_hessian_inverse_workspace_size(4097) >= 16 * 4160 ** 2
    assert C.crvq_workspace_size("hinv", N=65537) == 0
    assert L.crvq_workspace_size(99, 100, 16, 1, 1, 8, None, 1, 1, 1) == 0
    assert C.crvq_workspace_size("assign", n_vectors=100, d=8, K=65537) == 0
