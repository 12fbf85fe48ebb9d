"""CRVQ CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct fp64 implementation of what the GPU library
computes, used to check it.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package; the product path never
does.  It shares no code with the HIP library (``paper_2412_09282_amd``) and
imports nothing from it.

The heavy loops live in ``crvq_oracle.c`` (plain C, fp64, built with gcc
``-O2 -ffp-contract=off``); this module marshals numpy arrays into it and
holds the few steps that are easiest to read in Python (the stable sort that
defines the channel permutation, the column gather, storage rounding).

Paper: "CRVQ: Channel-Relaxed Vector Quantization for Extreme Compression of
LLMs" (arXiv 2412.09282).  Sections, equations and the algorithm are cited per
function.  Readings of points where the paper is silent are stated where they
are used.

Parity pins: every function here is pinned by ``tests/test_oracle_pins.py``
against brute force, closed forms, invariants or independent library routines.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "crvq_oracle.c")
_LIB_PATH = os.path.join(_HERE, "_crvq_oracle.so")
_lock = threading.Lock()
_lib = None

F32, BF16 = "f32", "bf16"


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (plain -O2, no fast-math, no FMA contraction, OpenMP)."""
    with _lock:
        if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            tmp = _LIB_PATH + f".tmp{os.getpid()}"
            subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
                                   "-shared", "-std=c11", "-o", tmp, _SRC, "-lm"])
            os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        P, I64, I32, D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_double
        lib.oracle_assign.argtypes = [P, I64, I32, P, I64, P, P]
        lib.oracle_kmeans_means.argtypes = [P, I64, I32, P, I64, P, P, P]
        lib.oracle_colreduce.argtypes = [P, I64, P, I64, I64, I64, P, I32, P]
        lib.oracle_beam.argtypes = [P, I64, I32, I32, P, P, I32, P, P]
        lib.oracle_reconstruct.argtypes = [I64, I32, I32, I32, P, P, P, P]
        lib.oracle_round_bf16.argtypes = [P, I64, P]
        lib.oracle_num_threads.restype = I32
        lib.oracle_set_num_threads.argtypes = [I32]
        _lib = lib
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Host threads the oracle's parallel loops use from now on (for timing it on fewer cores)."""
    _load().oracle_set_num_threads(int(n))


# ----------------------------------------------------------------------------------------------
# storage types
# ----------------------------------------------------------------------------------------------

def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Data as float32: fp32 unchanged, bf16 bit patterns (uint16) widened exactly."""
    if dtype == BF16:
        return (np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    return np.ascontiguousarray(x, dtype=np.float32)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 values to the storage type (round-to-nearest-even): float32, or bf16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    if dtype == BF16:
        out = np.empty(x.shape, dtype=np.uint16)
        _load().oracle_round_bf16(_p(x), x.size, _p(out))
        return out
    return x.astype(np.float32)  # numpy's float64 -> float32 cast rounds to nearest even


def vectors(W: np.ndarray, d: int) -> np.ndarray:
    """Sub-vector partition of Sec. 3.1 Eq. 1: row i of W cut into N/d contiguous pieces of length d,
    enumerated row-major (vector index = i * N/d + j/d).  Returns an (M*N/d) x d view."""
    M, N = W.shape
    assert N % d == 0
    return np.ascontiguousarray(W).reshape(M * (N // d), d)


# ----------------------------------------------------------------------------------------------
# the steps of the path
# ----------------------------------------------------------------------------------------------

def colreduce(A: np.ndarray, B: Optional[np.ndarray] = None, scale: Optional[np.ndarray] = None,
              reduce: str = "sum", dtype: str = F32) -> np.ndarray:
    """out[j] = s_j * R_i (A[i,j] - B[i,j])^2 in fp64 (R = sum in ascending i, or max).

    * Hessian diagonal of Appendix A.2 Eq. 9: A = X (tokens x N), no B, no scale, sum:
      h_j = sum_k x_jk^2 = [X X^T]_jj (the paper's X is N x tokens; here it is stored transposed).
    * W-only importance of Sec. 4.1: A = W, reduce = max  ->  I_j = max_i w_ij^2.
    * Reformulated W-A importance of Appendix A.2 Eq. 10: A = W, B = VQ(W), scale = h/2, max.
    * Eq. 7 with the OBS denominator: same with scale_j = 1 / (2 [(XX^T)^-1]_jj).
    * The importance used by the timed workloads: A = W, sum, scale = h  ->  I_j = h_j sum_i w_ij^2.
    Returns fp64; the GPU returns float32 (round with ``round_to``)."""
    A32 = widen(A, dtype)
    B32 = None if B is None else widen(B, dtype)
    M, N = A32.shape
    s = None if scale is None else np.ascontiguousarray(scale, dtype=np.float64)
    out = np.empty(N, dtype=np.float64)
    _load().oracle_colreduce(_p(A32), A32.strides[0] // 4, _p(B32), 0 if B32 is None else B32.strides[0] // 4,
                             M, N, _p(s), 0 if reduce == "sum" else 1, _p(out))
    return out


def hessian_inverse_diagonal(H: np.ndarray, damp: float = 0.01) -> np.ndarray:
    """Denominator of the W-A importance of Sec. 4.1 Eq. 7: [(X X^T)^-1]_jj for every channel j,
    in fp64.  H = X X^T (N x N; stored tokens x N activations give H = X^T X).

    Reading (the paper is silent): X X^T is singular whenever the calibration set has fewer tokens
    than channels or a channel is never active, so the inverse is taken of the damped matrix
    H + damp * mean_j(H_jj) * I, the dampening of the OBS-style quantizers the paper builds on
    (damp = 1 %).  If the damped matrix is not positive definite (for instance an all-zero H)
    every entry of the result is NaN.  The definition, written out: the diagonal of the inverse."""
    H = np.asarray(H, dtype=np.float64)
    N = H.shape[0]
    assert H.shape == (N, N)
    Hd = H + damp * np.mean(np.diag(H)) * np.eye(N) if N else H
    try:
        np.linalg.cholesky(Hd)  # positive definiteness check only
    except np.linalg.LinAlgError:
        return np.full(N, np.nan)
    return np.diag(np.linalg.inv(Hd)).copy()


def obs_scale(hinv: np.ndarray) -> np.ndarray:
    """Per-channel factor of Sec. 4.1 Eq. 7, 1 / (2 [(X X^T)^-1]_jj), rounded once to float32 (the
    form the importance reduction takes its scale in), returned as fp64."""
    return np.asarray(1.0 / (2.0 * np.asarray(hinv, np.float64)), np.float32).astype(np.float64)


def rank_perm(importance: np.ndarray) -> np.ndarray:
    """Channel reordering of Sec. 4.2 (Alg. 1 ReorderChannels): channels sorted by importance, most
    important first.  Reading: a stable sort -- equal importance keeps the lower channel index
    first -- with NaN last.  perm[k] = the original channel placed at position k."""
    I = np.asarray(importance, dtype=np.float32)
    keys = []
    for j in range(I.shape[0]):
        v = float(I[j])
        keys.append((1 if math.isnan(v) else 0, 0.0 if math.isnan(v) else -v, j))
    return np.array([k[2] for k in sorted(keys)], dtype=np.int32)


def gather_columns(W: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """W_sorted[:, k] = W[:, perm[k]] (Sec. 4.2)."""
    return np.ascontiguousarray(W[:, perm])


def scatter_columns(R: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """Reverse reordering at inference (Sec. 4.3, Fig. 3 right): out[:, perm[k]] = R[:, k]."""
    out = np.empty_like(R)
    out[:, perm] = R
    return out


def n_crit_columns(N: int, d: int, frac: float) -> int:
    """Critical groups of Sec. 4.3: the first ceil(lambda*N/d) groups of d reordered channels."""
    return min(N, d * int(math.ceil(frac * N / d - 1e-9)))


def assign(V: np.ndarray, C: np.ndarray, v_dtype: str = F32, c_dtype: str = F32):
    """Encoding of Sec. 3.1 Eq. 3-4: q_i = argmin_j ||w_i - c_j||, lowest j on equal distance.
    Returns (codes int32, squared distance fp64)."""
    V32 = widen(V, v_dtype)
    C32 = widen(C, c_dtype)
    n, d = V32.shape
    K = C32.shape[0]
    codes = np.empty(n, dtype=np.int32)
    dist = np.empty(n, dtype=np.float64)
    _load().oracle_assign(_p(V32), n, d, _p(C32), K, _p(codes), _p(dist))
    return codes, dist


def kmeans_update(V: np.ndarray, codes: np.ndarray, C_old: np.ndarray, v_dtype: str = F32,
                  c_dtype: str = F32):
    """One Lloyd step of the K-means of Sec. 3.1 Eq. 2: every centroid becomes the mean of its
    members (fp64, members in ascending index), rounded to the codebook's storage type.  Reading
    (the paper is silent): an empty cluster keeps its previous centroid.
    Returns (new codebook in c_dtype storage, counts int64, fp64 means)."""
    V32 = widen(V, v_dtype)
    C32 = widen(C_old, c_dtype)
    n, d = V32.shape
    K = C32.shape[0]
    q = np.ascontiguousarray(codes, dtype=np.int32)
    means = np.empty((K, d), dtype=np.float64)
    counts = np.empty(K, dtype=np.int64)
    _load().oracle_kmeans_means(_p(V32), n, d, _p(q), K, _p(C32), _p(means), _p(counts))
    return round_to(means, c_dtype), counts, means


def objective(V: np.ndarray, C: np.ndarray, codes: np.ndarray, v_dtype: str = F32, c_dtype: str = F32) -> float:
    """K-means objective J = sum_i ||w_i - c_{q_i}||^2 in fp64."""
    V64 = widen(V, v_dtype).astype(np.float64)
    C64 = widen(C, c_dtype).astype(np.float64)
    diff = V64 - C64[codes]
    return float(np.sum(diff * diff))


def beam(V: np.ndarray, books: Sequence[np.ndarray], width: int, v_dtype: str = F32,
         book_dtypes: Optional[Sequence[str]] = None):
    """Residual beam search over additive codebooks (Sec. 3.1 last paragraph, Sec. 4.3, Alg. 1
    BeamSearchOptimize).  Reading: sequential over the books in order (basic first), keeping the
    `width` best partial tuples under the squared Euclidean error of the residual, candidates
    keyed (error, parent rank, codeword index).  width = 1 is the greedy additive fit of Alg. 1's
    extended-codebook loop.  Returns (codes [n_books, n] int32, final error fp64)."""
    V32 = widen(V, v_dtype)
    n, d = V32.shape
    if book_dtypes is None:
        book_dtypes = [F32] * len(books)
    B32 = [widen(b, t) for b, t in zip(books, book_dtypes)]
    nb = len(B32)
    arr = (ctypes.c_void_p * nb)(*[b.ctypes.data for b in B32])
    Ks = np.array([b.shape[0] for b in B32], dtype=np.int64)
    codes = np.empty((nb, n), dtype=np.int32)
    err = np.empty(n, dtype=np.float64)
    _load().oracle_beam(_p(V32), n, d, nb, arr, _p(Ks), int(width), _p(codes), _p(err))
    return codes, err


def reconstruct(codes: Sequence[np.ndarray], books: Sequence[np.ndarray], crit: np.ndarray,
                book_dtypes: Optional[Sequence[str]] = None, n_full: int = 1) -> np.ndarray:
    """Additive reconstruction of Sec. 4.3: a critical vector is the sum (fp64, book order) of its
    codewords from the basic and every extended codebook; a non-critical one the sum of its codewords
    from the n_full basic books (one unless the layout has several).  codes[b] holds one code per
    vector for book b (entries of extended books are ignored where crit is 0).  Returns fp64 (n x d)."""
    if book_dtypes is None:
        book_dtypes = [F32] * len(books)
    B32 = [widen(b, t) for b, t in zip(books, book_dtypes)]
    nb = len(B32)
    n = len(codes[0])
    d = B32[0].shape[1]
    q = np.ascontiguousarray(np.stack([np.asarray(c, dtype=np.int32) for c in codes]))
    cr = np.ascontiguousarray(crit, dtype=np.uint8)
    arr = (ctypes.c_void_p * nb)(*[b.ctypes.data for b in B32])
    R = np.empty((n, d), dtype=np.float64)
    _load().oracle_reconstruct(n, d, nb, n_full, arr, _p(q), _p(cr), _p(R))
    return R


def gemv(M: int, N: int, d: int, n_crit: int, codes: Sequence[np.ndarray], books: Sequence[np.ndarray],
         perm: Optional[np.ndarray], x: np.ndarray, book_dtypes: Optional[Sequence[str]] = None,
         x_dtype: str = F32):
    """Matrix-vector product with a CRVQ-quantized layer (Sec. 4.3, Fig. 3 right: the reconstructed
    weights in original channel order), y = W_hat x, in fp64 from the exact (un-rounded) fp64 sum of
    the codewords.  codes[0] is the basic code array [M][N/d], codes[b] (b >= 1) the extended codes
    [M][n_crit/d] of the critical groups.  Returns (y, a) with a_i = sum_j |W_hat_ij x_j|, the scale
    against which the rounding of a product in lower precision is measured."""
    vpr, ncv = N // d, n_crit // d
    full = [np.asarray(codes[0], dtype=np.int32).reshape(M, vpr).ravel()]
    for c in codes[1:]:
        z = np.zeros((M, vpr), np.int32)
        z[:, :ncv] = np.asarray(c, dtype=np.int32).reshape(M, ncv)
        full.append(z.ravel())
    crit = (np.arange(M * vpr) % vpr < ncv).astype(np.uint8)
    R = reconstruct(full, books, crit, book_dtypes).reshape(M, N)
    Wh = scatter_columns(R, perm) if perm is not None else R
    x64 = widen(np.asarray(x), x_dtype).astype(np.float64)
    return Wh @ x64, np.abs(Wh) @ np.abs(x64)


def residual(minuend: np.ndarray, codes: np.ndarray, book: np.ndarray, m_dtype: str = F32,
             c_dtype: str = F32) -> np.ndarray:
    """ComputeError of Alg. 1: E = minuend - C[q] (per vector, fp64), rounded to float32."""
    Mv = widen(minuend, m_dtype).astype(np.float64)
    R = reconstruct([codes], [book], np.zeros(len(codes), np.uint8), [c_dtype])
    return (Mv - R).astype(np.float32)


def bits_per_weight_vq(m: int, e: int, d: int, rows: int = 4096, cols: int = 4096) -> float:
    """Average bits per weight of plain additive VQ (Sec. 3.2 Eq. 6, derived in Appendix A.1):
    codes m*e/d per weight plus m codebooks of 2^e FP16 d-vectors spread over the matrix."""
    n_w = rows * cols
    return (n_w * m * e / d + (2 ** e) * m * d * 16) / n_w


def bits_per_weight_crvq(m: int, e: int, d: int, lam: float, rows: int = 4096, cols: int = 4096,
                         include_perm: bool = False, m_base: int = 1) -> float:
    """Average bits per weight of CRVQ (Appendix A.1 Eq. 8): basic codes e/d, extended codes
    (m-1)*lambda*e/d, m codebooks, optionally the 16-bit channel-permutation indices.  With m_base
    basic books (Sec. 6.4's m = 2 setting) the basic codes take m_base*e/d and the extended ones
    (m-m_base)*lambda*e/d."""
    n_w = rows * cols
    bits = m_base * e / d + (m - m_base) * lam * e / d + (2 ** e) * m * d * 16 / n_w
    if include_perm:
        bits += cols * 16 / n_w
    return bits
