"""CRVQ per-layer quantization on the CPU oracle -- TEST INFRASTRUCTURE ONLY.

The steps of Alg. 1 that the GPU library implements, for one weight matrix, in
the paper's order:

  ComputeImportance -> ReorderChannels -> KMeansCodebook + VectorQuant (basic)
  -> for each extended codebook: ComputeError, KMeansCodebook, VectorQuant,
  Update (critical groups only) -> beam search over all books for the critical
  vectors -> reconstruction with the reverse reordering.

Readings where the paper is silent (each also listed in the design notes):
* importance (``importance=``): "energy" I_j = h_j * sum_i W_ij^2 with
  h = diag(X X^T) (the timed workloads' metric); "w_only" I_j = max_i W_ij^2
  (Sec. 4.1); "wa" the Hessian-proxy metric of Sec. 4.1 in the unpacked form of
  Appendix A.2 Eq. 10, I_j = h_j * max_i (W_ij - Wq_ij)^2 with Wq the
  prequantized W (Alg. 1 Prequantize: the basic VQ -- same K, init indices and
  iterations -- on the unsorted W); Eq. 10's factor 1/2 is the same for every
  channel and changes no ordering, so it is left out; "obs" Eq. 7 as printed,
  I_j = max_i (W_ij - Wq_ij)^2 / (2 [(X X^T)^-1]_jj), the inverse taken of the
  damped Hessian proxy (``hessian_inverse_diagonal``), the factor rounded to
  float32 before the reduction;
* critical channels: the first d * ceil(lambda N / d) reordered columns;
* K-means: initial codewords are the vectors at seeded indices (an input);
  one iteration = assign + update; ``iters`` iterations then a final assign;
  an empty cluster keeps its centroid;
* residuals are rounded to float32 when they are stored (E^t);
* the final codes of critical vectors come from the beam search (width 1 =
  greedy) over [basic, ext_1, ...] on the un-rounded (fp64) residual;
* several basic codebooks (``m_base`` > 1, the m = 2, d = 16 setting of
  Sec. 3.2 / Sec. 6.4): basic book b >= 1 is fitted (K-means from seeded
  indices) on the float32 residual of every vector after books < b and their
  final assignments; then the beam search over the basic books gives the codes
  of every vector; the extended books are fitted on the critical residual
  after those codes, and the critical vectors' final codes come from the beam
  over all books.  Basic books after the first are float32, like the residual
  they are fitted on.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from . import (F32, BF16, assign, beam, colreduce, gather_columns, hessian_inverse_diagonal, kmeans_update,
               n_crit_columns, objective, obs_scale, rank_perm, reconstruct, residual, round_to, scatter_columns,
               vectors, widen)
from .refine import gram


@dataclasses.dataclass
class LayerResult:
    hdiag: np.ndarray             # float32 [N]
    importance: np.ndarray        # float32 [N]
    perm: np.ndarray              # int32 [N]
    n_crit: int                   # critical columns (multiple of d)
    C_base: np.ndarray            # K_base x d, storage dtype of W
    C_ext: List[np.ndarray]       # float32 K_t x d
    codes_base: np.ndarray        # int32 [M * N/d]   (greedy basic codes; critical ones replaced by the beam)
    codes_ext: List[np.ndarray]   # int32 [M * n_crit/d] per extended book
    beam_err: np.ndarray          # fp64 [M * n_crit/d]
    W_hat: np.ndarray             # reconstruction in original channel order, storage dtype of W
    objectives: Dict[str, List[float]]
    C_basic: List[np.ndarray] = dataclasses.field(default_factory=list)      # all m_base basic books
    codes_basic: List[np.ndarray] = dataclasses.field(default_factory=list)  # their int32 [M * N/d] codes


def crit_mask(M: int, N: int, d: int, n_crit: int) -> np.ndarray:
    g = np.arange(N // d)
    return np.broadcast_to(g < n_crit // d, (M, N // d)).reshape(-1).astype(np.uint8)


def crit_slab(Ws: np.ndarray, n_crit: int) -> np.ndarray:
    return np.ascontiguousarray(Ws[:, :n_crit])


def kmeans(V: np.ndarray, C0: np.ndarray, iters: int, v_dtype: str, c_dtype: str):
    """KMeansCodebook + VectorQuant: `iters` Lloyd iterations then a final assignment."""
    C = C0
    J = []
    for _ in range(iters):
        q, _ = assign(V, C, v_dtype, c_dtype)
        J.append(objective(V, C, q, v_dtype, c_dtype))
        C, _, _ = kmeans_update(V, q, C, v_dtype, c_dtype)
    q, dist = assign(V, C, v_dtype, c_dtype)
    J.append(objective(V, C, q, v_dtype, c_dtype))
    return C, q, dist, J


def prequantize(W: np.ndarray, dtype: str, d: int, base_idx: np.ndarray, iters: int) -> np.ndarray:
    """Alg. 1 Prequantize: the basic VQ of the unsorted W (K-means from the vectors at base_idx,
    `iters` iterations, final assignment), reconstructed in W's storage type."""
    V = vectors(W, d)
    C, q, _, _ = kmeans(V, np.ascontiguousarray(V[base_idx]), iters, dtype, dtype)
    R = reconstruct([q], [C], np.zeros(len(q), np.uint8), [dtype])
    return round_to(R, dtype).reshape(W.shape)


def channel_importance(W: np.ndarray, h: np.ndarray, dtype: str, mode: str, d: int = 8,
                       base_idx: Optional[np.ndarray] = None, iters: int = 1,
                       H: Optional[np.ndarray] = None, damp: float = 0.01) -> np.ndarray:
    """Channel importance of Sec. 4.1 (modes as in the module notes), rounded to float32.  Mode
    "obs" needs H = X X^T (fp64, N x N)."""
    if mode == "obs":
        Wq = prequantize(W, dtype, d, base_idx, iters)
        s = obs_scale(hessian_inverse_diagonal(H, damp))
        I = colreduce(W, Wq, scale=s, reduce="max", dtype=dtype)
    elif mode == "energy":
        I = colreduce(W, scale=h.astype(np.float64), reduce="sum", dtype=dtype)
    elif mode == "w_only":
        I = colreduce(W, reduce="max", dtype=dtype)
    elif mode == "wa":
        Wq = prequantize(W, dtype, d, base_idx, iters)
        I = colreduce(W, Wq, scale=h.astype(np.float64), reduce="max", dtype=dtype)
    else:
        raise ValueError(mode)
    return round_to(I, F32)


def residual_books(minuend: np.ndarray, codes: List[np.ndarray], books: List[np.ndarray], m_dtype: str,
                   book_dtypes: List[str]) -> np.ndarray:
    """ComputeError over several books: E = minuend - sum_b C_b[q_b] (fp64, book order), rounded to float32."""
    Mv = widen(minuend, m_dtype).astype(np.float64)
    R = reconstruct(codes, books, np.zeros(len(codes[0]), np.uint8), book_dtypes, n_full=len(books))
    return (Mv - R).astype(np.float32)


def quantize_layer(W: np.ndarray, X: np.ndarray, dtype: str, d: int, K_base: int, K_ext: List[int],
                   crit_frac: float, width: int, iters: int, base_idx: np.ndarray,
                   ext_idx: List[np.ndarray], importance: str = "energy", m_base: int = 1,
                   base_idx_extra: List[np.ndarray] = (), damp: float = 0.01) -> LayerResult:
    M, N = W.shape
    h = round_to(colreduce(X, reduce="sum"), F32)
    H = gram(X) if importance == "obs" else None
    I = channel_importance(W, h, dtype, importance, d, base_idx, iters, H, damp)
    perm = rank_perm(I)
    Ws = gather_columns(W, perm)
    n_crit = n_crit_columns(N, d, crit_frac)
    V = vectors(Ws, d)
    objs: Dict[str, List[float]] = {}

    C_base, q_base, _, J = kmeans(V, np.ascontiguousarray(V[base_idx]), iters, dtype, dtype)
    objs["base"] = J
    C_basic, q_basic, basic_dt = [C_base], [q_base], [dtype]
    if m_base > 1:
        # further basic books on the residual of every vector, then the beam over the basic books
        Eall = residual(V, q_base, C_base, dtype, dtype)
        for b in range(1, m_base):
            Cb, qb, _, J = kmeans(Eall, np.ascontiguousarray(Eall[base_idx_extra[b - 1]]), iters, F32, F32)
            objs[f"base{b + 1}"] = J
            C_basic.append(Cb)
            q_basic.append(qb)
            basic_dt.append(F32)
            if b + 1 < m_base:
                Eall = residual(Eall, qb, Cb, F32, F32)
        q_basic, _ = beam(V, C_basic, width, dtype, basic_dt)
        q_base = q_basic[0]

    Vc = vectors(crit_slab(Ws, n_crit), d)
    crit_vec_idx = np.flatnonzero(crit_mask(M, N, d, n_crit))
    if m_base == 1:
        E = residual(Vc, q_base[crit_vec_idx], C_base, dtype, dtype)
    else:
        E = residual_books(Vc, [q[crit_vec_idx] for q in q_basic], C_basic, dtype, basic_dt)
    C_ext = []
    for t in range(1, len(K_ext) + 1):
        Ct, qt, _, J = kmeans(E, np.ascontiguousarray(E[ext_idx[t - 1]]), iters, F32, F32)
        objs[f"ext{t}"] = J
        objs[f"ext{t}_in"] = [float(np.sum(E.astype(np.float64) ** 2))]
        C_ext.append(Ct)
        if t < len(K_ext):
            E = residual(E, qt, Ct, F32, F32)

    books = C_basic + C_ext
    bdt = basic_dt + [F32] * len(C_ext)
    codes_b, err = beam(Vc, books, width, dtype, bdt)
    codes_basic = [q.copy() for q in q_basic]
    for b in range(m_base):
        codes_basic[b][crit_vec_idx] = codes_b[b]
    codes_ext = [codes_b[t] for t in range(m_base, len(books))]

    # reconstruction in sorted order (basic books on every vector, extended ones on the critical
    # groups), then reverse reordering
    n = M * N // d
    cm = crit_mask(M, N, d, n_crit)
    full_codes = codes_basic + [np.zeros(n, np.int32) for _ in C_ext]
    for t in range(len(C_ext)):
        full_codes[m_base + t][crit_vec_idx] = codes_ext[t]
    R = reconstruct(full_codes, books, cm, bdt, n_full=m_base)
    Rs = round_to(R, dtype).reshape(M, N)
    W_hat = scatter_columns(Rs, perm)
    return LayerResult(h, I, perm, n_crit, C_base, C_ext, codes_basic[0], codes_ext, err, W_hat, objs, C_basic,
                       codes_basic)


def frob_err(W: np.ndarray, W_hat: np.ndarray, dtype: str) -> float:
    a = widen(W, dtype).astype(np.float64)
    b = widen(W_hat, dtype).astype(np.float64)
    return float(np.sum((a - b) ** 2))
