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
  channel and changes no ordering, so it is left out;
* critical channels: the first d * ceil(lambda N / d) reordered columns;
* K-means: initial codewords are the vectors at seeded indices (an input);
  one iteration = assign + update; ``iters`` iterations then a final assign;
  an empty cluster keeps its centroid;
* residuals are rounded to float32 when they are stored (E^t);
* the final codes of critical vectors come from the beam search (width 1 =
  greedy) over [basic, ext_1, ...] on the un-rounded (fp64) residual.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from . import (F32, BF16, assign, beam, colreduce, gather_columns, kmeans_update, n_crit_columns,
               objective, rank_perm, reconstruct, residual, round_to, scatter_columns, vectors, widen)


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
                       base_idx: Optional[np.ndarray] = None, iters: int = 1) -> np.ndarray:
    """Channel importance of Sec. 4.1 (modes as in the module notes), rounded to float32."""
    if mode == "energy":
        I = colreduce(W, scale=h.astype(np.float64), reduce="sum", dtype=dtype)
    elif mode == "w_only":
        I = colreduce(W, reduce="max", dtype=dtype)
    elif mode == "wa":
        Wq = prequantize(W, dtype, d, base_idx, iters)
        I = colreduce(W, Wq, scale=h.astype(np.float64), reduce="max", dtype=dtype)
    else:
        raise ValueError(mode)
    return round_to(I, F32)


def quantize_layer(W: np.ndarray, X: np.ndarray, dtype: str, d: int, K_base: int, K_ext: List[int],
                   crit_frac: float, width: int, iters: int, base_idx: np.ndarray,
                   ext_idx: List[np.ndarray], importance: str = "energy") -> LayerResult:
    M, N = W.shape
    h = round_to(colreduce(X, reduce="sum"), F32)
    I = channel_importance(W, h, dtype, importance, d, base_idx, iters)
    perm = rank_perm(I)
    Ws = gather_columns(W, perm)
    n_crit = n_crit_columns(N, d, crit_frac)
    V = vectors(Ws, d)
    objs: Dict[str, List[float]] = {}

    C_base, q_base, _, J = kmeans(V, np.ascontiguousarray(V[base_idx]), iters, dtype, dtype)
    objs["base"] = J

    Vc = vectors(crit_slab(Ws, n_crit), d)
    crit_vec_idx = np.flatnonzero(crit_mask(M, N, d, n_crit))
    E = residual(Vc, q_base[crit_vec_idx], C_base, dtype, dtype)
    C_ext = []
    for t in range(1, len(K_ext) + 1):
        Ct, qt, _, J = kmeans(E, np.ascontiguousarray(E[ext_idx[t - 1]]), iters, F32, F32)
        objs[f"ext{t}"] = J
        objs[f"ext{t}_in"] = [float(np.sum(E.astype(np.float64) ** 2))]
        C_ext.append(Ct)
        if t < len(K_ext):
            E = residual(E, qt, Ct, F32, F32)

    books = [C_base] + C_ext
    bdt = [dtype] + [F32] * len(C_ext)
    codes_b, err = beam(Vc, books, width, dtype, bdt)
    codes_base = q_base.copy()
    codes_base[crit_vec_idx] = codes_b[0]
    codes_ext = [codes_b[t] for t in range(1, len(books))]

    # reconstruction in sorted order, then reverse reordering
    full_codes = [codes_base] + [np.zeros(M * N // d, np.int32) for _ in C_ext]
    for t in range(len(C_ext)):
        full_codes[t + 1][crit_vec_idx] = codes_ext[t]
    R = reconstruct(full_codes, books, crit_mask(M, N, d, n_crit), bdt)
    Rs = round_to(R, dtype).reshape(M, N)
    W_hat = scatter_columns(Rs, perm)
    return LayerResult(h, I, perm, n_crit, C_base, C_ext, codes_base, codes_ext, err, W_hat, objs)


def frob_err(W: np.ndarray, W_hat: np.ndarray, dtype: str) -> float:
    a = widen(W, dtype).astype(np.float64)
    b = widen(W_hat, dtype).astype(np.float64)
    return float(np.sum((a - b) ** 2))
