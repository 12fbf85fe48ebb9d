"""Loss-driven refinement of a quantized layer on the CPU oracle -- TEST INFRASTRUCTURE ONLY.

The loop that follows the codebook fitting in Alg. 1 (QuantLoss / FineTuneCodebook /
BeamSearchOptimize), in plain fp64 numpy.  Everything here works in the reordered (sorted) channel
order of the layer, where the critical channels are the first n_crit columns.

Notation (the paper writes W X with X of shape in-channels x tokens; the calibration activations
here are stored tokens x N, so the paper's X is ``X.T``):
  H = X^T X                                     (N x N, the paper's X X^T)
  R = W - W_hat                                 (M x N)
  QuantLoss = ||W X^T - W_hat X^T||_F^2 = sum_r R_r H R_r^T
  dL/dW_hat = -2 R H, so the gradient for codeword k of book b is the sum of -2 (R H)_v over the
  vectors v that book b covers and codes with k.

Readings where the paper is silent (each also listed in the design notes):
* FineTuneCodebook: ``steps`` full-batch Adam steps (Kingma & Ba, Algorithm 1 with bias correction;
  beta = (0.9, 0.95) as the paper's training setting, eps = 1e-8) on all codebooks at once, codes
  fixed, the gradient taken on the whole layer objective (H replaces the paper's mini-batches).
  Codebooks are fp32; Adam state m, v and the update are fp64, the new codeword is rounded to fp32.
* BeamSearchOptimize at the paper's width 1: books in order; for each book, the groups it covers in
  column order; for each row independently the code of that group becomes the one that minimises
  QuantLoss with every other code fixed (lowest index among equal losses).  The loss change of
  candidate k is -2 delta_k . (R H)_g + delta_k^T H_gg delta_k with delta_k = C[k] - C[current].
* The loop: while QuantLoss >= eps and fewer than ``max_rounds`` rounds ran: FineTuneCodebook, then
  BeamSearchOptimize over every book.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

from . import BF16, F32, reconstruct, round_to, widen


def gram(X: np.ndarray, x_dtype: str = F32) -> np.ndarray:
    """H = X^T X in fp64 for activations X stored tokens x N (the paper's X X^T, Appendix A.2)."""
    X64 = widen(np.asarray(X), x_dtype).astype(np.float64)
    return X64.T @ X64


def quant_loss(W: np.ndarray, W_hat: np.ndarray, X: np.ndarray, w_dtype: str = F32, x_dtype: str = F32) -> float:
    """QuantLoss of Alg. 1 by its definition: ||W X^T - W_hat X^T||_F^2 in fp64 (a float64 W_hat is
    taken as it is, e.g. the exact codeword sums)."""
    X64 = widen(np.asarray(X), x_dtype).astype(np.float64)
    Wh = W_hat if W_hat.dtype == np.float64 else widen(W_hat, w_dtype).astype(np.float64)
    D = widen(W, w_dtype).astype(np.float64) - Wh
    Y = D @ X64.T
    return float(np.sum(Y * Y))


def layout_codes(M: int, N: int, d: int, n_crit: int, codes: Sequence[np.ndarray], n_base: int) -> List[np.ndarray]:
    """Per-vector code arrays of every book (extended books' codes placed on the critical groups,
    zero elsewhere), the layout ``reconstruct`` takes."""
    vpr, ncv = N // d, n_crit // d
    full = [np.asarray(c, dtype=np.int32).ravel() for c in codes[:n_base]]
    for c in codes[n_base:]:
        z = np.zeros((M, vpr), np.int32)
        z[:, :ncv] = np.asarray(c, dtype=np.int32).reshape(M, ncv)
        full.append(z.ravel())
    return full


def crit_flags(M: int, N: int, d: int, n_crit: int) -> np.ndarray:
    g = np.arange(N // d)
    return np.broadcast_to(g < n_crit // d, (M, N // d)).reshape(-1).astype(np.uint8)


def residual_f64(Ws: np.ndarray, w_dtype: str, d: int, n_crit: int, codes: Sequence[np.ndarray],
                 books: Sequence[np.ndarray], book_dtypes: Sequence[str], n_base: int) -> np.ndarray:
    """R = W_s - W_hat_s in fp64 (sorted order): the exact codeword sums subtracted from W."""
    M, N = Ws.shape
    full = layout_codes(M, N, d, n_crit, codes, n_base)
    Rhat = reconstruct(full, books, crit_flags(M, N, d, n_crit), book_dtypes, n_full=n_base)
    return widen(Ws, w_dtype).astype(np.float64) - Rhat.reshape(M, N)


def codebook_grads(R: np.ndarray, H: np.ndarray, d: int, n_crit: int, codes: Sequence[np.ndarray],
                   Ks: Sequence[int], n_base: int):
    """Gradient of QuantLoss w.r.t. every codebook, codes fixed: -2 (R H) summed per code over the
    vectors each book covers.  Returns (grads [K_b x d fp64], loss)."""
    M, N = R.shape
    G = R @ H
    loss = float(np.sum(R * G))
    Gv = (-2.0 * G).reshape(M, N // d, d)
    grads = []
    for b, K in enumerate(Ks):
        cover = N // d if b < n_base else n_crit // d
        gb = np.zeros((K, d))
        q = np.asarray(codes[b], dtype=np.int64).reshape(M, cover)
        np.add.at(gb, q.ravel(), Gv[:, :cover, :].reshape(-1, d))
        grads.append(gb)
    return grads, loss


@dataclasses.dataclass
class AdamState:
    m: np.ndarray
    v: np.ndarray
    t: int = 0


def adam_step(C: np.ndarray, g: np.ndarray, st: AdamState, lr: float, beta1: float = 0.9, beta2: float = 0.95,
              eps: float = 1e-8) -> np.ndarray:
    """One step of Adam (Kingma & Ba, Algorithm 1): moments in fp64 with bias correction; the fp32
    codebook C moves by -lr * m_hat / (sqrt(v_hat) + eps), rounded once to fp32."""
    st.t += 1
    st.m = beta1 * st.m + (1.0 - beta1) * g
    st.v = beta2 * st.v + (1.0 - beta2) * (g * g)
    m_hat = st.m / (1.0 - beta1 ** st.t)
    v_hat = st.v / (1.0 - beta2 ** st.t)
    return (C.astype(np.float64) - lr * m_hat / (np.sqrt(v_hat) + eps)).astype(np.float32)


def refine_book(R: np.ndarray, H: np.ndarray, C: np.ndarray, codes: np.ndarray, d: int, n_cols: int,
                c_dtype: str = F32):
    """BeamSearchOptimize at width 1 for one book covering columns [0, n_cols): for every group in
    column order and every row, the code that minimises QuantLoss with the other codes fixed.
    R (M x N fp64) and codes (M x n_cols/d) are updated in place; returns the number of changes."""
    M, N = R.shape
    Cb = widen(C, c_dtype).astype(np.float64)
    q = codes.reshape(M, n_cols // d)
    rows = np.arange(M)
    changes = 0
    for g in range(n_cols // d):
        cols = slice(g * d, (g + 1) * d)
        s = R @ H[:, cols]                           # (R H)_g, M x d, from the current R
        Hgg = H[cols, cols]
        delta = Cb[None, :, :] - Cb[q[:, g]][:, None, :]          # M x K x d
        dL = -2.0 * np.einsum("mkt,mt->mk", delta, s) + np.einsum("mkt,tu,mku->mk", delta, Hgg, delta)
        k_new = np.argmin(dL, axis=1)                # lowest index among equal values
        moved = k_new != q[:, g]
        changes += int(moved.sum())
        R[:, cols] -= Cb[k_new] - Cb[q[:, g]]
        q[rows, g] = k_new
    return changes


@dataclasses.dataclass
class RefineResult:
    books: List[np.ndarray]
    codes: List[np.ndarray]
    losses: List[float]          # QuantLoss before the loop and after every round
    rounds: int
    changes: List[int]


def refine_layer(Ws: np.ndarray, Xs: np.ndarray, d: int, n_crit: int, books: Sequence[np.ndarray],
                 codes: Sequence[np.ndarray], n_base: int, lr: float, steps: int, max_rounds: int,
                 eps: float = 0.0, beta1: float = 0.9, beta2: float = 0.95, adam_eps: float = 1e-8,
                 w_dtype: str = F32) -> RefineResult:
    """The refinement loop of Alg. 1 on one layer in sorted order: while QuantLoss >= eps and rounds <
    max_rounds, ``steps`` Adam steps on the codebooks, then a width-1 code search over every book in
    order.  The first basic book has the layer's type (``w_dtype``), the others are fp32.

    Reading for bf16 layers (the paper fine-tunes a half-precision model without saying how): a bf16
    book is tuned through an fp32 master copy, set from the book when the loop starts; Adam moves the
    master exactly as it moves an fp32 book, and after every step the book is the master rounded to
    bf16 (nearest-even), which QuantLoss, the gradients and the code search then use."""
    M, N = Ws.shape
    dts = [w_dtype] + [F32] * (len(books) - 1)
    books = [np.asarray(b, dtype=np.uint16 if t == BF16 else np.float32).copy() for b, t in zip(books, dts)]
    masters = [widen(b, t).astype(np.float32) if t == BF16 else None for b, t in zip(books, dts)]
    codes = [np.asarray(c, dtype=np.int32).copy() for c in codes]
    H = gram(Xs)
    Ks = [b.shape[0] for b in books]
    adam = [AdamState(np.zeros(b.shape), np.zeros(b.shape)) for b in books]
    R = residual_f64(Ws, w_dtype, d, n_crit, codes, books, dts, n_base)
    losses = [float(np.sum(R * (R @ H)))]
    changes = []
    rounds = 0
    while losses[-1] >= eps and rounds < max_rounds:
        for _ in range(steps):
            grads, _ = codebook_grads(R, H, d, n_crit, codes, Ks, n_base)
            for b in range(len(books)):
                if dts[b] == BF16:
                    masters[b] = adam_step(masters[b], grads[b], adam[b], lr, beta1, beta2, adam_eps)
                    books[b] = round_to(masters[b].astype(np.float64), BF16)
                else:
                    books[b] = adam_step(books[b], grads[b], adam[b], lr, beta1, beta2, adam_eps)
            R = residual_f64(Ws, w_dtype, d, n_crit, codes, books, dts, n_base)
        ch = 0
        for b in range(len(books)):
            n_cols = N if b < n_base else n_crit
            ch += refine_book(R, H, books[b], codes[b], d, n_cols, dts[b])
        R = residual_f64(Ws, w_dtype, d, n_crit, codes, books, dts, n_base)
        changes.append(ch)
        losses.append(float(np.sum(R * (R @ H))))
        rounds += 1
    return RefineResult(books, codes, losses, rounds, changes)
