"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module only draws random numbers and lays them out; it holds none of the
quantization method's arithmetic.  Random choices the method makes (the K-means
initial codewords) are drawn here as index arrays and handed to both the GPU
path and the oracle, so the two see byte-identical inputs.

Every stream comes from ``numpy.random.Generator(PCG64(SeedSequence([241209282,
workload, layer, stream])))`` with the stream ids below.  The shapes and value
distributions stand in for the paper's LLaMA / OPT linear layers and its
RedPajama calibration activations (the paper's Sec. 5.1 setting), which are not
available here.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

ROOT_SEED = 241209282

S_W = 0          # weight matrix
S_X = 1          # calibration activations
S_XSCALE = 2     # per-channel activation scales / outlier columns
S_INIT_BASE = 3  # basic-codebook initial codeword indices
S_INIT_EXT = 4   # extended codebook t uses stream S_INIT_EXT + t - 1
S_SAMPLE = 9     # rows sampled for oracle checks on large layers
S_INIT_BASE_EXTRA = 10  # basic codebook b >= 1 (layouts with m_base > 1 basic books) uses stream 10 + b - 1


def rng(workload: int, layer: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, workload, layer, stream])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even) and return the bit patterns.

    Storage conversion for inputs that are specified as bf16 data; NaN is not expected."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class LayerSpec:
    name: str
    M: int                 # output rows of W
    N: int                 # input channels (columns) of W
    tokens: int            # calibration rows of X (tokens x N)
    dtype: str             # "f32" or "bf16" storage of W and the basic codebook
    w_dist: str            # "normal" or "t4_outliers"
    x_dist: str            # "normal" or "normal_scaled"


@dataclasses.dataclass
class Workload:
    wid: int
    name: str
    layers: List[LayerSpec]
    d: int
    K_base: int
    K_ext: List[int]        # one entry per extended codebook
    crit_frac: float        # lambda, fraction of input channels treated as critical
    beam: int
    iters: int              # Lloyd iterations per codebook (each = assign + update), then a final assign
    m_base: int = 1         # basic codebooks covering every vector (2 in the m = 2, d = 16 setting)


W_STD = 0.02


def _w(L: LayerSpec, wid: int, li: int) -> np.ndarray:
    g = rng(wid, li, S_W)
    if L.w_dist == "normal":
        W = g.standard_normal((L.M, L.N), dtype=np.float32) * np.float32(W_STD)
    elif L.w_dist == "t4_outliers":
        W = (g.standard_t(4.0, size=(L.M, L.N)) * W_STD).astype(np.float32)
        n_out = int(round(0.01 * L.N))
        cols = rng(wid, li, S_XSCALE).choice(L.N, size=n_out, replace=False)
        W[:, cols] *= np.float32(10.0)
    else:
        raise ValueError(L.w_dist)
    return W


def outlier_columns(wid: int, li: int, N: int) -> np.ndarray:
    n_out = int(round(0.01 * N))
    return np.sort(rng(wid, li, S_XSCALE).choice(N, size=n_out, replace=False))


def _x(L: LayerSpec, wid: int, li: int) -> np.ndarray:
    g = rng(wid, li, S_X)
    X = g.standard_normal((L.tokens, L.N), dtype=np.float32)
    if L.x_dist == "normal_scaled":
        s = np.power(10.0, rng(wid, li, S_XSCALE).uniform(-1.0, 1.0, size=L.N)).astype(np.float32)
        X *= s[None, :]
    return X


def make_weight(wl: Workload, li: int) -> np.ndarray:
    """W (M x N).  float32 array, or uint16 bf16 bit patterns for bf16 layers."""
    L = wl.layers[li]
    W = _w(L, wl.wid, li)
    return f32_to_bf16_bits(W) if L.dtype == "bf16" else W


def make_calib(wl: Workload, li: int) -> np.ndarray:
    """Calibration activations X (tokens x N), float32."""
    return _x(wl.layers[li], wl.wid, li)


def init_indices(n: int, K: int, g: np.random.Generator) -> np.ndarray:
    """K distinct vector indices drawn without replacement; if K > n, all n in random order, cycled."""
    if K <= n:
        return g.choice(n, size=K, replace=False).astype(np.int64)
    p = g.permutation(n).astype(np.int64)
    return np.resize(p, K)


def base_init_indices(wl: Workload, li: int, n: int) -> np.ndarray:
    return init_indices(n, wl.K_base, rng(wl.wid, li, S_INIT_BASE))


def extra_base_init_indices(wl: Workload, li: int, b: int, n: int) -> np.ndarray:
    """Indices for basic codebook b (b = 1 .. m_base-1) into the residual vectors of the whole layer."""
    return init_indices(n, wl.K_base, rng(wl.wid, li, S_INIT_BASE_EXTRA + b - 1))


def ext_init_indices(wl: Workload, li: int, t: int, n_crit_vec: int) -> np.ndarray:
    """Indices for extended codebook t (t = 1 .. m-1) into the critical residual vectors."""
    return init_indices(n_crit_vec, wl.K_ext[t - 1], rng(wl.wid, li, S_INIT_EXT + t - 1))


def sample_rows(wl: Workload, li: int, n: int, k: int) -> np.ndarray:
    k = min(k, n)
    return np.sort(rng(wl.wid, li, S_SAMPLE).choice(n, size=k, replace=False)).astype(np.int64)


def n_crit_columns(N: int, d: int, frac: float) -> int:
    """Critical input channels: the smallest multiple of d that covers frac * N, at most N."""
    return min(N, d * int(math.ceil(frac * N / d - 1e-9)))


WORKLOADS = {
    1: Workload(1, "toy 256x256 fp32, K=256 + 1 ext K=256 on top 2%, T=10",
                [LayerSpec("toy", 256, 256, 512, "f32", "normal", "normal")],
                d=8, K_base=256, K_ext=[256], crit_frac=0.02, beam=1, iters=10),
    2: Workload(2, "LLaMA-7B attention projection 4096x4096 fp32, K=65536 + 1 ext K=256 on top 3%",
                [LayerSpec("attn", 4096, 4096, 2048, "f32", "normal", "normal_scaled")],
                d=8, K_base=65536, K_ext=[256], crit_frac=0.03, beam=1, iters=1),
    3: Workload(3, "LLaMA-7B MLP up-projection 11008x4096 fp32, K=256 + 2 ext K=256 on top 5%, beam 8, T=20",
                [LayerSpec("up", 11008, 4096, 2048, "f32", "normal", "normal_scaled")],
                d=8, K_base=256, K_ext=[256, 256], crit_frac=0.05, beam=8, iters=20),
    4: Workload(4, "70B MLP projection 28672x8192 fp32 t4 + outliers, K=65536 + 1 ext K=65536 on top 2%",
                [LayerSpec("mlp70b", 28672, 8192, 1024, "f32", "t4_outliers", "normal")],
                d=8, K_base=65536, K_ext=[65536], crit_frac=0.02, beam=1, iters=1),
    5: Workload(5, "13B transformer block, 7 bf16 linears, K=65536 + 1 ext K=256 on top 5%, beam 4, T=20",
                [LayerSpec("q", 5120, 5120, 2048, "bf16", "normal", "normal"),
                 LayerSpec("k", 5120, 5120, 2048, "bf16", "normal", "normal"),
                 LayerSpec("v", 5120, 5120, 2048, "bf16", "normal", "normal"),
                 LayerSpec("o", 5120, 5120, 2048, "bf16", "normal", "normal"),
                 LayerSpec("gate", 13824, 5120, 2048, "bf16", "normal", "normal"),
                 LayerSpec("up", 13824, 5120, 2048, "bf16", "normal", "normal"),
                 LayerSpec("down", 5120, 13824, 2048, "bf16", "normal", "normal")],
                d=8, K_base=65536, K_ext=[256], crit_frac=0.05, beam=4, iters=20),
}


# Codebook-layout variants of Sec. 3.2 / Sec. 6.4 on the LLaMA-7B attention projection shape (the weights
# and activations of workload 2): e = 8 with three extended books (8+8x3), two basic books on d = 16
# vectors (m = 2) with three extended books, and wider basic books (e = 10, 12) with one extended book.
VARIANT_WORKLOADS = {
    21: Workload(2, "LLaMA-7B attention 4096x4096 fp32, 8+8x3: K=256 + 3 ext K=256 on top 2%",
                 [LayerSpec("attn", 4096, 4096, 2048, "f32", "normal", "normal_scaled")],
                 d=8, K_base=256, K_ext=[256, 256, 256], crit_frac=0.02, beam=1, iters=1),
    22: Workload(2, "LLaMA-7B attention 4096x4096 fp32, m=2 d=16: 2 basic K=256 + 3 ext K=256 on top 2%",
                 [LayerSpec("attn", 4096, 4096, 2048, "f32", "normal", "normal_scaled")],
                 d=16, K_base=256, K_ext=[256, 256, 256], crit_frac=0.02, beam=1, iters=1, m_base=2),
    23: Workload(2, "LLaMA-7B attention 4096x4096 fp32, e=10: K=1024 + 1 ext K=256 on top 2%",
                 [LayerSpec("attn", 4096, 4096, 2048, "f32", "normal", "normal_scaled")],
                 d=8, K_base=1024, K_ext=[256], crit_frac=0.02, beam=1, iters=1),
    24: Workload(2, "LLaMA-7B attention 4096x4096 fp32, e=12: K=4096 + 1 ext K=256 on top 2%",
                 [LayerSpec("attn", 4096, 4096, 2048, "f32", "normal", "normal_scaled")],
                 d=8, K_base=4096, K_ext=[256], crit_frac=0.02, beam=1, iters=1),
}


def workload(wid: int) -> Workload:
    """A timed workload (1-5) or a codebook-layout variant (21-24)."""
    return WORKLOADS[wid] if wid in WORKLOADS else VARIANT_WORKLOADS[wid]


def small_workload(M: int = 64, N: int = 64, tokens: int = 96, d: int = 8, K_base: int = 32,
                   K_ext: Sequence[int] = (16,), crit_frac: float = 0.1, beam: int = 2, iters: int = 3,
                   dtype: str = "f32", wid: int = 100, m_base: int = 1) -> Workload:
    """A tiny workload of the same structure, for fast parity and pin tests."""
    return Workload(wid, f"small {M}x{N}", [LayerSpec("small", M, N, tokens, dtype, "normal", "normal_scaled")],
                    d=d, K_base=K_base, K_ext=list(K_ext), crit_frac=crit_frac, beam=beam, iters=iters,
                    m_base=m_base)


def random_vectors(n: int, d: int, seed: int, scale: float = 0.02) -> np.ndarray:
    return (rng(999, seed, 0).standard_normal((n, d), dtype=np.float32) * np.float32(scale))
