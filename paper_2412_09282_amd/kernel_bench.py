"""Per-call timings of the library against its roofline, on one layer shape.

    python -m paper_2412_09282_amd.kernel_bench [--workload 4] [--reps 10] [--skip-assign] [--calibrate-copy]

Times every library call of the path with HIP events (median of --reps after warm-up) on the
workload's first layer and prints one JSON object per call with the algorithmic bytes (or flops)
of one call, the achieved rate and its fraction of the MI355X peak (HBM 8 TB/s; the d <= 8
nearest-codeword screen contracts split operands on the 16-bit matrix cores, 2.5 PFLOP/s dense).  Between repetitions of an HBM-bound call a 1 GiB buffer is overwritten so the
256 MiB last-level cache holds none of its data.
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np
import torch

from . import crvq as C
from . import inputs
from .crvq import VecSet

HBM_GBS = 8000.0
F16_MFMA_TFLOPS = 2500.0


def timed(fn, reps, flush=None):
    ts = []
    for r in range(reps + 2):
        if flush is not None:
            flush.fill_(r)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        if r >= 2:
            ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def report(name, ms, nbytes=None, flops=None, peak_tflops=F16_MFMA_TFLOPS, **extra):
    out = {"call": name, "ms": round(ms, 4)}
    if nbytes is not None:
        gbs = nbytes / (ms * 1e-3) / 1e9
        out.update({"bound": "hbm", "bytes": int(nbytes), "GB/s": round(gbs, 1), "frac": round(gbs / HBM_GBS, 4)})
    if flops is not None:
        tf = flops / (ms * 1e-3) / 1e12
        out.update({"bound": "mfma", "flop": int(flops), "TFLOP/s": round(tf, 2), "frac": round(tf / peak_tflops, 4),
                    "peak_tflops": peak_tflops})
    out.update(extra)
    print(json.dumps(out), flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, default=4)
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--skip-assign", action="store_true")
    ap.add_argument("--hinv", action="store_true",
                    help="also time the Eq. 7 pieces: the fp64 proxy and the diagonal of its damped inverse")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="start with a plain 1 GiB device-to-device copy (the reference for HBM counters)")
    a = ap.parse_args(argv)
    if a.calibrate_copy:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    wl = inputs.WORKLOADS[a.workload]
    L = wl.layers[0]
    M, N, d = L.M, L.N, wl.d
    n = M * N // d
    es = 2 if L.dtype == "bf16" else 4
    tdt = torch.bfloat16 if L.dtype == "bf16" else torch.float32
    print(f"[kernel_bench] workload {a.workload}: {L.name} {M}x{N} {L.dtype}, generating", file=sys.stderr, flush=True)
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    Wd = torch.from_numpy(W.view(np.int16)).view(torch.bfloat16).cuda() if L.dtype == "bf16" else torch.from_numpy(W).cuda()
    Xd = torch.from_numpy(X).cuda()
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB

    h = torch.empty(N, dtype=torch.float32, device="cuda")
    ms = timed(lambda: C.crvq_channel_importance(Xd, h), a.reps, flush)
    report("crvq_channel_importance (Hessian diagonal, X tokens x N)", ms, nbytes=X.size * 4 + N * 4, shape=[L.tokens, N])
    if a.hinv:
        # Eq. 7's denominator: the fp64 proxy H = X^T X, then the diagonal of its damped inverse
        H = torch.empty(N, N, dtype=torch.float64, device="cuda")
        ms = timed(lambda: C.crvq_gram(Xd, H), max(2, a.reps // 5), flush)
        report("crvq_gram (H = X^T X, fp64)", ms, flops=2.0 * L.tokens * N * N, peak_tflops=78.6, shape=[L.tokens, N])
        sc = torch.empty(N, dtype=torch.float32, device="cuda")
        ms = timed(lambda: C.crvq_hessian_inverse_diagonal(H, scale=sc, damp=0.01), max(2, a.reps // 5), flush)
        report("crvq_hessian_inverse_diagonal (fp64 Cholesky + inverse factor)", ms, flops=2.0 * N ** 3 / 3,
               peak_tflops=78.6, N=N)
        del H
    imp = torch.empty(N, dtype=torch.float32, device="cuda")
    ms = timed(lambda: C.crvq_channel_importance(Wd, imp, scale=h), a.reps, flush)
    report("crvq_channel_importance (W, scale = h)", ms, nbytes=M * N * es + 2 * N * 4, shape=[M, N])

    perm = torch.empty(N, dtype=torch.int32, device="cuda")
    Ws = torch.empty_like(Wd)
    ms = timed(lambda: C.crvq_reorder(None, None, perm, importance=imp), a.reps)
    report("crvq_reorder (rank sort only)", ms, N=N)
    C.crvq_reorder(None, None, perm, importance=imp)
    ms = timed(lambda: C.crvq_reorder(Wd, Ws, perm), a.reps, flush)
    report("crvq_reorder (column gather)", ms, nbytes=2 * M * N * es + N * 4, shape=[M, N])

    V = VecSet.of_matrix(Ws, d)
    K = wl.K_base
    idx = torch.from_numpy(inputs.base_init_indices(wl, 0, n)).cuda()
    Cb = torch.empty(K, d, dtype=tdt, device="cuda")
    C.crvq_gather_vectors(V, idx, Cb)
    codes = torch.empty(n, dtype=torch.int32, device="cuda")
    if not a.skip_assign:
        dist = torch.empty(n, dtype=torch.float32, device="cuda")
        ms = timed(lambda: C.crvq_assign(V, Cb, codes, dist), max(2, a.reps // 5))
        report("crvq_assign", ms, flops=2.0 * K * d * n, n=n, K=K)
    else:
        g = np.random.default_rng(0)
        codes.copy_(torch.from_numpy(g.integers(0, K, n).astype(np.int32)))
    C0 = Cb.clone()

    def upd():
        Cb.copy_(C0)
        C.crvq_kmeans_update(V, codes, Cb)
    t_copy = timed(lambda: Cb.copy_(C0), a.reps)
    ms = timed(upd, a.reps, flush) - t_copy
    report("crvq_kmeans_update", ms, nbytes=(d * es + 4) * n + K * d * es + 4 * K, n=n, K=K)

    n_crit = inputs.n_crit_columns(N, d, wl.crit_frac)
    # residual beam over the critical vectors: the basic book plus the workload's extended books
    # (residual-scale random codewords standing in for fitted ones), width wl.beam
    ncv = M * n_crit // d
    Vc = VecSet.of_matrix(Ws, d, n_cols=n_crit)
    # extended books initialised like the pipeline's: residual vectors of the critical slab drawn by
    # the workload's own seeded indices (the residual after the basic book for every extended book)
    Eb = torch.empty(M, n_crit, dtype=torch.float32, device="cuda")
    C.crvq_dequant(M, n_crit, d, codes, N // d, Cb, Eb, minuend=Ws)
    VE = VecSet.of_matrix(Eb, d)
    ext = []
    for t, Ke in enumerate(wl.K_ext):
        Ct = torch.empty(Ke, d, dtype=torch.float32, device="cuda")
        C.crvq_gather_vectors(VE, torch.from_numpy(inputs.ext_init_indices(wl, 0, t + 1, ncv)).cuda(), Ct)
        ext.append(Ct)
    books = [Cb] + ext
    bcodes = [torch.empty(ncv, dtype=torch.int32, device="cuda") for _ in books]
    berr = torch.empty(ncv, dtype=torch.float32, device="cuda")
    flops, width = 0.0, 1
    for Kt in [K] + list(wl.K_ext):  # step t screens min(beam, prod K before t) parents x K_t codewords
        flops += 2.0 * d * width * Kt
        width = min(wl.beam, width * Kt)
    if not a.skip_assign:
        ms = timed(lambda: C.crvq_assign_residual_beam(Vc, books, wl.beam, bcodes, berr), max(2, a.reps // 5))
        report("crvq_assign_residual_beam", ms, flops=flops * ncv, n=ncv, beam=wl.beam, K=[K] + list(wl.K_ext))
    E = torch.empty(M, n_crit, dtype=torch.float32, device="cuda")
    ms = timed(lambda: C.crvq_dequant(M, n_crit, d, codes, N // d, Cb, E, minuend=Ws), a.reps, flush)
    report("crvq_dequant (residual of the critical slab)", ms,
           nbytes=M * n_crit * (es + 4) + 4 * M * n_crit // d + K * d * es, shape=[M, n_crit])
    What = torch.empty_like(Wd)
    Ce = torch.zeros(wl.K_ext[0], d, dtype=torch.float32, device="cuda")
    qe = torch.zeros(M * n_crit // d, dtype=torch.int32, device="cuda")
    ms = timed(lambda: C.crvq_dequant(M, N, d, codes, N // d, Cb, What, n_crit=n_crit, q_ext=[qe], ldq_ext=n_crit // d,
                                      C_ext=[Ce], perm=perm), a.reps, flush)
    report("crvq_dequant (reconstruction + reverse reorder)", ms,
           nbytes=M * N * es + 4 * n + 4 * M * n_crit // d + (K + wl.K_ext[0]) * d * es + N * 4, shape=[M, N])


if __name__ == "__main__":
    main()
