"""Lockstep parity on the five benchmark workloads at their full sizes.

The GPU pipeline (`LayerQuantizer.run`, the product path) runs one layer; a hook re-computes every
library call on the CPU oracle from the GPU's own inputs (byte-identical), and compares:
  * perm, residuals, reconstruction: exactly (bitwise);
  * codes: exactly, except within 1e-6 relative distance ties; dist / beam error: bitwise (float of
    the same fp64 distance);
  * importance, Hessian diagonal: 1e-5 relative; centroids: 1e-5 (fp32) / 1e-2 (bf16) per d-vector,
    empty clusters unchanged bitwise.
Where the oracle would take minutes (K = 65536 assignments of millions of vectors), it checks a
seeded sample of rows at every call; everything else is checked in full."""
import zlib

import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline as opipe
from paper_2412_09282_amd import inputs
from paper_2412_09282_amd.pipeline import LayerConfig, LayerQuantizer

from gpu_util import check_codes, rel_close, say, to_host_bits

pytestmark = pytest.mark.gpu


def host(t):
    return to_host_bits(t)


class Lockstep:
    def __init__(self, wl, li, W, X, dtype, assign_sample, rows_sample):
        self.wl, self.li, self.W, self.X, self.dtype = wl, li, W, X, dtype
        self.d = wl.d
        self.assign_sample = assign_sample
        self.rows_sample = rows_sample
        self.snap = {}
        self.stats = {"calls": 0, "codes_checked": 0, "tie_substitutions": 0}
        self.Ws = None

    def sample(self, n, k, salt):
        g = np.random.default_rng([inputs.ROOT_SEED, self.wl.wid, self.li, salt])
        return np.sort(g.choice(n, size=min(n, k), replace=False))

    # ---------------------------------------------------------------------------------------------
    def pre(self, name, kw):
        if name.startswith("assign"):
            self.snap = {"C": host(kw["C"]), "X": kw["X"]}
        elif name.startswith("update"):
            self.snap = {"C": host(kw["C"]), "codes": host(kw["codes"]), "X": kw["X"]}
        elif name.startswith("residual"):
            self.snap = {"minuend": host(kw["minuend"]), "codes": host(kw["codes"]).ravel(), "book": host(kw["book"])}
        elif name == "beam":
            self.snap = {"books": [host(b) for b in kw["books"]]}
        elif name == "dequant":
            self.snap = {"codes": host(kw["codes"]), "codes_ext": [host(c) for c in kw["codes_ext"]],
                         "books": [host(b) for b in kw["books"]], "perm": host(kw["perm"])}
        elif name == "importance":
            self.snap = {"scale": host(kw["scale"])}
        elif name == "reorder":
            self.snap = {"importance": host(kw["importance"])}
        else:
            self.snap = {}

    def post(self, name, kw):
        torch.cuda.synchronize()
        self.stats["calls"] += 1
        d = self.d
        if name == "hdiag":
            rel_close(host(kw["out"]), oracle.colreduce(self.X), 1e-5, "hdiag")
        elif name == "importance":
            exp = oracle.colreduce(self.W, scale=self.snap["scale"].astype(np.float64), dtype=self.dtype)
            rel_close(host(kw["out"]), exp, 1e-5, "importance")
        elif name == "reorder":
            perm = host(kw["perm"])
            np.testing.assert_array_equal(perm, oracle.rank_perm(self.snap["importance"]))
            self.Ws = host(kw["out"])
            rows = self.sample(self.W.shape[0], self.rows_sample, 1)
            np.testing.assert_array_equal(self.Ws[rows], self.W[rows][:, perm])
        elif name.startswith("assign"):
            Xh = self.Ws if name.startswith("assign_base") else host(self.snap["X"])
            vdt = self.dtype if name.startswith("assign_base") else "f32"
            cdt = vdt
            V = oracle.vectors(np.ascontiguousarray(Xh), d)
            S = self.sample(V.shape[0], self.assign_sample, zlib.crc32(name.encode()) % 1000)
            exp, edist = oracle.assign(V[S], self.snap["C"], vdt, cdt)
            got = host(kw["codes"])[S]
            self.stats["tie_substitutions"] += check_codes(V[S], self.snap["C"], got, exp, vdt, cdt, name)
            self.stats["codes_checked"] += len(S)
            if "dist" in kw:
                np.testing.assert_array_equal(host(kw["dist"])[S], edist.astype(np.float32))
        elif name.startswith("update"):
            base = name.startswith("update_base")
            Xh = self.Ws if base else host(self.snap["X"])
            dt = self.dtype if base else "f32"
            V = oracle.vectors(np.ascontiguousarray(Xh), d)
            Cexp, cnt, _ = oracle.kmeans_update(V, self.snap["codes"], self.snap["C"], dt, dt)
            got = host(kw["C"])
            rel_close(oracle.widen(got, dt), oracle.widen(Cexp, dt), 1e-5 if dt == "f32" else 1e-2, name, axis_vec=True)
            np.testing.assert_array_equal(got[cnt == 0], self.snap["C"][cnt == 0])
        elif name.startswith("residual"):
            mdt = self.dtype if name == "residual_base" else "f32"
            Mv = oracle.vectors(np.ascontiguousarray(self.snap["minuend"]), d)
            exp = oracle.residual(Mv, self.snap["codes"], self.snap["book"], mdt, mdt)
            np.testing.assert_array_equal(oracle.vectors(host(kw["out"]), d), exp)
        elif name == "beam":
            M, N = self.W.shape
            n_crit = oracle.n_crit_columns(N, d, self.wl.crit_frac)
            Vc = oracle.vectors(np.ascontiguousarray(self.Ws[:, :n_crit]), d)
            S = self.sample(Vc.shape[0], self.assign_sample, 77)
            books = self.snap["books"]
            bdt = [self.dtype] + ["f32"] * (len(books) - 1)
            exp_codes, exp_err = oracle.beam(Vc[S], books, self.wl.beam, self.dtype, bdt)
            got = [host(kw["codes_base"]).ravel()[S]] + [host(c)[S] for c in kw["codes_ext"]]
            got = np.stack(got)
            bad = np.flatnonzero((got != exp_codes).any(0))
            if len(bad):
                R = oracle.reconstruct([g for g in got[:, bad]], books, np.ones(len(bad), np.uint8), bdt)
                e_got = ((oracle.widen(Vc[S][bad], self.dtype).astype(np.float64) - R) ** 2).sum(1)
                assert (e_got <= exp_err[bad] * (1 + 1e-6)).all(), f"beam: {len(bad)} tuples differ beyond ties"
            self.stats["tie_substitutions"] += len(bad)
            self.stats["codes_checked"] += len(S)
            ok = np.setdiff1d(np.arange(len(S)), bad)
            np.testing.assert_array_equal(host(kw["err"])[S][ok], exp_err[ok].astype(np.float32))
        elif name == "dequant":
            M, N = self.W.shape
            n_crit = oracle.n_crit_columns(N, d, self.wl.crit_frac)
            ncv, vpr = n_crit // d, N // d
            rows = self.sample(M, self.rows_sample, 3)
            books = self.snap["books"]
            bdt = [self.dtype] + ["f32"] * (len(books) - 1)
            qb = self.snap["codes"].reshape(M, vpr)[rows].ravel()
            qe = []
            for c in self.snap["codes_ext"]:
                z = np.zeros((len(rows), vpr), np.int32)
                z[:, :ncv] = c.reshape(M, ncv)[rows]
                qe.append(z.ravel())
            crit = opipe.crit_mask(len(rows), N, d, n_crit)
            R = oracle.reconstruct([qb] + qe, books, crit, bdt)
            Rs = oracle.round_to(R, self.dtype).reshape(len(rows), N)
            exp = oracle.scatter_columns(Rs, self.snap["perm"])
            np.testing.assert_array_equal(host(kw["out"])[rows], exp)


def run_layer(wid, li, assign_sample=4096, rows_sample=256):
    wl = inputs.WORKLOADS[wid]
    L = wl.layers[li]
    say(f"workload {wid} layer {li} ({L.name} {L.M}x{L.N} {L.dtype}): generating")
    W = inputs.make_weight(wl, li)
    X = inputs.make_calib(wl, li)
    d = wl.d
    n = L.M * L.N // d
    n_crit = inputs.n_crit_columns(L.N, d, wl.crit_frac)
    base_idx = inputs.base_init_indices(wl, li, n)
    ext_idx = [inputs.ext_init_indices(wl, li, t, L.M * n_crit // d) for t in range(1, len(wl.K_ext) + 1)]
    tdt = torch.bfloat16 if L.dtype == "bf16" else torch.float32
    if L.dtype == "bf16":
        Wd = torch.from_numpy(W.view(np.int16)).view(torch.bfloat16).cuda()
    else:
        Wd = torch.from_numpy(W).cuda()
    cfg = LayerConfig(d, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters)
    q = LayerQuantizer(L.M, L.N, tdt, cfg, L.tokens)
    chk = Lockstep(wl, li, W, X, L.dtype, assign_sample, rows_sample)
    say(f"workload {wid} layer {li}: running with lockstep checks")
    q.run(Wd, torch.from_numpy(X).cuda(), torch.from_numpy(base_idx).cuda(),
          [torch.from_numpy(e).cuda() for e in ext_idx], hooks=[chk])
    torch.cuda.synchronize()
    say(f"workload {wid} layer {li}: {chk.stats}")
    return chk.stats


def test_workload1_full_and_end_to_end():
    """Workload 1 is small enough to compare every call in full and the whole result with the
    oracle's own run of the same seeds."""
    st = run_layer(1, 0, assign_sample=10 ** 9, rows_sample=10 ** 9)
    assert st["calls"] > 20
    wl = inputs.WORKLOADS[1]
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    n_crit = inputs.n_crit_columns(256, 8, wl.crit_frac)
    ref = opipe.quantize_layer(W, X, "f32", 8, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters,
                               inputs.base_init_indices(wl, 0, 8192),
                               [inputs.ext_init_indices(wl, 0, 1, 256 * n_crit // 8)])
    cfg = LayerConfig(8, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters)
    q = LayerQuantizer(256, 256, torch.float32, cfg, 512)
    out = q.run(torch.from_numpy(W).cuda(), torch.from_numpy(X).cuda(),
                torch.from_numpy(inputs.base_init_indices(wl, 0, 8192)).cuda(),
                [torch.from_numpy(inputs.ext_init_indices(wl, 0, 1, 256)).cuda()])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.perm.cpu().numpy(), ref.perm)
    np.testing.assert_array_equal(out.codes_base.cpu().numpy(), ref.codes_base)
    np.testing.assert_array_equal(out.W_hat.cpu().numpy(), ref.W_hat)


@pytest.mark.parametrize("wid,li", [(2, 0), (3, 0), (4, 0)] + [(5, i) for i in range(7)])
def test_workload_lockstep(wid, li):
    st = run_layer(wid, li)
    assert st["calls"] > 5
