"""CRVQ per-layer quantization on the GPU, as a sequence of libcrvq calls.

The order follows Alg. 1 of the paper for one weight matrix:
ComputeImportance -> ReorderChannels -> KMeansCodebook + VectorQuant (basic)
-> for every extended codebook: ComputeError, KMeansCodebook, VectorQuant,
Update on the critical groups -> beam search over all codebooks for the
critical vectors -> reconstruction with the reverse reordering.

Readings where the paper leaves a choice open (shared with the design notes):
importance (LayerConfig.importance): "energy" I_j = h_j * sum_i W_ij^2 with
h = diag(X X^T) (the timed workloads), "w_only" I_j = max_i W_ij^2 (Sec. 4.1),
"wa" I_j = h_j * max_i (W_ij - Wq_ij)^2 with Wq the prequantized W (Alg. 1
Prequantize: the basic VQ of the unsorted W; the Hessian-proxy metric of
Sec. 4.1 in the unpacked form of Appendix A.2 Eq. 10 without its uniform
factor 1/2), "obs" Eq. 7 as printed, I_j = max_i (W_ij - Wq_ij)^2 /
(2 [(X X^T)^-1]_jj), the inverse taken of H + damp * mean(diag H) * I; the critical channels
are the first d * ceil(lambda N / d) reordered columns; K-means starts from the
vectors at given indices, one iteration is assign + update, `iters` iterations
are followed by a final assign, an empty cluster keeps its centroid; stored
residuals are float32; the critical vectors' final codes come from the beam
search (width 1 = greedy) on the exact residual.  With m_base > 1 basic books
(the m = 2, d = 16 setting of Sec. 3.2 / Sec. 6.4) basic book b >= 1 (fp32) is
fitted on the residual of every vector after books < b, the beam over the basic
books then codes every vector, and the extended books are fitted on the
critical residual after those codes.

Every arithmetic step runs in the library's kernels; this module only
allocates device tensors and sequences the calls.  Hooks see the device
tensors right around every call; passing `trace` (a list) records host copies
of every call's inputs and outputs, so a test can re-run each call from the
same bytes.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import torch

from . import crvq as C
from .crvq import VecSet


@dataclasses.dataclass
class LayerConfig:
    d: int
    K_base: int
    K_ext: List[int]
    crit_frac: float
    beam: int
    iters: int
    importance: str = "energy"  # "energy" | "w_only" | "wa" | "obs"
    m_base: int = 1             # basic codebooks covering every vector (2 in the m = 2, d = 16 setting)
    damp: float = 0.01          # "obs": the inverse is taken of H + damp * mean(diag H) * I


def n_crit_columns(N: int, d: int, frac: float) -> int:
    return min(N, d * int(math.ceil(frac * N / d - 1e-9)))


@dataclasses.dataclass
class LayerState:
    hdiag: torch.Tensor
    importance: torch.Tensor
    perm: torch.Tensor
    Ws: torch.Tensor
    n_crit: int
    C_base: torch.Tensor
    C_ext: List[torch.Tensor]
    codes_base: torch.Tensor     # [M * N/d]; critical entries hold the beam's basic codes at the end
    codes_ext: List[torch.Tensor]  # [M * n_crit/d] per extended book
    beam_err: torch.Tensor       # [M * n_crit/d]
    W_hat: torch.Tensor
    C_basic: List[torch.Tensor] = dataclasses.field(default_factory=list)      # all m_base basic books
    codes_basic: List[torch.Tensor] = dataclasses.field(default_factory=list)  # their codes [M * N/d]


class LayerQuantizer:
    """Holds the device buffers for one layer shape so repeated runs allocate nothing new."""

    def __init__(self, M: int, N: int, dtype: torch.dtype, cfg: LayerConfig, tokens: int, device="cuda"):
        d = cfg.d
        assert N % d == 0
        self.M, self.N, self.dtype, self.cfg, self.device = M, N, dtype, cfg, device
        self.n = M * N // d
        self.n_crit = n_crit_columns(N, d, cfg.crit_frac)
        self.ncv = self.n_crit // d
        f32, i32 = torch.float32, torch.int32
        self.hdiag = torch.empty(N, dtype=f32, device=device)
        self.imp = torch.empty(N, dtype=f32, device=device)
        self.perm = torch.empty(N, dtype=i32, device=device)
        self.Ws = torch.empty(M, N, dtype=dtype, device=device)
        self.C_base = torch.empty(cfg.K_base, d, dtype=dtype, device=device)
        self.codes = torch.empty(self.n, dtype=i32, device=device)
        self.dist = torch.empty(self.n, dtype=f32, device=device)
        self.E = [torch.empty(M, self.n_crit, dtype=f32, device=device) for _ in range(2)]
        self.C_ext = [torch.empty(K, d, dtype=f32, device=device) for K in cfg.K_ext]
        self.q_ext_fit = torch.empty(M * self.ncv, dtype=i32, device=device)
        self.codes_ext = [torch.empty(M * self.ncv, dtype=i32, device=device) for _ in cfg.K_ext]
        self.beam_err = torch.empty(M * self.ncv, dtype=f32, device=device)
        self.W_hat = torch.empty(M, N, dtype=dtype, device=device)
        if cfg.m_base < 1 or cfg.m_base + len(cfg.K_ext) > 8:
            raise ValueError(f"m_base {cfg.m_base} with {len(cfg.K_ext)} extended books")
        # basic books after the first are fp32, like the residual they are fitted on
        self.C_basic = [self.C_base] + [torch.empty(cfg.K_base, d, dtype=f32, device=device)
                                        for _ in range(cfg.m_base - 1)]
        self.codes_basic = [self.codes] + [torch.empty(self.n, dtype=i32, device=device)
                                           for _ in range(cfg.m_base - 1)]
        if cfg.m_base > 1:
            self.E_all = [torch.empty(M, N, dtype=f32, device=device) for _ in range(min(2, cfg.m_base - 1))]
        if cfg.importance not in ("energy", "w_only", "wa", "obs"):
            raise ValueError(f"importance {cfg.importance!r}")
        if cfg.importance in ("wa", "obs"):  # Prequantize buffers: the basic VQ of the unsorted W
            self.C_pre = torch.empty(cfg.K_base, d, dtype=dtype, device=device)
            self.codes_pre = torch.empty(self.n, dtype=i32, device=device)
            self.W_pre = torch.empty(M, N, dtype=dtype, device=device)
        if cfg.importance == "obs":  # Eq. 7: the Hessian proxy and its inverse's diagonal
            self.H = torch.empty(N, N, dtype=torch.float64, device=device)
            self.obs_scale = torch.empty(N, dtype=f32, device=device)

    def run(self, W: torch.Tensor, X: torch.Tensor, base_idx: torch.Tensor, ext_idx: List[torch.Tensor],
            trace: Optional[list] = None, hooks=(), base_idx_extra: Sequence[torch.Tensor] = ()) -> LayerState:
        """hooks: objects with pre(name, inputs) / post(name, outputs), called right around each library
        call; trace: a list that receives host copies of every call's inputs and outputs;
        base_idx_extra: initial-codeword indices of basic books 2 .. m_base."""
        cfg, d, M, N = self.cfg, self.cfg.d, self.M, self.N
        hooks = list(hooks) + ([TraceHook(trace)] if trace is not None else [])
        rec = _Recorder(hooks)

        rec.pre("hdiag", A=X)
        C.crvq_channel_importance(X, self.hdiag)
        rec.post("hdiag", out=self.hdiag)

        if cfg.importance == "energy":
            rec.pre("importance", A=W, scale=self.hdiag)
            C.crvq_channel_importance(W, self.imp, scale=self.hdiag)
        elif cfg.importance == "w_only":
            rec.pre("importance", A=W)
            C.crvq_channel_importance(W, self.imp, reduce=C.CRVQ_REDUCE_MAX)
        else:
            # Alg. 1 Prequantize: K-means + final assign + reconstruction of the unsorted W
            Vu = VecSet.of_matrix(W, d)
            C.crvq_gather_vectors(Vu, base_idx, self.C_pre)
            self._kmeans(Vu, self.C_pre, self.codes_pre, rec, "pre")
            rec.pre("assign_pre_final", X=W, C=self.C_pre)
            C.crvq_assign(Vu, self.C_pre, self.codes_pre)
            rec.post("assign_pre_final", codes=self.codes_pre)
            rec.pre("prequant", codes=self.codes_pre, book=self.C_pre)
            C.crvq_dequant(M, N, d, self.codes_pre, N // d, self.C_pre, self.W_pre)
            rec.post("prequant", out=self.W_pre)
            scale = self.hdiag
            if cfg.importance == "obs":
                rec.pre("gram", X=X)
                C.crvq_gram(X, self.H)
                rec.post("gram", H=self.H)
                rec.pre("hinv", H=self.H)
                C.crvq_hessian_inverse_diagonal(self.H, scale=self.obs_scale, damp=cfg.damp)
                rec.post("hinv", scale=self.obs_scale)
                scale = self.obs_scale
            rec.pre("importance", A=W, B=self.W_pre, scale=scale)
            C.crvq_channel_importance(W, self.imp, B=self.W_pre, scale=scale, reduce=C.CRVQ_REDUCE_MAX)
        rec.post("importance", out=self.imp)

        rec.pre("reorder", inp=W, importance=self.imp)
        C.crvq_reorder(W, self.Ws, self.perm, importance=self.imp)
        rec.post("reorder", perm=self.perm, out=self.Ws)

        V = VecSet.of_matrix(self.Ws, d)
        C.crvq_gather_vectors(V, base_idx, self.C_base)
        self._kmeans(V, self.C_base, self.codes, rec, "base")
        rec.pre("assign_base_final", X=self.Ws, C=self.C_base)
        C.crvq_assign(V, self.C_base, self.codes, self.dist)
        rec.post("assign_base_final", codes=self.codes, dist=self.dist)
        mb = cfg.m_base
        if mb > 1:
            # further basic books on the residual of every vector, then the beam over the basic books
            prev, src = (self.codes, self.C_base), self.Ws
            for b in range(1, mb):
                Eb = self.E_all[(b - 1) % 2]
                rec.pre(f"residual_all{b}", minuend=src, codes=prev[0], book=prev[1])
                C.crvq_dequant(M, N, d, prev[0], N // d, prev[1], Eb, minuend=src)
                rec.post(f"residual_all{b}", out=Eb)
                VE = VecSet.of_matrix(Eb, d)
                Cb, qb = self.C_basic[b], self.codes_basic[b]
                C.crvq_gather_vectors(VE, base_idx_extra[b - 1], Cb)
                self._kmeans(VE, Cb, qb, rec, f"base{b + 1}")
                rec.pre(f"assign_base{b + 1}_final", X=Eb, C=Cb)
                C.crvq_assign(VE, Cb, qb)
                rec.post(f"assign_base{b + 1}_final", codes=qb)
                prev, src = (qb, Cb), Eb
            rec.pre("beam_basic", X=self.Ws, books=self.C_basic, beam=cfg.beam)
            C.crvq_assign_residual_beam(V, self.C_basic, cfg.beam, self.codes_basic, None)
            rec.post("beam_basic", codes=list(self.codes_basic))

        # residual of the critical slab after the basic codebook(s) (Alg. 1 ComputeError)
        cur = 0
        if self.n_crit > 0:
            crit_codes = [q.view(M, N // d)[:, :self.ncv] for q in self.codes_basic]
            rec.pre("residual_base", minuend=self.Ws[:, :self.n_crit], codes=crit_codes[0] if mb == 1 else crit_codes,
                    book=self.C_base if mb == 1 else self.C_basic)
            C.crvq_dequant_books(M, self.n_crit, d, self.codes_basic, N // d, self.C_basic, self.E[cur],
                                 minuend=self.Ws)
            rec.post("residual_base", out=self.E[cur])
            for t, Ct in enumerate(self.C_ext):
                VE = VecSet.of_matrix(self.E[cur], d)
                C.crvq_gather_vectors(VE, ext_idx[t], Ct)
                self._kmeans(VE, Ct, self.q_ext_fit, rec, f"ext{t + 1}")
                rec.pre(f"assign_ext{t + 1}_final", X=self.E[cur], C=Ct)
                C.crvq_assign(VE, Ct, self.q_ext_fit)
                rec.post(f"assign_ext{t + 1}_final", codes=self.q_ext_fit)
                if t + 1 < len(self.C_ext):
                    rec.pre(f"residual_ext{t + 1}", minuend=self.E[cur], codes=self.q_ext_fit, book=Ct)
                    C.crvq_dequant(M, self.n_crit, d, self.q_ext_fit, self.ncv, Ct, self.E[cur ^ 1],
                                   minuend=self.E[cur])
                    rec.post(f"residual_ext{t + 1}", out=self.E[cur ^ 1])
                    cur ^= 1

            # beam over all books for the critical vectors; basic codes land in the full code arrays
            Vc = VecSet.of_matrix(self.Ws, d, self.n_crit)
            books = self.C_basic + self.C_ext
            rec.pre("beam", X=self.Ws[:, :self.n_crit], books=books, beam=cfg.beam)
            C.crvq_assign_residual_beam(Vc, books, cfg.beam, self.codes_basic + self.codes_ext, self.beam_err,
                                        ldc=[N // d] * mb + [self.ncv] * len(self.C_ext))
            rec.post("beam", codes_base=self.codes.view(M, N // d)[:, :self.ncv],
                     codes_basic=[q.view(M, N // d)[:, :self.ncv] for q in self.codes_basic],
                     codes_ext=list(self.codes_ext), err=self.beam_err)

        rec.pre("dequant", codes=self.codes, codes_basic=list(self.codes_basic), codes_ext=list(self.codes_ext),
                books=self.C_basic + self.C_ext, perm=self.perm)
        C.crvq_dequant_books(M, N, d, self.codes_basic, N // d, self.C_basic, self.W_hat, n_crit=self.n_crit,
                             q_ext=self.codes_ext, ldq_ext=self.ncv, C_ext=self.C_ext, perm=self.perm)
        rec.post("dequant", out=self.W_hat)

        return LayerState(self.hdiag, self.imp, self.perm, self.Ws, self.n_crit, self.C_base, self.C_ext, self.codes,
                          self.codes_ext, self.beam_err, self.W_hat, self.C_basic, self.codes_basic)

    def refine(self, X: torch.Tensor, rounds: int, steps: int, lr: float, eps: float = 0.0, beta1: float = 0.9,
               beta2: float = 0.95, adam_eps: float = 1e-8, trace: Optional[list] = None, hooks=()) -> List[float]:
        """The loss-driven refinement of Alg. 1 after run(): while QuantLoss >= eps and fewer than `rounds`
        rounds ran, `steps` Adam steps on every codebook (codes fixed), then the width-1 QuantLoss code
        search over every book in order.  Works in reordered channel order on the codebooks and codes
        run() left; a bf16 book (the first basic book of a bf16 layer) is tuned through an fp32 master
        copy and re-rounded after every step.  Rebuilds W_hat at the end.  Returns QuantLoss before the
        loop and after every round."""
        cfg, d, M, N = self.cfg, self.cfg.d, self.M, self.N
        hooks = list(hooks) + ([TraceHook(trace)] if trace is not None else [])
        rec = _Recorder(hooks)
        f64 = torch.float64
        dev = self.W_hat.device
        if not hasattr(self, "H"):
            self.H = torch.empty(N, N, dtype=f64, device=dev)
            self.Xs = torch.empty(X.shape[0], N, dtype=torch.float32, device=dev)
            self.R = torch.empty(M, N, dtype=f64, device=dev)
            self.G = torch.empty(M, N, dtype=f64, device=dev)
            self.row_loss = torch.empty(M, dtype=f64, device=dev)
            self.loss_total = torch.empty(1, dtype=f64, device=dev)
        books = self.C_basic + self.C_ext
        codes = self.codes_basic + self.codes_ext
        mb = cfg.m_base
        cover = [N] * mb + [self.n_crit] * len(self.C_ext)
        ldq = [N // d] * mb + [max(1, self.ncv)] * len(self.C_ext)
        sums = [torch.empty(b.shape[0], d, dtype=f64, device=dev) for b in books]
        moments = [(torch.zeros(b.shape[0], d, dtype=f64, device=dev), torch.zeros(b.shape[0], d, dtype=f64, device=dev))
                   for b in books]
        masters = [torch.empty(b.shape[0], d, dtype=torch.float32, device=dev) if b.dtype == torch.bfloat16 else None
                   for b in books]

        rec.pre("gram", X=X, perm=self.perm)
        C.crvq_reorder(X, self.Xs, self.perm)
        C.crvq_gram(self.Xs, self.H)
        rec.post("gram", Xs=self.Xs, H=self.H)

        def loss_now(tag):
            rec.pre(f"residual_{tag}", minuend=self.Ws, codes=list(codes), books=list(books))
            C.crvq_dequant_books(M, N, d, codes[:mb], N // d, books[:mb], self.R, n_crit=self.n_crit, q_ext=codes[mb:],
                                 ldq_ext=max(1, self.ncv), C_ext=books[mb:], minuend=self.Ws)
            rec.post(f"residual_{tag}", out=self.R)
            rec.pre(f"hessian_{tag}", R=self.R, H=self.H)
            C.crvq_hessian_product(self.R, self.H, self.G, self.row_loss, self.loss_total)
            rec.post(f"hessian_{tag}", G=self.G, row_loss=self.row_loss, loss_total=self.loss_total)

        def loss_value():
            # the only host read of the loop: QuantLoss for the guard, once per round
            return float(self.loss_total.item())

        loss_now("start")
        losses = [loss_value()]
        t = 0
        r = 0
        while losses[-1] >= eps and r < rounds:
            for s_ in range(steps):
                t += 1
                for b, Cb in enumerate(books):
                    Vg = VecSet.of_matrix(self.G, d, cover[b])
                    rec.pre(f"code_sums_{r}_{s_}_{b}", X=self.G[:, :cover[b]], codes=codes[b], K=Cb.shape[0])
                    C.crvq_code_sums(Vg, codes[b], Cb.shape[0], sums[b])
                    rec.post(f"code_sums_{r}_{s_}_{b}", sums=sums[b])
                    if masters[b] is not None:
                        rec.pre(f"adam_{r}_{s_}_{b}", C=Cb, master=masters[b], grad=sums[b], m=moments[b][0],
                                v=moments[b][1], step=t)
                        C.crvq_adam_step_bf16(Cb, masters[b], sums[b], -2.0, moments[b][0], moments[b][1], t, lr, beta1,
                                              beta2, adam_eps)
                        rec.post(f"adam_{r}_{s_}_{b}", C=Cb, master=masters[b], m=moments[b][0], v=moments[b][1])
                    else:
                        rec.pre(f"adam_{r}_{s_}_{b}", C=Cb, grad=sums[b], m=moments[b][0], v=moments[b][1], step=t)
                        C.crvq_adam_step(Cb, sums[b], -2.0, moments[b][0], moments[b][1], t, lr, beta1, beta2,
                                         adam_eps)
                        rec.post(f"adam_{r}_{s_}_{b}", C=Cb, m=moments[b][0], v=moments[b][1])
                loss_now(f"{r}_{s_}")
            for b, Cb in enumerate(books):
                rec.pre(f"refine_{r}_{b}", R=self.R, H=self.H, C=Cb, codes=codes[b], n_cols=cover[b])
                C.crvq_refine_codes(self.R, self.H, Cb, codes[b], d, cover[b], ldq[b])
                rec.post(f"refine_{r}_{b}", R=self.R, codes=codes[b])
            loss_now(f"round{r}")
            losses.append(loss_value())
            r += 1
        C.crvq_dequant_books(M, N, d, codes[:mb], N // d, books[:mb], self.W_hat, n_crit=self.n_crit,
                             q_ext=codes[mb:], ldq_ext=max(1, self.ncv), C_ext=books[mb:], perm=self.perm)
        return losses

    def _kmeans(self, V: VecSet, Cb: torch.Tensor, codes: torch.Tensor, rec, tag: str):
        for it in range(self.cfg.iters):
            rec.pre(f"assign_{tag}_{it}", X=V.t, C=Cb)
            C.crvq_assign(V, Cb, codes)
            rec.post(f"assign_{tag}_{it}", codes=codes)
            rec.pre(f"update_{tag}_{it}", X=V.t, codes=codes, C=Cb)
            C.crvq_kmeans_update(V, codes, Cb)
            rec.post(f"update_{tag}_{it}", C=Cb)


class TraceHook:
    """Copies the inputs and outputs of every call to the host, in call order."""

    def __init__(self, trace: list):
        self.trace = trace
        self.cur: Dict = {}

    @staticmethod
    def _host(v):
        if isinstance(v, torch.Tensor):
            return v.detach().to("cpu", copy=True)
        if isinstance(v, (list, tuple)):
            return [TraceHook._host(x) for x in v]
        return v

    def pre(self, name: str, kw: Dict):
        self.cur = {"name": name, "in": {k: self._host(v) for k, v in kw.items()}}

    def post(self, name: str, kw: Dict):
        self.cur["out"] = {k: self._host(v) for k, v in kw.items()}
        self.trace.append(self.cur)
        self.cur = {}


class _Recorder:
    """Calls every hook's pre(name, inputs) right before and post(name, outputs) right after each
    library call (inputs/outputs are the device tensors involved)."""

    def __init__(self, hooks):
        self.hooks = list(hooks)

    def pre(self, name: str, **kw):
        for h in self.hooks:
            h.pre(name, kw)

    def post(self, name: str, **kw):
        for h in reversed(self.hooks):
            h.post(name, kw)
