"""ctypes binding of libcrvq.so -- argument marshalling only.

Every function below has the name of the C entry point it wraps (include/crvq.h)
and does nothing but turn torch tensors into device pointers, sizes and dtype
codes, allocate the scratch workspace the C call asks for (torch's caching
allocator), pass the current HIP stream, and raise on a nonzero status.  All
computation happens in the library's HIP kernels.  If the library cannot be
loaded, every call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import threading
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcrvq.so")
_lock = threading.Lock()
_lib = None

CRVQ_F32, CRVQ_BF16, CRVQ_F64 = 0, 1, 2
CRVQ_REDUCE_SUM, CRVQ_REDUCE_MAX = 0, 1
STATUS = {0: "CRVQ_OK", 1: "CRVQ_ERR_INVALID", 2: "CRVQ_ERR_UNSUPPORTED", 3: "CRVQ_ERR_WORKSPACE", 4: "CRVQ_ERR_HIP"}


class CrvqError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: {STATUS.get(status, status)}: {msg}")
        self.status = status


def lib(build_if_missing: bool = True):
    """Load libcrvq.so (building it first only if no built library exists)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                if not build_if_missing:
                    raise OSError(f"{LIB_PATH} is not built")
                from . import build as _build
                _build.build(verbose=False)
            L = ctypes.CDLL(LIB_PATH)
            P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
            PP = ctypes.POINTER(ctypes.c_void_p)
            sigs = {
                "crvq_version": ([], ctypes.c_int),
                "crvq_last_error": ([], ctypes.c_char_p),
                "crvq_importance_workspace_size": ([I64, I64], SZ),
                "crvq_channel_importance": ([P, I64, P, I64, ctypes.c_int, I64, I64, P, ctypes.c_int, P, P, SZ, P], ctypes.c_int),
                "crvq_reorder_workspace_size": ([I64], SZ),
                "crvq_reorder": ([P, I64, P, I64, ctypes.c_int, I64, I64, P, P, ctypes.c_int, P, SZ, P], ctypes.c_int),
                "crvq_assign_workspace_size": ([I64, I32, I64], SZ),
                "crvq_assign": ([P, ctypes.c_int, I64, I64, I64, I32, P, ctypes.c_int, I64, P, P, P, SZ, P], ctypes.c_int),
                "crvq_assign_noalloc": ([P, ctypes.c_int, I64, I64, I64, I32, P, ctypes.c_int, I64, P, P, P],
                                        ctypes.c_int),
                "crvq_beam_workspace_size": ([I64, I32, I32, P, I32], SZ),
                "crvq_assign_residual_beam": ([P, ctypes.c_int, I64, I64, I64, I32, I32, PP, P, P, I32, PP, P, P, P, SZ, P],
                                              ctypes.c_int),
                "crvq_kmeans_workspace_size": ([I64, I32, I64], SZ),
                "crvq_kmeans_update": ([P, ctypes.c_int, I64, I64, I64, I32, P, I64, P, ctypes.c_int, P, P, SZ, P], ctypes.c_int),
                "crvq_gather_vectors": ([P, ctypes.c_int, I64, I64, I64, I32, P, I64, P, ctypes.c_int, P], ctypes.c_int),
                "crvq_dequant_workspace_size": ([I64], SZ),
                "crvq_dequant": ([I64, I64, I32, I64, P, I64, P, ctypes.c_int, I64, I32, PP, I64, PP, P, P, P, P, ctypes.c_int,
                                  I64, P, ctypes.c_int, I64, P, SZ, P], ctypes.c_int),
                "crvq_dequant_books": ([I64, I64, I32, I64, I32, I32, PP, I64, I64, PP, P, P, P, P, ctypes.c_int, I64,
                                        P, ctypes.c_int, I64, P, SZ, P], ctypes.c_int),
                "crvq_bits_per_weight": ([I64, I64, I32, I64, I32, I32, P, I32, I32, P], ctypes.c_int),
                "crvq_gram": ([P, ctypes.c_int, I64, I64, I64, P, I64, P], ctypes.c_int),
                "crvq_hessian_product": ([I64, I64, I64, P, I64, P, I64, P, I64, P, P, P], ctypes.c_int),
                "crvq_hessian_inverse_workspace_size": ([I64], SZ),
                "crvq_hessian_inverse_diagonal": ([P, I64, I64, ctypes.c_double, P, P, P, SZ, P], ctypes.c_int),
                "crvq_workspace_size": ([ctypes.c_int, I64, I64, I32, I32, I32, P, I64, I64, I64], SZ),
                "crvq_code_sums_workspace_size": ([I64, I32, I64], SZ),
                "crvq_code_sums": ([P, I64, I64, I64, I32, P, I64, P, P, P, SZ, P], ctypes.c_int),
                "crvq_adam_step_bf16": ([P, P, P, ctypes.c_double, P, P, I64, I64, ctypes.c_double, ctypes.c_double,
                                         ctypes.c_double, ctypes.c_double, P], ctypes.c_int),
                "crvq_adam_step": ([P, P, ctypes.c_double, P, P, I64, I64, ctypes.c_double, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_double, P], ctypes.c_int),
                "crvq_refine_workspace_size": ([I64, I64, I64], SZ),
                "crvq_refine_codes": ([I64, I64, I32, I64, P, I64, P, I64, P, ctypes.c_int, I64, P, I64, P, SZ, P],
                                      ctypes.c_int),
                "crvq_gemv_workspace_size": ([I64, I64, I64], SZ),
                "crvq_dequant_gemv": ([I64, I64, I64, P, I64, P, ctypes.c_int, I64, I32, PP, I64, PP, P, P, P, P,
                                       ctypes.c_int, P, P, SZ, P], ctypes.c_int),
                "crvq_pack_codes_u8": ([P, I64, P, P], ctypes.c_int),
            }
            for name, (args, res) in sigs.items():
                f = getattr(L, name)
                f.argtypes = args
                f.restype = res
            _lib = L
    return _lib


# ------------------------------------------------------------------------------------------------
# marshalling helpers
# ------------------------------------------------------------------------------------------------

def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return CRVQ_F32
    if t.dtype == torch.bfloat16:
        return CRVQ_BF16
    if t.dtype == torch.float64:
        return CRVQ_F64
    raise TypeError(f"unsupported element type {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(fn: str, status: int):
    if status != 0:
        raise CrvqError(fn, status, lib().crvq_last_error().decode())


def _workspace(nbytes: int, device) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return None
    ws = torch.empty(int(nbytes), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def _ptr_array(ts: Sequence[torch.Tensor]):
    arr = (ctypes.c_void_p * max(1, len(ts)))()
    for i, t in enumerate(ts):
        arr[i] = t.data_ptr()
    return arr


@dataclasses.dataclass
class VecSet:
    """The paper's sub-vector partition (Sec. 3.1 Eq. 1) of a row-major matrix view: n_rows rows of
    vecs_per_row contiguous d-vectors, row stride ld elements."""
    t: torch.Tensor
    n_rows: int
    vecs_per_row: int
    ld: int
    d: int

    @staticmethod
    def of_matrix(W: torch.Tensor, d: int, n_cols: Optional[int] = None) -> "VecSet":
        assert W.dim() == 2 and W.stride(1) == 1
        n_cols = W.shape[1] if n_cols is None else n_cols
        return VecSet(W, W.shape[0], n_cols // d, W.stride(0), d)

    @staticmethod
    def of_vectors(V: torch.Tensor) -> "VecSet":
        assert V.dim() == 2 and V.is_contiguous()
        return VecSet(V, V.shape[0], 1, V.shape[1], V.shape[1])

    @property
    def n(self) -> int:
        return self.n_rows * self.vecs_per_row

    def args(self):
        return (_ptr(self.t), dtype_code(self.t), self.n_rows, self.vecs_per_row, self.ld, self.d)


# ------------------------------------------------------------------------------------------------
# the C entry points
# ------------------------------------------------------------------------------------------------

def crvq_version() -> int:
    return int(lib().crvq_version())


def crvq_channel_importance(A: torch.Tensor, out: torch.Tensor, B: Optional[torch.Tensor] = None,
                            scale: Optional[torch.Tensor] = None, reduce: int = CRVQ_REDUCE_SUM, stream=None) -> None:
    L = lib()
    M, N = A.shape
    assert A.stride(1) == 1 and (B is None or (B.stride(1) == 1 and B.dtype == A.dtype))
    ws = _workspace(L.crvq_importance_workspace_size(M, N), A.device)
    _check("crvq_channel_importance", L.crvq_channel_importance(
        _ptr(A), A.stride(0), _ptr(B), 0 if B is None else B.stride(0), dtype_code(A), M, N, _ptr(scale), reduce,
        _ptr(out), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def crvq_reorder(inp: Optional[torch.Tensor], out: Optional[torch.Tensor], perm: torch.Tensor,
                 importance: Optional[torch.Tensor] = None, inverse: bool = False, stream=None) -> None:
    L = lib()
    N = perm.numel()
    M = 0 if inp is None else inp.shape[0]
    dev = perm.device
    ws = _workspace(L.crvq_reorder_workspace_size(N), dev) if (inverse or importance is not None) else None
    _check("crvq_reorder", L.crvq_reorder(
        _ptr(inp), 0 if inp is None else inp.stride(0), _ptr(out), 0 if out is None else out.stride(0),
        CRVQ_F32 if inp is None else dtype_code(inp), M, N, _ptr(importance), _ptr(perm), int(bool(inverse)),
        _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def crvq_assign(X: VecSet, C: torch.Tensor, codes: torch.Tensor, dist: Optional[torch.Tensor] = None,
                stream=None) -> None:
    L = lib()
    K = C.shape[0]
    ws = _workspace(L.crvq_assign_workspace_size(X.n, X.d, K), C.device)
    _check("crvq_assign", L.crvq_assign(*X.args(), _ptr(C), dtype_code(C), K, _ptr(codes), _ptr(dist), _ptr(ws),
                                        0 if ws is None else ws.numel(), _stream(stream)))


def crvq_assign_noalloc(X: VecSet, C: torch.Tensor, codes: torch.Tensor, dist: Optional[torch.Tensor] = None,
                        stream=None) -> None:
    """crvq_assign on the library's fixed per-GPU scratch: no workspace is allocated."""
    K = C.shape[0]
    _check("crvq_assign_noalloc", lib().crvq_assign_noalloc(*X.args(), _ptr(C), dtype_code(C), K, _ptr(codes),
                                                            _ptr(dist), _stream(stream)))


def crvq_assign_residual_beam(X: VecSet, books: Sequence[torch.Tensor], beam: int, codes: Sequence[torch.Tensor],
                              err: Optional[torch.Tensor] = None, ldc: Optional[Sequence[int]] = None,
                              stream=None) -> None:
    L = lib()
    nb = len(books)
    ldc_arr = None if ldc is None else (ctypes.c_int64 * nb)(*ldc)
    Ks = (ctypes.c_int64 * nb)(*[b.shape[0] for b in books])
    dts = (ctypes.c_int32 * nb)(*[dtype_code(b) for b in books])
    ws = _workspace(L.crvq_beam_workspace_size(X.n, X.d, nb, ctypes.cast(Ks, ctypes.c_void_p), beam), books[0].device)
    _check("crvq_assign_residual_beam", L.crvq_assign_residual_beam(
        *X.args(), nb, ctypes.cast(_ptr_array(books), ctypes.POINTER(ctypes.c_void_p)), ctypes.cast(dts, ctypes.c_void_p),
        ctypes.cast(Ks, ctypes.c_void_p), beam, ctypes.cast(_ptr_array(codes), ctypes.POINTER(ctypes.c_void_p)),
        None if ldc_arr is None else ctypes.cast(ldc_arr, ctypes.c_void_p),
        _ptr(err), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def crvq_kmeans_update(X: VecSet, codes: torch.Tensor, C: torch.Tensor, counts: Optional[torch.Tensor] = None,
                       stream=None) -> None:
    L = lib()
    K = C.shape[0]
    ws = _workspace(L.crvq_kmeans_workspace_size(X.n, X.d, K), C.device)
    _check("crvq_kmeans_update", L.crvq_kmeans_update(*X.args(), _ptr(codes), K, _ptr(C), dtype_code(C), _ptr(counts),
                                                      _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def crvq_gather_vectors(X: VecSet, idx: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    _check("crvq_gather_vectors", lib().crvq_gather_vectors(*X.args(), _ptr(idx), idx.numel(), _ptr(out),
                                                            dtype_code(out), _stream(stream)))


def crvq_dequant(M: int, n_cols: int, d: int, q_base: torch.Tensor, ldq_base: int, C_base: torch.Tensor,
                 out: torch.Tensor, n_crit: int = 0, q_ext: Sequence[torch.Tensor] = (), ldq_ext: int = 0,
                 C_ext: Sequence[torch.Tensor] = (), perm: Optional[torch.Tensor] = None,
                 minuend: Optional[torch.Tensor] = None, stream=None) -> None:
    L = lib()
    ne = len(C_ext)
    ws = _workspace(L.crvq_dequant_workspace_size(n_cols), out.device) if perm is not None else None
    dts = (ctypes.c_int32 * max(1, ne))(*[dtype_code(c) for c in C_ext])
    Ks = (ctypes.c_int64 * max(1, ne))(*[c.shape[0] for c in C_ext])
    _check("crvq_dequant", L.crvq_dequant(
        M, n_cols, d, n_crit, _ptr(q_base), ldq_base, _ptr(C_base), dtype_code(C_base), C_base.shape[0], ne,
        ctypes.cast(_ptr_array(q_ext), ctypes.POINTER(ctypes.c_void_p)) if ne else None, ldq_ext,
        ctypes.cast(_ptr_array(C_ext), ctypes.POINTER(ctypes.c_void_p)) if ne else None,
        ctypes.cast(dts, ctypes.c_void_p) if ne else None, ctypes.cast(Ks, ctypes.c_void_p) if ne else None,
        _ptr(perm), _ptr(minuend), CRVQ_F32 if minuend is None else dtype_code(minuend),
        0 if minuend is None else minuend.stride(0), _ptr(out), dtype_code(out), out.stride(0), _ptr(ws),
        0 if ws is None else ws.numel(), _stream(stream)))


def crvq_dequant_books(M: int, n_cols: int, d: int, q_base: Sequence[torch.Tensor], ldq_base: int,
                       C_base: Sequence[torch.Tensor], out: torch.Tensor, n_crit: int = 0,
                       q_ext: Sequence[torch.Tensor] = (), ldq_ext: int = 0, C_ext: Sequence[torch.Tensor] = (),
                       perm: Optional[torch.Tensor] = None, minuend: Optional[torch.Tensor] = None,
                       stream=None) -> None:
    """crvq_dequant with len(q_base) basic books covering every vector (see include/crvq.h)."""
    L = lib()
    assert len(q_base) == len(C_base) and len(q_ext) == len(C_ext)
    books = list(C_base) + list(C_ext)
    nb = len(books)
    ws = _workspace(L.crvq_dequant_workspace_size(n_cols), out.device) if perm is not None else None
    dts = (ctypes.c_int32 * nb)(*[dtype_code(c) for c in books])
    Ks = (ctypes.c_int64 * nb)(*[c.shape[0] for c in books])
    _check("crvq_dequant_books", L.crvq_dequant_books(
        M, n_cols, d, n_crit, len(C_base), len(C_ext),
        ctypes.cast(_ptr_array(list(q_base) + list(q_ext)), ctypes.POINTER(ctypes.c_void_p)), ldq_base, ldq_ext,
        ctypes.cast(_ptr_array(books), ctypes.POINTER(ctypes.c_void_p)), ctypes.cast(dts, ctypes.c_void_p),
        ctypes.cast(Ks, ctypes.c_void_p), _ptr(perm), _ptr(minuend),
        CRVQ_F32 if minuend is None else dtype_code(minuend), 0 if minuend is None else minuend.stride(0), _ptr(out),
        dtype_code(out), out.stride(0), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def crvq_bits_per_weight(rows: int, cols: int, d: int, n_crit: int, K_base: Sequence[int], K_ext: Sequence[int] = (),
                         codeword_bits: int = 16, perm_bits: int = 16) -> float:
    """Average bits per stored weight of a quantized layer (Eq. 6 / Eq. 8 for the exact layout); host only."""
    Ks = list(K_base) + list(K_ext)
    arr = (ctypes.c_int64 * max(1, len(Ks)))(*Ks)
    out = ctypes.c_double(0.0)
    _check("crvq_bits_per_weight", lib().crvq_bits_per_weight(
        rows, cols, d, n_crit, len(K_base), len(K_ext), ctypes.cast(arr, ctypes.c_void_p), codeword_bits, perm_bits,
        ctypes.byref(out)))
    return out.value


# ---- loss-driven refinement (fp64 operands) -------------------------------------------------------
def crvq_gram(X: torch.Tensor, H: torch.Tensor, stream=None) -> None:
    """H = X^T X (fp64) for activations X stored tokens x N (fp32 or fp64)."""
    assert X.dim() == 2 and X.stride(1) == 1 and H.dtype == torch.float64 and H.stride(1) == 1
    _check("crvq_gram", lib().crvq_gram(_ptr(X), dtype_code(X), X.shape[0], X.shape[1], X.stride(0), _ptr(H),
                                        H.stride(0), _stream(stream)))


def crvq_hessian_inverse_diagonal(H: torch.Tensor, hinv: Optional[torch.Tensor] = None,
                                  scale: Optional[torch.Tensor] = None, damp: float = 0.01, stream=None) -> None:
    """hinv = diag((H + damp * mean(diag H) I)^-1) (fp64) and/or scale = float32(1 / (2 hinv)), the
    factor of the W-A importance of Sec. 4.1 Eq. 7."""
    assert H.dim() == 2 and H.shape[0] == H.shape[1] and H.dtype == torch.float64 and H.stride(1) == 1
    assert hinv is None or (hinv.dtype == torch.float64 and hinv.is_contiguous())
    assert scale is None or (scale.dtype == torch.float32 and scale.is_contiguous())
    L = lib()
    N = H.shape[0]
    ws = _workspace(L.crvq_hessian_inverse_workspace_size(N), H.device)
    _check("crvq_hessian_inverse_diagonal", L.crvq_hessian_inverse_diagonal(
        _ptr(H), H.stride(0), N, float(damp), _ptr(hinv), _ptr(scale), _ptr(ws), 0 if ws is None else ws.numel(),
        _stream(stream)))


def crvq_hessian_product(R: torch.Tensor, H: torch.Tensor, G: torch.Tensor, row_loss: Optional[torch.Tensor] = None,
                         loss_total: Optional[torch.Tensor] = None, stream=None) -> None:
    """G = R H[:, :G.shape[1]], optionally the per-row QuantLoss sum_j R_rj G_rj and their total (fp64)."""
    M, N = R.shape
    _check("crvq_hessian_product", lib().crvq_hessian_product(
        M, N, G.shape[1], _ptr(R), R.stride(0), _ptr(H), H.stride(0), _ptr(G), G.stride(0), _ptr(row_loss),
        _ptr(loss_total), _stream(stream)))


CRVQ_OP = {"importance": 0, "reorder": 1, "assign": 2, "beam": 3, "kmeans": 4, "dequant": 5, "code_sums": 6,
           "refine": 7, "gemv": 8, "hinv": 9}


def crvq_workspace_size(op: str, n_vectors: int = 0, K: int = 0, beam: int = 0, Ks: Sequence[int] = (), d: int = 0,
                        M: int = 0, N: int = 0, n_cols: int = 0) -> int:
    """Workspace bytes of the call `op` names (a key of CRVQ_OP) at the given shape."""
    arr = (ctypes.c_int64 * max(1, len(Ks)))(*Ks)
    return int(lib().crvq_workspace_size(CRVQ_OP[op], n_vectors, K, beam, len(Ks), d, ctypes.cast(arr, ctypes.c_void_p),
                                         M, N, n_cols))


def crvq_code_sums(X: VecSet, codes: torch.Tensor, K: int, sums: torch.Tensor, counts: Optional[torch.Tensor] = None,
                   stream=None) -> None:
    """sums[k] = sum of the fp64 vectors coded k (see include/crvq.h)."""
    L = lib()
    assert X.t.dtype == torch.float64 and sums.dtype == torch.float64
    ws = _workspace(L.crvq_code_sums_workspace_size(X.n, X.d, K), sums.device)
    _check("crvq_code_sums", L.crvq_code_sums(_ptr(X.t), X.n_rows, X.vecs_per_row, X.ld, X.d, _ptr(codes), K,
                                              _ptr(sums), _ptr(counts), _ptr(ws), 0 if ws is None else ws.numel(),
                                              _stream(stream)))


def crvq_adam_step(C: torch.Tensor, grad: torch.Tensor, grad_scale: float, m: torch.Tensor, v: torch.Tensor,
                   step: int, lr: float, beta1: float = 0.9, beta2: float = 0.95, eps: float = 1e-8,
                   stream=None) -> None:
    assert C.dtype == torch.float32 and grad.dtype == m.dtype == v.dtype == torch.float64
    _check("crvq_adam_step", lib().crvq_adam_step(_ptr(C), _ptr(grad), grad_scale, _ptr(m), _ptr(v), C.numel(), step,
                                                  lr, beta1, beta2, eps, _stream(stream)))


def crvq_adam_step_bf16(C: torch.Tensor, master: torch.Tensor, grad: torch.Tensor, grad_scale: float, m: torch.Tensor,
                        v: torch.Tensor, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.95,
                        eps: float = 1e-8, stream=None) -> None:
    """Adam on the fp32 master of a bf16 codebook (set from it at step 1), the book re-rounded from it."""
    assert C.dtype == torch.bfloat16 and master.dtype == torch.float32 and master.numel() == C.numel()
    assert grad.dtype == m.dtype == v.dtype == torch.float64
    _check("crvq_adam_step_bf16", lib().crvq_adam_step_bf16(_ptr(C), _ptr(master), _ptr(grad), grad_scale, _ptr(m),
                                                            _ptr(v), C.numel(), step, lr, beta1, beta2, eps,
                                                            _stream(stream)))


def crvq_refine_codes(R: torch.Tensor, H: torch.Tensor, C: torch.Tensor, codes: torch.Tensor, d: int, n_cols: int,
                      ldq: int, stream=None) -> None:
    """Width-1 QuantLoss code search for one book covering columns [0, n_cols) (R, codes in/out)."""
    L = lib()
    M, N = R.shape
    ws = _workspace(L.crvq_refine_workspace_size(M, N, n_cols), R.device)
    _check("crvq_refine_codes", L.crvq_refine_codes(
        M, N, d, n_cols, _ptr(R), R.stride(0), _ptr(H), H.stride(0), _ptr(C), dtype_code(C), C.shape[0], _ptr(codes),
        ldq, _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))


def crvq_pack_codes_u8(codes: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    assert codes.dtype == torch.int32 and out.dtype == torch.uint8 and out.numel() >= codes.numel()
    _check("crvq_pack_codes_u8", lib().crvq_pack_codes_u8(_ptr(codes), codes.numel(), _ptr(out), _stream(stream)))


def crvq_dequant_gemv(M: int, N: int, q_base: torch.Tensor, ldq_base: int, C_base: torch.Tensor, x: torch.Tensor,
                      y: torch.Tensor, n_crit: int = 0, q_ext: Sequence[torch.Tensor] = (), ldq_ext: int = 0,
                      C_ext: Sequence[torch.Tensor] = (), perm: Optional[torch.Tensor] = None, stream=None) -> None:
    """y = W_hat x for a layer stored as 8-bit codes (uint8 tensors); see include/crvq.h."""
    L = lib()
    ne = len(C_ext)
    ws = _workspace(L.crvq_gemv_workspace_size(M, N, C_base.shape[0]), y.device)
    dts = (ctypes.c_int32 * max(1, ne))(*[dtype_code(c) for c in C_ext])
    Ks = (ctypes.c_int64 * max(1, ne))(*[c.shape[0] for c in C_ext])
    _check("crvq_dequant_gemv", L.crvq_dequant_gemv(
        M, N, n_crit, _ptr(q_base), ldq_base, _ptr(C_base), dtype_code(C_base), C_base.shape[0], ne,
        ctypes.cast(_ptr_array(q_ext), ctypes.POINTER(ctypes.c_void_p)) if ne else None, ldq_ext,
        ctypes.cast(_ptr_array(C_ext), ctypes.POINTER(ctypes.c_void_p)) if ne else None,
        ctypes.cast(dts, ctypes.c_void_p) if ne else None, ctypes.cast(Ks, ctypes.c_void_p) if ne else None,
        _ptr(perm), _ptr(x), dtype_code(x), _ptr(y), _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream)))
