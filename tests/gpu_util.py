"""Helpers shared by the GPU parity tests (comparison rules; no method arithmetic beyond the
oracle's own definitions)."""
import sys

import numpy as np
import torch

import oracle

TIE_REL = 1e-6  # codes may differ only where the distance gap is below this (relative)


def say(msg: str):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy; bf16 comes back as uint16 bit patterns (the oracle's bf16 format)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def dt(t: torch.Tensor) -> str:
    return "bf16" if t.dtype == torch.bfloat16 else "f32"


def dev(a: np.ndarray, dtype: str = "f32", device="cuda") -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def sqd(V64: np.ndarray, C64: np.ndarray, q: np.ndarray) -> np.ndarray:
    diff = V64 - C64[q]
    return (diff * diff).sum(1)


def check_codes(V: np.ndarray, C: np.ndarray, got: np.ndarray, exp: np.ndarray, v_dtype="f32", c_dtype="f32",
                what="codes") -> int:
    """Codes must equal the oracle's except where both choices are within TIE_REL of each other."""
    got = np.asarray(got)
    exp = np.asarray(exp)
    assert got.shape == exp.shape
    assert got.min() >= 0 and got.max() < len(C), f"{what}: code out of range"
    bad = np.flatnonzero(got != exp)
    if len(bad):
        V64 = oracle.widen(V, v_dtype).astype(np.float64)[bad]
        C64 = oracle.widen(C, c_dtype).astype(np.float64)
        dg = sqd(V64, C64, got[bad])
        de = sqd(V64, C64, exp[bad])
        ok = np.where(de == 0, dg == 0, dg <= de * (1 + TIE_REL))
        assert ok.all(), f"{what}: {int((~ok).sum())} of {len(got)} codes differ beyond ties, e.g. " \
                         f"{bad[~ok][:5]} got {got[bad[~ok][:5]]} want {exp[bad[~ok][:5]]}"
    return len(bad)


def rel_close(got: np.ndarray, exp: np.ndarray, tol: float, what: str, axis_vec: bool = False):
    got = np.asarray(got, dtype=np.float64)
    exp = np.asarray(exp, dtype=np.float64)
    if axis_vec:
        num = np.sqrt(((got - exp) ** 2).sum(-1))
        den = np.sqrt((exp ** 2).sum(-1))
    else:
        num = np.abs(got - exp)
        den = np.abs(exp)
    ok = num <= tol * den + 1e-30
    assert ok.all(), f"{what}: {int((~ok).sum())} entries beyond rel {tol}; worst {float((num / (den + 1e-300)).max())}"
