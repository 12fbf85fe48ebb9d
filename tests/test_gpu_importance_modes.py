"""GPU parity of the channel-importance strategies of Sec. 4.1 / Table 2 through the layer pipeline:
W-only (I_j = max_i W_ij^2), W-A in the unpacked form of Eq. 10 (I_j = h_j max_i (W_ij - Wq_ij)^2, Wq the
prequantized W of Alg. 1 Prequantize) and W-A as Eq. 7 prints it (I_j = max_i (W_ij - Wq_ij)^2 /
(2 [(X X^T)^-1]_jj), the proxy damped by 1 %).  Every call the pipeline makes for the strategy is re-run on the oracle from the
GPU's own inputs (lockstep), then the whole layer is compared with the oracle's pipeline: the same
permutation, critical set and reconstruction error."""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline as opipe
from paper_2412_09282_amd import inputs
from paper_2412_09282_amd.pipeline import LayerConfig, LayerQuantizer

from gpu_util import check_codes, dev, rel_close, say, to_host_bits

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode,dtype", [("w_only", "f32"), ("wa", "f32"), ("wa", "bf16"), ("obs", "f32"),
                                        ("obs", "bf16")])
def test_importance_strategy_lockstep(mode, dtype):
    M, N, d = 96, 128, 8
    say(f"importance strategy {mode} {dtype} {M}x{N}")
    wl = inputs.small_workload(M=M, N=N, tokens=64, d=d, K_base=64, K_ext=(16,), crit_frac=0.1, beam=2, iters=2,
                               dtype=dtype, wid=120)
    W = inputs.make_weight(wl, 0)
    X = inputs.make_calib(wl, 0)
    n = M * N // d
    n_crit = inputs.n_crit_columns(N, d, wl.crit_frac)
    base_idx = inputs.base_init_indices(wl, 0, n)
    ext_idx = [inputs.ext_init_indices(wl, 0, 1, M * n_crit // d)]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    cfg = LayerConfig(d, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters, importance=mode)
    q = LayerQuantizer(M, N, tdt, cfg, tokens=64, device="cuda")
    trace = []
    st = q.run(dev(W, dtype), torch.from_numpy(X).cuda(), torch.from_numpy(base_idx).cuda(),
               [torch.from_numpy(e).cuda() for e in ext_idx], trace=trace)
    torch.cuda.synchronize()
    calls = {c["name"]: c for c in trace}
    bits = lambda t: to_host_bits(t) if isinstance(t, torch.Tensor) else t
    h = bits(calls["hdiag"]["out"]["out"])
    # lockstep: the prequantization calls and the importance
    if mode in ("wa", "obs"):
        Vu = oracle.vectors(W, d)
        for name, c in calls.items():
            if name.startswith("assign_pre"):
                exp, _ = oracle.assign(Vu, bits(c["in"]["C"]), dtype, dtype)
                check_codes(Vu, bits(c["in"]["C"]), bits(c["out"]["codes"]), exp, dtype, dtype, name)
            elif name.startswith("update_pre"):
                Cexp, cnt, _ = oracle.kmeans_update(Vu, bits(c["in"]["codes"]), bits(c["in"]["C"]), dtype, dtype)
                got = bits(c["out"]["C"])
                tol = 1e-5 if dtype == "f32" else 1e-2
                rel_close(oracle.widen(got, dtype), oracle.widen(Cexp, dtype), tol, name, axis_vec=True)
        c = calls["prequant"]
        R = oracle.reconstruct([bits(c["in"]["codes"])], [bits(c["in"]["book"])], np.zeros(n, np.uint8), [dtype])
        Wq = oracle.round_to(R, dtype).reshape(M, N)
        np.testing.assert_array_equal(bits(c["out"]["out"]), Wq)
        scale = h.astype(np.float64)
        if mode == "obs":
            X64 = X.astype(np.float64)
            H = bits(calls["gram"]["out"]["H"])
            assert np.all(np.abs(H - X64.T @ X64) <= 1e-12 * (np.abs(X64).T @ np.abs(X64))), "gram"
            s_got = bits(calls["hinv"]["out"]["scale"]).astype(np.float64)
            s_exp = oracle.obs_scale(oracle.hessian_inverse_diagonal(bits(calls["hinv"]["in"]["H"]), 0.01))
            rel_close(s_got, s_exp, 1e-6, "Eq. 7 factor")
            scale = s_got
        exp_I = oracle.colreduce(W, Wq, scale=scale, reduce="max", dtype=dtype)
    else:
        exp_I = oracle.colreduce(W, reduce="max", dtype=dtype)
    got_I = bits(calls["importance"]["out"]["out"])
    rel_close(got_I, exp_I, 1e-6, f"importance ({mode})")
    # the whole layer against the oracle's own pipeline from the same seeds
    ref = opipe.quantize_layer(W, X, dtype, d, wl.K_base, wl.K_ext, wl.crit_frac, wl.beam, wl.iters, base_idx,
                               ext_idx, importance=mode)
    np.testing.assert_array_equal(st.perm.cpu().numpy(), ref.perm)
    err = opipe.frob_err(W, to_host_bits(st.W_hat), dtype)
    err_ref = opipe.frob_err(W, ref.W_hat, dtype)
    assert abs(err - err_ref) <= 1e-3 * err_ref, (err, err_ref)
    say(f"importance strategy {mode} {dtype}: perm identical, ||W - W_hat||^2 {err:.6e} (oracle {err_ref:.6e})")
