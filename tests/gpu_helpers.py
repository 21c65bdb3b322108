"""Shared helpers of the GPU parity tests: upload seeded inputs, call the HIP
path through the C-ABI binding, compare with the fp64 oracle at the stated
tolerances."""
from __future__ import annotations

import sys
import time

import numpy as np

# Tolerances: loss relative error; dh / dW / dgain max-abs error relative to max |ref|
TOL = {
    "bf16": {"loss": 1e-3, "grad": 2e-2},
    "f32": {"loss": 1e-5, "grad": 1e-5},
}


def log(msg: str) -> None:
    print(f"[gpu-test {time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def to_device(x: dict):
    import torch

    dev = torch.device("cuda:0")
    if x["cfg"].dtype == "bf16":
        def up(bits):
            return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

        h, gain, W = up(x["h_bits"]), up(x["gain_bits"]), up(x["W_bits"])
    else:
        h = torch.from_numpy(x["h"]).to(dev)
        gain = torch.from_numpy(x["gain"]).to(dev)
        W = torch.from_numpy(x["W"]).to(dev)
    targets = torch.from_numpy(x["targets"]).to(dev)
    return h, gain, W, targets


def run_gpu(x: dict, final_module_dW: bool = True, eps: float = 1e-6, dev_inputs=None):
    import torch

    from paper_2609_35440_amd import binding

    h, gain, W, targets = dev_inputs if dev_inputs is not None else to_device(x)
    out = binding.readout_fwd_bwd(h, gain, W, targets, final_module_dW, eps, row_loss=True)
    torch.cuda.synchronize()
    res = {
        "losses": out.losses.double().cpu().numpy(),
        "row_loss": out.row_loss.double().cpu().numpy(),
        "dh": out.dh.float().cpu().numpy().astype(np.float64),
        "dW": out.dW.double().cpu().numpy() if out.dW is not None else None,
        "dgain": out.dgain.double().cpu().numpy() if out.dgain is not None else None,
    }
    return res


def row_loss_error_bound(h, gain, R, targets, tau, dtype, bias=None, eps=1e-6):
    """Per-token bound on |row_loss_gpu - row_loss_oracle| of one module.

    The matrix-core kernels multiply the stored readout R by bf16(g * h_t), the
    exact product of two bf16 values rounded once to nearest even, and
    accumulate in fp32; the vector-ALU kernels multiply in fp32.  Write
    e_tj = rounded_tj - g_j h_tj for the operand's rounding.  The kernel's
    logit then differs from the exact one by
        tau r_t sum_j R_vj e_tj                      (the operand's rounding, exact)
      + tau r_t (an fp32 accumulation error of at most gamma sum_j |R_vj rounded_tj|)
    where gamma = n 2^-24 for n roundings along the accumulation: one per
    32-deep matrix instruction, the split-K tree and the scalings (d / 32 + 8)
    on the matrix cores, d for the vector-ALU kernels' sequential sums.  With
    B_tv the absolute value of the first term plus the second, a row loss
    lse_t - z_{t,y} moves by at most max_v B_tv (the log-sum-exp is
    1-Lipschitz in the largest change) plus B_{t,y}; the exp2/log2
    instructions and the fp32 bias add contribute a relative 2^-20 of the
    largest logit and of the loss.  Returns the bound per token, [T].
    """
    h = np.asarray(h, np.float64)
    g = np.asarray(gain, np.float64)
    R = np.asarray(R, np.float64)
    exact = h * g
    d = h.shape[-1]
    if dtype == "bf16":
        from solo_inputs import round_bf16

        rounded = round_bf16(exact.astype(np.float32)).astype(np.float64)
        gamma = (d / 32 + 8) * 2.0 ** -24
    else:
        rounded = exact.astype(np.float32).astype(np.float64)
        gamma = d * 2.0 ** -24
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1) + eps)
    scale = tau * r[:, None]
    B = scale * (np.abs((rounded - exact) @ R.T) + gamma * (np.abs(rounded) @ np.abs(R).T))   # [T, V]
    z = scale * (exact @ R.T) + (0.0 if bias is None else np.asarray(bias, np.float64)[None, :])
    rows = np.arange(h.shape[0])
    zabs = np.abs(z).max(axis=1)
    return B.max(axis=1) + B[rows, np.asarray(targets)] + 2.0 ** -20 * (1.0 + 2.0 * zabs)


def rel_max_err(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    scale = np.abs(b).max()
    if scale == 0.0:
        return float(np.abs(a - b).max())
    return float(np.abs(a - b).max() / scale)


def check_close(gpu: dict, ref: dict, dtype: str, modules=None, what=""):
    """Element-wise comparison at the tolerances of the workload's dtype."""
    tol = TOL[dtype]
    K = ref["losses"].shape[0]
    mods = range(K) if modules is None else modules
    errs = {}
    for k in mods:
        le = abs(gpu["losses"][k] - ref["losses"][k]) / max(abs(ref["losses"][k]), 1e-30)
        errs[f"loss{k}"] = le
        assert le <= tol["loss"], (what, k, gpu["losses"][k], ref["losses"][k], le)
        e = rel_max_err(gpu["dh"][k], ref["dh"][k])
        errs[f"dh{k}"] = e
        assert e <= tol["grad"], (what, "dh", k, e)
    if ref.get("dW") is not None:
        e = rel_max_err(gpu["dW"], ref["dW"])
        errs["dW"] = e
        assert e <= tol["grad"], (what, "dW", e)
        e = rel_max_err(gpu["dgain"], ref["dgain"])
        errs["dgain"] = e
        assert e <= tol["grad"], (what, "dgain", e)
    log(f"{what}: " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    return errs
