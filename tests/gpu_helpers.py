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
