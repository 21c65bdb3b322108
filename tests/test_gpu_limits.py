"""Parity at the largest token count the boundary accepts per module in one
tensor of more than 4 GiB: K = 1, T = 2^20 tokens at d = 2048 and d = 2560
(4 and 5 GiB of bf16 hidden states), with a small vocabulary.

Every streamed operand's buffer range and every offset must stay correct past
2^32 bytes.  The hidden states are zero outside the first 16 rows, so the
readout and gain gradients come from those rows alone (a zero row has zero
normalised states), which the oracle computes with the module's full T; a
few zero rows at both ends are compared too (their loss is log V, their input
gradient the mean readout row minus the target's, scaled by 1/sqrt(eps)).
"""
import numpy as np
import pytest

import oracle
from solo_inputs import bf16_bits, bf16_from_bits
from tests.gpu_helpers import TOL, log, rel_max_err

pytestmark = pytest.mark.gpu

T = 1 << 20
V = 64


@pytest.mark.parametrize("d", [2048, 2560])
def test_more_than_4gib_of_tokens(d):
    import torch

    from paper_2609_35440_amd import binding

    rng = np.random.default_rng(51)
    h16 = bf16_bits(rng.standard_normal((16, d)).astype(np.float32))
    W_bits = bf16_bits((0.05 * rng.standard_normal((V, d))).astype(np.float32))
    g_bits = bf16_bits((1.0 + 0.1 * rng.standard_normal(d)).astype(np.float32))
    targets = rng.integers(0, V, size=(1, T)).astype(np.int32)
    log(f"limits: K=1 T={T} d={d} V={V} ({T * d * 2 / 2**30:.1f} GiB of h)")
    dev = torch.device("cuda:0")
    h = torch.zeros((1, T, d), dtype=torch.bfloat16, device=dev)
    up = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to(dev)  # noqa: E731
    h[0, :16] = up(h16)
    out = binding.readout_fwd_bwd(h, up(g_bits), up(W_bits), torch.from_numpy(targets).to(dev), True, 1e-6,
                                  row_loss=True)
    torch.cuda.synchronize()
    rows = np.r_[0:24, T - 8:T]
    dh = out.dh[0, rows].float().cpu().numpy().astype(np.float64)
    rl = out.row_loss[0, rows].double().cpu().numpy()
    dW = out.dW.double().cpu().numpy()
    dgain = out.dgain.double().cpu().numpy()
    loss = float(out.losses[0])
    del out, h
    torch.cuda.empty_cache()

    W = bf16_from_bits(W_bits)
    gain = bf16_from_bits(g_bits)
    hr = np.zeros((len(rows), d), np.float32)
    hr[:16] = bf16_from_bits(h16)
    # the readout and gain gradients: only the first 16 rows contribute
    _, _, dW_ref, dg_ref = oracle.module_fwd_bwd(hr[:16], targets[0, :16], W, gain, want_readout_grads=True,
                                                  T_total=T)
    rl_ref, dh_ref, _, _ = oracle.module_fwd_bwd(hr, targets[0, rows], W, gain, T_total=T)
    tol = TOL["bf16"]
    e = {"dW": rel_max_err(dW, dW_ref), "dgain": rel_max_err(dgain, dg_ref), "dh": rel_max_err(dh, dh_ref),
         "row_loss": float(np.abs(rl - rl_ref).max() / np.abs(rl_ref).max())}
    # the module loss: 16 rows of their own and T - 16 rows of log V
    loss_ref = (oracle.module_fwd_bwd(hr[:16], targets[0, :16], W, gain)[0].sum() + (T - 16) * np.log(V)) / T
    e["loss"] = abs(loss - loss_ref) / loss_ref
    log(f"limits d={d}: " + " ".join(f"{k}={v:.2e}" for k, v in e.items()))
    assert e["dW"] <= tol["grad"] and e["dgain"] <= tol["grad"] and e["dh"] <= tol["grad"]
    assert e["row_loss"] <= 2 * tol["loss"] and e["loss"] <= tol["loss"]
