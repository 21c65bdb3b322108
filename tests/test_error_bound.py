"""The per-token error bound of the exit-evaluation and online-softmax GPU tests
(tests/gpu_helpers.row_loss_error_bound), checked on the CPU against an
emulation of the matrix-core arithmetic it bounds: bf16(g * h) formed once from
the stored bf16 values, each 32-deep block of exact products summed and rounded
once to fp32 (one matrix instruction), the blocks of each of 8 column slices
in fp32, the 8 slice partials in a fixed fp32 tree, the row scale
r tau log2(e) and the bias in fp32, and an fp32 log-sum-exp in base 2.  Every emulated row loss must lie within the bound of the exact fp64
one; without the bound's operand-rounding term some rows must fall outside
(the term is needed)."""
import numpy as np
import pytest

from solo_inputs import make_extras, make_inputs, round_bf16
from tests.gpu_helpers import row_loss_error_bound

LOG2E = np.float32(1.4426950408889634)
LN2 = np.float32(0.6931471805599453)


def _exact_row_loss(h, g, R, y, tau, bias, eps=1e-6):
    h = h.astype(np.float64)
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1) + eps)
    z = tau * r[:, None] * ((h * g.astype(np.float64)) @ R.astype(np.float64).T)
    if bias is not None:
        z = z + bias.astype(np.float64)[None, :]
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    return lse - z[np.arange(len(y)), y]


def _emulated_row_loss(h, g, R, y, tau, bias, eps=1e-6):
    T, d = h.shape
    f32 = np.float32
    # the stationary operand: the exact product of two bf16 values, rounded once
    x = round_bf16(h.astype(f32) * g.astype(f32))
    Rf = R.astype(f32)
    # 8 column slices (split-K), each summed over its 32-deep blocks in fp32
    nw = 8 if d % 256 == 0 else 1
    ds = d // nw
    parts = np.zeros((nw, T, R.shape[0]), f32)
    for w in range(nw):
        acc = np.zeros((T, R.shape[0]), f32)
        for k0 in range(w * ds, (w + 1) * ds, 32):
            # one 32-deep instruction: exact bf16 products, their sum rounded once to fp32
            blk = (x[:, k0:k0 + 32].astype(np.float64) @ Rf[:, k0:k0 + 32].astype(np.float64).T).astype(f32)
            acc = acc + blk
        parts[w] = acc
    if nw == 8:
        s = ((parts[0] + parts[1]) + (parts[2] + parts[3])) + ((parts[4] + parts[5]) + (parts[6] + parts[7]))
    else:
        s = parts[0]
    r = (1.0 / np.sqrt(np.mean(h.astype(np.float64) ** 2, axis=-1) + eps)).astype(f32)
    z2 = s * (r * f32(tau) * LOG2E)[:, None]
    if bias is not None:
        z2 = z2 + (bias.astype(f32) * LOG2E)[None, :]
    m = z2.max(axis=1)
    sumexp = np.exp2(z2 - m[:, None]).astype(f32).sum(axis=1, dtype=f32)
    lse2 = m + np.log2(sumexp).astype(f32)
    return ((lse2 - z2[np.arange(T), y]) * LN2).astype(np.float64)


CASES = [
    ("340m", dict(K=1, T=24, d=256, V=150), dict(), 1.0),
    ("340m", dict(K=1, T=20, d=1024, V=120), dict(bias=True), 1.9),
    ("1b", dict(K=1, T=16, d=2048, V=100), dict(), 0.7),
]


@pytest.mark.parametrize("cfg,ov,extras,tau", CASES, ids=["d256", "d1024_bias_tau", "d2048"])
def test_bound_covers_the_emulated_kernel_arithmetic(cfg, ov, extras, tau):
    x = make_extras(make_inputs(cfg, seed=5, **ov), 5, **extras)
    h, g, R, y = x["h"][0], x["gain"], x["W"], x["targets"][0]
    # larger logits than the workloads' (|z| of several units) so the rounding terms matter
    R = round_bf16((R * np.float32(25.0)).astype(np.float32))
    bias = None if x.get("bias") is None else x["bias"][0]
    exact = _exact_row_loss(h, g, R, y, tau, bias)
    emul = _emulated_row_loss(h, g, R, y, tau, bias)
    bound = row_loss_error_bound(h, g, R, y, tau, "bf16", bias)
    err = np.abs(emul - exact)
    assert np.all(err <= bound), float((err - bound).max())
    # the operand-rounding term is what most of the bound is made of: without it
    # (accumulation and instruction terms only) some rows fall outside
    d = h.shape[1]
    hh = h.astype(np.float64)
    r = 1.0 / np.sqrt(np.mean(hh * hh, axis=-1) + 1e-6)
    rounded = round_bf16((h.astype(np.float32) * g.astype(np.float32))).astype(np.float64)
    gamma = (d / 32 + 8) * 2.0 ** -24
    B = tau * r[:, None] * gamma * (np.abs(rounded) @ np.abs(R.astype(np.float64)).T)
    z = tau * r[:, None] * ((hh * g.astype(np.float64)) @ R.astype(np.float64).T)
    rows = np.arange(len(y))
    partial = B.max(axis=1) + B[rows, y] + 2.0 ** -20 * (1.0 + 2.0 * np.abs(z).max(axis=1))
    assert np.any(err > partial)
