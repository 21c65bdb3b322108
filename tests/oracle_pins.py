"""Pins of the fp64 oracle to things other than itself.

Every check takes the oracle module as an argument so that the same checks can
be run on deliberately broken copies of it (tests/test_oracle_mutations.py).
Each returns None on success and raises AssertionError on failure.

What pins what:
  * finite differences of the oracle's own loss -> dh, dW, dgain (the 1/T mean
    factor, the norm backward, the residual sign)
  * torch fp64 autograd of rms_norm / linear / cross_entropy, a library
    routine -> losses and every gradient, stop-gradient of the copies
  * W = 0 closed forms -> loss = log V exactly, dh = 0, dgain = 0, dW formula
  * T = 1, V = 2 -> loss = softplus(z_other - z_target)
  * V = 1 -> loss 0 and every gradient 0
  * invariants I1..I6 and softmax rows summing to one
  * torch fp64 softmax -> softmax_rows (ordinary, shifted to 1000, dominant entry)
  * the unblocked brute force agrees to 1e-12
"""
from __future__ import annotations

import math

import numpy as np


def tiny_case(seed=0, K=2, T=5, d=8, V=7, w_sigma=0.3, same_targets=False):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((K, T, d))
    W = rng.standard_normal((V, d)) * w_sigma
    gain = 1.0 + 0.3 * rng.standard_normal(d)
    y = rng.integers(0, V, size=(K, T))
    if same_targets:
        y[:] = y[0]
    return h, gain, W, y


def _module_loss(orc, hk, yk, W, gain, eps):
    rl, _, _, _ = orc.module_fwd_bwd(hk, yk, W, gain, eps, False)
    return rl.sum() / hk.shape[0]


def pin_finite_differences(orc, eps=1e-6, step=1e-6, seed=0):
    h, gain, W, y = tiny_case(seed)
    K, T, d = h.shape
    out = orc.readout_fwd_bwd(h, gain, W, y, True, eps)
    # dh of every module
    for k in range(K):
        fd = np.zeros((T, d))
        for t in range(T):
            for j in range(d):
                hp = h[k].copy()
                hm = h[k].copy()
                hp[t, j] += step
                hm[t, j] -= step
                fd[t, j] = (_module_loss(orc, hp, y[k], W, gain, eps) - _module_loss(orc, hm, y[k], W, gain, eps)) / (2 * step)
        err = np.abs(fd - out["dh"][k]).max() / max(np.abs(fd).max(), 1e-30)
        assert err < 1e-6, ("dh fd", k, err)
    # dW and dgain of the final module's loss
    kf = K - 1
    fdW = np.zeros_like(W)
    for v in range(W.shape[0]):
        for j in range(d):
            Wp = W.copy()
            Wm = W.copy()
            Wp[v, j] += step
            Wm[v, j] -= step
            fdW[v, j] = (_module_loss(orc, h[kf], y[kf], Wp, gain, eps) - _module_loss(orc, h[kf], y[kf], Wm, gain, eps)) / (2 * step)
    err = np.abs(fdW - out["dW"]).max() / np.abs(fdW).max()
    assert err < 1e-6, ("dW fd", err)
    fdg = np.zeros(d)
    for j in range(d):
        gp = gain.copy()
        gm = gain.copy()
        gp[j] += step
        gm[j] -= step
        fdg[j] = (_module_loss(orc, h[kf], y[kf], W, gp, eps) - _module_loss(orc, h[kf], y[kf], W, gm, eps)) / (2 * step)
    err = np.abs(fdg - out["dgain"]).max() / np.abs(fdg).max()
    assert err < 1e-6, ("dgain fd", err)


def pin_torch_autograd(orc, eps=1e-6, seed=1, K=3, T=9, d=16, V=11):
    import torch
    import torch.nn.functional as F

    h, gain, W, y = tiny_case(seed, K, T, d, V)
    out = orc.readout_fwd_bwd(h, gain, W, y, True, eps)
    th = torch.tensor(h, dtype=torch.float64, requires_grad=True)
    tW = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    tg = torch.tensor(gain, dtype=torch.float64, requires_grad=True)
    ty = torch.tensor(y, dtype=torch.long)
    total = 0.0
    losses = []
    for k in range(K):
        final = k == K - 1
        Wk = tW if final else tW.detach()          # read-only copy: stop-gradient
        gk = tg if final else tg.detach()
        hn = F.rms_norm(th[k], (d,), weight=gk, eps=eps)
        lk = F.cross_entropy(F.linear(hn, Wk), ty[k], reduction="mean")
        losses.append(lk.item())
        total = total + lk
    total.backward()
    np.testing.assert_allclose(out["losses"], np.array(losses), rtol=1e-12, atol=0)
    np.testing.assert_allclose(out["dh"], th.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(out["dW"], tW.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(out["dgain"], tg.grad.numpy(), rtol=1e-10, atol=1e-14)


def pin_w_zero_closed_form(orc, eps=1e-6, seed=2):
    h, gain, W, y = tiny_case(seed, K=2, T=6, d=8, V=5)
    W = np.zeros_like(W)
    out = orc.readout_fwd_bwd(h, gain, W, y, True, eps)
    V = W.shape[0]
    T = h.shape[1]
    np.testing.assert_allclose(out["losses"], math.log(V), rtol=0, atol=1e-15)
    assert np.abs(out["dh"]).max() == 0.0
    assert np.abs(out["dgain"]).max() == 0.0
    # dW_v = (1/T) [ (1/V) sum_t hhat_t - sum_{t: y_t = v} hhat_t ]
    x = h[-1]
    hhat = gain * x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps)
    want = np.tile(hhat.sum(0) / V, (V, 1))
    for t in range(T):
        want[y[-1, t]] -= hhat[t]
    want /= T
    np.testing.assert_allclose(out["dW"], want, rtol=1e-12, atol=1e-15)


def pin_softplus_v2(orc, eps=1e-6, seed=3):
    rng = np.random.default_rng(seed)
    for _ in range(5):
        d = 8
        h = rng.standard_normal((1, 1, d))
        W = rng.standard_normal((2, d))
        gain = 1.0 + 0.2 * rng.standard_normal(d)
        y = np.array([[rng.integers(0, 2)]])
        out = orc.readout_fwd_bwd(h, gain, W, y, True, eps)
        x = h[0, 0]
        hh = gain * x / math.sqrt(float(np.mean(x * x)) + eps)
        zy = float(W[y[0, 0]] @ hh)
        zo = float(W[1 - y[0, 0]] @ hh)
        want = math.log1p(math.exp(zo - zy))
        assert abs(out["losses"][0] - want) <= 1e-13 * max(1.0, want)
        # d loss / d z_other = sigmoid(zo - zy); dW_other = sigmoid * hhat, dW_y = -sigmoid * hhat
        sg = 1.0 / (1.0 + math.exp(zy - zo))
        np.testing.assert_allclose(out["dW"][1 - y[0, 0]], sg * hh, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(out["dW"][y[0, 0]], -sg * hh, rtol=1e-12, atol=1e-15)


def pin_v1_degenerate(orc, eps=1e-6, seed=4):
    h, gain, W, y = tiny_case(seed, K=2, T=4, d=8, V=1)
    y[:] = 0
    out = orc.readout_fwd_bwd(h, gain, W, y, True, eps)
    assert np.abs(out["losses"]).max() == 0.0
    assert np.abs(out["dh"]).max() < 1e-16
    assert np.abs(out["dW"]).max() < 1e-16 and np.abs(out["dgain"]).max() < 1e-16


def pin_invariants(orc, seed=5):
    h, gain, W, y = tiny_case(seed, K=3, T=7, d=12, V=9)
    # I3 at eps = 0: <dh_t, h_t> = 0 (scale invariance of the normalised input)
    out0 = orc.readout_fwd_bwd(h, gain, W, y, True, 0.0)
    assert np.abs(np.einsum("ktd,ktd->kt", out0["dh"], h)).max() < 1e-14
    # I5 at eps = 0: loss(c h) = loss(h), dh(c h) = dh(h) / c
    c = 2.75
    outc = orc.readout_fwd_bwd(c * h, gain, W, y, True, 0.0)
    np.testing.assert_allclose(outc["losses"], out0["losses"], rtol=1e-13)
    np.testing.assert_allclose(outc["dh"] * c, out0["dh"], rtol=1e-10, atol=1e-16)
    eps = 1e-6
    out = orc.readout_fwd_bwd(h, gain, W, y, True, eps)
    # I1: columns of dW sum to zero over the vocabulary
    assert np.abs(out["dW"].sum(0)).max() < 1e-15 * max(1.0, np.abs(out["dW"]).max()) * W.shape[0] * 10
    # I2: <dW, W> = <dgain, gain> (z is bilinear in W and gain)
    a = float(np.sum(out["dW"] * W))
    b = float(np.sum(out["dgain"] * gain))
    assert abs(a - b) < 1e-13 * max(1.0, abs(a))
    # I4: W -> W + 1 u^T leaves everything unchanged (sum_v delta_tv = 0)
    u = np.random.default_rng(seed).standard_normal(W.shape[1])
    outs = orc.readout_fwd_bwd(h, gain, W + u[None, :], y, True, eps)
    np.testing.assert_allclose(outs["losses"], out["losses"], rtol=1e-12)
    np.testing.assert_allclose(outs["dh"], out["dh"], rtol=1e-9, atol=1e-15)
    np.testing.assert_allclose(outs["dW"], out["dW"], rtol=1e-9, atol=1e-15)
    np.testing.assert_allclose(outs["dgain"], out["dgain"], rtol=1e-9, atol=1e-14)
    # I6 module independence and zero readout gradient from the read-only copies
    h2 = h.copy()
    h2[0] = np.random.default_rng(seed + 1).standard_normal(h[0].shape)
    out2 = orc.readout_fwd_bwd(h2, gain, W, y, True, eps)
    np.testing.assert_array_equal(out2["dW"], out["dW"])
    np.testing.assert_array_equal(out2["dgain"], out["dgain"])
    np.testing.assert_array_equal(out2["dh"][1:], out["dh"][1:])
    np.testing.assert_array_equal(out2["losses"][1:], out["losses"][1:])
    single = orc.readout_fwd_bwd(h[-1:], gain, W, y[-1:], True, eps)
    np.testing.assert_allclose(single["dW"], out["dW"], rtol=0, atol=0)
    # no readout gradient requested: None
    outn = orc.readout_fwd_bwd(h, gain, W, y, False, eps)
    assert outn["dW"] is None and outn["dgain"] is None
    np.testing.assert_array_equal(outn["dh"], out["dh"])
    # softmax rows sum to one
    hhat, _, _ = orc.rmsnorm_forward(h[0], gain, eps)
    p = orc.softmax_rows(hhat @ W.T)
    np.testing.assert_allclose(p.sum(1), 1.0, rtol=0, atol=1e-15)


def pin_softmax_rows(orc, seed=8):
    """softmax_rows against torch's fp64 softmax (a library routine), on
    ordinary logits, on logits near 1000 (where an unshifted exp overflows) and
    on a row with one dominant entry."""
    import torch

    rng = np.random.default_rng(seed)
    z = rng.standard_normal((5, 9)) * 3.0
    for zz in (z, z + 1000.0, np.concatenate([z[:1], [[40.0] + [0.0] * 8]])):
        ref = torch.softmax(torch.from_numpy(zz), dim=-1).numpy()
        got = orc.softmax_rows(zz)
        assert np.all(np.isfinite(got)), "softmax_rows not finite"
        assert np.abs(got - ref).max() <= 1e-14, ("softmax_rows", np.abs(got - ref).max())


def pin_bruteforce(orc, eps=1e-6, seed=6):
    h, gain, W, y = tiny_case(seed, K=2, T=4, d=6, V=5)
    a = orc.readout_fwd_bwd(h, gain, W, y, True, eps, row_chunk=3)
    b = orc.readout_bruteforce(h, gain, W, y, True, eps)
    for key in ("losses", "row_loss", "dh", "dW", "dgain"):
        scale = max(np.abs(b[key]).max(), 1e-300)
        assert np.abs(a[key] - b[key]).max() <= 1e-12 * scale, key


def pin_row_subset(orc, eps=1e-6, seed=7):
    """Rows are independent: a row subset with the module's T gives the same rows."""
    h, gain, W, y = tiny_case(seed, K=1, T=10, d=8, V=6)
    full = orc.readout_fwd_bwd(h, gain, W, y, False, eps)
    rows = np.array([0, 3, 9])
    rl, dh, _, _ = orc.module_fwd_bwd(h[0, rows], y[0, rows], W, gain, eps, False, T_total=10)
    np.testing.assert_allclose(rl, full["row_loss"][0, rows], rtol=1e-14)
    np.testing.assert_allclose(dh, full["dh"][0, rows], rtol=1e-12, atol=1e-18)


ALL_PINS = [
    pin_finite_differences,
    pin_torch_autograd,
    pin_w_zero_closed_form,
    pin_softplus_v2,
    pin_v1_degenerate,
    pin_invariants,
    pin_bruteforce,
    pin_row_subset,
    pin_softmax_rows,
]
