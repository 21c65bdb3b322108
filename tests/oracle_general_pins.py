"""Pins of the general fp64 oracle (temperatures, biases, per-module gains,
readout sources, exit evaluation) to things other than itself.

Every check takes the oracle module (``oracle.solo_oracle_general`` or a
mutated copy) as an argument and raises AssertionError on failure.

What pins what:
  * finite differences of each module's loss -> dh, dtau, dbias, dW, dWbar,
    per-module and shared dgain
  * torch fp64 autograd of Algorithm 1's readout lines (rms_norm with weight,
    linear, temperature, bias, cross_entropy; detached copies) -> every output
  * W = 0 closed form -> z = b_k: loss = lse(b_k) - b_k[y] averaged, dbias =
    softmax(b_k) - counts / T, dtau = dh = dgain = 0
  * invariants: a constant added to b_k changes nothing; sum_v dbias_k = 0;
    Euler identities tau dtau = <dW, W> = <dgain, gain>; (tau, g) -> (c tau,
    g / c) leaves the loss and dh unchanged; the readout-source spellings of
    SOLO agree; the headline special case agrees with the headline oracle
  * the per-element brute force agrees to 1e-12
  * exit evaluation: exact ties go to the lowest index, accuracy counts hits
"""
from __future__ import annotations

import math

import numpy as np


def case(seed=0, K=3, T=5, d=8, V=7, per_module_gain=True, wbar="per_module", with_tau=True, with_bias=True,
         w_sigma=0.4):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((K, T, d))
    W = rng.standard_normal((V, d)) * w_sigma
    gain = 1.0 + 0.3 * rng.standard_normal((K, d) if per_module_gain else d)
    if wbar == "per_module":
        Wbar = rng.standard_normal((K - 1, V, d)) * w_sigma
    elif wbar == "shared":
        Wbar = rng.standard_normal((V, d)) * w_sigma
    else:
        Wbar = None
    tau = (0.5 + rng.random(K)) if with_tau else None
    bias = (0.5 * rng.standard_normal((K, V))) if with_bias else None
    y = rng.integers(0, V, size=(K, T))
    return dict(h=h, gain=gain, W=W, Wbar=Wbar, tau=tau, bias=bias, targets=y)


def _loss_k(orc, c, k, **over):
    x = dict(c)
    x.update(over)
    out = orc.general_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], Wbar=x["Wbar"], tau=x["tau"],
                              bias=x["bias"], final_module_dW=False, heads_train_readout=False)
    return out["losses"][k]


def _fd(orc, c, k, name, idx, step=1e-6):
    arr_p = c[name].copy()
    arr_m = c[name].copy()
    arr_p[idx] += step
    arr_m[idx] -= step
    return (_loss_k(orc, c, k, **{name: arr_p}) - _loss_k(orc, c, k, **{name: arr_m})) / (2 * step)


def _rel(a, b):
    return float(np.abs(np.asarray(a) - np.asarray(b)).max() / max(np.abs(np.asarray(b)).max(), 1e-30))


def pin_fd_general(orc, seed=0):
    c = case(seed)
    K, T, d = c["h"].shape
    V = c["W"].shape[0]
    out = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], Wbar=c["Wbar"], tau=c["tau"],
                              bias=c["bias"], final_module_dW=True, heads_train_readout=True)
    for k in range(K):
        fd_dh = np.array([[_fd(orc, c, k, "h", (k, t, j)) for j in range(d)] for t in range(T)])
        assert _rel(out["dh"][k], fd_dh) < 1e-6, ("dh", k)
        assert abs(out["dtau"][k] - _fd(orc, c, k, "tau", (k,))) < 1e-7 * max(1.0, abs(out["dtau"][k])), ("dtau", k)
        fd_db = np.array([_fd(orc, c, k, "bias", (k, v)) for v in range(V)])
        assert _rel(out["dbias"][k], fd_db) < 1e-6, ("dbias", k)
        fd_dg = np.array([_fd(orc, c, k, "gain", (k, j)) for j in range(d)])
        assert _rel(out["dgain"][k], fd_dg) < 1e-6, ("dgain", k)
        if k < K - 1:
            fd_w = np.array([[_fd(orc, c, k, "Wbar", (k, v, j)) for j in range(d)] for v in range(V)])
            assert _rel(out["dWbar"][k], fd_w) < 1e-6, ("dWbar", k)
    fd_w = np.array([[_fd(orc, c, K - 1, "W", (v, j)) for j in range(d)] for v in range(V)])
    assert _rel(out["dW"], fd_w) < 1e-6, "dW"


def pin_fd_shared_gain(orc, seed=1):
    c = case(seed, per_module_gain=False, wbar="shared")
    K, T, d = c["h"].shape
    out = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], Wbar=c["Wbar"], tau=c["tau"],
                              bias=c["bias"], final_module_dW=True)
    # one shared gain: the heads read a frozen copy, so dgain is the terminal's loss only
    fd = np.array([_fd(orc, c, K - 1, "gain", (j,)) for j in range(d)])
    assert _rel(out["dgain"], fd) < 1e-6
    assert out["dWbar"] is None


def pin_torch_algorithm1(orc, seed=2, K=3, T=6, d=8, V=9):
    import torch
    import torch.nn.functional as F

    for pmg, wbar, priv in ((True, "per_module", True), (False, "shared", False), (True, None, False)):
        c = case(seed, K, T, d, V, per_module_gain=pmg, wbar=wbar)
        out = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], Wbar=c["Wbar"], tau=c["tau"],
                                  bias=c["bias"], final_module_dW=True, heads_train_readout=priv)
        T64 = torch.float64
        th = torch.tensor(c["h"], dtype=T64, requires_grad=True)
        tW = torch.tensor(c["W"], dtype=T64, requires_grad=True)
        tg = torch.tensor(c["gain"], dtype=T64, requires_grad=True)
        tt = torch.tensor(c["tau"], dtype=T64, requires_grad=True)
        tb = torch.tensor(c["bias"], dtype=T64, requires_grad=True)
        tWb = None if c["Wbar"] is None else torch.tensor(c["Wbar"], dtype=T64, requires_grad=True)
        ty = torch.tensor(c["targets"], dtype=torch.long)
        total = 0.0
        losses = []
        for k in range(K):
            final = k == K - 1
            if final:
                Wk = tW
            elif tWb is None:
                Wk = tW.detach()                      # SOLO: sg(W)
            elif tWb.dim() == 2:
                Wk = tWb.detach()                     # shared frozen copy
            else:
                Wk = tWb[k] if priv else tWb[k].detach()
            gk = tg[k] if pmg else (tg if final else tg.detach())
            hn = F.rms_norm(th[k], (d,), weight=gk, eps=1e-6)
            z = tt[k] * F.linear(hn, Wk) + tb[k]
            lk = F.cross_entropy(z, ty[k], reduction="mean")
            losses.append(lk.item())
            total = total + lk
        total.backward()
        np.testing.assert_allclose(out["losses"], losses, rtol=1e-12)
        np.testing.assert_allclose(out["dh"], th.grad.numpy(), rtol=1e-9, atol=1e-14)
        np.testing.assert_allclose(out["dW"], tW.grad.numpy(), rtol=1e-9, atol=1e-14)
        np.testing.assert_allclose(out["dgain"], tg.grad.numpy(), rtol=1e-9, atol=1e-14)
        np.testing.assert_allclose(out["dtau"], tt.grad.numpy(), rtol=1e-9, atol=1e-14)
        np.testing.assert_allclose(out["dbias"], tb.grad.numpy(), rtol=1e-9, atol=1e-14)
        if priv:
            np.testing.assert_allclose(out["dWbar"], tWb.grad.numpy(), rtol=1e-9, atol=1e-14)


def pin_bias_only_closed_form(orc, seed=3):
    c = case(seed, K=2, T=8, d=8, V=6)
    W0 = np.zeros_like(c["W"])
    Wb0 = np.zeros_like(c["Wbar"])
    out = orc.general_fwd_bwd(c["h"], c["gain"], W0, c["targets"], Wbar=Wb0, tau=c["tau"], bias=c["bias"],
                              final_module_dW=True, heads_train_readout=True)
    K, T, _ = c["h"].shape
    V = W0.shape[0]
    for k in range(K):
        b = c["bias"][k]
        lse = math.log(sum(math.exp(v) for v in b))
        want_loss = sum(lse - b[y] for y in c["targets"][k]) / T
        assert abs(out["losses"][k] - want_loss) < 1e-13
        p = [math.exp(v - lse) for v in b]
        counts = np.bincount(c["targets"][k], minlength=V)
        np.testing.assert_allclose(out["dbias"][k], np.array(p) - counts / T, rtol=0, atol=1e-15)
    assert np.abs(out["dtau"]).max() == 0.0
    assert np.abs(out["dh"]).max() == 0.0
    assert np.abs(out["dgain"]).max() == 0.0


def pin_general_invariants(orc, seed=4):
    c = case(seed, K=3, T=7, d=10, V=8)
    kw = dict(Wbar=c["Wbar"], tau=c["tau"], final_module_dW=True, heads_train_readout=True)
    out = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], bias=c["bias"], **kw)
    K = c["h"].shape[0]
    # a constant added to each module's bias changes nothing (softmax shift)
    shift = np.arange(K, dtype=np.float64)[:, None] * 3.25
    outs = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], bias=c["bias"] + shift, **kw)
    for key in ("losses", "dh", "dtau", "dbias", "dW", "dWbar", "dgain"):
        np.testing.assert_allclose(outs[key], out[key], rtol=1e-9, atol=1e-14)
    # the bias gradients of every module sum to zero over the vocabulary
    assert np.abs(out["dbias"].sum(axis=1)).max() < 1e-15
    # Euler: z - b is linear in tau and in each of (W_k, g_k): tau dtau = <dW_k, W_k> = <dg_k, g_k>
    for k in range(K):
        Wk = c["W"] if k == K - 1 else c["Wbar"][k]
        dWk = out["dW"] if k == K - 1 else out["dWbar"][k]
        a = c["tau"][k] * out["dtau"][k]
        assert abs(a - float(np.sum(dWk * Wk))) < 1e-13 * max(1.0, abs(a))
        assert abs(a - float(np.sum(out["dgain"][k] * c["gain"][k]))) < 1e-13 * max(1.0, abs(a))
    # temperature and gain trade off: (c tau_k, g_k / c) gives the same logits
    cc = 1.7
    g2 = c["gain"] / cc
    outc = orc.general_fwd_bwd(c["h"], g2, c["W"], c["targets"], bias=c["bias"], Wbar=c["Wbar"], tau=c["tau"] * cc,
                               final_module_dW=True, heads_train_readout=True)
    np.testing.assert_allclose(outc["losses"], out["losses"], rtol=1e-12)
    np.testing.assert_allclose(outc["dh"], out["dh"], rtol=1e-9, atol=1e-15)
    # spellings of SOLO's readout source agree: None, the shared copy W, one copy of W per head
    s = case(seed + 1, K=3, T=5, d=8, V=7, per_module_gain=False, wbar=None)
    base = dict(tau=s["tau"], bias=s["bias"], final_module_dW=True)
    a0 = orc.general_fwd_bwd(s["h"], s["gain"], s["W"], s["targets"], Wbar=None, **base)
    a1 = orc.general_fwd_bwd(s["h"], s["gain"], s["W"], s["targets"], Wbar=s["W"].copy(), **base)
    a2 = orc.general_fwd_bwd(s["h"], s["gain"], s["W"], s["targets"], Wbar=np.stack([s["W"]] * 2), **base)
    for key in ("losses", "dh", "dtau", "dbias", "dW", "dgain"):
        np.testing.assert_array_equal(a1[key], a0[key])
        np.testing.assert_array_equal(a2[key], a0[key])
    # module independence: a head's inputs only move that head's outputs
    h2 = s["h"].copy()
    h2[0] += 0.5
    a3 = orc.general_fwd_bwd(h2, s["gain"], s["W"], s["targets"], Wbar=None, **base)
    np.testing.assert_array_equal(a3["dW"], a0["dW"])
    np.testing.assert_array_equal(a3["dgain"], a0["dgain"])
    np.testing.assert_array_equal(a3["dtau"][1:], a0["dtau"][1:])
    np.testing.assert_array_equal(a3["dbias"][1:], a0["dbias"][1:])


def pin_headline_special_case(orc, seed=5):
    """tau = None, no bias, one gain, Wbar = None is the headline operation,
    which the headline oracle computes with its own code."""
    import oracle

    c = case(seed, K=3, T=6, d=8, V=7, per_module_gain=False, wbar=None, with_tau=False, with_bias=False)
    a = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], final_module_dW=True)
    b = oracle.readout_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], True)
    for key in ("losses", "row_loss", "dh", "dW", "dgain"):
        np.testing.assert_allclose(a[key], b[key], rtol=1e-12, atol=1e-16)
    # tau = 1 and b = 0 given explicitly are the same as leaving them out
    K, _, _ = c["h"].shape
    a1 = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], tau=np.ones(K),
                             bias=np.zeros((K, c["W"].shape[0])), final_module_dW=True)
    for key in ("losses", "dh", "dW", "dgain"):
        np.testing.assert_array_equal(a1[key], a[key])


def pin_general_bruteforce(orc, seed=6):
    for pmg, wbar, priv in ((True, "per_module", True), (False, "shared", False)):
        c = case(seed, K=3, T=4, d=6, V=5, per_module_gain=pmg, wbar=wbar)
        kw = dict(Wbar=c["Wbar"], tau=c["tau"], bias=c["bias"], final_module_dW=True, heads_train_readout=priv)
        a = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], row_chunk=3, **kw)
        b = orc.general_bruteforce(c["h"], c["gain"], c["W"], c["targets"], **kw)
        for key in ("losses", "row_loss", "dh", "dW", "dWbar", "dgain", "dtau", "dbias"):
            if b[key] is None:
                assert a[key] is None, key
                continue
            assert np.abs(a[key] - b[key]).max() <= 1e-12 * max(np.abs(b[key]).max(), 1e-300), key


def pin_exit_eval(orc, seed=7):
    c = case(seed, K=3, T=9, d=8, V=6)
    ev = orc.exit_eval(c["h"], c["gain"], c["W"], c["targets"], Wbar=c["Wbar"], tau=c["tau"], bias=c["bias"])
    full = orc.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], Wbar=c["Wbar"], tau=c["tau"],
                               bias=c["bias"], final_module_dW=False)
    np.testing.assert_allclose(ev["losses"], full["losses"], rtol=1e-13)
    np.testing.assert_allclose(ev["ppl"], np.exp(full["losses"]), rtol=1e-13)
    # the top-1 is a maximiser of the logits, checked per element by loops
    K, T, _ = c["h"].shape
    V = c["W"].shape[0]
    for k in range(K):
        for t in range(T):
            zs = [ev["logits_of"](k, t, v) for v in range(V)]
            tol = 1e-12 * max(1.0, max(abs(z) for z in zs))   # one row vs a block of rows: BLAS order
            assert zs[ev["top1"][k, t]] >= max(zs) - tol
            assert abs(ev["zmax"][k, t] - max(zs)) <= tol
    # exact ties go to the lowest index: duplicate readout rows, zero bias
    W = c["W"].copy()
    W[4] = W[1]
    W[5] = W[1]
    y = np.full((1, 5), 1)
    h = np.abs(c["h"][:1, :5]) + 0.1
    g = np.ones(h.shape[2])
    W[1] = np.full(h.shape[2], 2.0)
    W[4] = W[1]
    W[5] = W[1]
    evt = orc.exit_eval(h, g, W, y)
    assert (evt["top1"] == 1).all()
    assert evt["accuracy"][0] == 1.0
    y2 = np.full((1, 5), 4)
    assert orc.exit_eval(h, g, W, y2)["accuracy"][0] == 0.0


ALL_PINS = [
    pin_fd_general,
    pin_fd_shared_gain,
    pin_torch_algorithm1,
    pin_bias_only_closed_form,
    pin_general_invariants,
    pin_headline_special_case,
    pin_general_bruteforce,
    pin_exit_eval,
]
