"""Parity of the general call and of the exit evaluation at the full workload
sizes, in the launch configurations that the benchmark's variants time.

The general call's variants at the 1B and 340M shapes are checked in full
against the general fp64 oracle, element by element: losses, per-token
losses, every module's input gradient, the terminal's readout gradient, every
head's readout gradient (PRIV), every module's gain gradient (per-module
gains), temperature and bias gradients; ROT against the oracle handed
Wbar R_k as each head's readout.  The exit evaluation's per-token
outputs (row losses, top-1) are checked on a seeded sample of token rows of
every module against the oracle run on those rows alone, with bounds derived
from the kernel's operand rounding; the module losses against the oracle's
forward pass over every row."""
import numpy as np
import pytest

import oracle
from solo_inputs import make_extras, make_inputs
from tests.gpu_helpers import TOL, log, rel_max_err, row_loss_error_bound
from tests.test_gpu_general import _dev, compare, oracle_general, run_general

pytestmark = pytest.mark.gpu

N_SAMPLE = 32


def _sample(T, seed):
    rows = np.random.default_rng(seed).choice(T, size=min(N_SAMPLE, T), replace=False)
    return np.unique(np.concatenate([rows, [0, T - 1]]))


def _check_top1(top1_rows, ref, V, dtype, what):
    """The chosen column must maximise the fp64 logits within the error of the
    kernel's logits, and most sampled rows must agree with the oracle exactly."""
    ztol_rel = 1e-2 if dtype == "bf16" else 1e-5
    K, n = top1_rows.shape
    for k in range(K):
        for i in range(n):
            v = int(top1_rows[k, i])
            assert 0 <= v < V, (what, k, i, v)
            zv = ref["logits_of"](k, i, v)
            zm = ref["zmax"][k, i]
            assert zv >= zm - ztol_rel * (1.0 + abs(zm)), (what, k, i, v, zv, zm)
    agree = float((top1_rows == ref["top1"]).mean())
    log(f"{what}: top-1 agreement on the sample {agree:.4f}")
    assert agree >= 0.9


@pytest.mark.parametrize("name,extras", [("1b", dict()), ("2b", dict(tau=True, bias=True)),
                                         ("340m", dict(tau=True, bias=True))],
                         ids=["1b_plain", "2b_tau_bias", "340m_tau_bias"])
def test_fullsize_exit_eval(name, extras):
    import torch

    from paper_2609_35440_amd import binding

    x = make_extras(make_inputs(name, seed=0), 0, **extras)
    cfg = x["cfg"]
    log(f"full-size exit evaluation {name}: K={cfg.K} T={cfg.T} d={cfg.d} V={cfg.V} extras {extras}")
    f = _dev(x)
    out = binding.exit_eval(f["h"], f["gain"], f["W"], f["targets"], tau=f["tau"], bias=f["bias"])
    torch.cuda.synchronize()
    losses = out.losses.double().cpu().numpy()
    row_loss = out.row_loss.double().cpu().numpy()
    top1 = out.top1.cpu().numpy()
    del f, out
    torch.cuda.empty_cache()
    assert np.all(np.isfinite(row_loss)) and np.all(np.isfinite(losses))
    # module loss = mean of the per-token losses
    np.testing.assert_allclose(row_loss.mean(axis=1), losses, rtol=2e-6)
    rows = _sample(cfg.T, 300)
    ref = oracle.exit_eval(x["h"][:, rows], x["gain"], x["W"], x["targets"][:, rows], tau=x.get("tau"),
                           bias=x.get("bias"))
    for k in range(cfg.K):
        tk = 1.0 if x.get("tau") is None else float(x["tau"][k])
        bk = None if x.get("bias") is None else x["bias"][k]
        bound = row_loss_error_bound(x["h"][k, rows], x["gain"], x["W"], x["targets"][k, rows], tk, cfg.dtype, bk)
        err = np.abs(row_loss[k, rows] - ref["row_loss"][k])
        log(f"{name} module {k}: sampled rows {len(rows)}, row_loss err {err.max():.2e} (bound {bound.min():.2e}..)")
        assert np.all(err <= bound), (k, float((err - bound).max()))
    # module losses over every row against the oracle's forward pass
    full = oracle.exit_eval(x["h"], x["gain"], x["W"], x["targets"], tau=x.get("tau"), bias=x.get("bias"))
    rel = np.abs(losses - full["losses"]) / np.abs(full["losses"])
    log(f"{name}: module losses rel err {rel}")
    assert np.all(rel <= TOL[cfg.dtype]["loss"]), rel
    _check_top1(top1[:, rows], ref, cfg.V, cfg.dtype, f"exit eval {name}")


# the general call's variants, as bench.py --variant times them, in full against the oracle
VARIANTS = {
    "tau_bias": (dict(tau=True, bias=True), dict(final_module_dW=True, want_dtau=True, want_dbias=True)),
    "per_module_gain": (dict(per_module_gain=True), dict(final_module_dW=True)),
    "rand": (dict(wbar="per_head"), dict(final_module_dW=True)),
    "priv": (dict(wbar="per_head"), dict(final_module_dW=True, heads_train_readout=True)),
    "rot": (dict(rot=True), dict(final_module_dW=True)),
}


@pytest.mark.parametrize("name,variant", [("1b", v) for v in VARIANTS] + [("340m", "tau_bias")])
def test_fullsize_general_variant_in_full(name, variant):
    extras, flags = VARIANTS[variant]
    x = make_extras(make_inputs(name, seed=0), 0, **extras)
    cfg = x["cfg"]
    log(f"full-size general call {name} {variant}: K={cfg.K} T={cfg.T} d={cfg.d} V={cfg.V} flags {flags}")
    g = run_general(x, flags)
    for key, v in g.items():
        if v is not None:
            assert np.all(np.isfinite(v)), key
    ref = oracle_general(x, flags)
    log(f"{name} {variant}: oracle done")
    compare(g, ref, cfg.dtype, flags, f"{name} {variant} (full)")


def test_fullsize_rot_2b_wide():
    """ROT at the 2B shape (the wide family; seven rotated heads and the
    terminal as separate launches): every head's per-token losses and input
    gradients on seeded row samples against the oracle handed W R_k (formed in
    fp64) as that head's readout, with the module's full T in the mean; the
    terminal module (loss, dh, dW, dgain) in full."""
    from tests.gpu_helpers import check_close

    x = make_extras(make_inputs("2b", seed=0), 0, rot=True)
    cfg = x["cfg"]
    log(f"full-size ROT 2b: K={cfg.K} T={cfg.T} d={cfg.d} V={cfg.V}")
    g = run_general(x, dict(final_module_dW=True))
    for key, v in g.items():
        if v is not None:
            assert np.all(np.isfinite(v)), key
    tol = TOL[cfg.dtype]
    W64 = x["W"].astype(np.float64)
    for k in range(cfg.K - 1):
        rows = _sample(cfg.T, 400 + k)
        Wk = W64 @ x["rot"][k].astype(np.float64)
        rl, dh, _, _ = oracle.module_fwd_bwd(x["h"][k, rows], x["targets"][k, rows], Wk, x["gain"], T_total=cfg.T)
        e_rl = np.abs(g["row_loss"][k, rows] - rl).max() / max(1.0, np.abs(rl).max())
        e_dh = rel_max_err(g["dh"][k, rows], dh)
        log(f"rot 2b head {k}: sampled rows {len(rows)}, row_loss err {e_rl:.2e}, dh err {e_dh:.2e}")
        assert e_rl <= 2 * tol["loss"] and e_dh <= tol["grad"], (k, e_rl, e_dh)
    kf = cfg.K - 1
    rl, dh, dW, dgain = oracle.module_fwd_bwd(x["h"][kf], x["targets"][kf], x["W"], x["gain"], want_readout_grads=True)
    ref = {"losses": np.array([rl.mean()]), "dh": dh[None], "dW": dW, "dgain": dgain}
    gk = {"losses": g["losses"][kf:], "dh": g["dh"][kf:], "dW": g["dW"], "dgain": g["dgain"]}
    check_close(gk, ref, cfg.dtype, what="rot 2b terminal module (full)")


def test_fullsize_rot_exit_eval_1b():
    """ROT through the exit evaluation at the 1B shape (the forward-only
    register-fed pass on the rotated rows): sampled rows' losses and top-1
    against the oracle handed W R_k, and module losses equal to the training
    call's on the same inputs (the same forward on another tiling)."""
    import torch

    from paper_2609_35440_amd import binding
    from tests.test_gpu_general import oracle_view, run_exit_eval

    x = make_extras(make_inputs("1b", seed=0), 0, rot=True)
    cfg = x["cfg"]
    losses, row_loss, top1 = run_exit_eval(x)
    assert np.all(np.isfinite(row_loss))
    np.testing.assert_allclose(row_loss.mean(axis=1), losses, rtol=2e-6)
    g = run_general(x, dict(final_module_dW=False))
    np.testing.assert_allclose(losses, g["losses"], rtol=1e-5)
    torch.cuda.empty_cache()
    rows = _sample(cfg.T, 500)
    xo = oracle_view(x)
    ref = oracle.exit_eval(x["h"][:, rows], x["gain"], x["W"], x["targets"][:, rows], Wbar=xo["Wbar"])
    tol = TOL[cfg.dtype]
    rscale = max(np.abs(ref["row_loss"]).max(), 1.0)
    err = np.abs(row_loss[:, rows] - ref["row_loss"]).max()
    log(f"rot exit eval 1b: sampled rows {len(rows)}, row_loss err {err:.2e}")
    assert err <= 2 * tol["loss"] * rscale, err
    _check_top1(top1[:, rows], ref, cfg.V, cfg.dtype, "rot exit eval 1b")
