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
