"""Parity of the general call and of the exit evaluation at the full workload
sizes, in the launch configurations that the benchmark's variants time.

Per-token outputs (row losses, input gradients, top-1) are checked on a
seeded sample of token rows of every module, against the oracle run on those
rows alone; the input gradient carries the 1/T of the module mean, so the
oracle's rows are rescaled from the sample's T to the full T.  Sums over all
tokens (module losses, temperature and bias gradients) are checked through
identities that hold at any size."""
import numpy as np
import pytest

import oracle
from solo_inputs import make_extras, make_inputs
from tests.gpu_helpers import TOL, log, rel_max_err
from tests.test_gpu_general import _dev, run_general

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
    tol = TOL[cfg.dtype]
    err = np.abs(row_loss[:, rows] - ref["row_loss"]).max()
    log(f"{name}: sampled rows {len(rows)} per module, row_loss err {err:.2e}")
    assert err <= 2 * tol["loss"] * max(np.abs(ref["row_loss"]).max(), 1.0)
    _check_top1(top1[:, rows], ref, cfg.V, cfg.dtype, f"exit eval {name}")


@pytest.mark.parametrize("name", ["1b", "340m"])
def test_fullsize_general_tau_bias(name):
    x = make_extras(make_inputs(name, seed=0), 0, tau=True, bias=True)
    cfg = x["cfg"]
    K, T = cfg.K, cfg.T
    flags = dict(final_module_dW=True, want_dtau=True, want_dbias=True)
    log(f"full-size general call {name} with temperatures and biases: K={K} T={T} d={cfg.d} V={cfg.V}")
    g = run_general(x, flags)
    for key in ("losses", "row_loss", "dh", "dW", "dgain", "dtau", "dbias"):
        assert np.all(np.isfinite(g[key])), key
    np.testing.assert_allclose(g["row_loss"].mean(axis=1), g["losses"], rtol=2e-6)

    # sampled rows of every module against the oracle on those rows alone
    tol = TOL[cfg.dtype]
    rows = _sample(T, 301)
    ref = oracle.general_fwd_bwd(x["h"][:, rows], x["gain"], x["W"], x["targets"][:, rows], tau=x["tau"],
                                 bias=x["bias"], final_module_dW=False)
    e_rl = np.abs(g["row_loss"][:, rows] - ref["row_loss"]).max()
    assert e_rl <= 2 * tol["loss"] * max(np.abs(ref["row_loss"]).max(), 1.0), e_rl
    scale = len(rows) / T  # the oracle's dh carries 1/len(rows), the full call's 1/T
    for k in range(K):
        e = rel_max_err(g["dh"][k, rows], ref["dh"][k] * scale)
        log(f"module {k}: sampled rows {len(rows)} row_loss err {e_rl:.2e} dh err {e:.2e}")
        assert e <= tol["grad"], (k, e)

    # every module's bias gradient sums to zero over the vocabulary (softmax rows sum to one)
    for k in range(K):
        db = g["dbias"][k]
        assert abs(db.sum()) <= 1e-3 * np.abs(db).sum() + 1e-5, k
    # the final module's logits minus its bias are linear in tau, in R and in the gain:
    # tau dtau = <dR, R> = <dgain, gain>
    a = float(x["tau"][K - 1]) * g["dtau"][K - 1]
    b = float(np.sum(g["dW"] * x["W"].astype(np.float64)))
    c = float(np.sum(g["dgain"] * x["gain"].astype(np.float64)))
    log(f"final module: tau dtau {a:.6e} <dW,W> {b:.6e} <dgain,gain> {c:.6e}")
    s = max(abs(a), abs(b), abs(c), 1e-6)
    assert abs(a - b) <= 2e-2 * s and abs(a - c) <= 2e-2 * s
