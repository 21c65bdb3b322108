"""Parity at the full workload sizes, in the launch configuration the
benchmark times.  Rows are independent, so the read-only modules' per-token
outputs are checked on seeded row samples (the oracle computes those rows one
chunk at a time) and their module losses against the oracle's forward pass
over every row; the final module, whose readout gradient needs every row, is
checked in full; properties that hold at any size are checked as well."""
import numpy as np
import pytest

import oracle
from solo_inputs import make_inputs
from tests.gpu_helpers import TOL, check_close, log, rel_max_err, run_gpu

pytestmark = pytest.mark.gpu

N_SAMPLE = 48


def _check_sampled_rows(x, g, k, seed):
    cfg = x["cfg"]
    tol = TOL[cfg.dtype]
    rows = np.sort(np.random.default_rng(seed).choice(cfg.T, size=min(N_SAMPLE, cfg.T), replace=False))
    rows = np.unique(np.concatenate([rows, [0, cfg.T - 1]]))
    rl, dh, _, _ = oracle.module_fwd_bwd(x["h"][k, rows], x["targets"][k, rows], x["W"], x["gain"], T_total=cfg.T)
    e_rl = np.abs(g["row_loss"][k, rows] - rl).max() / max(1.0, np.abs(rl).max())
    e_dh = rel_max_err(g["dh"][k, rows], dh)
    log(f"{cfg.name} module {k}: sampled rows {len(rows)} row_loss err {e_rl:.2e} dh err {e_dh:.2e}")
    assert e_rl <= 2 * tol["loss"]
    assert e_dh <= tol["grad"]


def _check_head_losses(x, g):
    """Every read-only module's loss (the mean over all of its tokens) against
    the oracle's forward pass over every row."""
    cfg = x["cfg"]
    K = cfg.K
    if K < 2:
        return
    ref = oracle.exit_eval(x["h"][:K - 1], x["gain"], x["W"], x["targets"][:K - 1])["losses"]
    rel = np.abs(g["losses"][:K - 1] - ref) / np.abs(ref)
    log(f"{cfg.name}: head module losses rel err {rel}")
    assert np.all(rel <= TOL[cfg.dtype]["loss"]), rel


def _properties(x, g):
    cfg = x["cfg"]
    for key in ("losses", "row_loss", "dh", "dW", "dgain"):
        assert np.all(np.isfinite(g[key])), key
    # module loss = mean of the per-token losses (computed in fp64 on the host)
    np.testing.assert_allclose(g["row_loss"].mean(axis=1), g["losses"], rtol=2e-6)
    # Euler identity: <dW, W> = <dgain, gain>
    a = float(np.sum(g["dW"] * x["W"].astype(np.float64)))
    b = float(np.sum(g["dgain"] * x["gain"].astype(np.float64)))
    assert abs(a - b) <= 1e-3 * max(abs(a), abs(b), 1e-12), (a, b)
    # columns of dW sum to zero over the vocabulary (sum_v delta_tv = 0), up to bf16 rounding of delta
    colsum = np.abs(g["dW"].sum(axis=0))
    colabs = np.abs(g["dW"]).sum(axis=0)
    assert np.all(colsum <= 2e-2 * colabs + 1e-9), float((colsum / np.maximum(colabs, 1e-30)).max())
    log(f"{cfg.name}: properties ok (<dW,W>={a:.6e}, <dgain,gain>={b:.6e})")


@pytest.mark.parametrize("name", ["340m", "1b", "2b"])
def test_fullsize_final_module_in_full(name):
    x = make_inputs(name, seed=0)
    cfg = x["cfg"]
    log(f"full size {name}: K={cfg.K} T={cfg.T} d={cfg.d} V={cfg.V}")
    g = run_gpu(x, True)
    log(f"{name}: GPU done, losses {g['losses']}")
    _properties(x, g)
    for k in range(cfg.K - 1):
        _check_sampled_rows(x, g, k, seed=100 + k)
    _check_head_losses(x, g)
    kf = cfg.K - 1
    rl, dh, dW, dgain = oracle.module_fwd_bwd(x["h"][kf], x["targets"][kf], x["W"], x["gain"], want_readout_grads=True)
    ref = {"losses": np.array([rl.mean()]), "dh": dh[None], "dW": dW, "dgain": dgain}
    gk = {"losses": g["losses"][kf:], "dh": g["dh"][kf:], "dW": g["dW"], "dgain": g["dgain"]}
    check_close(gk, ref, cfg.dtype, what=f"{name} final module (full)")


def test_fullsize_large_vocab():
    x = make_inputs("large_vocab", seed=0)
    cfg = x["cfg"]
    log(f"full size large_vocab: K={cfg.K} T={cfg.T} d={cfg.d} V={cfg.V}")
    g = run_gpu(x, True)
    log(f"large_vocab: GPU done, losses {g['losses']}")
    _properties(x, g)
    for k in range(cfg.K):
        _check_sampled_rows(x, g, k, seed=200 + k)
    _check_head_losses(x, g)
    # the final module in full at T = 32768, V = 128256: loss, dh, dW, dgain
    kf = cfg.K - 1
    rl, dh, dW, dgain = oracle.module_fwd_bwd(x["h"][kf], x["targets"][kf], x["W"], x["gain"], want_readout_grads=True)
    ref = {"losses": np.array([rl.mean()]), "dh": dh[None], "dW": dW, "dgain": dgain}
    gk = {"losses": g["losses"][kf:], "dh": g["dh"][kf:], "dW": g["dW"], "dgain": g["dgain"]}
    check_close(gk, ref, cfg.dtype, what="large_vocab final module (full, T=32768)")
