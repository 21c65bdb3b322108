"""GPU parity of the general entry points (temperatures, biases, per-module
gains, readout sources, exit evaluation) with the general fp64 oracle,
element by element, on seeded inputs that span several tiles and ragged
tails, for both kernel families."""
import numpy as np
import pytest

import oracle
from solo_inputs import make_extras, make_inputs
from tests.gpu_helpers import TOL, log, rel_max_err, row_loss_error_bound

pytestmark = pytest.mark.gpu

ALL = dict(per_module_gain=True, wbar="per_head", tau=True, bias=True)
# (name, config, size overrides, input extras, call flags)
CASES = [
    ("mfma_d256_all", "340m", dict(K=3, T=70, d=256, V=300), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("mfma_d2048_all", "1b", dict(K=3, T=65, d=2048, V=515), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("mfma_d1024_shared_copy_bias", "340m", dict(K=3, T=40, d=1024, V=200),
     dict(wbar="shared", tau=True, bias=True), dict(final_module_dW=True, want_dtau=True, want_dbias=True)),
    ("mfma_d1536_tau_only", "340m", dict(K=2, T=33, d=1536, V=129), dict(tau=True),
     dict(final_module_dW=True, want_dtau=True)),
    ("mfma_d512_bias_only_frozen_heads", "340m", dict(K=3, T=45, d=512, V=97),
     dict(wbar="per_head", bias=True), dict(final_module_dW=True, want_dbias=True)),
    ("mfma_d256_bias_grad_three_tiles", "340m", dict(K=2, T=70, d=256, V=300), dict(bias=True),
     dict(final_module_dW=True, want_dbias=True)),
    ("mfma_d768_priv_without_terminal", "340m", dict(K=3, T=50, d=768, V=150), ALL,
     dict(final_module_dW=False, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("mfma_d2048_per_module_gain_frozen", "1b", dict(K=3, T=40, d=2048, V=100), dict(per_module_gain=True),
     dict(final_module_dW=False)),
    ("mfma_d2048_dbias_without_bias", "1b", dict(K=2, T=33, d=2048, V=70), dict(),
     dict(final_module_dW=True, want_dtau=True, want_dbias=True)),
    ("mfma_K1_all", "340m", dict(K=1, T=40, d=256, V=90), dict(per_module_gain=True, tau=True, bias=True),
     dict(final_module_dW=True, want_dtau=True, want_dbias=True)),
    ("mfma_V1_bias", "340m", dict(K=2, T=40, d=256, V=1), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("mfma_T1_all", "340m", dict(K=2, T=1, d=256, V=60), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("wide_d2560_all", "2b", dict(K=3, T=37, d=2560, V=300), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("wide_d2560_shared_copy_bias", "2b", dict(K=3, T=20, d=2560, V=70),
     dict(wbar="shared", tau=True, bias=True), dict(final_module_dW=True, want_dtau=True, want_dbias=True)),
    ("wide_d2560_bias_grad_V_below_tile", "2b", dict(K=2, T=20, d=2560, V=20), dict(bias=True),
     dict(final_module_dW=True, want_dbias=True)),
    ("valu_f32_all", "tiny", dict(K=3, T=37, d=24, V=45), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
    ("valu_f32_shared_copy", "tiny", dict(K=2, T=20, d=64, V=33), dict(wbar="shared", tau=True, bias=True),
     dict(final_module_dW=True, want_dtau=True, want_dbias=True)),
    ("valu_bf16_d72_all", "340m", dict(K=2, T=10, d=72, V=50), ALL,
     dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)),
]


def _dev(x):
    import torch

    dev = torch.device("cuda:0")
    bf = x["cfg"].dtype == "bf16"

    def up(name):
        if x.get(name) is None:
            return None
        if bf:
            return torch.from_numpy(np.ascontiguousarray(x[name + "_bits"]).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x[name])).to(dev)

    f = {n: up(n) for n in ("h", "gain", "W", "Wbar", "rot")}
    f["targets"] = torch.from_numpy(x["targets"]).to(dev)
    f["tau"] = torch.from_numpy(x["tau"]).to(dev) if x.get("tau") is not None else None
    f["bias"] = torch.from_numpy(x["bias"]).to(dev) if x.get("bias") is not None else None
    return f


def run_general(x, flags):
    import torch

    from paper_2609_35440_amd import binding

    f = _dev(x)
    out = binding.readout_general(f["h"], f["gain"], f["W"], f["targets"], Wbar=f["Wbar"], tau=f["tau"],
                                  bias=f["bias"], rot=f["rot"], row_loss=True, **flags)
    torch.cuda.synchronize()
    return {k: (None if v is None else v.double().cpu().numpy()) for k, v in out._asdict().items()}


def oracle_view(x):
    """The inputs as the oracle reads them.  ROT (head k reads Wbar R_k, with
    Wbar = W when there is no separate copy): the oracle gets one readout per
    head, the product formed here in fp64 from the stored values."""
    if x.get("rot") is None:
        return x
    base = (x["W"] if x.get("Wbar") is None else x["Wbar"]).astype(np.float64)
    xo = dict(x)
    xo["rot"] = None
    xo["Wbar"] = np.stack([base @ r.astype(np.float64) for r in x["rot"]])
    return xo


def oracle_general(x, flags):
    x = oracle_view(x)
    return oracle.general_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], Wbar=x.get("Wbar"), tau=x.get("tau"),
                                  bias=x.get("bias"), final_module_dW=flags.get("final_module_dW", True),
                                  heads_train_readout=flags.get("heads_train_readout", False))


def compare(g, ref, dtype, flags, what):
    tol = TOL[dtype]
    K = ref["losses"].shape[0]
    errs = {}
    for k in range(K):
        le = abs(g["losses"][k] - ref["losses"][k]) / max(abs(ref["losses"][k]), 1e-30)
        errs[f"loss{k}"] = le
        assert le <= tol["loss"], (what, "loss", k, g["losses"][k], ref["losses"][k])
        e = rel_max_err(g["dh"][k], ref["dh"][k])
        errs[f"dh{k}"] = e
        assert e <= tol["grad"], (what, "dh", k, e)
    rscale = max(np.abs(ref["row_loss"]).max(), 1.0)
    assert np.abs(g["row_loss"] - ref["row_loss"]).max() <= 2 * tol["loss"] * rscale, (what, "row_loss")
    if flags.get("final_module_dW", True):
        errs["dW"] = e = rel_max_err(g["dW"], ref["dW"])
        assert e <= tol["grad"], (what, "dW", e)
    else:
        assert g["dW"] is None
    if flags.get("heads_train_readout") and K > 1:
        for k in range(K - 1):
            errs[f"dWbar{k}"] = e = rel_max_err(g["dWbar"][k], ref["dWbar"][k])
            assert e <= tol["grad"], (what, "dWbar", k, e)
    if ref["dgain"] is not None:
        if ref["dgain"].ndim == 2:
            for k in range(K):
                errs[f"dg{k}"] = e = rel_max_err(g["dgain"][k], ref["dgain"][k])
                assert e <= tol["grad"], (what, "dgain", k, e)
        else:
            errs["dg"] = e = rel_max_err(g["dgain"], ref["dgain"])
            assert e <= tol["grad"], (what, "dgain", e)
    if flags.get("want_dtau"):
        # one scalar per module: error relative to the largest |dtau_k|
        errs["dtau"] = e = rel_max_err(g["dtau"], ref["dtau"])
        assert e <= tol["grad"], (what, "dtau", g["dtau"], ref["dtau"])
    if flags.get("want_dbias"):
        for k in range(K):
            errs[f"db{k}"] = e = rel_max_err(g["dbias"][k], ref["dbias"][k])
            assert e <= tol["grad"], (what, "dbias", k, e)
        # every module's bias gradient sums to zero over the vocabulary (softmax rows sum to one)
        for k in range(K):
            assert abs(g["dbias"][k].sum()) <= 1e-3 * np.abs(g["dbias"][k]).sum() + 1e-5, (what, "sum dbias", k)
    log(f"{what}: " + " ".join(f"{k}={v:.1e}" for k, v in errs.items()))


@pytest.mark.parametrize("name,cfg,ov,extras,flags", CASES, ids=[c[0] for c in CASES])
def test_general_parity(name, cfg, ov, extras, flags):
    x = make_extras(make_inputs(cfg, seed=21, **ov), 21, **extras)
    log(f"case {name}: {x['cfg']} extras {extras} flags {flags}")
    g = run_general(x, flags)
    ref = oracle_general(x, flags)
    compare(g, ref, x["cfg"].dtype, flags, name)


def test_general_headline_options_match_headline_entry_point():
    """The general entry point with the headline options computes what
    solo_readout_fwd_bwd computes, bit for bit (one code path)."""
    from tests.gpu_helpers import run_gpu

    x = make_inputs("1b", seed=22, K=3, T=48, d=2048, V=333)
    a = run_gpu(x, True)
    b = run_general(make_extras(x, 22), dict(final_module_dW=True))
    for key in ("losses", "dh", "dW", "dgain"):
        np.testing.assert_array_equal(a[key], b[key])


@pytest.mark.parametrize("cfg,d", [("1b", 2048), ("2b", 2560)])
def test_general_bitwise_determinism(cfg, d):
    x = make_extras(make_inputs(cfg, seed=23, K=3, T=64, d=d, V=400), 23, **ALL)
    flags = dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True)
    a = run_general(x, flags)
    b = run_general(x, flags)
    for key, v in a.items():
        if v is not None:
            np.testing.assert_array_equal(v, b[key])


def test_euler_identities_on_gpu():
    # z - b is linear in tau_k and in each of (R_k, g_k): tau dtau = <dR, R> = <dg, g>, within bf16 tolerance
    x = make_extras(make_inputs("1b", seed=24, K=3, T=64, d=2048, V=256), 24, **ALL)
    g = run_general(x, dict(final_module_dW=True, heads_train_readout=True, want_dtau=True, want_dbias=True))
    K = 3
    for k in range(K):
        R = x["W"] if k == K - 1 else x["Wbar"][k]
        dR = g["dW"] if k == K - 1 else g["dWbar"][k]
        a = float(x["tau"][k]) * g["dtau"][k]
        b = float(np.sum(dR * R))
        c = float(np.sum(g["dgain"][k] * x["gain"][k]))
        scale = max(abs(a), abs(b), abs(c), 1e-6)
        log(f"euler k={k}: tau dtau {a:.6e} <dR,R> {b:.6e} <dg,g> {c:.6e}")
        assert abs(a - b) <= 2e-2 * scale and abs(a - c) <= 2e-2 * scale


# ---- exit evaluation

EVAL_CASES = [
    ("mfma_d2048", "1b", dict(K=3, T=65, d=2048, V=515), ALL),
    ("mfma_d256_plain", "340m", dict(K=2, T=70, d=256, V=300), dict()),
    ("mfma_d1024_shared", "340m", dict(K=3, T=40, d=1024, V=1000), dict(wbar="shared", tau=True)),
    ("mfma_d512_three_tiles", "340m", dict(K=2, T=300, d=512, V=211), dict(tau=True, bias=True)),
    ("wide_d2560", "2b", dict(K=3, T=37, d=2560, V=300), ALL),
    ("wide_d2560_T1", "2b", dict(K=2, T=1, d=2560, V=77), dict(tau=True, bias=True)),
    ("wide_d2560_two_tiles", "2b", dict(K=2, T=60, d=2560, V=130), dict()),
    ("valu_f32", "tiny", dict(K=3, T=37, d=24, V=45), ALL),
    ("valu_bf16_d72", "340m", dict(K=2, T=10, d=72, V=50), ALL),
]


def run_exit_eval(x):
    import torch

    from paper_2609_35440_amd import binding

    f = _dev(x)
    out = binding.exit_eval(f["h"], f["gain"], f["W"], f["targets"], Wbar=f["Wbar"], tau=f["tau"], bias=f["bias"],
                            rot=f["rot"])
    torch.cuda.synchronize()
    return out.losses.double().cpu().numpy(), out.row_loss.double().cpu().numpy(), out.top1.cpu().numpy()


def check_exit_eval(x, losses, row_loss, top1, what, min_rows_for_agreement=1):
    """Exit-evaluation outputs against the oracle at the tolerances of the dtype."""
    ref = oracle.exit_eval(x["h"], x["gain"], x["W"], x["targets"], Wbar=x.get("Wbar"), tau=x.get("tau"),
                           bias=x.get("bias"))
    dtype = x["cfg"].dtype
    tol = TOL[dtype]
    # per-token losses within the bound derived from the kernel's operand rounding
    # (tests/gpu_helpers.row_loss_error_bound); a module loss, the mean of its
    # tokens, within the mean of their bounds, and within the relative 1e-3 of
    # the loss wherever that bound allows it
    K = losses.shape[0]
    for k in range(K):
        R = oracle.solo_oracle_general.readout_matrix(k, K, x["W"], x.get("Wbar"))
        gk = x["gain"][k] if x["gain"].ndim == 2 else x["gain"]
        tk = 1.0 if x.get("tau") is None else float(x["tau"][k])
        bk = None if x.get("bias") is None else x["bias"][k]
        bound = row_loss_error_bound(x["h"][k], gk, R, x["targets"][k], tk, dtype, bk)
        err = np.abs(row_loss[k] - ref["row_loss"][k])
        assert np.all(err <= bound), (what, k, float((err - bound).max()))
        lerr = abs(losses[k] - ref["losses"][k])
        assert lerr <= bound.mean(), (what, k, lerr, bound.mean())
        if bound.mean() <= tol["loss"] * abs(ref["losses"][k]):
            assert lerr <= tol["loss"] * abs(ref["losses"][k]), (what, k, lerr)
    # the top-1 is unique only up to ties and rounding: the chosen column must be a
    # maximiser of the fp64 logits within the error of the kernel's logits
    # (bf16 operands: about 2^-8 of |z|; fp32: 1e-5), and most rows agree exactly
    K, T = top1.shape
    ztol_rel = 1e-2 if dtype == "bf16" else 1e-5
    for k in range(K):
        for t in range(T):
            v = int(top1[k, t])
            assert 0 <= v < x["cfg"].V, (what, k, t, v)
            zv = ref["logits_of"](k, t, v)
            assert zv >= ref["zmax"][k, t] - ztol_rel * (1.0 + abs(ref["zmax"][k, t])), (what, k, t, v, zv,
                                                                                        ref["zmax"][k, t])
    agree = float((top1 == ref["top1"]).mean())
    log(f"{what}: top-1 agreement {agree:.4f}")
    if K * T >= min_rows_for_agreement:
        assert agree >= (0.95 if dtype == "bf16" else 0.99), (what, agree)
    # the eval losses equal the training call's losses (same forward)
    g = run_general(x, dict(final_module_dW=False))
    np.testing.assert_allclose(losses, g["losses"], rtol=1e-6, err_msg=what)


@pytest.mark.parametrize("name,cfg,ov,extras", EVAL_CASES, ids=[c[0] for c in EVAL_CASES])
def test_exit_eval_parity(name, cfg, ov, extras):
    x = make_extras(make_inputs(cfg, seed=31, **ov), 31, **extras)
    log(f"eval case {name}: {x['cfg']} extras {extras}")
    losses, row_loss, top1 = run_exit_eval(x)
    check_exit_eval(x, losses, row_loss, top1, name)


def test_exit_eval_ties_go_to_lowest_index():
    import torch

    from paper_2609_35440_amd import binding

    # duplicated readout rows give exactly equal logits; the lowest index must win
    x = make_inputs("340m", seed=33, K=2, T=40, d=256, V=64)
    W_bits = x["W_bits"].copy()
    W_bits[40] = W_bits[7]
    W_bits[63] = W_bits[7]
    W_bits[7] = np.uint16(0x4000)   # 2.0 everywhere: row 7 dominates, copied to 40 and 63
    W_bits[40] = W_bits[7]
    W_bits[63] = W_bits[7]
    h_bits = (x["h_bits"] & np.uint16(0x7FFF))   # |h| > 0: every logit of rows 7, 40, 63 is the largest
    dev = torch.device("cuda:0")
    up = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to(dev)
    gain = torch.ones(256, dtype=torch.bfloat16, device=dev)
    out = binding.exit_eval(up(h_bits), gain, up(W_bits), torch.from_numpy(x["targets"]).to(dev))
    torch.cuda.synchronize()
    top1 = out.top1.cpu().numpy()
    assert (top1 == 7).all(), np.unique(top1)
