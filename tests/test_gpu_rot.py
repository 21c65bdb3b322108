"""GPU parity of the ROT readout source (Appendix D, the table of readout
content and basis): head k reads the shared readout in a fixed basis R_k,
Wbar R_k.  The library rotates the heads' normalised rows instead of forming
Wbar R_k; the oracle is handed Wbar R_k itself (formed in fp64 from the stored
values) as one readout per head, so the two sides share nothing but the
inputs.  Element by element, on seeded inputs that span several tiles and
ragged tails, for every kernel family."""
import numpy as np
import pytest

import oracle
from solo_inputs import make_extras, make_inputs
from tests.gpu_helpers import TOL, log
from tests.test_gpu_general import compare, oracle_general, oracle_view, run_exit_eval, run_general

pytestmark = pytest.mark.gpu

ALL_ROT = dict(per_module_gain=True, tau=True, bias=True, rot=True)
ALL_FLAGS = dict(final_module_dW=True, want_dtau=True, want_dbias=True)
# (name, config, size overrides, input extras, call flags)
CASES = [
    ("mfma_d256_all", "340m", dict(K=3, T=70, d=256, V=300), ALL_ROT, ALL_FLAGS),
    ("mfma_d2048_shared_copy_tau", "1b", dict(K=3, T=65, d=2048, V=515), dict(wbar="shared", tau=True, rot=True),
     dict(final_module_dW=True, want_dtau=True)),
    ("mfma_d1024_frozen", "340m", dict(K=4, T=40, d=1024, V=200), dict(rot=True), dict(final_module_dW=False)),
    ("mfma_d2048_gain_per_module_bias", "1b", dict(K=2, T=33, d=2048, V=70),
     dict(per_module_gain=True, bias=True, rot=True), dict(final_module_dW=True, want_dbias=True)),
    ("mfma_d1536_dbias_without_bias", "340m", dict(K=3, T=45, d=1536, V=97), dict(rot=True),
     dict(final_module_dW=False, want_dbias=True, want_dtau=True)),
    ("mfma_T1", "340m", dict(K=2, T=1, d=256, V=60), ALL_ROT, ALL_FLAGS),
    ("wide_d2560_all", "2b", dict(K=3, T=37, d=2560, V=300), ALL_ROT, ALL_FLAGS),
    ("valu_f32_all", "tiny", dict(K=3, T=37, d=24, V=45), ALL_ROT, ALL_FLAGS),
    ("valu_bf16_d72_all", "340m", dict(K=2, T=10, d=72, V=50), ALL_ROT, ALL_FLAGS),
    # vector-ALU passes at a width whose rotation products run on the matrix cores
    ("valu_bf16_d3072_all", "1b", dict(K=2, T=20, d=3072, V=40), ALL_ROT, ALL_FLAGS),
    ("valu_f32_d256", "tiny", dict(K=3, T=21, d=256, V=30), dict(tau=True, rot=True),
     dict(final_module_dW=True, want_dtau=True)),
]


@pytest.mark.parametrize("name,cfg,ov,extras,flags", CASES, ids=[c[0] for c in CASES])
def test_rot_parity(name, cfg, ov, extras, flags):
    x = make_extras(make_inputs(cfg, seed=41, **ov), 41, **extras)
    log(f"rot case {name}: {x['cfg']} extras {extras} flags {flags}")
    g = run_general(x, flags)
    ref = oracle_general(x, flags)
    compare(g, ref, x["cfg"].dtype, flags, f"rot {name}")


@pytest.mark.parametrize("cfg,ov", [("1b", dict(K=3, T=70, d=2048, V=300)), ("2b", dict(K=3, T=37, d=2560, V=130)),
                                    ("tiny", dict(K=3, T=37, d=24, V=45))], ids=["mfma", "wide", "valu_f32"])
def test_identity_rotation_is_solo(cfg, ov):
    """R_k = I turns ROT into SOLO.  On the matrix-core families the rotated rows
    are bf16(g * h) itself, the operand the plain call rounds, so every logit,
    loss, row loss, readout and bias gradient is bit for bit the plain call's
    (the vector-ALU family multiplies r, g and h in another order: to fp32
    rounding).  The input and gain gradients go through the rotate-back product
    (e split into two bf16 parts) and agree to its rounding (dh to one unit of
    its storage dtype's last place); the temperature
    gradient sums e * u over the rounded rows instead of the unrounded g * h."""
    x = make_extras(make_inputs(cfg, seed=42, **ov), 42, per_module_gain=True, tau=True, bias=True)
    flags = dict(final_module_dW=True, want_dtau=True, want_dbias=True)
    a = run_general(x, flags)
    xi = dict(x)
    K, d = x["cfg"].K, x["cfg"].d
    eye = np.broadcast_to(np.eye(d, dtype=np.float32), (K - 1, d, d)).copy()
    xi["rot"] = eye
    xi["rot_bits"] = (eye.view(np.uint32) >> 16).astype(np.uint16)
    b = run_general(xi, flags)
    exact = x["cfg"].dtype == "bf16"
    for key in ("losses", "row_loss", "dW", "dbias"):
        if exact:
            np.testing.assert_array_equal(a[key], b[key], err_msg=key)
        else:
            np.testing.assert_allclose(b[key], a[key], rtol=1e-5, atol=1e-6 * np.abs(a[key]).max(), err_msg=key)
    # dh is stored in the dtype: the two fp32 values may round to neighbouring bf16 values
    ulp = 2.0 ** -7 if exact else 2.0 ** -22  # one unit in the last place is at most this relative
    diff = np.abs(a["dh"] - b["dh"])
    slack = diff - ulp * np.abs(a["dh"]) - 1e-4 * np.abs(a["dh"]).max()
    log(f"identity rotation {cfg}: dh max diff {diff.max():.2e} (max |dh| {np.abs(a['dh']).max():.2e})")
    assert slack.max() <= 0, float(slack.max())
    for key, tol in (("dgain", 1e-4), ("dtau", TOL["bf16"]["grad"])):
        err = np.abs(a[key] - b[key]).max() / np.abs(a[key]).max()
        log(f"identity rotation {cfg}: {key} rel diff {err:.2e}")
        assert err <= tol, (key, err)


def test_rot_bitwise_determinism():
    x = make_extras(make_inputs("1b", seed=44, K=3, T=64, d=2048, V=400), 44, **ALL_ROT)
    a = run_general(x, ALL_FLAGS)
    b = run_general(x, ALL_FLAGS)
    for key, v in a.items():
        if v is not None:
            np.testing.assert_array_equal(v, b[key], err_msg=key)


EVAL_CASES = [
    ("mfma_d2048", "1b", dict(K=3, T=65, d=2048, V=515), dict(tau=True, bias=True, rot=True)),
    ("mfma_d512_shared", "340m", dict(K=3, T=300, d=512, V=211), dict(wbar="shared", rot=True)),
    ("wide_d2560", "2b", dict(K=3, T=37, d=2560, V=300), dict(per_module_gain=True, tau=True, rot=True)),
    ("valu_f32", "tiny", dict(K=3, T=37, d=24, V=45), dict(tau=True, bias=True, rot=True)),
    ("valu_bf16_d72", "340m", dict(K=2, T=10, d=72, V=50), dict(bias=True, rot=True)),
]


@pytest.mark.parametrize("name,cfg,ov,extras", EVAL_CASES, ids=[c[0] for c in EVAL_CASES])
def test_rot_exit_eval(name, cfg, ov, extras):
    x = make_extras(make_inputs(cfg, seed=45, **ov), 45, **extras)
    dtype = x["cfg"].dtype
    tol = TOL[dtype]
    losses, row_loss, top1 = run_exit_eval(x)
    xo = oracle_view(x)
    ref = oracle.exit_eval(xo["h"], xo["gain"], xo["W"], xo["targets"], Wbar=xo["Wbar"], tau=xo.get("tau"),
                           bias=xo.get("bias"))
    rel = np.abs(losses - ref["losses"]) / np.abs(ref["losses"])
    assert np.all(rel <= tol["loss"]), (name, rel)
    rscale = max(np.abs(ref["row_loss"]).max(), 1.0)
    assert np.abs(row_loss - ref["row_loss"]).max() <= 2 * tol["loss"] * rscale, name
    # the chosen column maximises the fp64 logits within the error of the kernel's logits
    ztol_rel = 1e-2 if dtype == "bf16" else 1e-5
    K, T = top1.shape
    for k in range(K):
        for t in range(T):
            v = int(top1[k, t])
            zv, zm = ref["logits_of"](k, t, v), ref["zmax"][k, t]
            assert zv >= zm - ztol_rel * (1.0 + abs(zm)), (name, k, t, v, zv, zm)
    agree = float((top1 == ref["top1"]).mean())
    log(f"rot eval {name}: loss rel err {rel.max():.2e}, top-1 agreement {agree:.4f}")
    assert agree >= (0.95 if dtype == "bf16" else 0.99)
    # the forward of the training call computes the same losses
    g = run_general(x, dict(final_module_dW=False))
    np.testing.assert_allclose(losses, g["losses"], rtol=1e-6, err_msg=name)


@pytest.mark.parametrize("cfg,ov", [("1b", dict(K=3, T=45, d=2048, V=300)), ("2b", dict(K=2, T=30, d=2560, V=90))],
                         ids=["mfma", "wide"])
def test_rot_needs_no_orthogonality(cfg, ov):
    """The library applies R_k forward and R_k^T backward as given (the gradient
    of <Wbar_v R_k, hhat> is R_k^T Wbar_v^T, whatever R_k is), so a matrix that
    is far from orthogonal (Gaussian entries of variance 1/d) must match the
    oracle handed Wbar R_k just as well."""
    from solo_inputs import bf16_bits, bf16_from_bits

    x = make_extras(make_inputs(cfg, seed=47, **ov), 47, tau=True, per_module_gain=True, rot=True)
    K, d = x["cfg"].K, x["cfg"].d
    r = (np.random.default_rng(47).standard_normal((K - 1, d, d)) / np.sqrt(d)).astype(np.float32)
    x["rot_bits"] = bf16_bits(r)
    x["rot"] = bf16_from_bits(x["rot_bits"])
    flags = dict(final_module_dW=True, want_dtau=True)
    compare(run_general(x, flags), oracle_general(x, flags), x["cfg"].dtype, flags, f"rot {cfg} gaussian R")
