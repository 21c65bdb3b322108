"""GPU parity of the HIP path with the fp64 oracle, element by element, on
seeded inputs at sizes that span several tiles and ragged tails, for every
kernel family and slice width; plus edge and degenerate cases."""
import math

import numpy as np
import pytest

import oracle
from solo_inputs import make_inputs
from tests.gpu_helpers import check_close, log, run_gpu, to_device

pytestmark = pytest.mark.gpu

# (name, config, overrides, final_module_dW): small shapes, ragged in T and V
CASES = [
    ("tiny_f32", "tiny", {}, True),
    ("f32_ragged", "tiny", dict(K=3, T=37, d=24, V=45), True),
    ("f32_d2048", "tiny", dict(K=2, T=19, d=2048, V=70), True),
    ("mfma_d256", "340m", dict(K=2, T=100, d=256, V=1000), True),
    ("mfma_d512_K1", "340m", dict(K=1, T=33, d=512, V=33), True),
    ("mfma_d768", "340m", dict(K=2, T=40, d=768, V=200), True),
    ("mfma_d1024", "340m", dict(K=2, T=70, d=1024, V=777), True),
    ("mfma_d1536", "340m", dict(K=2, T=35, d=1536, V=129), True),
    ("mfma_d2048", "1b", dict(K=2, T=65, d=2048, V=515), True),
    ("mfma_d2048_frozen_only", "1b", dict(K=3, T=64, d=2048, V=320), False),
    ("mfma_large_vocab_hot", "large_vocab", dict(K=2, T=256, d=2048, V=4099), True),
    ("mfma_2b_scaled", "2b", dict(K=3, T=50, d=2048, V=100), True),
    ("wide_d2560", "2b", dict(K=2, T=40, d=2560, V=300), True),
    ("wide_d2560_ragged", "2b", dict(K=3, T=37, d=2560, V=515), True),
    ("wide_d2560_frozen_only", "2b", dict(K=2, T=33, d=2560, V=129), False),
    ("wide_d2560_V1", "2b", dict(K=2, T=20, d=2560, V=1), True),
    ("wide_d2560_T1", "2b", dict(K=2, T=1, d=2560, V=77), True),
    ("valu_d72", "340m", dict(K=2, T=10, d=72, V=50), True),
    ("valu_d3072", "2b", dict(K=2, T=9, d=3072, V=37), True),
    ("valu_d4096_max", "1b", dict(K=2, T=5, d=4096, V=33), True),
    ("f32_d4096_max", "tiny", dict(K=2, T=4, d=4096, V=19), True),
    ("mfma_V1", "340m", dict(K=2, T=40, d=256, V=1), True),
    ("mfma_V2", "340m", dict(K=2, T=40, d=256, V=2), True),
    ("mfma_T1", "340m", dict(K=2, T=1, d=256, V=60), True),
    ("mfma_V17_T33", "1b", dict(K=2, T=33, d=2048, V=17), True),
]


@pytest.mark.parametrize("name,cfg,ov,fdw", CASES, ids=[c[0] for c in CASES])
def test_parity(name, cfg, ov, fdw):
    x = make_inputs(cfg, seed=11, **ov)
    log(f"case {name}: {x['cfg']}")
    g = run_gpu(x, fdw)
    ref = oracle.readout_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], fdw)
    check_close(g, ref, x["cfg"].dtype, what=name)
    # per-token losses too, and the module loss is their mean
    tol = 1e-3 if x["cfg"].dtype == "bf16" else 1e-5
    scale = max(np.abs(ref["row_loss"]).max(), 1e-30)
    assert np.abs(g["row_loss"] - ref["row_loss"]).max() <= 2 * tol * max(scale, 1.0)
    np.testing.assert_allclose(g["row_loss"].mean(axis=1), g["losses"], rtol=1e-5, atol=1e-6)
    if not fdw:
        assert g["dW"] is None and g["dgain"] is None


def test_w_zero_closed_form():
    # W = 0: loss = log V exactly, dh = 0, dgain = 0, dW = (1/T)[(1/V) sum_t hhat_t - sum_{t: y_t = v} hhat_t]
    x = make_inputs("1b", seed=3, K=2, T=64, d=2048, V=300)
    x["W"][:] = 0.0
    x["W_bits"][:] = 0
    g = run_gpu(x, True)
    log(f"W=0: losses {g['losses']} vs log V {math.log(300)}")
    np.testing.assert_allclose(g["losses"], math.log(300), rtol=1e-6)
    assert np.abs(g["dh"]).max() == 0.0
    assert np.abs(g["dgain"]).max() == 0.0
    ref = oracle.readout_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], True)
    assert np.abs(ref["dh"]).max() == 0.0
    check_close(g, ref, "bf16", what="W=0")


def test_identical_targets_across_modules():
    # the paper's setting: every head sees the minibatch's targets
    x = make_inputs("1b", seed=5, K=3, T=48, d=2048, V=400)
    x["targets"][:] = x["targets"][0]
    g = run_gpu(x, True)
    ref = oracle.readout_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], True)
    check_close(g, ref, "bf16", what="same targets")


def test_bitwise_determinism_and_module_independence():
    import torch

    x = make_inputs("340m", seed=7, K=3, T=96, d=1024, V=700)
    a = run_gpu(x, True)
    b = run_gpu(x, True)
    for key in ("losses", "row_loss", "dh", "dW", "dgain"):
        np.testing.assert_array_equal(a[key], b[key])
    # a read-only copy's module does not touch the readout gradient
    x2 = dict(x)
    h_bits = x["h_bits"].copy()
    rng = np.random.default_rng(99)
    h_bits[0] = rng.integers(0, 2 ** 15, size=h_bits[0].shape, dtype=np.uint16) & 0x3FFF
    x2["h_bits"] = h_bits
    c = run_gpu(x2, True)
    np.testing.assert_array_equal(c["dW"], a["dW"])
    np.testing.assert_array_equal(c["dgain"], a["dgain"])
    np.testing.assert_array_equal(c["dh"][1:], a["dh"][1:])
    np.testing.assert_array_equal(c["losses"][1:], a["losses"][1:])
    torch.cuda.synchronize()


def test_invalid_target_reports_nan_without_fault():
    x = make_inputs("340m", seed=8, K=2, T=40, d=256, V=100)
    x["targets"][0, 5] = 100      # out of range
    x["targets"][0, 6] = -3
    g = run_gpu(x, True)
    assert np.isnan(g["row_loss"][0, 5]) and np.isnan(g["row_loss"][0, 6])
    assert np.isnan(g["losses"][0])
    assert np.isfinite(g["losses"][1]) and np.all(np.isfinite(g["dh"][1]))
    ref = oracle.readout_fwd_bwd(x["h"][1:], x["gain"], x["W"], x["targets"][1:], True)
    g1 = {k: (v[1:] if k in ("losses", "row_loss", "dh") else v) for k, v in g.items()}
    check_close(g1, ref, "bf16", what="valid module next to invalid targets")


def test_scale_invariance_on_gpu():
    # I5: loss(c h) = loss(h), dh(c h) = dh(h) / c (eps << mean h^2); exact powers of two keep bf16 exact
    x = make_inputs("1b", seed=9, K=2, T=64, d=2048, V=256)
    a = run_gpu(x, True)
    x4 = dict(x)
    x4["h_bits"] = (x["h_bits"].astype(np.uint32) + (2 << 7)).astype(np.uint16)  # multiply by 4 via exponent
    x4["h"] = x["h"] * 4
    b = run_gpu(x4, True)
    np.testing.assert_allclose(b["losses"], a["losses"], rtol=1e-5)
    assert np.abs(b["dh"] * 4 - a["dh"]).max() <= 2e-2 * np.abs(a["dh"]).max()


def test_shift_invariance_on_gpu():
    # I4: W -> W + 1 u^T leaves loss and gradients unchanged (within bf16 tolerance)
    x = make_inputs("1b", seed=10, K=2, T=64, d=2048, V=256)
    a = run_gpu(x, True)
    from solo_inputs import bf16_bits, bf16_from_bits

    u = bf16_from_bits(bf16_bits(np.random.default_rng(4).standard_normal(2048).astype(np.float32) * 0.02))
    Ws = bf16_from_bits(bf16_bits(x["W"] + u[None, :]))
    xs = dict(x)
    xs["W"], xs["W_bits"] = Ws, bf16_bits(Ws)
    b = run_gpu(xs, True)
    ref = oracle.readout_fwd_bwd(xs["h"], xs["gain"], xs["W"], xs["targets"], True)
    check_close(b, ref, "bf16", what="shifted W")
    np.testing.assert_allclose(b["losses"], a["losses"], rtol=2e-3)
