"""The fp64 oracle against what the paper and the mathematics fix (CPU only)."""
import numpy as np
import pytest

import oracle
from tests import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle)


def test_w_zero_log_v_values():
    # loss = log V exactly at W = 0, for the vocabularies of the workloads
    import math

    for V in (512, 32000, 128256):
        want = math.log(V)
        h = np.random.default_rng(0).standard_normal((1, 3, 8))
        out = oracle.readout_fwd_bwd(h, np.ones(8), np.zeros((V, 8)), np.zeros((1, 3), np.int64), False)
        assert abs(out["losses"][0] - want) < 1e-12


def test_identical_targets_across_modules():
    # the paper's setting: every head sees the same minibatch targets
    h, gain, W, y = pins.tiny_case(11, K=3, T=6, d=8, V=7, same_targets=True)
    out = oracle.readout_fwd_bwd(h, gain, W, y, True)
    for k in range(3):
        rl, dh, _, _ = oracle.module_fwd_bwd(h[k], y[0], W, gain, want_readout_grads=False)
        np.testing.assert_allclose(out["dh"][k], dh, rtol=1e-14, atol=0)


def test_rejects_bad_inputs():
    h, gain, W, y = pins.tiny_case(0)
    with pytest.raises(ValueError):
        oracle.readout_fwd_bwd(h, gain, W, y + 100, True)
    h2 = h.copy()
    h2[0, 0, 0] = np.nan
    with pytest.raises(ValueError):
        oracle.readout_fwd_bwd(h2, gain, W, y, True)


def test_random_init_loss_sanity():
    # sanity, not parity: for random init, loss ~ log V + var(z)/2
    from solo_inputs import make_inputs

    x = make_inputs("340m", seed=0, K=1, T=256)
    out = oracle.readout_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], False)
    d = x["cfg"].d
    var_z = d * 0.02 ** 2 * float(np.mean(x["gain"].astype(np.float64) ** 2))
    assert abs(out["losses"][0] - (np.log(32000) + var_z / 2)) < 0.15
