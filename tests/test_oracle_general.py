"""The general fp64 oracle against what the paper and the mathematics fix (CPU only)."""
import importlib.util
import os
import types

import numpy as np
import pytest

import oracle
from tests import oracle_general_pins as gp


@pytest.mark.parametrize("pin", gp.ALL_PINS, ids=lambda p: p.__name__)
def test_general_pin(pin):
    pin(oracle.solo_oracle_general)


def test_general_rejects_bad_inputs():
    c = gp.case(0)
    g = oracle.solo_oracle_general
    with pytest.raises(ValueError):
        g.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"] + 100, Wbar=c["Wbar"])
    with pytest.raises(ValueError):   # PRIV needs one readout per head
        g.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], Wbar=None, heads_train_readout=True)
    with pytest.raises(ValueError):
        g.general_fwd_bwd(c["h"], c["gain"], c["W"], c["targets"], tau=np.ones(2))


SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "solo_oracle_general.py")

MUTANTS = {
    "tau_missing_in_backward": ("dhhat = tk * (delta @ Wk)", "dhhat = delta @ Wk"),
    "dtau_uses_z": ("dtau[k] += float(np.sum(delta * u))", "dtau[k] += float(np.sum(delta * z))"),
    "dbias_sign": ("dbias[k] += delta.sum(axis=0)", "dbias[k] -= delta.sum(axis=0)"),
    "bias_dropped": ("z = tk * u + bk ", "z = tk * u "),
    "priv_missing_tau": ("dWbar[k] += tk * (delta.T @ hhat)", "dWbar[k] += delta.T @ hhat"),
    "head_reads_wrong_copy": ("return Wbar if Wbar.ndim == 2 else Wbar[k]",
                              "return Wbar if Wbar.ndim == 2 else Wbar[(k + 1) % Wbar.shape[0]]"),
    "gain_of_module_zero": ("gk = gain[k] if per_module_gain else gain", "gk = gain[0] if per_module_gain else gain"),
    "dgain_uses_hhat": ("dgain[k] += np.sum(dhhat * n, axis=0)", "dgain[k] += np.sum(dhhat * hhat, axis=0)"),
    "terminal_uses_copy": ("if k == K - 1 or Wbar is None:\n        return W", "if Wbar is None:\n        return W"),
    "top1_last_index": ("top1[k, t0:t1] = np.argmax(z, axis=1)",
                        "top1[k, t0:t1] = z.shape[1] - 1 - np.argmax(z[:, ::-1], axis=1)"),
}


def _load(edits):
    text = open(SRC).read()
    for old, new in ([edits] if isinstance(edits, tuple) else edits):
        assert old in text, old
        text = text.replace(old, new)
    mod = types.ModuleType("oracle_general_mutant")
    exec(compile(text, "<mutant>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_general_mutant_is_caught(name):
    mod = _load(MUTANTS[name])
    caught = []
    for pin in gp.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
