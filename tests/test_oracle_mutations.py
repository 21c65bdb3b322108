"""Planted mistakes in a copy of the oracle must each fail at least one pin.

The oracle's source is copied, one plausible mistake is applied to the copy
(a dropped term, a wrong sign, a wrong factor or operand), the copy is loaded
as a separate module and the pins of tests/oracle_pins.py are run on it.  Only
the copy is changed, on the CPU.
"""
import importlib.util
import os
import sys
import types

import pytest

from tests import oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "solo_oracle.py")

MUTANTS = {
    "drop_norm_projection": ("dh[t0:t1] = r[:, None] * (dn - c[:, None] * n)", "dh[t0:t1] = r[:, None] * dn"),
    "onehot_sign": ("delta[rows, yc] -= 1.0", "delta[rows, yc] += 1.0"),
    "drop_mean_factor": ("delta /= float(T_total)", "pass"),
    "drop_gain_in_backward": ("dn = dhhat * g", "dn = dhhat"),
    "dgain_wrong_operand": ("dgain += np.sum(dhhat * n, axis=0)", "dgain += np.sum(dhhat * hhat, axis=0)"),
    "sum_not_mean_square": ("ms = np.mean(h * h, axis=-1)", "ms = np.sum(h * h, axis=-1)"),
    "lse_drops_shift": ("lse = m + np.log(", "lse = np.log("),
    "eps_outside_sqrt": ("r = 1.0 / np.sqrt(ms + float(eps))", "r = 1.0 / (np.sqrt(ms) + float(eps))"),
    "wrong_target_index": ("row_loss[t0:t1] = lse - z[rows, yc]", "row_loss[t0:t1] = lse - z[rows, (yc + 1) % z.shape[1]]"),
    "dW_uses_n_not_hhat": ("dW += delta.T @ hhat", "dW += delta.T @ n"),
    "softmax_without_exp": ("e = np.exp(z - m)", "e = z - m"),
    "softmax_without_shift": ("e = np.exp(z - m)", "e = np.exp(z)"),
    "frozen_gets_dW": [
        ("want = bool(final_module_dW) and k == K - 1", "want = bool(final_module_dW)"),
        ("dW, dgain = dWk, dgk", "dW, dgain = (dWk, dgk) if dW is None else (dW + dWk, dgain + dgk)"),
    ],
}


def _load_mutant(name, edits):
    with open(SRC) as f:
        text = f.read()
    if isinstance(edits, tuple):
        edits = [edits]
    for old, new in edits:
        assert text.count(old) >= 1, f"mutation anchor not found: {old}"
        text = text.replace(old, new)
    mod = types.ModuleType(f"oracle_mutant_{name}")
    mod.__file__ = f"<mutant {name}>"
    exec(compile(text, mod.__file__, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _load_mutant(name, MUTANTS[name])
    failures = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, FloatingPointError) as e:  # a pin rejected the mutant
            failures.append(pin.__name__)
    assert failures, f"mutant {name} passed every pin"


def test_unmutated_copy_passes():
    mod = _load_mutant("identity", ("import numpy as np", "import numpy as np"))
    for pin in pins.ALL_PINS:
        pin(mod)
