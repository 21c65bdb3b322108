"""The FLOP accounting helper against the values printed in the paper.

Fixtures: tests/golden/flops_table.json (FLOP table, rho sweep, per-stage check,
Eq. "win", pipe-shapes table; each entry cites its table or equation).
"""
import json
import os

import pytest

from paper_2609_35440_amd import costmodel as cm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "flops_table.json")


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_flops_table_rows(golden):
    for row in golden["flops_rows"]:
        got = cm.flops_per_token(row["L"], row["d"], row["K"], row["H"], row["T"], row["V"])
        for key in ("bp_total", "bp_layers", "solo_total", "aux_blocks"):
            assert abs(got[key] - row[key]) <= 0.0051, (row["model"], key, got[key], row[key])
        # 2B readout: printed 1.48 vs 1.4746 without the V bias entries
        tol = 0.01 if row["model"] == "2B" else 0.0051
        assert abs(got["readouts"] - row["readouts"]) <= tol, (row["model"], got["readouts"])
        assert abs(got["rho"] - row["rho"]) <= 0.00051, (row["model"], got["rho"])


def test_rho_sweep_340m(golden):
    s = golden["rho_340m_sweep"]
    for H in (1, 2):
        for K, want in s[f"H{H}"].items():
            got = cm.rho(s["L"], s["d"], int(K), H, s["T"], s["V"])
            assert abs(got - want) <= 0.00051, (H, K, got, want)


def test_stage_check_prediction(golden):
    s = golden["stage_check"]
    assert abs(cm.rho(s["L"], s["d"], s["K"], 1, s["T"], s["V"]) - s["rho_H1"]) < 5e-5
    assert abs(cm.rho(s["L"], s["d"], s["K"], 2, s["T"], s["V"]) - s["rho_H2"]) < 5e-5


def test_mstar(golden):
    a = golden["mstar_config_A"]
    assert abs(cm.mstar(a["L"], a["d"], a["H"], a["T"], a["V"]) - a["mstar"]) < 0.05
    for row in golden["pipe_shapes"]:
        for H in (1, 2):
            got = cm.mstar(row["L"], row["d"], H, row["T"], row["V"])
            assert abs(got - row[f"H{H}"]) <= 0.051, (row, H, got)
    s = golden["shallow_eight_modules"]
    assert abs(cm.rho(s["L"], s["d"], s["K"], s["H"], s["T"], s["V"]) - s["rho"]) < 0.005
    assert round(cm.mstar(s["L"], s["d"], s["H"], s["T"], s["V"])) == s["mstar"]


def test_readout_flops_matches_table_units():
    # per token, the readout column of the FLOP table equals readout_flops / T
    for L, d, K, H in [(24, 1024, 2, 2), (24, 2048, 2, 2), (24, 2560, 4, 2)]:
        t = cm.flops_per_token(L, d, K, H, 2048, 32000)
        assert abs(cm.readout_flops(K, 1, 32000, d) * 1e-9 - t["readouts"]) < 1e-9


def test_readout_flops_headline_value():
    # K=4, T=16384, d=2048, V=32000: 2 * 9 * T * V * d
    assert cm.readout_flops(4, 16384, 32000, 2048) == 2 * 9 * 16384 * 32000 * 2048
    assert cm.readout_flops(4, 16384, 32000, 2048, final_module_dW=False) == 2 * 8 * 16384 * 32000 * 2048
    assert cm.readout_bytes(1, 1, 1, 8, 2) == 2 * 8 * 2 + 8 * 2 + 8 * 2 + 4 + 4 + 8 * 4 + 8 * 4


def test_general_flops_special_cases():
    from paper_2609_35440_amd import costmodel as cm

    K, T, V, d = 4, 16384, 32000, 2048
    r2 = 2 * T * V * d          # one readout unit (r MACs per token) in FLOPs
    # the headline call is the paper's FLOP-table count: 2r per head, 3r for the terminal
    assert cm.general_flops(K, T, V, d) == cm.readout_flops(K, T, V, d, True) == (2 * K + 1) * r2
    assert cm.general_flops(K, T, V, d, final_module_dW=False) == cm.readout_flops(K, T, V, d, False)
    # PRIV: every module pays 3r
    assert cm.general_flops(K, T, V, d, heads_train_readout=True) == 3 * K * r2
    # exit evaluation: the forward product of every exit
    assert cm.general_flops(K, T, V, d, exit_eval=True) == K * r2
    # executed: local pass 2r per module, readout-gradient pass 2r per trained readout,
    # bias-gradient pass 1r for each other module
    assert cm.executed_flops(K, T, V, d) == (2 * K + 2) * r2
    assert cm.executed_flops(K, T, V, d, bias_grad=True) == (2 * K + 2 + (K - 1)) * r2
    assert cm.executed_flops(K, T, V, d, heads_train_readout=True, bias_grad=True) == 4 * K * r2
    assert cm.executed_flops(K, T, V, d, final_module_dW=False, bias_grad=True) == 3 * K * r2
    assert cm.executed_flops(K, T, V, d, exit_eval=True) == K * r2
    # ROT: the heads' rows rotated (2 T d^2 each), and their gradients rotated back
    assert cm.executed_flops(K, T, V, d, rot=True) - cm.executed_flops(K, T, V, d) == 2 * (K - 1) * 2 * T * d * d
    assert cm.executed_flops(K, T, V, d, rot=True, exit_eval=True) - K * r2 == (K - 1) * 2 * T * d * d
    assert cm.executed_flops(1, T, V, d, rot=True) == cm.executed_flops(1, T, V, d)
    # 1B headline: 19.33 TFLOP algorithmic, 21.47 executed
    assert abs(cm.general_flops(K, T, V, d) / 1e12 - 19.33) < 0.01
    assert abs(cm.executed_flops(K, T, V, d) / 1e12 - 21.47) < 0.01
