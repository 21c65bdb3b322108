"""The seeded input generator: determinism, bf16 rounding, distributions."""
import numpy as np
import pytest

from solo_inputs import CONFIGS, bf16_bits, bf16_from_bits, make_inputs, round_bf16, zipf_targets


def test_bf16_rne_known_values():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 0.0, -0.0, 65504.0,
                  3.0e38, np.inf, -np.inf], dtype=np.float32)
    got = bf16_from_bits(bf16_bits(x))
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: ties to even -> 1
    # 1 + 3*2^-8 is a tie between 1+2^-7 and 1+2^-6: ties to even -> 1 + 2^-6
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5, 0.0, -0.0, 65536.0, 2.9999e38, np.inf, -np.inf],
                    dtype=np.float32)
    np.testing.assert_array_equal(got[:8], want[:8])
    assert np.isinf(got[9]) and got[9] > 0 and np.isinf(got[10]) and got[10] < 0
    assert abs(got[8] - 3.0e38) / 3.0e38 < 2 ** -8
    assert np.isnan(bf16_from_bits(bf16_bits(np.array([np.nan], np.float32))))[0]


def test_bf16_rounding_error_bound():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(100000).astype(np.float32)
    y = round_bf16(x)
    rel = np.abs(y - x) / np.abs(x)
    # unit roundoff of an 8-bit significand: 2^-8
    assert rel.max() <= 2.0 ** -8 * (1 + 1e-6)
    assert rel.max() > 2.0 ** -9
    # idempotent
    np.testing.assert_array_equal(round_bf16(y), y)


def test_determinism_and_seed_dependence():
    a = make_inputs("tiny", seed=3)
    b = make_inputs("tiny", seed=3)
    c = make_inputs("tiny", seed=4)
    for key in ("h", "gain", "W", "targets"):
        np.testing.assert_array_equal(a[key], b[key])
    assert not np.array_equal(a["h"], c["h"])


def test_shapes_and_overrides():
    x = make_inputs("340m", seed=0, K=2, T=100, V=1007)
    assert x["h"].shape == (2, 100, 1024) and x["W"].shape == (1007, 1024)
    assert x["targets"].shape == (2, 100) and x["targets"].dtype == np.int32
    assert x["targets"].min() >= 0 and x["targets"].max() < 1007
    # bf16 values are exactly their bit patterns
    np.testing.assert_array_equal(bf16_from_bits(x["h_bits"]), x["h"])


def test_distribution_moments():
    x = make_inputs("340m", seed=0, K=1, T=2048)
    assert abs(x["h"].std() - 1.0) < 0.01
    assert abs(x["W"].std() - 0.02) < 0.0005
    assert abs(x["gain"].mean() - 1.0) < 0.02 and abs(x["gain"].std() - 0.1) < 0.01
    x2 = make_inputs("2b", seed=0, T=64, V=64)
    for k in range(8):
        assert abs(x2["h"][k].std() - (1 + 0.25 * k)) < 0.02 * (1 + 0.25 * k)


def test_zipf_mass():
    rng = np.random.default_rng(0)
    y = zipf_targets(rng, (400000,), 32000, 1.1)
    ranks = np.arange(1, 32001, dtype=np.float64) ** -1.1
    p0 = 1.0 / ranks.sum()
    assert abs((y == 0).mean() - p0) < 0.003
    assert abs(p0 - 0.142) < 0.001
    # monotone-ish: token 0 more frequent than token 1 more frequent than token 10
    counts = np.bincount(y, minlength=32000)
    assert counts[0] > counts[1] > counts[10]


def test_hot_token_fraction():
    x = make_inputs("large_vocab", seed=0, T=4096, V=1000, d=64)
    for k in range(x["cfg"].K):
        frac = (x["targets"][k] == 999).mean()
        assert 0.01 <= frac < 0.02


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_config_table(name):
    cfg = CONFIGS[name]
    assert cfg.d % 8 == 0 and cfg.K >= 1 and cfg.T >= 1 and cfg.V >= 1


def test_random_rotations():
    # orthogonal to fp64 rounding before storage; rounded once to the dtype; seeded
    from solo_inputs import make_extras, random_orthogonal

    q = random_orthogonal(np.random.default_rng(0), 3, 64)
    for r in q:
        assert np.abs(r.T @ r - np.eye(64)).max() < 1e-12
    x = make_extras(make_inputs("340m", seed=1, K=3, T=8, d=256, V=16), 1, rot=True)
    r = x["rot"]
    assert r.shape == (2, 256, 256) and r.dtype == np.float32
    np.testing.assert_array_equal(r, round_bf16(r))
    # bf16 storage keeps each R_k orthogonal to about 2^-8
    for rk in r.astype(np.float64):
        assert np.abs(rk.T @ rk - np.eye(256)).max() < 2e-2
    y = make_extras(make_inputs("340m", seed=1, K=3, T=8, d=256, V=16), 1, rot=True)
    np.testing.assert_array_equal(x["rot_bits"], y["rot_bits"])
    z = make_extras(make_inputs("340m", seed=1, K=3, T=8, d=256, V=16), 2, rot=True)
    assert not np.array_equal(x["rot_bits"], z["rot_bits"])
    assert make_extras(make_inputs("340m", seed=1, K=3, T=8, d=256, V=16), 1)["rot"] is None
