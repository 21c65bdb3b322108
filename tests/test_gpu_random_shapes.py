"""GPU parity on a seeded sweep of random shapes: every kernel family and
tiling (32- and 64-row matrix-core tiles, the wide tiling, the vector-ALU
family in bf16 and fp32), random module counts, ragged token and vocabulary
counts, with and without the final module's readout gradient, the general
entry point with random option sets, and exit evaluation across the
forward-only tilings (128, 64 and 48 rows).  Each case is compared element by
element with the fp64 oracle at the tolerances of its dtype."""
import zlib

import numpy as np
import pytest

import oracle
from solo_inputs import make_extras, make_inputs
from tests.gpu_helpers import check_close, log, run_gpu
from tests.test_gpu_general import check_exit_eval, compare, oracle_general, run_exit_eval, run_general

pytestmark = pytest.mark.gpu

# widths per family: 64-row tiles (d <= 1024), 32-row tiles, the wide tiling,
# bf16 widths of the vector-ALU family, fp32 (always vector-ALU)
WIDTHS_BF16 = [256, 512, 768, 1024, 1280, 1536, 1792, 2048, 2560, 40, 136]
WIDTHS_F32 = [16, 64, 200]


def _cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        f32 = rng.random() < 0.2
        d = int(rng.choice(WIDTHS_F32 if f32 else WIDTHS_BF16))
        K = int(rng.integers(1, 4))
        T = int(rng.integers(1, 150))
        V = int(rng.integers(1, 700))
        fdw = bool(rng.random() < 0.75)
        out.append((f"r{i}_{'f32' if f32 else 'bf16'}_K{K}_T{T}_d{d}_V{V}_{'dW' if fdw else 'frozen'}",
                    "tiny" if f32 else "1b", dict(K=K, T=T, d=d, V=V), fdw))
    return out


CASES = _cases(24, 2026)


@pytest.mark.parametrize("name,cfg,ov,fdw", CASES, ids=[c[0] for c in CASES])
def test_random_shape_parity(name, cfg, ov, fdw):
    x = make_inputs(cfg, seed=zlib.crc32(name.encode()) % 1000, **ov)
    log(f"case {name}")
    g = run_gpu(x, fdw)
    ref = oracle.readout_fwd_bwd(x["h"], x["gain"], x["W"], x["targets"], fdw)
    check_close(g, ref, x["cfg"].dtype, what=name)
    np.testing.assert_allclose(g["row_loss"].mean(axis=1), g["losses"], rtol=1e-5, atol=1e-6)


def _general_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        d = [256, 1024, 2048, 2560, 72][i % 5]  # every family in turn
        K = int(rng.integers(1, 4))
        T = int(rng.integers(1, 90))
        V = int(rng.integers(1, 400))
        extras = dict(per_module_gain=bool(rng.random() < 0.5), tau=bool(rng.random() < 0.5),
                      bias=bool(rng.random() < 0.5),
                      wbar=str(rng.choice(["none", "shared", "per_head"] if K > 1 else ["none", "shared"])))
        if extras["wbar"] == "none":
            extras.pop("wbar")
        priv = extras.get("wbar") == "per_head" and bool(rng.random() < 0.5)
        flags = dict(final_module_dW=bool(rng.random() < 0.75), heads_train_readout=priv,
                     want_dtau=bool(rng.random() < 0.5), want_dbias=bool(rng.random() < 0.5))
        out.append((f"g{i}_K{K}_T{T}_d{d}_V{V}", dict(K=K, T=T, d=d, V=V), extras, flags))
    return out


GENERAL_CASES = _general_cases(12, 7)


@pytest.mark.parametrize("name,ov,extras,flags", GENERAL_CASES, ids=[c[0] for c in GENERAL_CASES])
def test_random_general_parity(name, ov, extras, flags):
    cfg = "2b" if ov["d"] == 2560 else "1b"
    x = make_extras(make_inputs(cfg, seed=zlib.crc32(name.encode()) % 1000, **ov), 5, **extras)
    log(f"general case {name}: extras {extras} flags {flags}")
    g = run_general(x, flags)
    ref = oracle_general(x, flags)
    compare(g, ref, x["cfg"].dtype, flags, name)


def _rot_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        d = [256, 1024, 2048, 2560, 72, 1536][i % 6]  # both matrix-core tilings, vector-ALU bf16
        K = int(rng.integers(2, 5))
        T = int(rng.integers(1, 90))
        V = int(rng.integers(1, 400))
        extras = dict(per_module_gain=bool(rng.random() < 0.5), tau=bool(rng.random() < 0.5),
                      bias=bool(rng.random() < 0.5), wbar=str(rng.choice(["none", "shared"])), rot=True)
        if extras["wbar"] == "none":
            extras.pop("wbar")
        flags = dict(final_module_dW=bool(rng.random() < 0.75), want_dtau=bool(rng.random() < 0.5),
                     want_dbias=bool(rng.random() < 0.5))
        out.append((f"r{i}_K{K}_T{T}_d{d}_V{V}", dict(K=K, T=T, d=d, V=V), extras, flags))
    return out


ROT_CASES = _rot_cases(8, 31)


@pytest.mark.parametrize("name,ov,extras,flags", ROT_CASES, ids=[c[0] for c in ROT_CASES])
def test_random_rot_parity(name, ov, extras, flags):
    # ROT: the oracle is handed W R_k (or the shared copy's) as each head's readout
    cfg = "2b" if ov["d"] == 2560 else "1b"
    x = make_extras(make_inputs(cfg, seed=zlib.crc32(name.encode()) % 1000, **ov), 7, **extras)
    log(f"rot case {name}: extras {extras} flags {flags}")
    g = run_general(x, flags)
    ref = oracle_general(x, flags)
    compare(g, ref, x["cfg"].dtype, flags, name)


def _eval_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        d = [256, 1024, 2048, 2560, 72, 24][i % 6]  # 128-, 64-, 48-row tiles, vector-ALU bf16 and fp32
        K = int(rng.integers(1, 4))
        T = int(rng.integers(1, 400))  # up to four 128-row tiles, ragged
        V = int(rng.integers(1, 600))
        extras = dict(tau=bool(rng.random() < 0.5), bias=bool(rng.random() < 0.5),
                      per_module_gain=bool(rng.random() < 0.3),
                      wbar=str(rng.choice(["none", "shared", "per_head"])))
        if K == 1:
            extras["wbar"] = "none"  # no heads
        cfg = "tiny" if d == 24 else ("2b" if d == 2560 else "1b")
        out.append((f"e{i}_K{K}_T{T}_d{d}_V{V}", cfg, dict(K=K, T=T, d=d, V=V), extras))
    return out


EVAL_CASES = _eval_cases(12, 2027)


@pytest.mark.parametrize("name,cfg,ov,extras", EVAL_CASES, ids=[c[0] for c in EVAL_CASES])
def test_random_exit_eval_parity(name, cfg, ov, extras):
    seed = zlib.crc32(name.encode()) % 1000
    x = make_extras(make_inputs(cfg, seed=seed, **ov), seed, **extras)
    log(f"eval case {name}: extras {extras}")
    losses, row_loss, top1 = run_exit_eval(x)
    check_exit_eval(x, losses, row_loss, top1, name, min_rows_for_agreement=50)
