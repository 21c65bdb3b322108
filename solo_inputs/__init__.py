"""Seeded synthetic inputs for the SOLO shared-readout local loss.

This module is shared by the tests, ``bench.py`` and the oracle's checks.  It
holds no arithmetic of the method itself: it only draws random numbers, rounds
them once to the storage dtype (bf16, round-to-nearest-even) and returns the
exact values that both the GPU path and the fp64 oracle read.

Workload shapes stand in for the paper's SlimPajama pretraining runs
(context 2048, a 32k vocabulary, per-GPU micro-batch 8; Section 4 and the
systems appendix) and its own synthetic Zipf-token systems runs (appendix on
pipeline parallelism: bf16, synthetic Zipf-distributed tokens).  No dataset is
read.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

__all__ = [
    "Config",
    "CONFIGS",
    "bf16_bits",
    "bf16_from_bits",
    "round_bf16",
    "zipf_targets",
    "make_inputs",
    "make_extras",
    "random_orthogonal",
    "make_profile_inputs",
]


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload shape.

    K modules, T tokens per module, width d, vocabulary V.  ``h_scale_step``
    multiplies module k's hidden states by ``1 + h_scale_step * k`` (k zero
    based) to mimic a residual stream whose norm grows with depth.
    ``hot_fraction`` of the positions of every module get token ``V - 1``
    (stresses the online softmax with one very frequent class).
    """

    name: str
    config_id: int
    K: int
    T: int
    d: int
    V: int
    dtype: str  # "bf16" or "f32"
    w_sigma: float = 0.02
    gain_sigma: float = 0.1
    h_scale_step: float = 0.0
    targets: str = "zipf"  # "zipf" or "uniform"
    zipf_s: float = 1.1
    hot_fraction: float = 0.0

    @property
    def tokens(self) -> int:
        return self.T


CONFIGS: Dict[str, Config] = {
    # correctness config: fp32 storage, uniform targets
    "tiny": Config("tiny", 0, K=2, T=256, d=64, V=512, dtype="f32", targets="uniform"),
    # 340M-class model: micro-batch 4 x context 2048, width 1024
    "340m": Config("340m", 1, K=4, T=8192, d=1024, V=32000, dtype="bf16"),
    # 1B-class model: micro-batch 8 x context 2048, width 2048 (headline shape)
    "1b": Config("1b", 2, K=4, T=16384, d=2048, V=32000, dtype="bf16"),
    # 2B-class model: width 2560, eight modules, growing residual norm
    "2b": Config("2b", 3, K=8, T=16384, d=2560, V=32000, dtype="bf16", h_scale_step=0.25),
    # large-vocabulary stress: V not a multiple of large tiles, larger logits
    "large_vocab": Config(
        "large_vocab", 4, K=2, T=32768, d=2048, V=128256, dtype="bf16", w_sigma=0.05, hot_fraction=0.01
    ),
}

# tensor ids inside one (seed, config) stream family
_H, _W, _GAIN, _TARGETS, _HOT = 0, 1, 2, 3, 4
_GAIN_K, _WBAR, _TAU, _BIAS = 5, 6, 7, 8
_DIR, _PH, _PW, _PT = 9, 10, 11, 12
_ROT = 13
# stream family of the structured inputs (make_profile_inputs)
_PROFILE_ID = 100


def _rng(seed: int, config_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, config_id, tensor_id])))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even.

    NaN stays NaN (quiet); infinities and overflow to infinity follow IEEE.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded = rounded.copy()
        rounded[nan] = ((u[nan] >> 16).astype(np.uint16)) | np.uint16(0x0040)
    return rounded


def bf16_from_bits(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> the fp32 values they encode (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 value, returned as fp32."""
    return bf16_from_bits(bf16_bits(x))


def zipf_targets(rng: np.random.Generator, shape, V: int, s: float) -> np.ndarray:
    """Bounded Zipf on ranks 1..V with P(rank r) proportional to r**-s.

    Sampled by inverse CDF from seeded uniforms; token id = rank - 1, so
    token 0 is the most frequent.
    """
    ranks = np.arange(1, V + 1, dtype=np.float64)
    pmf = ranks ** (-s)
    cdf = np.cumsum(pmf)
    cdf /= cdf[-1]
    u = rng.random(size=shape)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def _normal_f32(rng: np.random.Generator, shape, sigma: float = 1.0) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        out *= np.float32(sigma)
    return out


def make_inputs(cfg: Config | str, seed: int = 0, *, K: Optional[int] = None, T: Optional[int] = None,
                d: Optional[int] = None, V: Optional[int] = None) -> dict:
    """Draw the inputs of one call.

    Returns a dict with
      ``h``       float32 [K, T, d]   values exactly representable in cfg.dtype
      ``gain``    float32 [d]
      ``W``       float32 [V, d]
      ``targets`` int32   [K, T]
      ``h_bits``, ``gain_bits``, ``W_bits`` uint16 bf16 patterns (bf16 configs)
      ``cfg``     the Config (with any size override applied)

    Sizes may be overridden (for ragged or reduced cases); the distributions
    stay those of ``cfg``.
    """
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    cfg = dataclasses.replace(
        cfg,
        K=cfg.K if K is None else K,
        T=cfg.T if T is None else T,
        d=cfg.d if d is None else d,
        V=cfg.V if V is None else V,
    )
    Kc, Tc, dc, Vc = cfg.K, cfg.T, cfg.d, cfg.V

    h = _normal_f32(_rng(seed, cfg.config_id, _H), (Kc, Tc, dc))
    if cfg.h_scale_step:
        scale = (1.0 + cfg.h_scale_step * np.arange(Kc, dtype=np.float32)).astype(np.float32)
        h *= scale[:, None, None]
    W = _normal_f32(_rng(seed, cfg.config_id, _W), (Vc, dc), cfg.w_sigma)
    gain = np.float32(1.0) + _normal_f32(_rng(seed, cfg.config_id, _GAIN), (dc,), cfg.gain_sigma)

    trng = _rng(seed, cfg.config_id, _TARGETS)
    if cfg.targets == "uniform":
        targets = trng.integers(0, Vc, size=(Kc, Tc), dtype=np.int64).astype(np.int32)
    else:
        targets = zipf_targets(trng, (Kc, Tc), Vc, cfg.zipf_s)
    if cfg.hot_fraction > 0.0:
        hrng = _rng(seed, cfg.config_id, _HOT)
        n_hot = int(round(cfg.hot_fraction * Tc))
        for k in range(Kc):
            pos = hrng.choice(Tc, size=n_hot, replace=False)
            targets[k, pos] = Vc - 1

    out = {"cfg": cfg, "targets": np.ascontiguousarray(targets, dtype=np.int32)}
    if cfg.dtype == "bf16":
        out["h_bits"] = bf16_bits(h)
        out["gain_bits"] = bf16_bits(gain)
        out["W_bits"] = bf16_bits(W)
        out["h"] = bf16_from_bits(out["h_bits"])
        out["gain"] = bf16_from_bits(out["gain_bits"])
        out["W"] = bf16_from_bits(out["W_bits"])
    elif cfg.dtype == "f32":
        out["h"] = np.ascontiguousarray(h)
        out["gain"] = np.ascontiguousarray(gain)
        out["W"] = np.ascontiguousarray(W)
    else:
        raise ValueError(f"unknown dtype {cfg.dtype!r}")
    return out


def random_orthogonal(rng: np.random.Generator, n: int, d: int) -> np.ndarray:
    """n random d x d orthogonal matrices (Haar measure), fp64.

    QR of a matrix of seeded standard normals, with the signs of R's diagonal
    moved into Q so that the distribution does not depend on the QR routine's
    sign convention.
    """
    out = np.empty((n, d, d), dtype=np.float64)
    for i in range(n):
        q, r = np.linalg.qr(rng.standard_normal((d, d)))
        out[i] = q * np.where(np.diag(r) < 0, -1.0, 1.0)[None, :]
    return out


def make_extras(x: dict, seed: int = 0, *, per_module_gain: bool = False, wbar: str = "none",
                tau: bool = False, bias: bool = False, rot: bool = False) -> dict:
    """Extra inputs of the general call for the workload ``x`` (from make_inputs).

    ``per_module_gain``: ``gain`` becomes [K, d], 1 + N(0, gain_sigma^2) per module.
    ``wbar``: "none" (the heads read W), "shared" (one [V, d] matrix, drawn like W:
    an earlier step's copy or a shared random readout) or "per_head" ([K-1, V, d]).
    ``tau``: temperatures [K] uniform on [0.5, 2) (learned logit scales), fp32.
    ``bias``: biases [K, V], N(0, 0.5^2), fp32.
    ``rot``: [K-1, d, d] random orthogonal matrices (the ROT variant's fixed
    per-head bases), rounded once to the dtype (so only nearly orthogonal in bf16).
    Returns a dict with the same keys as make_inputs (``gain``, ``gain_bits``
    replaced when per-module) plus ``Wbar`` (and ``Wbar_bits``), ``tau``, ``bias``,
    ``rot`` (and ``rot_bits``) (None when absent).  Tensor values are exactly
    representable in the dtype.
    """
    cfg = x["cfg"]
    K, d, V = cfg.K, cfg.d, cfg.V
    out = dict(x)
    bf = cfg.dtype == "bf16"

    def stored(a):
        return (bf16_bits(a), bf16_from_bits(bf16_bits(a))) if bf else (None, np.ascontiguousarray(a))

    if per_module_gain:
        g = np.float32(1.0) + _normal_f32(_rng(seed, cfg.config_id, _GAIN_K), (K, d), cfg.gain_sigma)
        out["gain_bits"], out["gain"] = stored(g)
    out["Wbar"] = out["Wbar_bits"] = None
    if wbar == "shared":
        out["Wbar_bits"], out["Wbar"] = stored(_normal_f32(_rng(seed, cfg.config_id, _WBAR), (V, d), cfg.w_sigma))
    elif wbar == "per_head":
        out["Wbar_bits"], out["Wbar"] = stored(
            _normal_f32(_rng(seed, cfg.config_id, _WBAR), (max(K - 1, 0), V, d), cfg.w_sigma))
    elif wbar != "none":
        raise ValueError(f"unknown wbar {wbar!r}")
    out["tau"] = (np.float32(0.5) + np.float32(1.5) * _rng(seed, cfg.config_id, _TAU).random(K, dtype=np.float32)
                  ) if tau else None
    out["bias"] = _normal_f32(_rng(seed, cfg.config_id, _BIAS), (K, V), 0.5) if bias else None
    out["rot"] = out["rot_bits"] = None
    if rot:
        r = random_orthogonal(_rng(seed, cfg.config_id, _ROT), max(K - 1, 0), d).astype(np.float32)
        out["rot_bits"], out["rot"] = stored(r)
    return out


def make_profile_inputs(dtype: str, K: int, T: int, d: int, V: int, profile: np.ndarray, targets: np.ndarray,
                        seed: int = 0, row_jitter: float = 0.1, w_noise: float = 0.02) -> dict:
    """Structured inputs whose logits follow a chosen profile over the vocabulary.

    A seeded random sign vector s (entries +1 or -1) is shared by the hidden
    states and the readout rows:

      h[k, t] = s * (1 + row_jitter * N(0, 1))          (elementwise)
      gain    = 1 + 0.1 * N(0, 1)
      W[v]    = profile[v] * s / d + N(0, w_noise^2)

    so that a row's logit at column v is close to ``profile[v]`` (the hidden
    states have root-mean-square close to one and the gain close to one), with
    seeded noise of a few tenths that makes every row and column different.
    Profiles that climb by many nats across the vocabulary, or that put one
    column far above the others, steer the online softmax through re-basing
    and through rows whose target holds nearly all of the probability.
    ``targets`` [K, T] (int32) is used as given.  Returns the keys of
    make_inputs (a Config named "profile" of the given sizes and dtype).
    """
    cfg = Config("profile", _PROFILE_ID, K=K, T=T, d=d, V=V, dtype=dtype)
    profile = np.asarray(profile, dtype=np.float32)
    if profile.shape != (V,) or targets.shape != (K, T):
        raise ValueError("profile must be [V] and targets [K, T]")
    sgn = np.where(_rng(seed, _PROFILE_ID, _DIR).random(d) < 0.5, -1.0, 1.0).astype(np.float32)
    h = sgn[None, None, :] * (np.float32(1.0) + _normal_f32(_rng(seed, _PROFILE_ID, _PH), (K, T, d), row_jitter))
    gain = np.float32(1.0) + _normal_f32(_rng(seed, _PROFILE_ID, _GAIN), (d,), 0.1)
    W = profile[:, None] * sgn[None, :] / np.float32(d) + _normal_f32(_rng(seed, _PROFILE_ID, _PW), (V, d), w_noise)
    out = {"cfg": cfg, "targets": np.ascontiguousarray(targets, dtype=np.int32)}
    if dtype == "bf16":
        for name, a in (("h", h), ("gain", gain), ("W", W)):
            out[name + "_bits"] = bf16_bits(a.astype(np.float32))
            out[name] = bf16_from_bits(out[name + "_bits"])
    elif dtype == "f32":
        out["h"], out["gain"], out["W"] = (np.ascontiguousarray(a, dtype=np.float32) for a in (h, gain, W))
    else:
        raise ValueError(f"unknown dtype {dtype!r}")
    return out
