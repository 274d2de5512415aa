"""Seeded synthetic inputs for the Sliding Window Recurrence.

This module is shared by the tests, the benchmark and the smoke check.  It
holds input generation only (random draws, the decay-coefficient recipes and
rounding to the I/O dtype) and none of the recurrence's arithmetic.

Recipe (every tensor is drawn on the host with numpy's PCG64 generator seeded
with the configuration's seed, in this fixed order):

* ``x, b, c`` and, for backward workloads, ``dy``: float32 standard normals of
  shape ``[B, T, H, D]`` (``D`` channels per head, channels contiguous).
  For the Phalanx-layer shape (model width 2048) ``x`` is instead the product
  ``Z @ W`` of float32 normals ``Z [B*T, width]`` and ``W [width, width]`` with
  standard deviation ``1/sqrt(width)`` (a random-init linear projection, drawn
  before everything else), reshaped to ``[B, T, H, D]``.
* ``a`` (shape ``[B, T, H]``: one decay per token and head, shared by the
  head's channels as in the paper's Phalanx layer, Sec. 5):
  ``sigmoid(N(mu, 1))`` or ``exp(-softplus(N(0, 1)) * Delta)`` with ``Delta``
  uniform in ``[1e-3, 1e-1]``, drawn per (b, t, h).  Per-channel-decay
  workloads draw ``a`` with the same recipe per (b, t, h, channel), shape
  ``[B, T, H, D]``.  Workloads fed through the fused sigmoid featurisation
  (``logits``) store the normal ``N(mu, 1)`` itself, the decay's logit.
* Every tensor is then rounded to the I/O dtype with round-to-nearest-even;
  the GPU library and the oracle both consume exactly these rounded values.
"""
from dataclasses import dataclass, replace
from typing import Dict, Optional

import numpy as np

# ----------------------------------------------------------------------------
# bfloat16 storage helpers (round-to-nearest-even, NaN kept quiet)
# ----------------------------------------------------------------------------


def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to bfloat16 (RNE); returns the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    out = bits + (np.uint32(0x7FFF) + ((bits >> np.uint32(16)) & np.uint32(1)))
    out >>= np.uint32(16)
    out = out.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = ((bits[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
    return out


def bf16_bits_to_f32(bits) -> np.ndarray:
    """Exact float32 values of bfloat16 bit patterns."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to(x, dtype: str) -> np.ndarray:
    """float32 array holding ``x`` rounded to ``dtype`` ('f32' or 'bf16')."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(x))
    raise ValueError(f"unknown dtype {dtype!r}")


def storage(x_rounded: np.ndarray, dtype: str) -> np.ndarray:
    """Storage array for already-rounded float32 values: float32 or uint16 bits."""
    if dtype == "f32":
        return np.ascontiguousarray(x_rounded, dtype=np.float32)
    return f32_to_bf16_bits(x_rounded)


# ----------------------------------------------------------------------------
# Workload definitions
# ----------------------------------------------------------------------------


@dataclass(frozen=True)
class Config:
    id: int
    name: str
    B: int
    T: int
    H: int
    D: int
    block: int
    dtype: str            # 'f32' or 'bf16' (I/O dtype; accumulation is always fp32)
    a_kind: str           # 'sigmoid' or 'exp_softplus'
    a_mu: float = 0.0     # mean of the normal fed to the sigmoid
    seed: int = 0
    backward: bool = True
    width: Optional[int] = None   # model width of the projected-x recipe
    per_channel: bool = False     # one decay per token, head and channel ([B, T, H, D])
    logits: bool = False          # a holds the sigmoid's argument instead of the decay

    @property
    def tokens(self) -> int:
        return self.B * self.T

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


CONFIGS: Dict[int, Config] = {
    1: Config(1, "tiny_fp32_B1_T1024_H4_d64_l64", 1, 1024, 4, 64, 64, "f32", "sigmoid", 2.0,
              seed=0, backward=False),
    2: Config(2, "bf16_B8_T4096_H16_d128_l64", 8, 4096, 16, 128, 64, "bf16", "sigmoid", 3.0,
              seed=1),
    3: Config(3, "bf16_B8_T16384_H16_d128_l128", 8, 16384, 16, 128, 128, "bf16",
              "exp_softplus", seed=2),
    4: Config(4, "bf16_B1_T131072_H32_d64_l128", 1, 131072, 32, 64, 128, "bf16",
              "exp_softplus", seed=3),
    5: Config(5, "bf16_B16_T8192_H32_d64_l64_width2048", 16, 8192, 32, 64, 64, "bf16",
              "sigmoid", 5.0, seed=4, width=2048),
}

HEADLINE = 3

# The same shapes with one decay per token, head and channel (the diagonal
# transition with a full diagonal): the tiny workload read with its decay
# "per-token per-channel", and the headline shape.
PER_CHANNEL: Dict[int, Config] = {
    1: CONFIGS[1].with_(name=CONFIGS[1].name + "_perchannel", per_channel=True),
    3: CONFIGS[3].with_(name=CONFIGS[3].name + "_perchannel", per_channel=True),
}


@dataclass
class Problem:
    """Rounded inputs as float32 arrays (exact values of the I/O dtype) plus the
    storage arrays the GPU library reads (float32, or uint16 bf16 bit patterns)."""
    cfg: Config
    x: np.ndarray
    a: np.ndarray
    b: np.ndarray
    c: np.ndarray
    dy: Optional[np.ndarray]

    def stored(self, name: str) -> np.ndarray:
        return storage(getattr(self, name), self.cfg.dtype)


def _sigmoid(z):
    z = np.asarray(z, np.float64)
    return 1.0 / (1.0 + np.exp(-z))


def _softplus(z):
    z = np.asarray(z, np.float64)
    return np.logaddexp(0.0, z)


def draw_decay(rng: np.random.Generator, shape, kind: str, mu: float = 0.0) -> np.ndarray:
    """Decay coefficients in [0, 1] as float32 (before I/O rounding)."""
    z = rng.standard_normal(shape, dtype=np.float32)
    if kind == "sigmoid":
        a = _sigmoid(z.astype(np.float64) + mu)
    elif kind == "exp_softplus":
        delta = rng.uniform(1e-3, 1e-1, size=shape)
        a = np.exp(-_softplus(z) * delta)
    elif kind == "uniform":
        a = rng.uniform(0.0, 1.0, size=shape)
    else:
        raise ValueError(f"unknown decay recipe {kind!r}")
    return a.astype(np.float32)


def generate(cfg: Config, with_dy: Optional[bool] = None) -> Problem:
    """Draw the seeded inputs of a workload (see the module docstring)."""
    if with_dy is None:
        with_dy = cfg.backward
    rng = np.random.Generator(np.random.PCG64(cfg.seed))
    shape = (cfg.B, cfg.T, cfg.H, cfg.D)
    if cfg.width is not None:
        if cfg.width != cfg.H * cfg.D:
            raise ValueError("width must equal H * D")
        Z = rng.standard_normal((cfg.B * cfg.T, cfg.width), dtype=np.float32)
        W = rng.standard_normal((cfg.width, cfg.width), dtype=np.float32)
        W *= np.float32(1.0 / np.sqrt(cfg.width))
        x = (Z @ W).reshape(shape)
        del Z, W
    else:
        x = rng.standard_normal(shape, dtype=np.float32)
    x = round_to(x, cfg.dtype)
    b = round_to(rng.standard_normal(shape, dtype=np.float32), cfg.dtype)
    c = round_to(rng.standard_normal(shape, dtype=np.float32), cfg.dtype)
    dy = round_to(rng.standard_normal(shape, dtype=np.float32), cfg.dtype) if with_dy else None
    a_shape = shape if cfg.per_channel else shape[:3]
    if cfg.logits:     # the decay's logit z ~ N(mu, 1): the decay is sigmoid(z)
        if cfg.a_kind != "sigmoid":
            raise ValueError("logit inputs need the sigmoid decay recipe")
        z = rng.standard_normal(a_shape, dtype=np.float32) + np.float32(cfg.a_mu)
        a = round_to(z, cfg.dtype)
    else:
        a = round_to(draw_decay(rng, a_shape, cfg.a_kind, cfg.a_mu), cfg.dtype)
    return Problem(cfg, x, a, b, c, dy)


def random_problem(seed: int, B: int, T: int, H: int, D: int, block: int, dtype: str = "bf16",
                   a_kind: str = "sigmoid", a_mu: float = 2.0, with_dy: bool = True,
                   per_channel: bool = False, logits: bool = False) -> Problem:
    """A small ad-hoc workload with the same recipe (used by parity tests)."""
    cfg = Config(0, f"adhoc_B{B}_T{T}_H{H}_d{D}_l{block}_{dtype}", B, T, H, D, block, dtype,
                 a_kind, a_mu, seed=seed, backward=with_dy, per_channel=per_channel,
                 logits=logits)
    return generate(cfg, with_dy=with_dy)
