"""Input generation: bf16 rounding, determinism and the workload shapes."""
import numpy as np
import pytest
import torch

import workloads as W


def test_bf16_rounding_is_round_to_nearest_even():
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 20000),
        # exact ties: bit 15 set, lower bits clear -> rounds to even
        (np.arange(1 << 12, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, 1e-40, -1e-42], np.float32),
    ]).astype(np.float32)
    ours = W.f32_to_bf16_bits(vals)
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = W.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16)
                                  .float().numpy())


def test_bf16_nan_stays_nan():
    bits = W.f32_to_bf16_bits(np.array([np.nan], np.float32))
    assert np.isnan(W.bf16_bits_to_f32(bits))[0]


def test_generation_is_deterministic_and_rounded():
    cfg = W.CONFIGS[2].with_(B=1, T=128, H=2)
    p1, p2 = W.generate(cfg), W.generate(cfg)
    for name in ("x", "a", "b", "c", "dy"):
        v1, v2 = getattr(p1, name), getattr(p2, name)
        np.testing.assert_array_equal(v1, v2)
        np.testing.assert_array_equal(W.round_to(v1, "bf16"), v1)   # already bf16 values
    assert p1.x.shape == (1, 128, 2, 128) and p1.a.shape == (1, 128, 2)
    assert p1.stored("x").dtype == np.uint16
    assert 0.0 <= p1.a.min() and p1.a.max() <= 1.0


@pytest.mark.parametrize("cid", sorted(W.CONFIGS))
def test_config_shapes(cid):
    cfg = W.CONFIGS[cid]
    assert cfg.T % cfg.block == 0 and cfg.D % 16 == 0
    small = cfg.with_(B=1, T=2 * cfg.block, H=min(cfg.H, 2),
                      width=None if cfg.width is None else min(cfg.H, 2) * cfg.D)
    p = W.generate(small)
    assert p.x.shape == (1, 2 * cfg.block, small.H, cfg.D)
    assert (p.dy is None) == (not cfg.backward)
    assert np.all(np.isfinite(p.x)) and np.all((p.a >= 0) & (p.a <= 1))


def test_decay_recipes_ranges():
    rng = np.random.Generator(np.random.PCG64(7))
    a = W.draw_decay(rng, (4096,), "exp_softplus")
    # exp(-softplus(z) * Delta) with Delta <= 0.1 stays close to 1
    assert a.min() > 0.5 and a.max() < 1.0
    s = W.draw_decay(rng, (4096,), "sigmoid", 5.0)
    assert np.median(s) > 0.98
