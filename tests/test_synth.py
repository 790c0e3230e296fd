"""Seeded input generators: determinism, shapes, statistics, bf16 rounding."""
import numpy as np
import torch

from paper_2608_04401_amd import synth


def test_bf16_rounding_matches_torch():
    a = np.random.default_rng(1).standard_normal(200_000, dtype=np.float32) * np.float32(7)
    a[:6] = [1.00390625, 1.01171875, -1.00390625, 0.0, -0.0, 3.0e-39]   # ties, zeros, denormal
    ref = torch.from_numpy(a.copy()).to(torch.bfloat16).float().numpy()
    assert np.array_equal(synth.round_bf16(a).view(np.uint32), ref.view(np.uint32))
    b = a.copy()
    synth.round_bf16(b, inplace=True)
    assert np.array_equal(b.view(np.uint32), ref.view(np.uint32))


def test_layer_is_deterministic_and_shaped():
    a = synth.moe_layer(32, 64, 4, 48, dtype="bf16", seed=7)
    b = synth.moe_layer(32, 64, 4, 48, dtype="bf16", seed=7)
    for x, y in ((a.x, b.x), (a.W_router, b.W_router), (a.W_gu, b.W_gu), (a.W_down, b.W_down)):
        assert np.array_equal(x, y)
    assert a.W_gu.shape == (4, 96, 64) and a.W_down.shape == (4, 64, 48)
    assert (a.T, a.d, a.N, a.m) == (32, 64, 4, 48)
    # bf16-representable: the low 16 bits are zero
    assert (a.W_gu.view(np.uint32) & 0xFFFF).max() == 0
    c = synth.moe_layer(32, 64, 4, 48, dtype="bf16", seed=8)
    assert not np.array_equal(a.x, c.x)


def test_weight_std():
    L = synth.moe_layer(256, 512, 4, 256, dtype="f32", seed=0)
    assert abs(L.W_gu.std() - 0.02) < 0.0005
    assert abs(L.x.std() - 1.0) < 0.01


def test_planted_logits_structure():
    lg = synth.planted_logits(T=4000, N=64, seed=2)
    assert lg.shape == (4000, 64) and lg.dtype == np.float32
    base = np.random.default_rng(2).standard_normal(size=(4000, 64), dtype=np.float32)
    planted = lg != base
    m = planted.sum(axis=1)
    assert m.min() >= 1 and m.max() <= 8
    # one shared offset per token in [2, 6)
    off = np.where(planted, lg - base, np.nan)
    spread = np.nanmax(off, axis=1) - np.nanmin(off, axis=1)
    assert np.nanmax(spread) < 1e-5
    assert np.nanmin(off) >= 2 - 1e-5 and np.nanmax(off) < 6 + 1e-5
