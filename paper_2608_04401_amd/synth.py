"""Seeded synthetic inputs shared by the GPU path's tests/bench and the oracle.

This module only draws random numbers and rounds them to the storage dtype.  It holds
none of the routing or expert arithmetic, so both sides can consume the same arrays
without sharing any of the method's code.

Recipe (all draws from ``numpy.random.default_rng``, PCG64):

* normal draws are taken in float32 (``standard_normal(dtype=float32)``) and scaled in
  float32; ``N(0, 0.02)`` means standard deviation 0.02;
* bf16 tensors are the float32 draws rounded to nearest-even bf16 (values returned as
  float32 arrays that are exactly representable in bf16);
* draw order inside one layer: x, W_router, W_gate, W_up, W_down; layer ``l`` of a
  stack uses ``default_rng([seed, l])`` and the stack input ``default_rng([seed, 10**6])``.

Shapes follow the OLMoE-1B-7B MoE block (64 experts, top-8, d_model 2048, SwiGLU
intermediate 1024); the paper evaluates that model (Implementation Details section).
The public benchmark suites the paper measures on are not available: these synthetic
draws stand in for them.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def round_bf16(a: np.ndarray, inplace: bool = False) -> np.ndarray:
    """Round a float32 array to the nearest bf16 value (ties to even), kept as float32.

    Finite inputs only (the draws never produce NaN/Inf).  Works in place on uint32 views,
    in chunks, so that large weight tensors need no 64-bit temporaries.
    """
    out = np.ascontiguousarray(a, dtype=np.float32)
    if not inplace or out is not a:
        out = out.copy() if out is a else out
    u = out.reshape(-1).view(np.uint32)
    step = 1 << 24
    for s in range(0, u.size, step):
        c = u[s:s + step]
        bias = (c >> 16) & np.uint32(1)
        bias += np.uint32(0x7FFF)
        c += bias
        c &= np.uint32(0xFFFF0000)
    return out


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


@dataclass
class LayerInputs:
    """One MoE layer's inputs.  Weights follow the nn.Linear (out, in) convention.

    x        [T, d]
    W_router [N, d]
    W_gu     [N, 2m, d]   rows [0, m) are the gate projection, rows [m, 2m) the up one
    W_down   [N, d, m]
    """
    x: np.ndarray
    W_router: np.ndarray
    W_gu: np.ndarray
    W_down: np.ndarray
    dtype: str  # "f32" or "bf16" (values already rounded for bf16)

    @property
    def T(self) -> int:
        return self.x.shape[0]

    @property
    def d(self) -> int:
        return self.x.shape[1]

    @property
    def N(self) -> int:
        return self.W_router.shape[0]

    @property
    def m(self) -> int:
        return self.W_down.shape[2]


def moe_layer(T: int, d: int, N: int, m: int, dtype: str = "bf16", seed=0,
              x_std: float = 1.0, w_std: float = 0.02, with_x: bool = True) -> LayerInputs:
    """x ~ N(0, x_std), all weights ~ N(0, w_std); rounded to bf16 when dtype == "bf16"."""
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    rng = np.random.default_rng(seed)
    x = _normal(rng, (T, d), x_std) if with_x else np.zeros((0, d), np.float32)
    W_router = _normal(rng, (N, d), w_std)
    W_gu = np.empty((N, 2 * m, d), np.float32)
    W_gu[:, :m] = _normal(rng, (N, m, d), w_std)     # gate projection
    W_gu[:, m:] = _normal(rng, (N, m, d), w_std)     # up projection
    W_down = _normal(rng, (N, d, m), w_std)
    if dtype == "bf16":
        for a in (x, W_router, W_gu, W_down):
            round_bf16(a, inplace=True)
    return LayerInputs(x, W_router, W_gu, W_down, dtype)


def tiny_layer(seed=0) -> LayerInputs:
    """Tiny fp32 layer: T=256, d=128, N=8 experts, SwiGLU intermediate 256."""
    return moe_layer(256, 128, 8, 256, dtype="f32", seed=seed)


def olmoe_layer(T: int = 4096, seed=0) -> LayerInputs:
    """OLMoE-shaped bf16 layer: d=2048, N=64, intermediate 1024 (prefill T=4096, decode T=64)."""
    return moe_layer(T, 2048, 64, 1024, dtype="bf16", seed=seed)


def stack_layer(l: int, T: int = 16384, seed=0, d=2048, N=64, m=1024) -> LayerInputs:
    """Weights of layer ``l`` of a residual stack of OLMoE-shaped layers (no x drawn)."""
    return moe_layer(T, d, N, m, dtype="bf16", seed=[seed, l], with_x=False)


def stack_input(T: int = 16384, d: int = 2048, seed=0) -> np.ndarray:
    rng = np.random.default_rng([seed, 10 ** 6])
    return round_bf16(_normal(rng, (T, d), 1.0))


# ---- device-side draws for the 16-layer stack (12.9 GB of weights: host draws would take
# minutes).  torch's seeded Philox generator on the GPU, fp32 normal draws scaled in fp32,
# bf16 by round-to-nearest-even; the same (seed, stream) gives the same tensor on the same
# torch build.  Both the GPU run and the oracle read these tensors (the oracle a host copy).

def device_normal_bf16(shape, stream: int, std: float, seed: int = 0, device="cuda"):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + stream)
    a = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32) * std
    return a.to(torch.bfloat16)


def device_stack_layer(l: int, d: int = 2048, N: int = 64, m: int = 1024, seed: int = 0,
                       device="cuda"):
    """(W_router [N, d], W_gate_up [N, 2m, d], W_down [N, d, m]) of stack layer l, bf16 on
    the device, weights ~ N(0, 0.02)."""
    import torch
    base = 16 * (l + 1)
    Wr = device_normal_bf16((N, d), base + 1, 0.02, seed, device)
    Wgu = torch.cat([device_normal_bf16((N, m, d), base + 2, 0.02, seed, device),
                     device_normal_bf16((N, m, d), base + 3, 0.02, seed, device)], dim=1)
    Wd = device_normal_bf16((N, d, m), base + 4, 0.02, seed, device)
    return Wr, Wgu, Wd


def device_stack_input(T: int = 16384, d: int = 2048, seed: int = 0, device="cuda"):
    """x [T, d] ~ N(0, 1), bf16 on the device."""
    return device_normal_bf16((T, d), 0, 1.0, seed, device)


def planted_logits(T: int = 65536, N: int = 64, seed=0, m_max: int = 8,
                   delta_lo: float = 2.0, delta_hi: float = 6.0) -> np.ndarray:
    """Routing-only workload: fp32 logits [T, N].

    Each row is N(0,1) noise; m_t ~ Uniform{1..m_max} experts, drawn without replacement,
    get one shared offset delta_t ~ Uniform(delta_lo, delta_hi) added (sharp and gradual
    elbows mixed).
    """
    rng = np.random.default_rng(seed)
    base = rng.standard_normal(size=(T, N), dtype=np.float32)
    m_t = rng.integers(1, m_max + 1, size=T)
    delta = rng.uniform(delta_lo, delta_hi, size=T).astype(np.float32)
    perm = np.argsort(rng.random((T, N)), axis=1)
    planted = np.arange(N)[None, :] < m_t[:, None]          # first m_t positions of perm
    rows = np.repeat(np.arange(T), N).reshape(T, N)
    add = np.zeros((T, N), np.float32)
    add[rows[planted], perm[planted]] = delta[rows[planted]]
    return (base + add).astype(np.float32)


def gaussian_logits(T: int, N: int, seed=0, std: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return _normal(rng, (T, N), std)


def uniform_draws(T: int, N: int, seed=0) -> np.ndarray:
    """Uniform [0, 1) float32 draws [T, N], one per (token, expert): the random numbers of
    tail randomisation, passed in to both sides."""
    rng = np.random.default_rng([seed, 2 * 10 ** 6])
    return rng.random((T, N), dtype=np.float32)
