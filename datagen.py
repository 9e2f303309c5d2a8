"""Seeded synthetic inputs for the fused-MLP workloads.

This module is shared by the CPU oracle's tests, the GPU parity tests and the
benchmark.  It only draws numbers; it holds none of the MLP's arithmetic.

Every element is a pure function of (seed, stream, index), so any slice of
any tensor can be regenerated on its own and the same values come out on the
CPU and on a GPU:

    u = (splitmix64(seed ^ (stream << 56) ^ idx) >> 40) * 2**-24   in [0, 1)

splitmix64 is Sebastiano Vigna's public-domain output function (add the
golden-ratio increment, then two xor-shift-multiply rounds and a final
xor-shift).  ``idx`` runs row-major over the logical tensor.  Streams:
weights 1, inputs 2, targets 3, auxiliary 4.

Derived distributions:
    uniform[lo, hi]   lo + (hi - lo) * u           (computed in fp32; exact
                                                    for [-1, 1] and [0, 1])
    Xavier-uniform    bf16(a * (2u - 1)), a = sqrt(6 / (fan_in + fan_out)),
                      over the real (unpadded) fan_in and fan_out, fp32 then
                      round-to-nearest-even to bf16
    Gaussian          Box-Muller on index pairs (2i, 2i + 1):
                      sqrt(-2 ln(1 - u1)) * cos(2 pi u2), fp64
Inputs X are rounded to bf16; targets stay fp32.
"""
from __future__ import annotations

import math

import torch

STREAM_W = 1
STREAM_X = 2
STREAM_T = 3
STREAM_AUX = 4

_GOLDEN = 0x9E3779B97F4A7C15
_MUL1 = 0xBF58476D1CE4E5B9
_MUL2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1


def _as_i64(v: int) -> int:
    """Two's-complement int64 value with the same 64 bits as ``v``."""
    v &= _MASK64
    return v - (1 << 64) if v >= (1 << 63) else v


def _shr(z: torch.Tensor, s: int) -> torch.Tensor:
    """Logical right shift of int64 bit patterns."""
    return (z >> s) & ((1 << (64 - s)) - 1)


def splitmix64(x: torch.Tensor) -> torch.Tensor:
    """splitmix64 of int64 bit patterns; wrapping int64 arithmetic."""
    z = x + _as_i64(_GOLDEN)
    z = (z ^ _shr(z, 30)) * _as_i64(_MUL1)
    z = (z ^ _shr(z, 27)) * _as_i64(_MUL2)
    return z ^ _shr(z, 31)


def splitmix64_scalar(x: int) -> int:
    """Reference scalar splitmix64 on Python integers (for self-checks)."""
    z = (x + _GOLDEN) & _MASK64
    z = ((z ^ (z >> 30)) * _MUL1) & _MASK64
    z = ((z ^ (z >> 27)) * _MUL2) & _MASK64
    return z ^ (z >> 31)


def uniform01(seed: int, stream: int, start: int, count: int,
              device: str | torch.device = "cpu") -> torch.Tensor:
    """u in [0, 1) as float64, for flat indices start .. start+count-1."""
    base = _as_i64((seed ^ (stream << 56)) & _MASK64)
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    bits = splitmix64(idx ^ base)
    return _shr(bits, 40).to(torch.float64) * (2.0 ** -24)


def uniform(seed: int, stream: int, shape, lo: float = -1.0, hi: float = 1.0,
            device: str | torch.device = "cpu", start: int = 0) -> torch.Tensor:
    """fp32 uniform[lo, hi] tensor of the given shape."""
    n = math.prod(shape)
    u = uniform01(seed, stream, start, n, device).to(torch.float32)
    return (lo + (hi - lo) * u).reshape(shape)


def gaussian(seed: int, stream: int, shape,
             device: str | torch.device = "cpu") -> torch.Tensor:
    """fp32 standard normal tensor (Box-Muller over index pairs)."""
    n = math.prod(shape)
    u = uniform01(seed, stream, 0, 2 * n, device).reshape(n, 2)
    r = torch.sqrt(-2.0 * torch.log1p(-u[:, 0]))
    return (r * torch.cos(2.0 * math.pi * u[:, 1])).to(torch.float32).reshape(shape)


def layer_shapes(width: int, depth: int, in_dim: int, out_dim: int):
    """(fan_in, fan_out) of each of the depth + 1 weight matrices."""
    L = depth + 1
    return [(in_dim if l == 0 else width, out_dim if l == L - 1 else width)
            for l in range(L)]


def xavier_weights(seed: int, width: int, depth: int, in_dim: int,
                   out_dim: int, device: str | torch.device = "cpu"):
    """Concatenated bf16 weights, layer-major, each row-major [fan_in, fan_out]."""
    parts = []
    start = 0
    for fi, fo in layer_shapes(width, depth, in_dim, out_dim):
        a = torch.tensor(math.sqrt(6.0 / (fi + fo)), dtype=torch.float32)
        u = uniform01(seed, STREAM_W, start, fi * fo, device).to(torch.float32)
        parts.append((a.to(device) * (2.0 * u - 1.0)).to(torch.bfloat16))
        start += fi * fo
    return torch.cat(parts)


def inputs_uniform(seed: int, M: int, in_dim: int,
                   device: str | torch.device = "cpu") -> torch.Tensor:
    """bf16 inputs [M, in_dim], uniform[-1, 1] rounded to bf16."""
    return uniform(seed, STREAM_X, (M, in_dim), -1.0, 1.0, device).to(torch.bfloat16)


def targets_uniform(seed: int, M: int, out_dim: int, lo: float = -1.0,
                    hi: float = 1.0, device: str | torch.device = "cpu") -> torch.Tensor:
    """fp32 targets [M, out_dim], uniform[lo, hi]."""
    return uniform(seed, STREAM_T, (M, out_dim), lo, hi, device)


def image_features(seed: int, M: int, n_freq: int = 8, pad_to: int = 64,
                   device: str | torch.device = "cpu") -> torch.Tensor:
    """Image-compression-like inputs: pixel coordinates (x, y) ~ U[0, 1]^2
    expanded to sin/cos(2^k pi x), k < n_freq, for both coordinates, zero
    padded to ``pad_to`` features and rounded to bf16."""
    xy = uniform(seed, STREAM_X, (M, 2), 0.0, 1.0, device).to(torch.float64)
    freqs = (2.0 ** torch.arange(n_freq, dtype=torch.float64, device=device)) * math.pi
    ang = xy[:, :, None] * freqs[None, None, :]              # [M, 2, F]
    feats = torch.cat([torch.sin(ang), torch.cos(ang)], dim=2).reshape(M, -1)
    out = torch.zeros(M, pad_to, dtype=torch.float64, device=device)
    out[:, : feats.shape[1]] = feats
    return out.to(torch.float32).to(torch.bfloat16)


def pinn_inputs(seed: int, M: int, device: str | torch.device = "cpu") -> torch.Tensor:
    """PINN-like inputs: 3-D points uniform[-1, 1], bf16 [M, 3]."""
    return inputs_uniform(seed, M, 3, device)


def gaussian_features(seed: int, stream: int, M: int, dim: int,
                      device: str | torch.device = "cpu") -> torch.Tensor:
    """NeRF-like features: N(0, 1), bf16 [M, dim]."""
    return gaussian(seed, stream, (M, dim), device).to(torch.bfloat16)
