"""Seeded synthetic inputs, shared by the HIP path's harness and the oracle.

Every tensor is drawn with numpy's PCG64 generator as standard normals in
float64, in C order over its logical NCHW / OIHW shape, and then quantised to
the run's storage type: float64 -> float32 (round to nearest even) for fp32
runs, and float64 -> float32 -> bfloat16 (round to nearest even at each step)
for bf16 runs.  Both sides consume the same quantised values, so input
quantisation never counts against a tolerance.

Seeds: input x = 1; target (or upstream gradient k of a stage run) = 2 + k;
layer l weight = 100 + l; layer l bias = 200 + l.  Weights are He-normal
(N(0,1) * sqrt(2 / fan_in), not truncated); biases are 0.1 * N(0,1).

Nothing here computes any step of the method.
"""
from __future__ import annotations

import numpy as np

from .specs import BF16, FP32, Net

SEED_X = 1
SEED_TARGET = 2
SEED_W = 100
SEED_B = 200


def normal(seed: int, shape) -> np.ndarray:
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape)


def f32_to_bf16_bits(a32: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits.
    Inputs here are finite normals, so NaN handling is not needed."""
    u = np.ascontiguousarray(a32, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & 1
    r = (u + np.uint32(0x7FFF) + lsb) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def quantize(a64: np.ndarray, dtype: int):
    """Returns (values as float64, raw storage array).  Raw storage is float32
    for fp32 runs and uint16 bfloat16 bits for bf16 runs."""
    a32 = a64.astype(np.float32)
    if dtype == FP32:
        return a32.astype(np.float64), a32
    bits = f32_to_bf16_bits(a32)
    return bf16_bits_to_f64(bits), bits


def input_x(net: Net, batch: int, dtype: int, seed: int = SEED_X):
    return quantize(normal(seed, (batch, net.in_channels, net.height, net.width)), dtype)


def target_like(shape, dtype: int, k: int = 0):
    return quantize(normal(SEED_TARGET + k, shape), dtype)


def layer_params(net: Net, idx: int, dtype: int, index_offset: int = 0):
    """He-normal weight (logical OIHW) and 0.1*N(0,1) bias for layer idx.
    `index_offset` is added to the seed index so a partition run as its own
    network draws the same values as inside the full network.
    Weights follow the storage type; biases stay float32 (accumulation
    precision) in every run."""
    L = net.layers[idx]
    g = idx + index_offset
    w64 = normal(SEED_W + g, L.weight_shape()) * np.sqrt(2.0 / L.fan_in())
    w = quantize(w64, dtype)
    if L.bias:
        b32 = (0.1 * normal(SEED_B + g, (L.cout,))).astype(np.float32)
        b = (b32.astype(np.float64), b32)
    else:
        b = None
    return w, b
