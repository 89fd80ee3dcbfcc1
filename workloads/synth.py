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

A second family, EXACT, draws small integers instead: inputs in
{-2..2}, targets in {-2..2}, upstream gradients in {-1, 0, 1} (half of them
zero), biases in {-1, 0, 1}, and weights that are zero except for three +-1
entries per output channel (three of a depthwise filter's nine taps).  Its
values are chosen so that a bf16 run of the benchmark networks stays inside
the range where float32 sums of such values are exact whatever the order,
which makes every ReLU and max-pool decision, and every bf16 store, the same
on any correct implementation.  Whether a given run stays in that range is
checked by the tests, not assumed here.

Nothing here computes any step of the method.
"""
from __future__ import annotations

import numpy as np

from .specs import BF16, FP32, Net

SEED_X = 1
SEED_TARGET = 2
SEED_W = 100
SEED_B = 200

NORMAL = "normal"
EXACT = "exact"
FAMILIES = (NORMAL, EXACT)
EXACT_NNZ = 3          # nonzero weights per output channel in the EXACT family


def normal(seed: int, shape) -> np.ndarray:
    return np.random.Generator(np.random.PCG64(seed)).standard_normal(shape)


def ints(seed: int, shape, lo: int, hi: int) -> np.ndarray:
    """Uniform integers in [lo, hi] as float64."""
    g = np.random.Generator(np.random.PCG64(seed))
    return g.integers(lo, hi + 1, size=shape).astype(np.float64)


def signs(seed: int, shape, density: float = 0.5) -> np.ndarray:
    """Values in {-1, 0, 1}: +-1 with probability `density`, else 0."""
    g = np.random.Generator(np.random.PCG64(seed))
    v = g.choice(np.array([-1.0, 1.0]), size=shape)
    return v * (g.random(shape) < density)


def sparse_signs(seed: int, shape, nnz: int = EXACT_NNZ) -> np.ndarray:
    """For each index of the first axis, `nnz` distinct positions of the
    flattened remaining axes hold +-1; the rest is zero.  Positions are drawn
    per row and rows with a repeated position are drawn again."""
    g = np.random.Generator(np.random.PCG64(seed))
    rows, fan = shape[0], int(np.prod(shape[1:]))
    k = min(nnz, fan)
    pos = g.integers(0, fan, size=(rows, k))
    while True:
        srt = np.sort(pos, axis=1)
        bad = np.any(srt[:, 1:] == srt[:, :-1], axis=1) if k > 1 else np.zeros(rows, bool)
        if not bad.any():
            break
        pos[bad] = g.integers(0, fan, size=(int(bad.sum()), k))
    out = np.zeros((rows, fan))
    np.put_along_axis(out, pos, g.choice(np.array([-1.0, 1.0]), size=(rows, k)), axis=1)
    return out.reshape(shape)


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


def input_x(net: Net, batch: int, dtype: int, seed: int = SEED_X, family: str = NORMAL):
    return tensor(seed, (batch, net.in_channels, net.height, net.width), dtype, family)


def tensor(seed: int, shape, dtype: int, family: str = NORMAL):
    """A seeded input-like tensor: N(0,1), or integers in {-2..2} (EXACT)."""
    assert family in FAMILIES, family
    a = normal(seed, shape) if family == NORMAL else ints(seed, shape, -2, 2)
    return quantize(a, dtype)


def target_like(shape, dtype: int, k: int = 0, family: str = NORMAL):
    """Target of a network run: N(0,1), or integers in {-2..2} (EXACT)."""
    return tensor(SEED_TARGET + k, shape, dtype, family)


def upstream_grad(shape, dtype: int, k: int = 0, family: str = NORMAL):
    """Upstream gradient k of a stage run (main output k = 0, exported skip
    k >= 1): N(0,1), or values in {-1, 0, 1} with half of them zero (EXACT)."""
    assert family in FAMILIES, family
    if family == NORMAL:
        return quantize(normal(SEED_TARGET + k, shape), dtype)
    return quantize(signs(SEED_TARGET + k, shape), dtype)


def layer_params(net: Net, idx: int, dtype: int, index_offset: int = 0, family: str = NORMAL):
    """Weight (logical OIHW) and bias for layer idx: He-normal and
    0.1*N(0,1) (NORMAL), or sparse +-1 and {-1, 0, 1} (EXACT).
    `index_offset` is added to the seed index so a partition run as its own
    network draws the same values as inside the full network.
    Weights follow the storage type; biases stay float32 (accumulation
    precision) in every run."""
    assert family in FAMILIES, family
    L = net.layers[idx]
    g = idx + index_offset
    if family == NORMAL:
        w64 = normal(SEED_W + g, L.weight_shape()) * np.sqrt(2.0 / L.fan_in())
    else:
        w64 = sparse_signs(SEED_W + g, L.weight_shape())
    w = quantize(w64, dtype)
    if L.bias:
        if family == NORMAL:
            b32 = (0.1 * normal(SEED_B + g, (L.cout,))).astype(np.float32)
        else:
            b32 = ints(SEED_B + g, (L.cout,), -1, 1).astype(np.float32)
        b = (b32.astype(np.float64), b32)
    else:
        b = None
    return w, b
