"""Seeded synthetic inputs for the SPHQuant decode path.

Shared by the oracle tests, the GPU parity tests and the benchmark. This module only
draws random numbers and describes workload shapes: it holds none of the quantisation
method's arithmetic (no decomposition, direction assignment, radius fitting, packing or
decoding). Every array is derived from ``numpy.random.default_rng`` with an explicit
integer key, so a (config, layer, matrix, stream) tuple always yields the same bytes.

Code arrays use the logical layout of the C ABI:

* ``signs``  uint8  [n][k/8]    bit j set  <=> element 8v+j of the vector is negative
* ``dir``    uint16 [n][k/8]    direction index, < 2**D
* ``q``      uint8  [n][k/8]    radius level, < 2**V
* ``gmin``   uint16 [n][k/128]  fp16 bit patterns of the group offsets
* ``gstep``  uint16 [n][k/128]  fp16 bit patterns of the group steps
* codebook   uint16 [2**D][8]   fp16 bit patterns, entries non-negative
* x          uint16 [m][k]      fp16 bit patterns of the activations
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

VEC = 8
GROUP = 128

# Random-stream identifiers inside one (config, layer, matrix) key.
STREAM_CODEBOOK = 0
STREAM_WEIGHTS = 1
STREAM_CODES = 2
STREAM_X = 3

# (dir_bits, radius_bits) of every representation the library accepts.
FORMATS = {
    "W2": (6, 4),       # 8 sign + 6-bit direction + 4-bit radius (the W2 kernel format)
    "W3": (13, 3),      # 8 sign + 13-bit direction + 3-bit radius (3.00 bpw payload)
    "W2_cfg": (4, 4),   # 8 sign + 4-bit direction + 4-bit radius (16 bits per vector)
    "W3_cfg": (8, 8),   # 8 sign + 8-bit direction + 8-bit radius (24 bits per vector)
    "W2_16": (6, 2),    # 8 sign + 6-bit direction + 2-bit radius (2.00 bpw payload)
    "W3_25": (13, 4),   # 8 sign + 13-bit direction + 4-bit radius (3.125 bpw payload)
    "W2_63": (6, 3),    # bit-allocation splits of the W2 budget: 8 sign + 6 direction + 3 radius,
    "W2_72": (7, 2),    # 8 + 7 + 2,
    "W2_82": (8, 2),    # 8 + 8 + 2
    "V4": (2, 3),       # 4-D vectors: 4 sign + 2-bit direction + 3-bit radius (2.25 bpw payload)
    "V16": (14, 6),     # 16-D vectors: 16 sign + 14-bit direction + 6-bit radius (2.25 bpw payload)
}

# Vector size of each format (8 unless listed).
FORMAT_DIM = {"V4": 4, "V16": 16}


def fmt_dim(fmt: str) -> int:
    return FORMAT_DIM.get(fmt, VEC)


def rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(v) for v in key])


def f16_bits(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float16).view(np.uint16))


def random_codebook(dir_bits: int, g: np.random.Generator, dim: int = VEC) -> np.ndarray:
    """2**dir_bits positive unit directions |g|/||g|| with g ~ N(0, I), stored as fp16 bits."""
    a = np.abs(g.standard_normal((1 << dir_bits, dim)))
    a /= np.linalg.norm(a, axis=1, keepdims=True)
    return f16_bits(a)


def uniform_codes(n: int, k: int, dir_bits: int, radius_bits: int, g: np.random.Generator,
                  dim: int = VEC) -> dict:
    """Independent uniform signs, direction indices and radius levels (signs are one byte per
    vector for 4-D and 8-D vectors, 16 bits for 16-D)."""
    nv = k // dim
    return {
        "signs": g.integers(0, 1 << dim, (n, nv)).astype(np.uint8 if dim <= 8 else np.uint16),
        "dir": g.integers(0, 1 << dir_bits, (n, nv), dtype=np.uint16),
        "q": g.integers(0, 1 << radius_bits, (n, nv), dtype=np.uint8),
    }


def row_scale_group_params(n: int, k: int, radius_bits: int, g: np.random.Generator):
    """Per-row scale s ~ U(0.5, 2) whose radius levels sit at s*(level+0.5)/2**V.

    Expressed as the per-group (offset, step) pair: offset s/2**(V+1), step s/2**V,
    repeated over every group of the row. Both are exact in fp16 once s is.
    """
    s = g.uniform(0.5, 2.0, n).astype(np.float16).astype(np.float64)
    ng = k // GROUP
    off = np.repeat((s / 2.0 ** (radius_bits + 1))[:, None], ng, axis=1)
    step = np.repeat((s / 2.0 ** radius_bits)[:, None], ng, axis=1)
    return f16_bits(off), f16_bits(step)


def varied_group_params(n: int, k: int, radius_bits: int, g: np.random.Generator):
    """An independent (offset, step) pair for every group of every row, so that neighbouring
    groups of one row never share parameters: offsets of either sign (about a quarter negative),
    about one step in eight exactly zero, and magnitudes spread over eight binary orders
    (2^-4 ... 2^3 times a U(0.5, 2) mantissa), all finite fp16."""
    ng = k // GROUP
    mag = g.uniform(0.5, 2.0, (n, ng)) * 2.0 ** g.integers(-4, 4, (n, ng))
    off = np.where(g.random((n, ng)) < 0.25, -1.0, 1.0) * mag
    step = g.uniform(0.5, 2.0, (n, ng)) * 2.0 ** g.integers(-4, 4, (n, ng)) / 2.0 ** radius_bits
    step[g.random((n, ng)) < 0.125] = 0.0
    return f16_bits(off), f16_bits(step)


def extreme_group_params(n: int, k: int, radius_bits: int, g: np.random.Generator):
    """Group parameters at the edges of fp16: rows cycle through three kinds.

    * row % 3 == 0: radii beyond the fp16 range, offsets in [2^14, 2^15.9] and steps in
      [2^10, 2^15], so min + q * step reaches far past 65504;
    * row % 3 == 1: radii among the fp16 subnormals and smallest normals (offsets and steps in
      [2^-24, 2^-13]);
    * row % 3 == 2: huge and ordinary groups alternating inside the row.
    """
    ng = k // GROUP
    big_off = 2.0 ** g.uniform(14.0, 15.9, (n, ng))
    big_step = 2.0 ** g.uniform(10.0, 15.0, (n, ng))
    tiny_off = 2.0 ** g.uniform(-24.0, -13.0, (n, ng))
    tiny_step = 2.0 ** g.uniform(-24.0, -13.0, (n, ng))
    mid_off = g.uniform(0.01, 0.1, (n, ng))
    mid_step = g.uniform(0.001, 0.01, (n, ng))
    kind = (np.arange(n) % 3)[:, None] * np.ones((1, ng), dtype=np.int64)
    alt = (np.arange(ng) % 2)[None, :] == 0
    use_big = (kind == 0) | ((kind == 2) & alt)
    off = np.where(use_big, big_off, np.where(kind == 1, tiny_off, mid_off))
    step = np.where(use_big, big_step, np.where(kind == 1, tiny_step, mid_step))
    off = np.where(g.random((n, ng)) < 0.25, -off, off)
    return f16_bits(off), f16_bits(step)


def outlier_gaussian_weights(n: int, k: int, g: np.random.Generator, sigma: float = 0.02,
                             p: float = 1e-3, scale: float = 20.0, nu: float = 3.0) -> np.ndarray:
    """N(0, sigma^2) weights; each entry is replaced with probability p by scale*sigma*t_nu."""
    w = g.normal(0.0, sigma, (n, k))
    mask = g.random((n, k)) < p
    w[mask] = scale * sigma * g.standard_t(nu, int(mask.sum()))
    return w


def activations(m: int, k: int, g: np.random.Generator) -> np.ndarray:
    """fp16 N(0, 1) activations, row-major [m][k], as fp16 bits."""
    return f16_bits(g.standard_normal((m, k)))


# ---------------------------------------------------------------------------------------
# Workloads: backbone-shaped matrix sets at batch 1..32.
# ---------------------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    name: str
    fmt: str
    shapes: tuple          # ((label, n, k), ...) for one layer
    layers: int
    batches: tuple
    codes: str             # "uniform" (random codes + row-scale params) or "encoded"


LLM8B_SHAPES = (("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
                ("gate", 12288, 4096), ("up", 12288, 4096), ("down", 4096, 12288))
LLM32B_SHAPES = (("q", 5120, 5120), ("k", 1024, 5120), ("v", 1024, 5120), ("o", 5120, 5120),
                 ("gate", 25600, 5120), ("up", 25600, 5120), ("down", 5120, 25600))

WORKLOADS = {
    0: Workload("w2-1024x1024", "W2", (("w", 1024, 1024),), 1, (1,), "uniform"),
    1: Workload("w2-4096x4096", "W2", (("w", 4096, 4096),), 1, (1,), "encoded"),
    2: Workload("w3-8b-class-36L", "W3", LLM8B_SHAPES, 36, (1,), "encoded"),
    3: Workload("w2-32b-class-64L", "W2", LLM32B_SHAPES, 64, (1, 2, 4, 8), "encoded"),
    4: Workload("w2w3-12288x4096-4096x12288", "W2",
                (("up", 12288, 4096), ("down", 4096, 12288)), 1, (16, 32), "encoded"),
}
