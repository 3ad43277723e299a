"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module only draws random numbers and rounds them to the storage type the
device path consumes.  It holds none of the method's arithmetic: no policy,
no attention, no RoPE, no GEMM.  Both the CPU oracle and the HIP path read the
values it returns, so the two sides always see bit-identical inputs.

Keys.  Every tensor is addressed by a tuple of non-negative integers
``(seed, cfg, tag, layer, chunk, level, ...)`` fed to ``numpy.random.SeedSequence``.
A tensor therefore never depends on the order in which tensors are drawn.

bf16.  ``bf16_bits`` rounds fp32 to bfloat16 with round-to-nearest-even and
returns the raw 16-bit patterns (what the device buffers hold);
``bf16_value`` turns those patterns back into the exactly representable fp32
values (what the oracle upcasts to fp64).
"""
from __future__ import annotations

import concurrent.futures as _cf
import os as _os

import numpy as np

# Tensor tags (the third key component).  Fixed numbers so stored keys stay valid.
TAG_Q = 1
TAG_K = 2
TAG_V = 3
TAG_X = 4
TAG_W_QKV = 10
TAG_W_O = 11
TAG_W_UP = 12
TAG_W_DOWN = 13
TAG_NOISE = 20
TAG_CTX = 40       # condition sequence (e.g. text tokens)
TAG_W_CQ = 41      # cross-attention projections
TAG_W_CK = 42
TAG_W_CV = 43
TAG_W_CO = 44
TAG_GAIN = 45      # RMSNorm gains (qk-norm)


def normal(shape, key, scale: float = 1.0) -> np.ndarray:
    """Standard normal fp32 of ``shape`` times ``scale``, drawn from ``key``."""
    rng = np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))
    x = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x


def normal_parallel(shape, key, scale: float = 1.0, parts: int = 0) -> np.ndarray:
    """Like ``normal`` but drawn in row blocks on a thread pool (large weights).

    Block ``b`` of the leading axis is drawn from ``key + (b,)``; the result
    depends on ``parts`` only through that split, which callers keep fixed.
    """
    shape = tuple(int(s) for s in shape)
    parts = parts or 16
    rows = shape[0]
    bounds = [rows * b // parts for b in range(parts + 1)]
    out = np.empty(shape, dtype=np.float32)

    def fill(b):
        lo, hi = bounds[b], bounds[b + 1]
        if hi > lo:
            out[lo:hi] = normal((hi - lo,) + shape[1:], tuple(key) + (b,), scale)

    workers = min(parts, max(1, len(_os.sched_getaffinity(0))))
    with _cf.ThreadPoolExecutor(workers) as ex:
        list(ex.map(fill, range(parts)))
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even.

    Inputs here are finite (normal draws), so no NaN handling is needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> the fp32 values they encode."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bfloat16, returned as fp32."""
    return bf16_value(bf16_bits(x))
