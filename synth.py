"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the method: it only draws random arrays (numpy PCG64,
one child stream per named tensor) with the shapes and value distributions of the
paper's workloads, and converts fp32 draws to bf16 bit patterns by dropping the low 16
bits (so the bf16 values are exactly representable and need no rounding rule).
Nothing here is shared with the oracle's or the GPU library's arithmetic.

The datasets the paper trains on (ImageNet, Sec. 4) and the MNIST/CIFAR-shaped inputs of
the smaller workloads are not used: these generators stand in for them by shape only.
"""
from __future__ import annotations

import zlib

import numpy as np

BASE_SEED = 1701_00485


def rng(stream: int, name: str) -> np.random.Generator:
    """Independent generator for tensor `name` of workload `stream`."""
    ss = np.random.SeedSequence([BASE_SEED + int(stream), zlib.crc32(name.encode())])
    return np.random.Generator(np.random.PCG64(ss))


def normal(stream: int, name: str, shape, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    return (rng(stream, name).standard_normal(size=shape, dtype=np.float32) * np.float32(std)
            + np.float32(mean)).astype(np.float32)


def uniform(stream: int, name: str, shape, lo: float = 0.0, hi: float = 1.0) -> np.ndarray:
    return rng(stream, name).uniform(lo, hi, size=shape).astype(np.float32)


def labels(stream: int, name: str, n: int, classes: int) -> np.ndarray:
    return rng(stream, name).integers(0, classes, size=n, dtype=np.int64)


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of fp32 draws, keeping the top 16 bits of each value."""
    return (np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def bf16_values(bits: np.ndarray) -> np.ndarray:
    """The fp32 values of bf16 bit patterns (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(stream: int, name: str, shape, std: float = 1.0) -> np.ndarray:
    return bf16_bits(normal(stream, name, shape, std))


def sample_indices(stream: int, name: str, total: int, count: int) -> np.ndarray:
    """`count` distinct flat indices in [0, total), sorted, always including both ends."""
    count = min(count, total)
    g = rng(stream, name)
    idx = g.choice(total, size=count, replace=False) if count < total else np.arange(total)
    idx = np.unique(np.concatenate([idx, [0, total - 1]]).astype(np.int64))
    return idx
