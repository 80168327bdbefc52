"""Palettization of clustered weights in plain numpy — test infrastructure only.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The compressed artefact of weight clustering (the paper's Sec. 2: a model
stored as a lookup table of k centroids plus a b-bit index per weight): each
weight takes the index of its nearest lookup-table entry.

  index_i = the j minimising |v_i - lut_j|  (lowest j on ties),

with v_i the weight's value.  This integer is decided in fp32, the precision
the GPU path computes it in: v_i is exact in fp32 (a 16-bit float), and
|v_i - lut_j| is one fp32 subtraction, so both sides round identically.
Non-finite weights get index 0.  Packing: index i occupies bits [b i, b i + b)
of a little-endian bit stream (byte m holds stream bits 8m .. 8m+7, least
significant first), ceil(n b / 8) bytes.
"""
from __future__ import annotations

import numpy as np


def values32(keys: np.ndarray, fmt: str = "fp16") -> np.ndarray:
    u = np.asarray(keys, dtype=np.uint16).ravel()
    if fmt == "bf16":
        return (u.astype(np.uint32) << 16).view(np.float32)
    return u.view(np.float16).astype(np.float32)


def indices(keys: np.ndarray, lut, fmt: str = "fp16") -> np.ndarray:
    """Nearest-entry index per weight (uint8), decided in fp32."""
    v = values32(keys, fmt)
    c = np.asarray(lut, dtype=np.float32).ravel()
    d = np.abs(v[:, None] - c[None, :])          # float32 subtraction and abs
    idx = np.argmin(d, axis=1).astype(np.uint8)  # first minimum: lowest j on ties
    idx[~np.isfinite(v)] = 0
    return idx


def pack(idx: np.ndarray, bits: int) -> np.ndarray:
    """b-bit little-endian packing of indices."""
    idx = np.asarray(idx, dtype=np.uint8).ravel()
    stream = ((idx[:, None] >> np.arange(bits, dtype=np.uint8)[None, :]) & 1).astype(np.uint8).ravel()
    return np.packbits(stream, bitorder="little")


def unpack(packed: np.ndarray, n: int, bits: int) -> np.ndarray:
    """Inverse of ``pack``."""
    stream = np.unpackbits(np.asarray(packed, dtype=np.uint8), bitorder="little")[: n * bits]
    w = (1 << np.arange(bits, dtype=np.uint32)).astype(np.uint32)
    return (stream.reshape(n, bits).astype(np.uint32) @ w).astype(np.uint8)


def palettize(keys: np.ndarray, lut, bits: int, fmt: str = "fp16") -> np.ndarray:
    return pack(indices(keys, lut, fmt), bits)
