"""After refinement: canonical positive scales, dequantized weights, packed
codes and activation ordering (test oracle).

TEST INFRASTRUCTURE ONLY: used by the tests; never by the product path.

* canonicalize: App. E.3, eq. (canonicalization): a group with s < 0 becomes
  s' = -s, q' = qmax - q, z' = qmax - z (same weights, eq.
  (canonicalization_equivalence)).
* dequantize: eq. (1), what = s (q - z) in fp32, rounded once to the target
  dtype; with an activation-order permutation the weights return to the
  original column order (App. A.1, App. E.2).
* pack / unpack: row-wise little-endian bit streams of b-bit codes, 32-bit
  words (the library's deployment layout).
* act_order: channels by decreasing diag(H), ties by increasing index.
"""

from __future__ import annotations

import numpy as np


def canonicalize(codes, scales, zeros, g, bits):
    qmax = (1 << bits) - 1
    codes = np.array(codes, dtype=np.uint8, copy=True)
    scales = np.array(scales, dtype=np.float32, copy=True)
    zeros = np.array(zeros, dtype=np.int32, copy=True)
    rows, G = scales.shape
    for r in range(rows):
        for i in range(G):
            if scales[r, i] < 0:
                scales[r, i] = -scales[r, i]
                zeros[r, i] = qmax - zeros[r, i]
                codes[r, i * g:(i + 1) * g] = qmax - codes[r, i * g:(i + 1) * g]
    return codes, scales, zeros


def bf16_bits(x):
    """fp32 -> bf16 bit patterns, round to nearest even (NaN stays NaN)."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.asarray(x, np.float32))
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), r)


def dequantize(codes, scales, zeros, g, dtype="f32", perm=None):
    """s (q - z) in fp32, then rounded to dtype ('f32', 'f16' or 'bf16', the
    last as uint16 bit patterns); with perm, column perm[k] receives position k."""
    s = np.repeat(np.asarray(scales, np.float32), g, axis=1)
    zq = (np.asarray(codes, np.int64) - np.repeat(np.asarray(zeros, np.int64), g, axis=1))
    w = (s * zq.astype(np.float32)).astype(np.float32)
    if dtype == "f16":
        w = w.astype(np.float16)
    elif dtype == "bf16":
        w = bf16_bits(w)
    if perm is not None:
        out = np.empty_like(w)
        out[:, np.asarray(perm)] = w
        w = out
    return w


def pack(codes, bits):
    """uint32 [rows, ceil(cols bits / 32)]: bit j of code k is stream bit k bits + j."""
    codes = np.asarray(codes, np.uint64)
    rows, cols = codes.shape
    wpr = (cols * bits + 31) // 32
    stream = np.zeros((rows, wpr * 32), dtype=np.uint64)
    for j in range(bits):
        stream[:, np.arange(cols) * bits + j] = (codes >> j) & 1
    words = (stream.reshape(rows, wpr, 32) << np.arange(32, dtype=np.uint64)).sum(axis=2)
    return words.astype(np.uint32)


def unpack(packed, cols, bits):
    packed = np.asarray(packed, np.uint32).astype(np.uint64)
    rows, wpr = packed.shape
    stream = (packed[:, :, None] >> np.arange(32, dtype=np.uint64)) & 1
    stream = stream.reshape(rows, wpr * 32)
    codes = np.zeros((rows, cols), dtype=np.uint64)
    for j in range(bits):
        codes |= stream[:, np.arange(cols) * bits + j] << j
    return codes.astype(np.uint8)


def act_order(H):
    return np.argsort(-np.diag(np.asarray(H, np.float32)), kind="stable").astype(np.int32)


def permute(W, H, perm):
    perm = np.asarray(perm)
    return (np.ascontiguousarray(np.asarray(W)[:, perm]),
            np.ascontiguousarray(np.asarray(H)[np.ix_(perm, perm)]))


__all__ = ["canonicalize", "bf16_bits", "dequantize", "pack", "unpack", "act_order", "permute"]
