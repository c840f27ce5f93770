"""IsoQuant KV compression, Algorithm 1 (Sec. 3.2 Steps 1-4).  Test
infrastructure only.

For one key or value vector x in R^d:

1. Normalize (Alg. 1 first step; Step 1): s = ||x||_2, x_hat = x / s; s is
   kept as the vector's scale.
2. Rotate (Step 2, Eq. 2): x_tilde = R_SO(4)(H_d x_hat) = R x_hat.
3. Quantize (Step 3): each coordinate to the nearest codebook level.
4. Bit-pack (Step 4): d codes of b bits into d*b/8 bytes (48 bytes at
   d = 128, b = 3; 32 at b = 2, 64 at b = 4).  Algorithm 1 is stated for a
   general b with its codebook C_b; the bit width is read off the codebook
   (2^b levels, 2^b - 1 thresholds).

Readings of what the paper leaves open:

* Precision: x is taken exactly into fp64, s and x_tilde are computed in
  fp64, and the stored scale is s rounded to fp32 (round to nearest even).
* Zero vector: s = 0 gives x_hat = 0 and every coordinate 0.
* Code of a coordinate y: the number of thresholds t_j with t_j <= y, i.e.
  levels are numbered in ascending order and a value exactly on a threshold
  goes to the upper level (-0.0 counts as 0).  With thresholds at the level
  midpoints this is the nearest level, ties upward.
* Packed layout: code i occupies bits b*i .. b*i+b-1 of a little-endian bit
  string (bit n is bit n % 8 of byte n // 8), least significant bit first;
  at b = 3 dims 8g .. 8g+7 fill bytes 3g .. 3g+2.  Keys and values use the
  same record format, one d*b/8-byte record per token, records of
  consecutive tokens contiguous, scales stored in a separate fp32 array.
"""

from __future__ import annotations

import numpy as np

BITS = 3


def bits_of(codebook) -> int:
    """Bit width b of a codebook given by its levels (2^b) or thresholds
    (2^b - 1)."""
    n = len(codebook)
    n = n + 1 if n % 2 else n
    b = int(n).bit_length() - 1
    if n != 1 << b or b < 1:
        raise ValueError(f"codebook of {len(codebook)} entries is not 2^b levels")
    return b


def normalize(x):
    """Step 1: fp64 norm and unit vector.  x: [..., d]."""
    x64 = np.asarray(x).astype(np.float64)
    s = np.sqrt(np.sum(x64 * x64, axis=-1))
    safe = np.where(s > 0, s, 1.0)
    xhat = np.where((s > 0)[..., None], x64 / safe[..., None], 0.0)
    return s, xhat


def rotate(xhat, r):
    """Step 2: x_tilde = R x_hat for each row of xhat ([..., d]); r: [d, d]."""
    return np.asarray(xhat, dtype=np.float64) @ np.asarray(r, dtype=np.float64).T


def quantize(y, thresholds):
    """Step 3: code = #{j : t_j <= y} per coordinate (uint8)."""
    y = np.asarray(y, dtype=np.float64)
    t = np.asarray(thresholds, dtype=np.float64)
    return np.sum(y[..., None] >= t, axis=-1).astype(np.uint8)


def pack(codes, bits: int = BITS):
    """Step 4: [..., d] codes of ``bits`` bits -> [..., d*bits/8] bytes, code i
    at bits bits*i .. bits*i + bits-1, LSB first, little-endian bit string."""
    codes = np.asarray(codes, dtype=np.uint8)
    d = codes.shape[-1]
    if (d * bits) % 8:
        raise ValueError("d * bits must be a multiple of 8")
    shifts = np.arange(bits, dtype=np.uint8)
    bitplanes = (codes[..., :, None] >> shifts) & 1          # [..., d, bits]
    flat = bitplanes.reshape(codes.shape[:-1] + (d * bits,))
    return np.packbits(flat, axis=-1, bitorder="little")


def unpack(packed, d: int = 128, bits: int = BITS):
    """Inverse of :func:`pack`."""
    packed = np.asarray(packed, dtype=np.uint8)
    flat = np.unpackbits(packed, axis=-1, bitorder="little")
    bitplanes = flat.reshape(packed.shape[:-1] + (d, bits)).astype(np.uint8)
    weights = (1 << np.arange(bits)).astype(np.uint8)
    return np.sum(bitplanes * weights, axis=-1).astype(np.uint8)


def compress(x, r, thresholds):
    """Algorithm 1 for a batch of vectors that share one rotation.

    x: [..., d] (any float dtype, taken exactly); r: [d, d]; thresholds of
    C_b (2^b - 1 of them).  Returns (packed [..., d*b/8] uint8, scale fp32
    [...], codes [..., d], x_tilde fp64 [..., d], scale fp64 [...]).  The
    last three are for analysis (boundary distances, reconstruction).
    """
    s, xhat = normalize(x)
    y = rotate(xhat, r)
    codes = quantize(y, thresholds)
    return pack(codes, bits_of(thresholds)), s.astype(np.float32), codes, y, s


def compress_kv(x, rots, thresholds):
    """Compress a cache tensor x: [B][H_kv][T][d] with one rotation per KV
    head (rots: [H_kv][d][d]).  Returns (packed [B][H][T][d*b/8], scale
    fp32 [B][H][T], codes, x_tilde, scale64)."""
    x = np.asarray(x)
    b, h, t, d = x.shape
    packed = np.empty((b, h, t, d * bits_of(thresholds) // 8), dtype=np.uint8)
    norms = np.empty((b, h, t), dtype=np.float32)
    codes = np.empty((b, h, t, d), dtype=np.uint8)
    ys = np.empty((b, h, t, d), dtype=np.float64)
    s64 = np.empty((b, h, t), dtype=np.float64)
    for hh in range(h):
        p, s, c, y, s_ = compress(x[:, hh], rots[hh], thresholds)
        packed[:, hh], norms[:, hh], codes[:, hh], ys[:, hh], s64[:, hh] = p, s, c, y, s_
    return packed, norms, codes, ys, s64


def dequantize_rotated(codes, scale, levels):
    """Rotated-space reconstruction s * C[code] (no renormalization)."""
    lv = np.asarray(levels, dtype=np.float64)
    return np.asarray(scale, dtype=np.float64)[..., None] * lv[np.asarray(codes)]


def reconstruct(codes, scale, levels, r):
    """Original-space reconstruction x_hat' = s * R^T C[code] (what the
    reconstruct-then-compute path materializes)."""
    return dequantize_rotated(codes, scale, levels) @ np.asarray(r, dtype=np.float64)


def reconstruct_kv(packed, norms, rots, levels, d: int = 128):
    """Materialize a packed cache [B][H_kv][T][d*b/8] with scales [B][H_kv][T]
    as original-space vectors [B][H_kv][T][d] (fp64): the dequantization and
    R^T of the reconstruct-then-compute pipeline (Fig. 1 top), one rotation
    per KV head."""
    packed = np.asarray(packed)
    b, h, t, _ = packed.shape
    out = np.empty((b, h, t, d), dtype=np.float64)
    for hh in range(h):
        out[:, hh] = reconstruct(unpack(packed[:, hh], d, bits_of(levels)), norms[:, hh], levels,
                                 rots[hh])
    return out
