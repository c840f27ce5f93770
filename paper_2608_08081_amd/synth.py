"""Seeded synthetic workloads shaped like the paper's MoE attention layers.

This module only draws random inputs; it holds none of the compression or
attention arithmetic.  Both the GPU library's tests/benchmark and the CPU
oracle consume what it produces, so the two sides always see identical bytes.

Recipe (stands in for the KV activations of the MoE models the paper
evaluates, which are not available; head_dim 128 as in App. C):

* "anisotropic" keys/values: entries N(0, 1) times a per-channel scale drawn
  log-normal(0, 0.5) (i.e. ln scale ~ N(0, 0.25)), with 4 distinct random
  outlier channels multiplied by 20; scales are drawn independently for keys
  and values and for every KV head.
* "heavy-tailed" keys/values: Student-t (4 degrees of freedom) entries times
  the same kind of log-normal channel scales, no outlier channels.
* queries: N(0, 1) fp32.
* needle: at one seeded position of each KV head the key is replaced by
  8 * sqrt(d) times the unit direction of the group's first query head, so
  that head's softmax argmax is that position by a wide margin.
* variable lengths: per-sequence context lengths uniform on the integers
  [2048, 32768].

Streams: numpy ``default_rng([seed, workload_id, stream])`` with stream
0 = key channel scales, 1 = value channel scales, 2 = keys, 3 = values,
4 = queries, 5 = needle positions / appended tokens, 6 = context lengths,
7 = the standard normal matrices of the dense-random rotation design.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

HEAD_DIM = 128


@dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic workload."""
    wid: int
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    context: int                      # tokens per sequence (max for varlen)
    dtype: str                        # "f32" | "f16" (K/V input precision)
    kv_dist: str = "anisotropic"      # | "heavy_tailed"
    varlen: tuple | None = None       # (lo, hi) inclusive, per-sequence length
    needle: bool = False
    decode_steps: int = 1             # appended tokens + decode steps
    rotation_seed: int = 0
    notes: str = field(default="", compare=False)

    @property
    def group(self) -> int:
        return self.n_q_heads // max(self.n_kv_heads, 1)


WORKLOADS = {
    0: Workload(0, "tiny_g1_t1024", 1, 1, 1, 1024, "f32", rotation_seed=1000,
                notes="single head, fp32 K/V, compress all then one decode step"),
    1: Workload(1, "gqa8_t8192_append1000", 1, 32, 4, 8192, "f16", decode_steps=1000,
                rotation_seed=1001,
                notes="bulk compress 8192 tokens, then 1000 x (append one token, decode)"),
    2: Workload(2, "gqa8_t32768_needle", 1, 32, 4, 32768, "f16", needle=True,
                rotation_seed=1002, notes="32K context decode with a planted key"),
    3: Workload(3, "varlen_b64_g8", 64, 16, 2, 32768, "f16", varlen=(2048, 32768),
                rotation_seed=1003, notes="batched serving decode, varlen split-K"),
    4: Workload(4, "compress_4x32768x8", 4, 8, 8, 32768, "f16", kv_dist="heavy_tailed",
                rotation_seed=1004, notes="prefill-scale compression only"),
}


def rng(seed: int, wid: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([seed, wid, stream])


def channel_scales(g: np.random.Generator, n_heads: int, d: int = HEAD_DIM,
                   n_outliers: int = 4, outlier_factor: float = 20.0) -> np.ndarray:
    """[n_heads][d] fp32 per-channel scales: log-normal(0, 0.5), with
    ``n_outliers`` distinct channels per head multiplied by ``outlier_factor``."""
    sc = g.lognormal(0.0, 0.5, size=(n_heads, d))
    for h in range(n_heads):
        if n_outliers:
            idx = g.choice(d, size=n_outliers, replace=False)
            sc[h, idx] *= outlier_factor
    return sc.astype(np.float32)


def _draw_entries(g: np.random.Generator, shape, dist: str) -> np.ndarray:
    if dist == "anisotropic":
        return g.standard_normal(size=shape, dtype=np.float32)
    if dist == "heavy_tailed":
        return g.standard_t(4.0, size=shape).astype(np.float32)
    raise ValueError(dist)


def kv_tensor(seed: int, w: Workload, which: str, n_tokens: int | None = None,
              batch: int | None = None) -> np.ndarray:
    """Keys (``which='k'``) or values (``'v'``): [B][H_kv][T][d] in the
    workload's input dtype (fp16 values are the RNE rounding of the fp32
    draw)."""
    t = w.context if n_tokens is None else n_tokens
    b = w.batch if batch is None else batch
    scale_stream, data_stream = (0, 2) if which == "k" else (1, 3)
    n_out = 4 if w.kv_dist == "anisotropic" else 0
    sc = channel_scales(rng(seed, w.wid, scale_stream), w.n_kv_heads, n_outliers=n_out)
    x = _draw_entries(rng(seed, w.wid, data_stream), (b, w.n_kv_heads, t, HEAD_DIM),
                      w.kv_dist)
    x *= sc[None, :, None, :]
    return x.astype(np.float16) if w.dtype == "f16" else x


def queries(seed: int, w: Workload, n_steps: int = 1) -> np.ndarray:
    """[n_steps][B][H_q][d] fp32 queries."""
    g = rng(seed, w.wid, 4)
    return g.standard_normal(size=(n_steps, w.batch, w.n_q_heads, HEAD_DIM),
                             dtype=np.float32)


def appended_tokens(seed: int, w: Workload, n_steps: int, batch: int | None = None):
    """Keys and values appended during decode: two arrays
    [n_steps][B][H_kv][d], same distribution (and channel scales) as the
    cache, drawn from stream 5."""
    b = w.batch if batch is None else batch
    n_out = 4 if w.kv_dist == "anisotropic" else 0
    sk = channel_scales(rng(seed, w.wid, 0), w.n_kv_heads, n_outliers=n_out)
    sv = channel_scales(rng(seed, w.wid, 1), w.n_kv_heads, n_outliers=n_out)
    g = rng(seed, w.wid, 5)
    shape = (n_steps, b, w.n_kv_heads, HEAD_DIM)
    k = _draw_entries(g, shape, w.kv_dist) * sk[None, None]
    v = _draw_entries(g, shape, w.kv_dist) * sv[None, None]
    if w.dtype == "f16":
        return k.astype(np.float16), v.astype(np.float16)
    return k.astype(np.float32), v.astype(np.float32)


def context_lengths(seed: int, w: Workload) -> np.ndarray:
    """Per-sequence context lengths (int32 [B])."""
    if w.varlen is None:
        return np.full(w.batch, w.context, dtype=np.int32)
    lo, hi = w.varlen
    return rng(seed, w.wid, 6).integers(lo, hi + 1, size=w.batch).astype(np.int32)


def plant_needle(seed: int, w: Workload, k: np.ndarray, q: np.ndarray,
                 factor: float = 8.0):
    """Replace, in place, one seeded key position per (sequence, KV head) by
    factor * sqrt(d) * q_h0 / ||q_h0||, h0 = first query head of the group.
    k: [B][H_kv][T][d]; q: [B][H_q][d].  Returns positions [B][H_kv]."""
    g = rng(seed, w.wid, 5)
    bsz, hkv, t, d = k.shape
    pos = g.integers(0, t, size=(bsz, hkv))
    for b in range(bsz):
        for h in range(hkv):
            qv = q[b, h * w.group].astype(np.float64)
            u = qv / np.sqrt(np.dot(qv, qv))
            k[b, h, pos[b, h]] = (factor * np.sqrt(d) * u).astype(k.dtype)
    return pos


def gaussian_matrices(seed: int, n: int, d: int = HEAD_DIM) -> np.ndarray:
    """[n][d][d] independent standard normal entries (fp64): the input of the
    dense-random rotation design of the rotation study (one matrix per KV
    head)."""
    return rng(seed, 90, 7).standard_normal((n, d, d))
