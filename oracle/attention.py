"""Single-token decode attention on the packed cache (App. A; Table 2;
Sec. 3.4 "Fused Metal Decode Pipeline").  Test infrastructure only.

Compressed-space path (App. A), for query head h of KV head g = h // G with
G = H_q / H_kv and one rotation R_g shared by the keys, values and the G
query heads of the group:

    q_tilde   = R_g q_h                                  (forward rotation)
    score_j   = s^K_j * (q_tilde . C[codeK_j]) * scale    (fused QK, Kernel A)
    alpha     = softmax_j(score)                          (Kernel B)
    o_tilde   = sum_j alpha_j s^V_j C[codeV_j]             (fused V, Kernel C)
    o         = R_g^T o_tilde                              (one inverse, Kernel D)

Reconstruct-then-compute path (Sec. 1, Fig. 1 top): materialize
k_hat_j = s^K_j R_g^T C[codeK_j] and v_hat_j likewise, then ordinary attention
with the unrotated query.  Because R_g is orthogonal the two paths are equal
in exact arithmetic (App. A: <Rq, Rk> = <q, k> and sum alpha R v = R sum alpha v).

Readings: scale defaults to 1/sqrt(d); the softmax is the max-subtracted
one; no mask inside the cache (single-token decode attends to every cached
position j < seq_len[b]); a sequence of length 0 yields a zero output.
All arithmetic is fp64.
"""

from __future__ import annotations

import numpy as np

from . import compress as _cz
from . import rotation as _rot


def softmax(x):
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(x - np.max(x, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def _default_scale(d, scale):
    return 1.0 / np.sqrt(d) if (scale is None or scale <= 0) else float(scale)


def fused_scores(q, k_packed, k_norms, r, levels, scale=None):
    """Compressed-space scores for one KV head: q [G][d] (original space),
    k_packed [T][d*b/8], k_norms [T] -> scores [G][T] (fp64)."""
    q = np.asarray(q, dtype=np.float64)
    d = q.shape[-1]
    qt = q @ np.asarray(r).T                                   # R q per head
    bits = _cz.bits_of(levels)
    kt = _cz.dequantize_rotated(_cz.unpack(k_packed, d, bits), k_norms, levels)
    return (qt @ kt.T) * _default_scale(d, scale)


def decode_fused(q, k_packed, k_norms, v_packed, v_norms, seq_lens, quats,
                 levels, scale=None, skip_inverse=False):
    """Compressed-space decode attention for a batch (App. A).

    q: [B][H_q][d]; k_packed/v_packed: [B][H_kv][cap][d*b/8] uint8 (b from
    the codebook: 48 bytes at b = 3);
    k_norms/v_norms: [B][H_kv][cap] fp32; seq_lens: [B]; quats:
    [H_kv][d/4][2][4].  Returns out [B][H_q][d] fp64 in the original space.
    ``skip_inverse`` returns o_tilde without R^T (the negative control of
    Sec. 5, "Inverse rotation is mandatory")."""
    rots = _rot.rotation_matrices(np.asarray(quats))
    return decode_fused_rotations(q, k_packed, k_norms, v_packed, v_norms, seq_lens, rots,
                                  levels, scale, skip_inverse)


def decode_fused_rotations(q, k_packed, k_norms, v_packed, v_norms, seq_lens, rots, levels,
                           scale=None, skip_inverse=False):
    """decode_fused with the rotation of each KV head given as a d x d
    orthogonal matrix ([H_kv][d][d]): App. A holds for any orthogonal R, so
    the designs of the rotation ablation run through the same steps."""
    q = np.asarray(q, dtype=np.float64)
    bsz, hq, d = q.shape
    hkv = k_packed.shape[1]
    if hq % hkv:
        raise ValueError("H_q must be a multiple of H_kv")
    group = hq // hkv
    out = np.zeros((bsz, hq, d))
    bits = _cz.bits_of(levels)
    for b in range(bsz):
        n = int(seq_lens[b])
        if n == 0:
            continue
        for g in range(hkv):
            heads = slice(g * group, (g + 1) * group)
            scores = fused_scores(q[b, heads], k_packed[b, g, :n], k_norms[b, g, :n],
                                  rots[g], levels, scale)
            alpha = softmax(scores)                                   # [G][n]
            vt = _cz.dequantize_rotated(_cz.unpack(v_packed[b, g, :n], d, bits),
                                        v_norms[b, g, :n], levels)     # [n][d]
            o_tilde = alpha @ vt                                      # [G][d]
            out[b, heads] = o_tilde if skip_inverse else o_tilde @ rots[g]
    return out


def decode_multi(q, k_packed, k_norms, v_packed, v_norms, seq_lens, quats, levels,
                 scale=None):
    """Decode of T query tokens per sequence over one cache (the verification
    step of speculative decoding; App. A applied per token): the T tokens
    occupy the last T of the seq_lens[b] cached positions, and token t
    attends positions 0 .. seq_lens[b] - T + t (causal among the new tokens),
    i.e. it is single-token decode with length max(seq_lens[b] - T + 1 + t, 0).

    q: [B][T][H_q][d]; caches and quats as for decode_fused.  Returns
    [B][T][H_q][d] fp64."""
    q = np.asarray(q, dtype=np.float64)
    bsz, t_new, hq, d = q.shape
    out = np.zeros((bsz, t_new, hq, d))
    for t in range(t_new):
        lens = [max(int(n) - t_new + 1 + t, 0) for n in seq_lens]
        out[:, t] = decode_fused(q[:, t], k_packed, k_norms, v_packed, v_norms, lens, quats,
                                 levels, scale)
    return out


def decode_reconstruct(q, k_packed, k_norms, v_packed, v_norms, seq_lens, quats,
                       levels, scale=None):
    """Reconstruct-then-compute decode: dequantize, apply R^T per token, then
    standard attention in the original space (Fig. 1 top)."""
    q = np.asarray(q, dtype=np.float64)
    bsz, hq, d = q.shape
    hkv = k_packed.shape[1]
    group = hq // hkv
    rots = _rot.rotation_matrices(np.asarray(quats))
    sc = _default_scale(d, scale)
    out = np.zeros((bsz, hq, d))
    bits = _cz.bits_of(levels)
    for b in range(bsz):
        n = int(seq_lens[b])
        if n == 0:
            continue
        for g in range(hkv):
            k_hat = _cz.reconstruct(_cz.unpack(k_packed[b, g, :n], d, bits), k_norms[b, g, :n],
                                    levels, rots[g])
            v_hat = _cz.reconstruct(_cz.unpack(v_packed[b, g, :n], d, bits), v_norms[b, g, :n],
                                    levels, rots[g])
            for h in range(g * group, (g + 1) * group):
                alpha = softmax((k_hat @ q[b, h]) * sc)
                out[b, h] = alpha @ v_hat
    return out


def attention_exact(q, k, v, seq_lens, n_kv_heads, scale=None):
    """Plain fp64 attention on unquantized K/V ([B][H_kv][T][d]); context for
    the error the 3-bit cache introduces, not a target."""
    q = np.asarray(q, dtype=np.float64)
    bsz, hq, d = q.shape
    group = hq // n_kv_heads
    sc = _default_scale(d, scale)
    out = np.zeros((bsz, hq, d))
    for b in range(bsz):
        n = int(seq_lens[b])
        if n == 0:
            continue
        for h in range(hq):
            g = h // group
            kk = np.asarray(k[b, g, :n], dtype=np.float64)
            vv = np.asarray(v[b, g, :n], dtype=np.float64)
            out[b, h] = softmax((kk @ q[b, h]) * sc) @ vv
    return out


def decode_fused_rope(q, q_rope, k_packed, k_norms, k_rope, v_packed, v_norms, seq_lens, quats,
                      levels, scale=None):
    """Decode attention with the content / RoPE sub-block split that the
    paper names as the missing piece for latent-attention models (Sec. 5,
    "MLA/RoPE hard blocker"; Sec. 6): each key is a content part of d dims,
    compressed as every other key (Alg. 1), and a positional part of d_r
    dims that carries the rotary phase and therefore is neither rotated nor
    quantized, stored as given.  Values are content only.  For query head h
    of KV head g:

        score_j = scale * ( s^K_j (R_g q_h) . C[codeK_j]  +  q_rope_h . k_rope_j )
        o       = R_g^T sum_j softmax_j(score) s^V_j C[codeV_j]

    q: [B][H_q][d]; q_rope: [B][H_q][d_r]; k_rope: [B][H_r][cap][d_r] with
    H_r = 1 (one positional key per token shared by every head, as in
    latent attention) or H_r = H_kv; other arguments as for decode_fused.
    scale defaults to 1/sqrt(d + d_r).  Returns [B][H_q][d] fp64."""
    q = np.asarray(q, dtype=np.float64)
    qr = np.asarray(q_rope, dtype=np.float64)
    kr = np.asarray(k_rope, dtype=np.float64)
    bsz, hq, d = q.shape
    d_r = qr.shape[-1]
    hkv = k_packed.shape[1]
    group = hq // hkv
    sc = _default_scale(d + d_r, scale)
    rots = _rot.rotation_matrices(np.asarray(quats))
    bits = _cz.bits_of(levels)
    out = np.zeros((bsz, hq, d))
    for b in range(bsz):
        n = int(seq_lens[b])
        if n == 0:
            continue
        for g in range(hkv):
            heads = slice(g * group, (g + 1) * group)
            kt = _cz.dequantize_rotated(_cz.unpack(k_packed[b, g, :n], d, bits),
                                        k_norms[b, g, :n], levels)     # [n][d] rotated space
            qt = q[b, heads] @ rots[g].T                                # [G][d]
            pos = kr[b, g if kr.shape[1] > 1 else 0, :n]                # [n][d_r]
            scores = (qt @ kt.T + qr[b, heads] @ pos.T) * sc
            alpha = softmax(scores)
            vt = _cz.dequantize_rotated(_cz.unpack(v_packed[b, g, :n], d, bits),
                                        v_norms[b, g, :n], levels)
            out[b, heads] = (alpha @ vt) @ rots[g]
    return out
