"""Pins for the oracle's decode with the content / RoPE sub-block split
(Sec. 5 "MLA/RoPE hard blocker", Sec. 6): the positional part of each key
is neither rotated nor quantized, the content part is compressed."""

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import codebook as ocb
from oracle import compress as ocz
from oracle import rotation as orot

LEVELS, THR = ocb.isoquant_codebook(128, 3)
D, DR = 128, 64


def _case(seed, bsz, hq, hkv, n, shared=True):
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((bsz, hkv, n, D)) * rng.lognormal(0, 0.5, D)
    v = rng.standard_normal((bsz, hkv, n, D))
    quats = orot.make_quaternions(seed + 3, hkv)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    kr = rng.standard_normal((bsz, 1 if shared else hkv, n, DR))
    q = rng.standard_normal((bsz, hq, D))
    qr = rng.standard_normal((bsz, hq, DR))
    return q, qr, kp, kn, kr, vp, vn, quats, rots


def test_equals_loop_form_over_reconstructed_keys():
    """Against a plain loop: key j = [s R^T C[code] ; k_rope_j] (the content
    part reconstructed, the positional part as stored), value j = s R^T
    C[code], query [q ; q_rope], softmax of the scaled dot products."""
    bsz, hq, hkv, n = 2, 4, 2, 9
    q, qr, kp, kn, kr, vp, vn, quats, rots = _case(1, bsz, hq, hkv, n, shared=False)
    lens = [9, 5]
    got = oatt.decode_fused_rope(q, qr, kp, kn, kr, vp, vn, lens, quats, LEVELS)
    sc = 1.0 / np.sqrt(D + DR)
    for b in range(bsz):
        for h in range(hq):
            g = h // (hq // hkv)
            s = []
            vals = []
            for j in range(lens[b]):
                kc = ocz.reconstruct(ocz.unpack(kp[b, g, j]), kn[b, g, j], LEVELS, rots[g])
                key = np.concatenate([kc, kr[b, g, j]])
                s.append(np.dot(np.concatenate([q[b, h], qr[b, h]]), key) * sc)
                vals.append(ocz.reconstruct(ocz.unpack(vp[b, g, j]), vn[b, g, j], LEVELS,
                                            rots[g]))
            s = np.array(s)
            w = np.exp(s - s.max())
            want = (w / w.sum()) @ np.array(vals)
            np.testing.assert_allclose(got[b, h], want, rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("which", ["q_rope", "k_rope"])
def test_zero_positional_part_is_plain_decode(which):
    """With a zero positional query or key the scores are the content scores
    alone: decode_fused at the same scale 1/sqrt(d + d_r)."""
    q, qr, kp, kn, kr, vp, vn, quats, _ = _case(2, 1, 8, 1, 40)
    if which == "q_rope":
        qr = np.zeros_like(qr)
    else:
        kr = np.zeros_like(kr)
    got = oatt.decode_fused_rope(q, qr, kp, kn, kr, vp, vn, [40], quats, LEVELS)
    want = oatt.decode_fused(q, kp, kn, vp, vn, [40], quats, LEVELS, scale=1 / np.sqrt(D + DR))
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_positional_scores_alone():
    """A zero content query: the weights are the softmax of the positional
    dot products only (brute force), the output their weighted values."""
    q, qr, kp, kn, kr, vp, vn, quats, rots = _case(3, 1, 2, 1, 30)
    q = np.zeros_like(q)
    got = oatt.decode_fused_rope(q, qr, kp, kn, kr, vp, vn, [30], quats, LEVELS, scale=0.3)
    vals = ocz.reconstruct(ocz.unpack(vp[0, 0, :30]), vn[0, 0, :30], LEVELS, rots[0])
    for h in range(2):
        s = np.array([0.3 * sum(qr[0, h, i] * kr[0, 0, j, i] for i in range(DR))
                      for j in range(30)])
        w = np.exp(s - s.max())
        np.testing.assert_allclose(got[0, h], (w / w.sum()) @ vals, rtol=1e-11, atol=1e-13)


def _rotary(x, pos, base=10000.0):
    """Rotary position embedding (pairs (2i, 2i+1) rotated by pos * base^(-2i/d_r))."""
    x = np.asarray(x, dtype=np.float64)
    half = x.shape[-1] // 2
    theta = pos * base ** (-np.arange(half) * 2.0 / x.shape[-1])
    c, s = np.cos(theta), np.sin(theta)
    out = x.copy()
    out[..., 0::2] = x[..., 0::2] * c - x[..., 1::2] * s
    out[..., 1::2] = x[..., 0::2] * s + x[..., 1::2] * c
    return out


def test_positional_part_keeps_relative_position():
    """Why the split is needed: keys and query carrying rotary phases of
    positions j and m score by m - j only; kept exact, shifting every
    position by the same offset leaves the output unchanged."""
    q, qr, kp, kn, kr, vp, vn, quats, _ = _case(4, 1, 8, 1, 50)
    raw_k = np.random.default_rng(5).standard_normal((50, DR))
    raw_q = np.random.default_rng(6).standard_normal((8, DR))
    outs = []
    for shift in (0, 1000):
        krot = np.stack([_rotary(raw_k[j], j + shift) for j in range(50)])[None, None]
        qrot = _rotary(raw_q, 50 + shift)[None]
        outs.append(oatt.decode_fused_rope(q, qrot, kp, kn, krot, vp, vn, [50], quats, LEVELS))
    np.testing.assert_allclose(outs[0], outs[1], rtol=1e-9, atol=1e-12)


def test_shared_positional_key_equals_per_head_copies():
    q, qr, kp, kn, kr, vp, vn, quats, _ = _case(7, 2, 8, 4, 20, shared=True)
    per = np.repeat(kr, 4, axis=1)
    a = oatt.decode_fused_rope(q, qr, kp, kn, kr, vp, vn, [20, 11], quats, LEVELS)
    b = oatt.decode_fused_rope(q, qr, kp, kn, per, vp, vn, [20, 11], quats, LEVELS)
    np.testing.assert_array_equal(a, b)
