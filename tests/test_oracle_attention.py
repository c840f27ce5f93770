"""Pins for the oracle's decode attention (App. A; Table 2; Sec. 5 "Inverse
rotation is mandatory"; App. F NIAH stand-in)."""

import math

import numpy as np
import pytest

from oracle import attention as att
from oracle import codebook as cb
from oracle import compress as cz
from oracle import rotation as rot
from paper_2608_08081_amd import synth

LEVELS, THR = cb.isoquant_codebook(128, 3)


def _make_cache(seed, b, hkv, t, hq, cap=None):
    g = np.random.default_rng(seed)
    cap = t if cap is None else cap
    quats = rot.make_quaternions(seed, hkv)
    rots = rot.rotation_matrices(quats)
    k = (g.standard_normal((b, hkv, cap, 128)) * g.lognormal(0, 0.5, 128)).astype(np.float32)
    v = (g.standard_normal((b, hkv, cap, 128)) * g.lognormal(0, 0.5, 128)).astype(np.float32)
    kp, kn, *_ = cz.compress_kv(k, rots, THR)
    vp, vn, *_ = cz.compress_kv(v, rots, THR)
    q = g.standard_normal((b, hq, 128)).astype(np.float32)
    return q, kp, kn, vp, vn, quats, rots, k, v


@pytest.mark.parametrize("hq,hkv", [(1, 1), (4, 2), (8, 1)])
def test_fused_equals_reconstruct(hq, hkv):
    """Orthogonality invariant q . R^T k_hat = (R q) . k_hat: the fused
    compressed-space path equals reconstruct-then-compute to 1e-12."""
    q, kp, kn, vp, vn, quats, *_ = _make_cache(1, 2, hkv, 37, hq)
    seq = np.array([37, 20])
    a = att.decode_fused(q, kp, kn, vp, vn, seq, quats, LEVELS)
    b = att.decode_reconstruct(q, kp, kn, vp, vn, seq, quats, LEVELS)
    assert np.max(np.abs(a - b)) <= 1e-12 * np.max(np.abs(b))


def test_fused_brute_force_loops():
    """Tiny case recomputed with explicit Python loops from App. A's
    formulas (no matrix library calls), so a transposed R or a wrong sign
    in the oracle's vectorized code would show."""
    q, kp, kn, vp, vn, quats, rots, *_ = _make_cache(2, 1, 1, 5, 2)
    d = 128
    r = rots[0]
    kc = cz.unpack(kp[0, 0])
    vc = cz.unpack(vp[0, 0])
    got = att.decode_fused(q, kp, kn, vp, vn, [5], quats, LEVELS)
    for h in range(2):
        qt = [sum(r[i][j] * float(q[0, h, j]) for j in range(d)) for i in range(d)]
        scores = []
        for t in range(5):
            dot = sum(qt[i] * float(LEVELS[kc[t, i]]) for i in range(d))
            scores.append(float(kn[0, 0, t]) * dot / math.sqrt(d))
        m = max(scores)
        e = [math.exp(s - m) for s in scores]
        z = sum(e)
        ot = [sum(e[t] / z * float(vn[0, 0, t]) * float(LEVELS[vc[t, i]]) for t in range(5))
              for i in range(d)]
        o = [sum(r[i][j] * ot[i] for i in range(d)) for j in range(d)]   # R^T o_tilde
        np.testing.assert_allclose(got[0, h], o, rtol=0, atol=1e-12 * max(map(abs, o)))


def test_single_token_returns_its_value():
    """T = 1: softmax weight 1, output = reconstructed v_0 = s R^T C[code]."""
    q, kp, kn, vp, vn, quats, rots, *_ = _make_cache(3, 1, 1, 1, 3, cap=4)
    out = att.decode_fused(q, kp, kn, vp, vn, [1], quats, LEVELS)
    v0 = cz.reconstruct(cz.unpack(vp[0, 0, :1]), vn[0, 0, :1], LEVELS, rots[0])[0]
    for h in range(3):
        np.testing.assert_allclose(out[0, h], v0, rtol=0, atol=1e-13 * np.max(np.abs(v0)))


def test_zero_query_averages_values_and_empty_sequence():
    q, kp, kn, vp, vn, quats, rots, *_ = _make_cache(4, 2, 1, 9, 1)
    q[:] = 0
    out = att.decode_fused(q, kp, kn, vp, vn, [9, 0], quats, LEVELS)
    v_hat = cz.reconstruct(cz.unpack(vp[0, 0]), vn[0, 0], LEVELS, rots[0])
    np.testing.assert_allclose(out[0, 0], v_hat.mean(axis=0), atol=1e-13)
    assert np.all(out[1] == 0)


def test_skipping_inverse_rotation_is_wrong():
    """Sec. 5: the aggregated output must be mapped back by R^T; leaving it
    in the rotated domain gives an unrelated vector."""
    q, kp, kn, vp, vn, quats, rots, k, v = _make_cache(5, 1, 1, 64, 2)
    seq = [64]
    good = att.decode_fused(q, kp, kn, vp, vn, seq, quats, LEVELS)
    bad = att.decode_fused(q, kp, kn, vp, vn, seq, quats, LEVELS, skip_inverse=True)
    exact = att.attention_exact(q, k, v, seq, 1)
    rel = lambda a: np.linalg.norm(a - exact) / np.linalg.norm(exact)
    assert rel(good) < 0.5
    assert rel(bad) > 0.9 and rel(bad) > 2 * rel(good)


def test_compressed_attention_error_context():
    """Context (not a target): output error of 3-bit compressed attention
    against fp64 attention on the unquantized cache, averaged over seeds, is
    clearly smaller with the isotropizing rotation than with none (the
    motivation of Sec. 3.2; the paper's quality numbers need real models)."""
    w = synth.WORKLOADS[0]
    t = 512
    quats = rot.make_quaternions(w.rotation_seed, 1)
    rots = rot.rotation_matrices(quats)
    ident = np.eye(128)[None]
    errs_rot, errs_none = [], []
    for seed in range(8):
        k = synth.kv_tensor(seed, w, "k", n_tokens=t)
        v = synth.kv_tensor(seed, w, "v", n_tokens=t)
        q = synth.queries(seed, w)[0]
        exact = att.attention_exact(q, k, v, [t], 1)
        kp, kn, *_ = cz.compress_kv(k, rots, THR)
        vp, vn, *_ = cz.compress_kv(v, rots, THR)
        out = att.decode_fused(q, kp, kn, vp, vn, [t], quats, LEVELS)
        errs_rot.append(np.linalg.norm(out - exact) / np.linalg.norm(exact))
        _, kn0, kc0, _, _ = cz.compress_kv(k, ident, THR)
        _, vn0, vc0, _, _ = cz.compress_kv(v, ident, THR)
        kh = cz.dequantize_rotated(kc0[0, 0], kn0[0, 0], LEVELS)
        vh = cz.dequantize_rotated(vc0[0, 0], vn0[0, 0], LEVELS)
        o0 = att.softmax(kh @ q[0, 0].astype(np.float64) / np.sqrt(128)) @ vh
        errs_none.append(np.linalg.norm(o0 - exact[0, 0]) / np.linalg.norm(exact))
    assert np.all(np.isfinite(errs_rot))
    assert np.mean(errs_rot) < 0.8 * np.mean(errs_none)


def test_needle_argmax_survives_compression():
    """Stand-in for the NIAH check (App. F): the planted key stays the
    softmax argmax of its query head after 3-bit compression.  Reduced
    context here; the full 32K case runs with the GPU parity tests."""
    w = synth.WORKLOADS[2]
    seed = 0
    t = 4096
    k = synth.kv_tensor(seed, w, "k", n_tokens=t)
    q = synth.queries(seed, w)[0]
    pos = synth.plant_needle(seed, w, k, q)
    quats = rot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = rot.rotation_matrices(quats)
    kp, kn, *_ = cz.compress_kv(k, rots, THR)
    for g in range(w.n_kv_heads):
        h0 = g * w.group
        s = att.fused_scores(q[0, h0:h0 + 1], kp[0, g], kn[0, g], rots[g], LEVELS)[0]
        assert int(np.argmax(s)) == int(pos[0, g])
        exact = k[0, g].astype(np.float64) @ q[0, h0].astype(np.float64)
        assert int(np.argmax(exact)) == int(pos[0, g])


def test_exact_attention_matches_library_attention():
    """The unquantized-cache attention (the fp16 baseline's reference, Fig. 1
    top after materialization) against PyTorch's CPU scaled-dot-product
    attention in fp64, grouped query heads expanded per KV head, ragged
    lengths, one empty sequence and a non-default scale."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(9)
    b, hkv, grp, cap = 3, 2, 4, 40
    k = g.standard_normal((b, hkv, cap, 128)) * 3.0
    v = g.standard_normal((b, hkv, cap, 128))
    q = g.standard_normal((b, hkv * grp, 128))
    lens = [40, 17, 0]
    for scale in (None, 0.2):
        got = att.attention_exact(q, k, v, lens, hkv, scale)
        for bb in range(b):
            n = lens[bb]
            if n == 0:
                assert np.all(got[bb] == 0)
                continue
            kt = torch.from_numpy(k[bb, :, :n]).repeat_interleave(grp, dim=0)
            vt = torch.from_numpy(v[bb, :, :n]).repeat_interleave(grp, dim=0)
            qt = torch.from_numpy(q[bb])[:, None, :]
            ref = torch.nn.functional.scaled_dot_product_attention(
                qt, kt, vt, scale=scale)[:, 0, :].numpy()
            np.testing.assert_allclose(got[bb], ref, rtol=0, atol=1e-12)


def test_decode_multi_brute_force_causal():
    """Multi-token decode recomputed in explicit loops: token t attends the
    cached positions before seq - T + 1 + t, so the last token sees every
    position and the first sees all but the T - 1 newer ones."""
    q1, kp, kn, vp, vn, quats, rots, *_ = _make_cache(4, 1, 1, 6, 2)
    g = np.random.default_rng(9)
    t_new, seq = 3, 6
    q = g.standard_normal((1, t_new, 2, 128)).astype(np.float32)
    got = att.decode_multi(q, kp, kn, vp, vn, [seq], quats, LEVELS)
    d = 128
    r = rots[0]
    kc = cz.unpack(kp[0, 0])
    vc = cz.unpack(vp[0, 0])
    for t in range(t_new):
        n = seq - t_new + 1 + t
        for h in range(2):
            qt = [sum(r[i][j] * float(q[0, t, h, j]) for j in range(d)) for i in range(d)]
            scores = [float(kn[0, 0, p]) * sum(qt[i] * float(LEVELS[kc[p, i]]) for i in range(d))
                      / math.sqrt(d) for p in range(n)]
            m = max(scores)
            e = [math.exp(s - m) for s in scores]
            z = sum(e)
            ot = [sum(e[p] / z * float(vn[0, 0, p]) * float(LEVELS[vc[p, i]]) for p in range(n))
                  for i in range(d)]
            o = [sum(r[i][j] * ot[i] for i in range(d)) for j in range(d)]
            np.testing.assert_allclose(got[0, t, h], o, rtol=0, atol=1e-12 * max(map(abs, o)))


def test_decode_multi_special_cases():
    """T = 1 is single-token decode; a token whose causal length is 0 (seq < T)
    gives a zero row; a token sees nothing past its own position (changing
    the last cached record moves only the last token's output)."""
    q, kp, kn, vp, vn, quats, *_ = _make_cache(6, 2, 2, 12, 4)
    one = att.decode_multi(q[:, None], kp, kn, vp, vn, [12, 5], quats, LEVELS)
    ref = att.decode_fused(q, kp, kn, vp, vn, [12, 5], quats, LEVELS)
    assert np.array_equal(one[:, 0], ref)
    g = np.random.default_rng(3)
    qm = g.standard_normal((2, 3, 4, 128))
    out = att.decode_multi(qm, kp, kn, vp, vn, [12, 2], quats, LEVELS)
    assert np.all(out[1, 0] == 0) and np.any(out[1, 1] != 0)
    kp2 = kp.copy()
    kp2[0, :, 11] ^= 0xFF
    out2 = att.decode_multi(qm, kp2, kn, vp, vn, [12, 2], quats, LEVELS)
    assert np.array_equal(out2[0, :2], out[0, :2]) and not np.array_equal(out2[0, 2], out[0, 2])
