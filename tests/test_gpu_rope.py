"""GPU parity of decode with the content / RoPE sub-block split
(iq_decode_attention_rope; Sec. 5 "MLA/RoPE hard blocker") against the
oracle: content keys and values compressed (Alg. 1), positional keys kept
in fp16 with rotary phases, at a DeepSeek-V2-like per-head shape (128
content dims + 64 positional dims, one positional key per token shared by
every head, one query head per KV head) and at a grouped shape with one
positional key per KV head."""

import numpy as np
import pytest
import torch

from oracle import attention as oatt
from oracle import codebook as ocb
from oracle import compress as ocz
from oracle import rotation as orot
from paper_2608_08081_amd import api, synth
from tests.parity import check_attention

pytestmark = pytest.mark.gpu

LEVELS, THR = ocb.isoquant_codebook(128, 3)
DEV = torch.device("cuda:0")
DR = 64


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _rotary(x, pos, base=10000.0):
    half = x.shape[-1] // 2
    theta = np.asarray(pos, np.float64)[..., None] * base ** (-np.arange(half) * 2.0 / x.shape[-1])
    c, s = np.cos(theta), np.sin(theta)
    out = np.empty_like(x, dtype=np.float64)
    out[..., 0::2] = x[..., 0::2] * c - x[..., 1::2] * s
    out[..., 1::2] = x[..., 0::2] * s + x[..., 1::2] * c
    return out


def _case(seed, bsz, hq, hkv, hr, cap, lens):
    w = synth.Workload(101, "rope", bsz, hq, hkv, cap, "f16", rotation_seed=700 + seed)
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap)
    quats = orot.make_quaternions(w.rotation_seed, hkv)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    rng = np.random.default_rng(seed + 50)
    raw = rng.standard_normal((bsz, hr, cap, DR)) * rng.lognormal(0.0, 0.5, DR)
    kr = _rotary(raw, np.arange(cap)).astype(np.float16)
    q = synth.queries(seed, w)[0]
    qr_raw = rng.standard_normal((bsz, hq, DR)).astype(np.float32)
    qr = np.stack([_rotary(qr_raw[b], lens[b]) for b in range(bsz)]).astype(np.float32)
    return q, qr, kp, kn, kr, vp, vn, quats


@pytest.mark.parametrize("bsz,hq,hkv,hr,cap,lens", [
    (2, 16, 16, 1, 4096, [4000, 1234]),          # DeepSeek-V2-like: group 1, shared key
    (1, 32, 4, 4, 8192, [8192]),                 # grouped, one positional key per KV head
    (1, 8, 8, 1, 1024, [0]),                     # empty sequence
    (12, 16, 2, 2, 2048, [int(x) for x in np.linspace(1, 2048, 12)]),   # several rounds
])
def test_rope_decode_matches_oracle(bsz, hq, hkv, hr, cap, lens):
    q, qr, kp, kn, kr, vp, vn, quats = _case(11, bsz, hq, hkv, hr, cap, lens)
    print(f"[rope] b={bsz} hq={hq} hkv={hkv} hr={hr} cap={cap}", flush=True)
    out = api.iq_decode_attention_rope(_dev(q), _dev(qr), _dev(kp), _dev(kn), _dev(kr),
                                       _dev(vp), _dev(vn), _dev(np.asarray(lens, np.int32)),
                                       _dev(quats), max_seq_len=cap)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = oatt.decode_fused_rope(q, qr, kp, kn, kr.astype(np.float64), vp, vn, lens, quats,
                                 LEVELS)
    check_attention(got, ref, f"rope hq{hq} hkv{hkv} hr{hr}")
    for b, n in enumerate(lens):
        if n == 0:
            assert np.all(got[b] == 0)


def test_rope_positional_part_matters_and_zero_query_part_is_plain_decode():
    """The positional scores change the output; with a zero positional
    query the result is plain decode at scale 1/sqrt(192)."""
    lens = [3000]
    q, qr, kp, kn, kr, vp, vn, quats = _case(12, 1, 16, 2, 2, 3008, lens)
    args = [_dev(kp), _dev(kn), _dev(kr), _dev(vp), _dev(vn), _dev(np.asarray(lens, np.int32)),
            _dev(quats)]
    with_r = api.iq_decode_attention_rope(_dev(q), _dev(qr), *args).cpu().numpy()
    zero_r = api.iq_decode_attention_rope(_dev(q), _dev(np.zeros_like(qr)), *args).cpu().numpy()
    plain = api.iq_decode_attention(_dev(q), _dev(kp), _dev(kn), _dev(vp), _dev(vn),
                                    _dev(np.asarray(lens, np.int32)), _dev(quats),
                                    softmax_scale=1.0 / np.sqrt(192.0)).cpu().numpy()
    torch.cuda.synchronize()
    err = np.max(np.abs(zero_r - plain)) / np.max(np.abs(plain))
    assert err < 1e-5, err
    assert np.max(np.abs(with_r - zero_r)) > 1e-2 * np.max(np.abs(zero_r))
