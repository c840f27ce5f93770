"""GPU checks at the largest sizes the matrix-core path accepts: a cache row
of the most positions whose byte offsets fit in 32 bits (44,739,232
positions of 48-byte records; 33,554,416 of 64-byte 4-bit records), one KV
head and its 8 query heads, about 4.6 GB per cache.  Only the last 16
positions hold records (compressed at the end of the row); every other
record is all-zero with scale 0, so its score is exactly 0 and its value
contributes nothing.  The exact output then has a closed form in terms of
the oracle's scores and values of the 16 records:
    o_h = R^T sum_j e^(s_hj - m) v_j / (sum_j e^(s_hj - m) + (L - 16) e^(-m)),
m = max(0, max_j s_hj).  Heads 0-3 use small queries (the zero positions
dominate the softmax), heads 4-7 large ones (the records dominate)."""

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

DEV = torch.device("cuda:0")


def _expected(q, kp, kn, vp, vn, rot, levels, total):
    bits = ocz.bits_of(levels)
    scores = oatt.fused_scores(q, kp, kn, rot, levels)             # [8][16]
    vt = ocz.dequantize_rotated(ocz.unpack(vp, 128, bits), vn, levels)
    m = np.maximum(scores.max(axis=1, keepdims=True), 0.0)
    e = np.exp(scores - m)
    den = e.sum(axis=1, keepdims=True) + (total - scores.shape[1]) * np.exp(-m)
    return ((e @ vt) / den) @ rot


@pytest.mark.parametrize("bits", [3, 4])
def test_decode_at_largest_row(bits):
    levels, thr = ocb.isoquant_codebook(128, bits)
    rb = 16 * bits
    cap = ((2 ** 31 - 1) // rb) // 16 * 16
    assert cap * rb < 2 ** 31 and (cap + 16) * rb >= 2 ** 31
    w = synth.Workload(89, "limits", 1, 8, 1, 16, "f16", rotation_seed=1089)
    k = synth.kv_tensor(9, w, "k", n_tokens=16)
    v = synth.kv_tensor(9, w, "v", n_tokens=16)
    quats = api.iq_make_rotation(w.rotation_seed, 1).to(DEV)
    print(f"[limits] b={bits} capacity={cap} ({2 * cap * (rb + 4) / 2**30:.2f} GiB)", flush=True)
    cache = api.alloc_cache(1, 1, cap, DEV, bits=bits)
    api.iq_compress_kv_bits(torch.from_numpy(k).to(DEV), torch.from_numpy(v).to(DEV), quats,
                            cache["k_codes"], cache["k_norms"], cache["v_codes"],
                            cache["v_norms"], dst_offset=cap - 16, bits=bits)
    cache["seq_lens"].fill_(cap)
    g = np.random.default_rng(10)
    q = g.standard_normal((1, 8, 128)).astype(np.float32)
    q[0, 4:] *= 400.0
    got = api.iq_decode_attention_bits(torch.from_numpy(q).to(DEV), cache["k_codes"],
                                       cache["k_norms"], cache["v_codes"], cache["v_norms"],
                                       cache["seq_lens"], quats, bits=bits).cpu().numpy()
    # the records the GPU wrote at the end of the row, against the oracle's
    rot = orot.rotation_matrices(orot.make_quaternions(w.rotation_seed, 1))[0]
    kp, kn, kc, *_ = ocz.compress(k[0, 0], rot, thr)
    vp, vn, *_ = ocz.compress(v[0, 0], rot, thr)
    gk = cache["k_codes"][0, 0, cap - 16:].cpu().numpy()
    assert np.count_nonzero(ocz.unpack(gk, 128, bits) != kc) <= 1
    ref = _expected(q[0], kp, kn, vp, vn, rot, levels, cap)
    check_attention(got[0], ref, f"largest row b{bits}")
    del cache
    torch.cuda.empty_cache()
