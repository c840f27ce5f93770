"""GPU parity of multi-token decode (iq_decode_attention_multi: T query
tokens per sequence over one packed cache, causal among the new tokens;
App. A per token) against the oracle's decode_multi, on oracle-packed caches
and end to end, for grids of one round, several rounds and one split."""

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


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _oracle_cache(w, seed, cap):
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    return quats, kp, kn, vp, vn


def _queries(seed, b, t, hq):
    g = np.random.default_rng([seed, 17])
    return g.standard_normal((b, t, hq, 128), dtype=np.float32)


@pytest.mark.parametrize("n_tok", [2, 3, 4])
@pytest.mark.parametrize("hkv,seq,cap", [
    (4, [3000], 3008),                                              # one round
    (1, [0, 1, 2, 3, 4, 15, 16, 17, 64, 65, 129, 560, 561, 640], 640),  # edges, T > length
    (2, [int(x) for x in np.linspace(0, 4090, 24)], 4096),            # several rounds
    (8, [int(x) for x in np.linspace(0, 128, 160)], 128),             # one split per (b, g)
])
def test_multi_parity_on_oracle_cache(n_tok, hkv, seq, cap):
    w = synth.Workload(93, "multi", len(seq), 8 * hkv, hkv, cap, "f16", rotation_seed=1093)
    quats, kp, kn, vp, vn = _oracle_cache(w, 3, cap)
    q = _queries(3, len(seq), n_tok, 8 * hkv)
    print(f"[multi] T={n_tok} hkv={hkv} batch={len(seq)} cap={cap}", flush=True)
    got = api.iq_decode_attention_multi(_dev(q), _dev(kp), _dev(kn), _dev(vp), _dev(vn),
                                        _dev(np.asarray(seq, np.int32)), _dev(quats),
                                        max_seq_len=cap).cpu().numpy()
    ref = oatt.decode_multi(q, kp, kn, vp, vn, seq, quats, LEVELS)
    check_attention(got.reshape(-1, 128), ref.reshape(-1, 128), f"T{n_tok} hkv{hkv}")
    for b, n in enumerate(seq):
        for t in range(n_tok):
            if n - n_tok + 1 + t <= 0:
                assert np.all(got[b, t] == 0)


def test_multi_one_token_is_single_decode():
    seq, hkv, cap = [1000, 7], 2, 1024
    w = synth.Workload(92, "multi1", len(seq), 16, hkv, cap, "f16", rotation_seed=1092)
    quats, kp, kn, vp, vn = _oracle_cache(w, 4, cap)
    q = _queries(4, len(seq), 1, 16)
    args = (_dev(kp), _dev(kn), _dev(vp), _dev(vn), _dev(np.asarray(seq, np.int32)),
            _dev(quats))
    a = api.iq_decode_attention_multi(_dev(q), *args)
    b = api.iq_decode_attention(_dev(q[:, 0]), *args)
    torch.cuda.synchronize()
    assert torch.equal(a[:, 0], b)


def test_multi_full_size_32k():
    """The 32K shape with 4 tokens (batch 1, 32 query heads, 4 KV heads),
    every output against the oracle."""
    w = synth.WORKLOADS[2]
    cap = 32768
    quats, kp, kn, vp, vn = _oracle_cache(w, 5, cap)
    q = _queries(5, 1, 4, 32)
    got = api.iq_decode_attention_multi(_dev(q), _dev(kp), _dev(kn), _dev(vp), _dev(vn),
                                        _dev(np.asarray([cap], np.int32)), _dev(quats),
                                        max_seq_len=cap).cpu().numpy()
    ref = oatt.decode_multi(q, kp, kn, vp, vn, [cap], quats, LEVELS)
    check_attention(got.reshape(-1, 128), ref.reshape(-1, 128), "32K T4")


def test_multi_end_to_end_and_determinism():
    """GPU-compressed cache holding the new tokens, multi-token decode against
    the oracle; two calls give identical outputs."""
    seq, hkv, cap, n_tok = [2000, 513, 3], 2, 2048, 3
    w = synth.Workload(91, "multi_e2e", len(seq), 16, hkv, cap, "f16", rotation_seed=1091)
    k = synth.kv_tensor(6, w, "k")
    v = synth.kv_tensor(6, w, "v")
    quats = api.iq_make_rotation(w.rotation_seed, hkv).to(DEV)
    cache = api.alloc_cache(len(seq), hkv, cap, DEV)
    api.iq_compress_kv(_dev(k), _dev(v), quats, cache["k_codes"], cache["k_norms"],
                       cache["v_codes"], cache["v_norms"])
    cache["seq_lens"].copy_(torch.tensor(seq, dtype=torch.int32))
    q = _dev(_queries(6, len(seq), n_tok, 16))
    args = (cache["k_codes"], cache["k_norms"], cache["v_codes"], cache["v_norms"],
            cache["seq_lens"], quats)
    o1 = api.iq_decode_attention_multi(q, *args)
    o2 = api.iq_decode_attention_multi(q, *args)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    rots = orot.rotation_matrices(orot.make_quaternions(w.rotation_seed, hkv))
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    ref = oatt.decode_multi(q.cpu().numpy(), kp, kn, vp, vn, seq,
                            orot.make_quaternions(w.rotation_seed, hkv), LEVELS)
    check_attention(o1.cpu().numpy().reshape(-1, 128), ref.reshape(-1, 128), "e2e T3")
