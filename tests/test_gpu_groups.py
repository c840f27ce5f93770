"""GPU parity of the matrix-core decode path at group sizes other than 8
(query heads per KV head 1 .. 16, served in head groups of 8 with unused
rows left empty): decode attention, the fused step and the paged and 2/4-bit
variants against the oracle's compressed-space attention (App. A) on
oracle-packed caches, capacities multiples of 16."""

import numpy as np
import pytest
import torch

from oracle import attention as oatt
from oracle import codebook as ocb
from oracle import compress as ocz
from oracle import rotation as orot
from paper_2608_08081_amd import api, synth
from tests.parity import check_attention, check_codes, check_norms

pytestmark = pytest.mark.gpu

LEVELS, THR = ocb.isoquant_codebook(128, 3)
DEV = torch.device("cuda:0")


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _oracle_cache(w, seed, cap, bits=3):
    thr = ocb.isoquant_codebook(128, bits)[1]
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, kc, ky, ks = ocz.compress_kv(k, rots, thr)
    vp, vn, vc, vy, vs = ocz.compress_kv(v, rots, thr)
    return k, v, quats, dict(kp=kp, kn=kn, kc=kc, ky=ky, ks=ks, vp=vp, vn=vn, vc=vc, vy=vy,
                             vs=vs)


@pytest.mark.parametrize("hq,hkv,seq", [
    (1, 1, [1024]),                         # the single-head workload's shape
    (2, 2, [15, 16, 17, 640]),
    (4, 2, [1, 63, 64, 65, 0, 1000]),
    (6, 2, [300, 511]),
    (12, 1, [999]),                         # two head groups, the second of 4 heads
    (16, 2, [2000, 129, 0]),                # two full head groups
    (16, 1, [4096]),
    (32, 8, [int(x) for x in np.linspace(0, 3000, 40)]),  # group 4, several rounds
])
def test_decode_any_group_matches_oracle(hq, hkv, seq):
    cap = (max(max(seq), 1) + 15) // 16 * 16
    w = synth.Workload(97, "groups", len(seq), hq, hkv, cap, "f16", rotation_seed=300 + hq)
    _, _, quats, o = _oracle_cache(w, 7, cap)
    q = synth.queries(7, w)[0]
    print(f"[groups] decode hq={hq} hkv={hkv} n={len(seq)} cap={cap}", flush=True)
    out = api.iq_decode_attention(_dev(q), _dev(o["kp"]), _dev(o["kn"]), _dev(o["vp"]),
                                  _dev(o["vn"]), _dev(np.asarray(seq, np.int32)), _dev(quats),
                                  max_seq_len=cap)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = oatt.decode_fused(q, o["kp"], o["kn"], o["vp"], o["vn"], seq, quats, LEVELS)
    check_attention(got, ref, f"group {hq // hkv}")
    for b, n in enumerate(seq):
        if n == 0:
            assert np.all(got[b] == 0)


@pytest.mark.parametrize("hq,hkv,seq0,cap", [
    (1, 1, [1023], 1024),
    (4, 2, [0, 17, 500, 1007], 1024),
    (16, 2, [3000, 64], 3008),
    (12, 3, [int(x) for x in np.linspace(1, 990, 30)], 1008),   # several rounds
])
def test_step_any_group_matches_oracle(hq, hkv, seq0, cap):
    """Fused step: the new records written once per KV head (by its first
    head group), every query head attending them; poisoned tails."""
    w = synth.Workload(98, "groups_s", len(seq0), hq, hkv, cap, "f16", rotation_seed=400 + hq)
    k, v, quats, o = _oracle_cache(w, 8, cap)
    rng = np.random.default_rng(8)
    gk, gv, gkn, gvn = o["kp"].copy(), o["vp"].copy(), o["kn"].copy(), o["vn"].copy()
    for i, n in enumerate(seq0):
        gk[i, :, n:] = rng.integers(0, 256, size=gk[i, :, n:].shape, dtype=np.uint8)
        gv[i, :, n:] = rng.integers(0, 256, size=gv[i, :, n:].shape, dtype=np.uint8)
        gkn[i, :, n:] = np.nan
        gvn[i, :, n:] = np.nan
    cache = dict(k_codes=_dev(gk), k_norms=_dev(gkn), v_codes=_dev(gv), v_norms=_dev(gvn),
                 seq_lens=_dev(np.asarray(seq0, np.int32)))
    k_new = np.stack([k[i, :, n] for i, n in enumerate(seq0)])
    v_new = np.stack([v[i, :, n] for i, n in enumerate(seq0)])
    q = synth.queries(8, w)[0]
    print(f"[groups] step hq={hq} hkv={hkv} n={len(seq0)} cap={cap}", flush=True)
    out = api.iq_decode_step(_dev(q), _dev(k_new), _dev(v_new), cache["k_codes"],
                             cache["k_norms"], cache["v_codes"], cache["v_norms"],
                             cache["seq_lens"], _dev(quats), max_seq_len=cap)
    torch.cuda.synchronize()
    seq1 = [n + 1 for n in seq0]
    assert cache["seq_lens"].cpu().numpy().tolist() == seq1
    for i, n in enumerate(seq0):
        for side in ("k", "v"):
            got = cache[f"{side}_codes"][i, :, n].cpu().numpy()
            check_codes(got[None, :, None], o[f"{side}c"][i:i + 1, :, n:n + 1],
                        o[f"{side}y"][i:i + 1, :, n:n + 1], THR, f"new {side}")
            check_norms(cache[f"{side}_norms"][i, :, n].cpu().numpy(), o[f"{side}s"][i, :, n],
                        "new scale")
            # the slot after the new one keeps its poison
            if n + 1 < cap:
                assert np.isnan(cache[f"{side}_norms"][i, :, n + 1].cpu().numpy()).all()
    ref = oatt.decode_fused(q, o["kp"], o["kn"], o["vp"], o["vn"], seq1, quats, LEVELS)
    check_attention(out.cpu().numpy(), ref, f"step group {hq // hkv}")


@pytest.mark.parametrize("bits", [2, 4])
def test_bits_group_4(bits):
    levels = ocb.isoquant_codebook(128, bits)[0]
    cap, seq = 768, [700, 5, 768]
    w = synth.Workload(99, "groups_b", len(seq), 8, 2, cap, "f16", rotation_seed=500)
    _, _, quats, o = _oracle_cache(w, 9, cap, bits)
    q = synth.queries(9, w)[0]
    out = api.iq_decode_attention_bits(_dev(q), _dev(o["kp"]), _dev(o["kn"]), _dev(o["vp"]),
                                       _dev(o["vn"]), _dev(np.asarray(seq, np.int32)),
                                       _dev(quats), max_seq_len=cap, bits=bits)
    torch.cuda.synchronize()
    ref = oatt.decode_fused(q, o["kp"], o["kn"], o["vp"], o["vn"], seq, quats, levels)
    check_attention(out.cpu().numpy(), ref, f"{bits}-bit group 4")


def test_paged_group_2_equals_contiguous():
    """Paged pools at group 2 give the contiguous result bit for bit."""
    cap, page, seq = 1024, 64, [1000, 130, 64]
    w = synth.Workload(100, "groups_p", len(seq), 4, 2, cap, "f16", rotation_seed=600)
    _, _, quats, o = _oracle_cache(w, 10, cap)
    max_pages = cap // page
    n_pages = len(seq) * max_pages
    perm = np.random.default_rng(3).permutation(n_pages).astype(np.int32)
    tables = perm.reshape(len(seq), max_pages)
    pool = api.alloc_paged_cache(n_pages, 2, page, DEV)
    for s in range(len(seq)):
        for j in range(max_pages):
            p = int(tables[s, j])
            for side in ("k", "v"):
                pool[f"{side}_codes"][p] = _dev(o[f"{side}p"][s, :, j * page:(j + 1) * page])
                pool[f"{side}_norms"][p] = _dev(o[f"{side}n"][s, :, j * page:(j + 1) * page])
    q = _dev(synth.queries(10, w)[0])
    lens = _dev(np.asarray(seq, np.int32))
    got = api.iq_decode_attention_paged(q, pool, _dev(tables), lens, _dev(quats),
                                        max_seq_len=cap)
    ref = api.iq_decode_attention(q, _dev(o["kp"]), _dev(o["kn"]), _dev(o["vp"]), _dev(o["vn"]),
                                  lens, _dev(quats), max_seq_len=cap)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
