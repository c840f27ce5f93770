"""Paged cache (page pools + per-sequence page tables): decode, fused step and
bulk compression on the pools against the contiguous entry points on the
same records (bit-identical: the same kernels, placed through the page
table), and decode against the oracle.  Unmapped table entries (-1) past a
sequence's length are read only speculatively (one-round grids) and fall
back to page 0, inside the pools."""

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


def _tables(lens, page, max_pages, n_pages, seed):
    """Random physical pages for the logical pages each sequence uses
    (ceil(len / page) + 1 for the step's new token), -1 elsewhere."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(n_pages)
    t = np.full((len(lens), max_pages), -1, np.int32)
    k = 0
    for b, n in enumerate(lens):
        need = min(max_pages, n // page + 1)
        t[b, :need] = perm[k:k + need]
        k += need
    assert k <= n_pages
    return t


def _scatter(cache, tables, page, n_pages):
    """Pools holding the contiguous cache's records at the mapped pages."""
    b, hkv, cap, _ = cache["k_codes"].shape
    pool = api.alloc_paged_cache(n_pages, hkv, page, DEV)
    for s in range(b):
        for j in range(tables.shape[1]):
            p = int(tables[s, j])
            if p < 0 or j * page >= cap:
                continue
            for side in ("k", "v"):
                pool[f"{side}_codes"][p] = cache[f"{side}_codes"][s, :, j * page:(j + 1) * page]
                pool[f"{side}_norms"][p] = cache[f"{side}_norms"][s, :, j * page:(j + 1) * page]
    return pool


def _filled(w, lens, cap, seed):
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(DEV)
    k = torch.from_numpy(synth.kv_tensor(seed, w, "k", n_tokens=cap)).to(DEV)
    v = torch.from_numpy(synth.kv_tensor(seed, w, "v", n_tokens=cap)).to(DEV)
    cache = api.alloc_cache(w.batch, w.n_kv_heads, cap, DEV)
    api.iq_compress_kv(k, v, quats, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                       cache["v_norms"])
    cache["seq_lens"].copy_(torch.tensor(lens, dtype=torch.int32))
    return cache, quats, k, v


@pytest.mark.parametrize("lens,hkv,page,cap", [
    ([4000], 4, 256, 4096),                                      # one-round grid
    ([0, 17, 255, 256, 257, 1000, 2047, 4095], 4, 64, 4096),     # edges, one round
    ([int(x) for x in np.linspace(1, 2040, 48)], 2, 128, 2048),  # several rounds
])
def test_paged_decode_equals_contiguous(lens, hkv, page, cap):
    w = synth.Workload(97, "paged", len(lens), 8 * hkv, hkv, cap, "f16", rotation_seed=1097)
    cache, quats, _, _ = _filled(w, lens, cap, 6)
    max_pages = cap // page
    n_pages = len(lens) * max_pages + 3
    tables = _tables(lens, page, max_pages, n_pages, 1)
    pool = _scatter(cache, tables, page, n_pages)
    bt = torch.from_numpy(tables).to(DEV)
    q = torch.from_numpy(synth.queries(6, w)[0]).to(DEV)
    ref = api.iq_decode_attention(q, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                                  cache["v_norms"], cache["seq_lens"], quats, max_seq_len=cap)
    got = api.iq_decode_attention_paged(q, pool, bt, cache["seq_lens"], quats, max_seq_len=cap)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)


def test_paged_decode_matches_oracle():
    lens, hkv, page, cap = [3000, 1], 4, 128, 3072
    w = synth.Workload(98, "paged_o", len(lens), 32, hkv, cap, "f16", rotation_seed=1098)
    cache, quats, k, v = _filled(w, lens, cap, 7)
    tables = _tables(lens, page, cap // page, 2 * (cap // page), 2)
    pool = _scatter(cache, tables, page, 2 * (cap // page))
    q = synth.queries(7, w)[0]
    got = api.iq_decode_attention_paged(torch.from_numpy(q).to(DEV), pool,
                                        torch.from_numpy(tables).to(DEV), cache["seq_lens"],
                                        quats, max_seq_len=cap)
    torch.cuda.synchronize()
    oq = orot.make_quaternions(w.rotation_seed, hkv)
    rots = orot.rotation_matrices(oq)
    kp, kn, *_ = ocz.compress_kv(k.cpu().numpy(), rots, THR)
    vp, vn, *_ = ocz.compress_kv(v.cpu().numpy(), rots, THR)
    ref = oatt.decode_fused(q, kp, kn, vp, vn, lens, oq, LEVELS)
    check_attention(got.cpu().numpy(), ref, "paged decode")


@pytest.mark.parametrize("lens,hkv,page,cap", [
    ([4000], 4, 256, 4096),
    ([0, 63, 64, 65, 511, 1023], 2, 64, 1024),
    ([int(x) for x in np.linspace(0, 2046, 40)], 4, 128, 2048),  # several rounds
])
def test_paged_step_equals_contiguous(lens, hkv, page, cap):
    """Fused step on the pools and on the contiguous cache: identical outputs
    and lengths, and the new records land in the mapped page slot."""
    w = synth.Workload(99, "paged_s", len(lens), 8 * hkv, hkv, cap, "f16", rotation_seed=1099)
    cache, quats, _, _ = _filled(w, lens, cap, 8)
    max_pages = cap // page
    n_pages = len(lens) * max_pages + 1
    tables = _tables(lens, page, max_pages, n_pages, 3)
    pool = _scatter(cache, tables, page, n_pages)
    bt = torch.from_numpy(tables).to(DEV)
    seq_p = cache["seq_lens"].clone()
    kn_new, vn_new = synth.appended_tokens(8, w, 1)
    k_new, v_new = torch.from_numpy(kn_new[0]).to(DEV), torch.from_numpy(vn_new[0]).to(DEV)
    q = torch.from_numpy(synth.queries(8, w)[0]).to(DEV)
    ref = api.iq_decode_step(q, k_new, v_new, cache["k_codes"], cache["k_norms"],
                             cache["v_codes"], cache["v_norms"], cache["seq_lens"], quats,
                             max_seq_len=cap)
    got = api.iq_decode_step_paged(q, k_new, v_new, pool, bt, seq_p, quats, max_seq_len=cap)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    assert torch.equal(seq_p, cache["seq_lens"])
    for s, n in enumerate(lens):
        if n >= cap:
            continue
        p, slot = int(tables[s, n // page]), n % page
        for side in ("k", "v"):
            assert torch.equal(pool[f"{side}_codes"][p, :, slot], cache[f"{side}_codes"][s, :, n])
            assert torch.equal(pool[f"{side}_norms"][p, :, slot], cache[f"{side}_norms"][s, :, n])


@pytest.mark.parametrize("lens,hkv,page,cap", [
    ([128, 100], 2, 64, 256),                                    # one-round grid
    ([128] + [int(x) for x in np.linspace(0, 1000, 39)], 4, 64, 1024),  # several rounds
])
def test_paged_step_unmapped_append_slot(lens, hkv, page, cap):
    """A fused step whose new position lies on an unmapped page (sequence 0,
    length on a page boundary, that page's entry -1): nothing is written to
    the pools, the token is not attended, the length stays and the capacity
    flag is raised; the other sequences step as usual."""
    w = synth.Workload(98, "paged_u", len(lens), 8 * hkv, hkv, cap, "f16", rotation_seed=1098)
    cache, quats, _, _ = _filled(w, lens, cap, 12)
    max_pages = cap // page
    n_pages = len(lens) * max_pages + 1
    tables = _tables(lens, page, max_pages, n_pages, 5)
    assert lens[0] % page == 0
    tables[0, lens[0] // page] = -1
    pool = _scatter(cache, tables, page, n_pages)
    before = {k: t.clone() for k, t in pool.items()}
    bt = torch.from_numpy(tables).to(DEV)
    seq_p = cache["seq_lens"].clone()
    kn_new, vn_new = synth.appended_tokens(12, w, 1)
    k_new, v_new = torch.from_numpy(kn_new[0]).to(DEV), torch.from_numpy(vn_new[0]).to(DEV)
    q = torch.from_numpy(synth.queries(12, w)[0]).to(DEV)
    # reference: sequence 0 attends its cache as it is, the others step
    ref0 = api.iq_decode_attention(q, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                                   cache["v_norms"], cache["seq_lens"], quats, max_seq_len=cap)
    ref = api.iq_decode_step(q, k_new, v_new, cache["k_codes"], cache["k_norms"],
                             cache["v_codes"], cache["v_norms"], cache["seq_lens"], quats,
                             max_seq_len=cap)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    got = api.iq_decode_step_paged(q, k_new, v_new, pool, bt, seq_p, quats, max_seq_len=cap,
                                   status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 5
    want_lens = [lens[0]] + [n + 1 for n in lens[1:]]
    assert seq_p.cpu().numpy().tolist() == want_lens
    err0 = (got[0] - ref0[0]).abs().max() / ref0[0].abs().max()
    assert float(err0) < 1e-5, float(err0)
    assert torch.equal(got[1:], ref[1:])
    # the pools changed only at the other sequences' new slots
    touched = {(int(tables[s, n // page]), n % page) for s, n in enumerate(lens) if s > 0}
    for side in ("k", "v"):
        diff = (pool[f"{side}_norms"].view(torch.int32) !=
                before[f"{side}_norms"].view(torch.int32)).nonzero().cpu().numpy()
        assert {(int(p), int(sl)) for p, _, sl in diff} <= touched


def test_paged_compress_equals_contiguous():
    """Bulk compression into the pools writes the records the contiguous
    compression writes, at the mapped pages; unmapped pages stay untouched."""
    lens, hkv, page, cap = [1000, 300, 7], 2, 64, 1024
    w = synth.Workload(100, "paged_c", len(lens), 16, hkv, cap, "f32", rotation_seed=1100)
    quats = api.iq_make_rotation(w.rotation_seed, hkv).to(DEV)
    t, off = 700, 128
    k = torch.from_numpy(synth.kv_tensor(9, w, "k", n_tokens=t)).to(DEV)
    v = torch.from_numpy(synth.kv_tensor(9, w, "v", n_tokens=t)).to(DEV)
    cache = api.alloc_cache(len(lens), hkv, cap, DEV)
    api.iq_compress_kv(k, v, quats, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                       cache["v_norms"], dst_offset=off)
    max_pages = cap // page
    n_pages = len(lens) * max_pages + 2
    rng = np.random.default_rng(4)
    tables = rng.permutation(n_pages)[:len(lens) * max_pages].reshape(len(lens), max_pages)
    tables = tables.astype(np.int32)
    pool = api.alloc_paged_cache(n_pages, hkv, page, DEV)
    api.iq_compress_kv_paged(k, v, quats, pool, torch.from_numpy(tables).to(DEV),
                             dst_offset=off)
    torch.cuda.synchronize()
    for s in range(len(lens)):
        for j in range(max_pages):
            p = int(tables[s, j])
            for side in ("k", "v"):
                assert torch.equal(pool[f"{side}_codes"][p],
                                   cache[f"{side}_codes"][s, :, j * page:(j + 1) * page])
                assert torch.equal(pool[f"{side}_norms"][p],
                                   cache[f"{side}_norms"][s, :, j * page:(j + 1) * page])
    unused = sorted(set(range(n_pages)) - set(tables.ravel().tolist()))
    for p in unused:
        assert int(pool["k_codes"][p].abs().sum()) == 0


@pytest.mark.parametrize("n_tok,lens,hkv,page,cap", [
    (3, [4000], 4, 256, 4096),                                        # one round
    (4, [int(x) for x in np.linspace(0, 2040, 40)], 2, 64, 2048),     # several rounds
])
def test_paged_multi_equals_contiguous(n_tok, lens, hkv, page, cap):
    """Multi-token decode on the pools equals it on the contiguous cache."""
    w = synth.Workload(87, "paged_mt", len(lens), 8 * hkv, hkv, cap, "f16", rotation_seed=1087)
    cache, quats, _, _ = _filled(w, lens, cap, 12)
    max_pages = cap // page
    n_pages = len(lens) * max_pages + 2
    tables = _tables(lens, page, max_pages, n_pages, 6)
    pool = _scatter(cache, tables, page, n_pages)
    g = np.random.default_rng(13)
    q = torch.from_numpy(g.standard_normal((len(lens), n_tok, 8 * hkv, 128),
                                           dtype=np.float32)).to(DEV)
    ref = api.iq_decode_attention_multi(q, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                                        cache["v_norms"], cache["seq_lens"], quats,
                                        max_seq_len=cap)
    got = api.iq_decode_attention_multi_paged(q, pool, torch.from_numpy(tables).to(DEV),
                                              cache["seq_lens"], quats, max_seq_len=cap)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
