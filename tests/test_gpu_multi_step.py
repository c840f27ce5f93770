"""GPU parity of multi-token decode on 2- and 4-bit records
(iq_decode_attention_multi with bits) and of the fused multi-token step
(iq_decode_step_multi: the T new tokens compressed and appended at
seq_lens[b], attended causally, the length advanced by T) against the
oracle: Algorithm 1 with C_b for the new records, App. A per token for the
outputs (decode_multi over the cache holding the new records)."""

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

DEV = torch.device("cuda:0")
BOOKS = {b: ocb.isoquant_codebook(128, b) for b in (2, 3, 4)}


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _oracle_cache(w, seed, cap, bits):
    """Records of `cap` positions packed by the oracle at b bits."""
    _, thr = BOOKS[bits]
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, thr)
    vp, vn, *_ = ocz.compress_kv(v, rots, thr)
    return quats, kp, kn, vp, vn


def _queries(seed, b, t, hq):
    g = np.random.default_rng([seed, 29])
    return g.standard_normal((b, t, hq, 128), dtype=np.float32)


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("n_tok", [2, 4])
@pytest.mark.parametrize("hkv,seq,cap", [
    (4, [3000], 3008),                                                # one round
    (1, [0, 1, 2, 3, 15, 16, 17, 64, 65, 560, 561, 640], 640),          # edges, T > length
    (2, [int(x) for x in np.linspace(0, 4090, 24)], 4096),              # several rounds
])
def test_multi_bits_parity_on_oracle_cache(bits, n_tok, hkv, seq, cap):
    levels, _ = BOOKS[bits]
    w = synth.Workload(96, "multibits", len(seq), 8 * hkv, hkv, cap, "f16", rotation_seed=1096)
    quats, kp, kn, vp, vn = _oracle_cache(w, 6, cap, bits)
    q = _queries(6, len(seq), n_tok, 8 * hkv)
    print(f"[multi-bits] b={bits} T={n_tok} hkv={hkv} batch={len(seq)}", flush=True)
    got = api.iq_decode_attention_multi(_dev(q), _dev(kp), _dev(kn), _dev(vp), _dev(vn),
                                        _dev(np.asarray(seq, np.int32)), _dev(quats),
                                        max_seq_len=cap, bits=bits).cpu().numpy()
    ref = oatt.decode_multi(q, kp, kn, vp, vn, seq, quats, levels)
    check_attention(got.reshape(-1, 128), ref.reshape(-1, 128), f"b{bits} T{n_tok} hkv{hkv}")
    for b, n in enumerate(seq):
        for t in range(n_tok):
            if n - n_tok + 1 + t <= 0:
                assert np.all(got[b, t] == 0)


def _step_case(bits, n_tok, hkv, seq0, cap, seed, dtype="f16"):
    """An oracle-packed cache (positions past each length poisoned with
    random codes and NaN scales), the new tokens and queries."""
    w = synth.Workload(97, "multistep", len(seq0), 8 * hkv, hkv, cap, dtype,
                       rotation_seed=1097 + bits)
    quats, kp, kn, vp, vn = _oracle_cache(w, seed, cap, bits)
    g = np.random.default_rng([seed, 31])
    for b, n in enumerate(seq0):
        n = max(n, 0)
        for arr in (kp, vp):
            arr[b, :, n:] = g.integers(0, 256, arr[b, :, n:].shape, dtype=np.uint8)
        for arr in (kn, vn):
            arr[b, :, n:] = np.nan
    kx = synth.kv_tensor(seed + 1, w, "k", n_tokens=n_tok)     # [B][H_kv][T][d]
    vx = synth.kv_tensor(seed + 1, w, "v", n_tokens=n_tok)
    q = _queries(seed, len(seq0), n_tok, 8 * hkv)
    return w, quats, kp, kn, vp, vn, kx, vx, q


def _run_step(bits, q, kx, vx, quats, kp, kn, vp, vn, seq0, max_seq_len, status=None):
    cache = {n: _dev(a) for n, a in (("kp", kp), ("kn", kn), ("vp", vp), ("vn", vn))}
    lens = _dev(np.asarray(seq0, np.int32))
    kn_new = _dev(np.ascontiguousarray(kx.transpose(0, 2, 1, 3)))   # [B][T][H_kv][d]
    vn_new = _dev(np.ascontiguousarray(vx.transpose(0, 2, 1, 3)))
    out = api.iq_decode_step_multi(_dev(q), kn_new, vn_new, cache["kp"], cache["kn"],
                                   cache["vp"], cache["vn"], lens, _dev(quats),
                                   max_seq_len=max_seq_len, status=status, bits=bits)
    torch.cuda.synchronize()
    return (out.cpu().numpy(), lens.cpu().numpy(),
            {n: t.cpu().numpy() for n, t in cache.items()})


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("n_tok,hkv,seq0,cap", [
    (2, 4, [3000], 3008),                                        # one round
    (4, 4, [28000], 28032),                                       # one round, long
    (3, 1, [0, 1, 15, 16, 17, 63, 64, 559, 560, 636], 640),       # batch / split edges
    (4, 2, [int(x) for x in np.linspace(0, 4000, 20)], 4096),    # several rounds
])
def test_multi_step_parity(bits, n_tok, hkv, seq0, cap):
    levels, thr = BOOKS[bits]
    _, quats, kp, kn, vp, vn, kx, vx, q = _step_case(bits, n_tok, hkv, seq0, cap, 8)
    print(f"[multi-step] b={bits} T={n_tok} hkv={hkv} batch={len(seq0)} cap={cap}", flush=True)
    got, lens, cache = _run_step(bits, q, kx, vx, quats, kp, kn, vp, vn, seq0, cap)
    assert np.array_equal(lens, np.asarray(seq0) + n_tok)
    # the new records: Algorithm 1 on the new tokens, at seq0 .. seq0 + T - 1
    rots = orot.rotation_matrices(quats)
    ref_cache = {"kp": kp.copy(), "kn": kn.copy(), "vp": vp.copy(), "vn": vn.copy()}
    for name, x in (("k", kx), ("v", vx)):
        packed, norms, codes, y, s64 = ocz.compress_kv(x, rots, thr)
        for b, n in enumerate(seq0):
            gp = cache[name + "p"][b:b + 1, :, n:n + n_tok]
            check_codes(gp, codes[b:b + 1], y[b:b + 1], thr, f"{name} b{bits} seq {b}")
            check_norms(cache[name + "n"][b:b + 1, :, n:n + n_tok], s64[b:b + 1], f"{name}")
            ref_cache[name + "p"][b, :, n:n + n_tok] = packed[b]
            ref_cache[name + "n"][b, :, n:n + n_tok] = norms[b]
        # every other position untouched
        for b, n in enumerate(seq0):
            assert np.array_equal(cache[name + "p"][b, :, :n], ref_cache[name + "p"][b, :, :n])
            assert np.array_equal(cache[name + "p"][b, :, n + n_tok:],
                                  ref_cache[name + "p"][b, :, n + n_tok:])
    ref = oatt.decode_multi(q, ref_cache["kp"], ref_cache["kn"], ref_cache["vp"],
                            ref_cache["vn"], list(np.asarray(seq0) + n_tok), quats, levels)
    check_attention(got.reshape(-1, 128), ref.reshape(-1, 128), f"step b{bits} T{n_tok}")


def test_multi_step_capacity_and_max_seq_len():
    """Sequences whose T records do not fit: nothing written, the length
    kept, the capacity flag raised, and every token attends the cached
    positions only.  max_seq_len below the new positions: those are written
    but not attended."""
    bits, n_tok, hkv, cap = 3, 3, 2, 640
    levels, thr = BOOKS[bits]
    seq0 = [638, 637, 500, 0]      # 638: does not fit; 637: fits exactly
    _, quats, kp, kn, vp, vn, kx, vx, q = _step_case(bits, n_tok, hkv, seq0, cap, 9)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    got, lens, cache = _run_step(bits, q, kx, vx, quats, kp, kn, vp, vn, seq0, cap,
                                 status=status)
    assert status.item() == 5, status.item()      # IQ_ERR_CAPACITY
    assert list(lens) == [638, 640, 503, 3]
    assert np.array_equal(cache["kp"][0], kp[0]) and np.array_equal(cache["vp"][0], vp[0])
    rots = orot.rotation_matrices(quats)
    kpk, knk, *_ = ocz.compress_kv(kx, rots, thr)
    vpk, vnk, *_ = ocz.compress_kv(vx, rots, thr)
    ref_cache = {"kp": kp.copy(), "kn": kn.copy(), "vp": vp.copy(), "vn": vn.copy()}
    for b in range(1, 4):
        n = seq0[b]
        ref_cache["kp"][b, :, n:n + n_tok] = kpk[b]
        ref_cache["kn"][b, :, n:n + n_tok] = knk[b]
        ref_cache["vp"][b, :, n:n + n_tok] = vpk[b]
        ref_cache["vn"][b, :, n:n + n_tok] = vnk[b]
    for t in range(n_tok):
        lens_t = [638] + [seq0[b] + 1 + t for b in range(1, 4)]
        ref = oatt.decode_fused(q[:, t], ref_cache["kp"], ref_cache["kn"], ref_cache["vp"],
                                ref_cache["vn"], lens_t, quats, levels)
        check_attention(got[:, t], ref, f"capacity token {t}")

    # max_seq_len 502: the sequence of 500 cached positions attends its new
    # positions 0 and 1 only, the one of 510 none of them
    seq0 = [500, 510]
    _, quats, kp, kn, vp, vn, kx, vx, q = _step_case(bits, n_tok, hkv, seq0, cap, 10)
    got, lens, _ = _run_step(bits, q, kx, vx, quats, kp, kn, vp, vn, seq0, 502)
    assert list(lens) == [503, 513]
    rots = orot.rotation_matrices(quats)
    kpk, knk, *_ = ocz.compress_kv(kx, rots, thr)
    vpk, vnk, *_ = ocz.compress_kv(vx, rots, thr)
    ref_cache = {"kp": kp.copy(), "kn": kn.copy(), "vp": vp.copy(), "vn": vn.copy()}
    for b, n in enumerate(seq0):
        ref_cache["kp"][b, :, n:n + n_tok] = kpk[b]
        ref_cache["kn"][b, :, n:n + n_tok] = knk[b]
        ref_cache["vp"][b, :, n:n + n_tok] = vpk[b]
        ref_cache["vn"][b, :, n:n + n_tok] = vnk[b]
    for t in range(n_tok):
        lens_t = [min(n + 1 + t, 502) for n in seq0]
        ref = oatt.decode_fused(q[:, t], ref_cache["kp"], ref_cache["kn"], ref_cache["vp"],
                                ref_cache["vn"], lens_t, quats, levels)
        check_attention(got[:, t], ref, f"max_seq_len token {t}")


def test_multi_step_equals_compress_then_multi_decode():
    """The fused step against iq_compress_kv_bits of the new tokens at the
    length followed by iq_decode_attention_multi on the advanced lengths:
    identical records, outputs within the attention bar of each other."""
    bits, n_tok, hkv, cap = 4, 2, 4, 2048
    seq0 = [1500]
    _, quats, kp, kn, vp, vn, kx, vx, q = _step_case(bits, n_tok, hkv, seq0, cap, 11)
    got, lens, cache = _run_step(bits, q, kx, vx, quats, kp, kn, vp, vn, seq0, cap)
    c2 = {n: _dev(a) for n, a in (("kp", kp), ("kn", kn), ("vp", vp), ("vn", vn))}
    api.iq_compress_kv_bits(_dev(kx), _dev(vx), _dev(quats), c2["kp"], c2["kn"], c2["vp"],
                            c2["vn"], dst_offset=seq0[0], bits=bits)
    out2 = api.iq_decode_attention_multi(_dev(q), c2["kp"], c2["kn"], c2["vp"], c2["vn"],
                                         _dev(np.asarray(lens, np.int32)), _dev(quats),
                                         max_seq_len=cap, bits=bits).cpu().numpy()
    for n in ("kp", "kn", "vp", "vn"):
        a, b = cache[n][0, :, :1502], c2[n].cpu().numpy()[0, :, :1502]
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), n
    check_attention(got.reshape(-1, 128), out2.reshape(-1, 128), "fused vs separate")
