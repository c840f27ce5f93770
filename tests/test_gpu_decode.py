"""GPU parity of iq_decode_attention against the oracle's compressed-space
decode (App. A), through the C ABI via the PyTorch binding."""

import numpy as np
import pytest
import torch

from oracle import attention as oatt
from oracle import codebook as ocb
from oracle import compress as ocz
from oracle import rotation as orot
from paper_2608_08081_amd import api, synth
from tests.parity import check_attention, check_codes

pytestmark = pytest.mark.gpu

LEVELS, THR = ocb.isoquant_codebook(128, 3)
DEV = torch.device("cuda:0")


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _oracle_cache(w, seed, t, batch, cap):
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap, batch=batch)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap, batch=batch)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    return k, v, quats, kp, kn, vp, vn


def _gpu_decode(q, kp, kn, vp, vn, seq, quats, max_seq_len, scale=0.0, ws=None):
    out = api.iq_decode_attention(_dev(q), _dev(kp), _dev(kn), _dev(vp), _dev(vn),
                                  _dev(np.asarray(seq, np.int32)), _dev(quats),
                                  max_seq_len=max_seq_len, softmax_scale=scale, workspace=ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("hq,hkv,seq", [
    (1, 1, [1024]),
    (8, 1, [1, 63, 64, 65]),
    (32, 4, [777, 0, 513]),
    (16, 2, [2, 1000]),
    (6, 2, [300]),
    (2, 2, [129]),
])
def test_decode_parity_on_oracle_cache(hq, hkv, seq):
    """Decode over caches packed by the oracle (identical packed input on both
    sides); ragged lengths, an empty sequence, several group sizes."""
    w = synth.Workload(9, "test", len(seq), hq, hkv, max(seq), "f16", rotation_seed=77)
    cap = max(max(seq), 1) + 3
    k, v, quats, kp, kn, vp, vn = _oracle_cache(w, 1, max(seq), len(seq), cap)
    q = synth.queries(1, w)[0]
    got = _gpu_decode(q, kp, kn, vp, vn, seq, quats, cap)
    ref = oatt.decode_fused(q, kp, kn, vp, vn, seq, quats, LEVELS)
    check_attention(got, ref, f"hq{hq} hkv{hkv}")
    for b, n in enumerate(seq):
        if n == 0:
            assert np.all(got[b] == 0)


@pytest.mark.parametrize("hkv,ctx", [(1, 32768), (2, 20000)])
def test_many_splits_per_row(hkv, ctx):
    """One sequence over one or two KV heads: the planner fills the chip with
    short splits (229 of 144 positions at 32K over one KV head), so each row
    has more than 64 partials, which the merge reads in one wide pass."""
    from tests.test_gpu_bench_shapes import g8_instance

    assert g8_instance(1, hkv, ctx, append=False)[1] > 64
    w = synth.Workload(9, "many splits", 1, 8 * hkv, hkv, ctx, "f16", rotation_seed=91)
    k, v, quats, kp, kn, vp, vn = _oracle_cache(w, 3, ctx, 1, ctx)
    q = synth.queries(3, w)[0]
    got = _gpu_decode(q, kp, kn, vp, vn, [ctx], quats, ctx)
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [ctx], quats, LEVELS)
    check_attention(got, ref, f"many splits hkv{hkv} T{ctx}")
    got2 = _gpu_decode(q, kp, kn, vp, vn, [ctx - 1000], quats, ctx)
    ref2 = oatt.decode_fused(q, kp, kn, vp, vn, [ctx - 1000], quats, LEVELS)
    check_attention(got2, ref2, f"many splits hkv{hkv} T{ctx - 1000}")


def test_decode_custom_scale_and_determinism():
    w = synth.WORKLOADS[1]
    t = 2000
    k, v, quats, kp, kn, vp, vn = _oracle_cache(w, 4, t, 1, t)
    q = synth.queries(4, w)[0]
    got1 = _gpu_decode(q, kp, kn, vp, vn, [t], quats, t, scale=0.05)
    got2 = _gpu_decode(q, kp, kn, vp, vn, [t], quats, t, scale=0.05)
    assert np.array_equal(got1.view(np.uint32), got2.view(np.uint32))
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [t], quats, LEVELS, scale=0.05)
    check_attention(got1, ref, "scale 0.05")


def test_end_to_end_tiny_config():
    """Workload 0: fp32 K/V, G = 1, T = 1024: GPU compress then GPU decode,
    against the oracle's compress + decode."""
    w = synth.WORKLOADS[0]
    seed = 0
    k = synth.kv_tensor(seed, w, "k")
    v = synth.kv_tensor(seed, w, "v")
    q = synth.queries(seed, w)[0]
    quats_t = api.iq_make_rotation(w.rotation_seed, 1).to(DEV)
    cache = api.alloc_cache(1, 1, w.context, DEV)
    api.iq_compress_kv(_dev(k), _dev(v), quats_t, cache["k_codes"], cache["k_norms"],
                       cache["v_codes"], cache["v_norms"])
    cache["seq_lens"].fill_(w.context)
    out = api.iq_decode_attention(_dev(q), cache["k_codes"], cache["k_norms"],
                                  cache["v_codes"], cache["v_norms"], cache["seq_lens"],
                                  quats_t)
    torch.cuda.synchronize()
    quats = orot.make_quaternions(w.rotation_seed, 1)
    rots = orot.rotation_matrices(quats)
    kp, kn, kc, ky, _ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    check_codes(cache["k_codes"].cpu().numpy(), kc, ky, THR, "w0 k")
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [w.context], quats, LEVELS)
    check_attention(out.cpu().numpy(), ref, "w0")


@pytest.mark.timeout(300)
def test_gqa_append_decode_steps():
    """Workload 1 shape: bulk-compress 8192 tokens, then (append one token,
    decode) steps; every decode checked against the oracle on the oracle's
    own cache of the same tokens."""
    w = synth.WORKLOADS[1]
    seed, steps = 2, 6
    t0 = w.context
    cap = t0 + 8
    k = synth.kv_tensor(seed, w, "k")
    v = synth.kv_tensor(seed, w, "v")
    kn_new, vn_new = synth.appended_tokens(seed, w, steps)
    qs = synth.queries(seed, w, steps)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    quats_t = _dev(quats)
    cache = api.alloc_cache(1, w.n_kv_heads, cap, DEV)
    api.iq_compress_kv(_dev(k), _dev(v), quats_t, cache["k_codes"], cache["k_norms"],
                       cache["v_codes"], cache["v_norms"])
    cache["seq_lens"].fill_(t0)
    ws = api.alloc_workspace(1, w.n_q_heads, w.n_kv_heads, cap, DEV)
    k_all = np.concatenate([k, kn_new.transpose(1, 2, 0, 3)], axis=2)
    v_all = np.concatenate([v, vn_new.transpose(1, 2, 0, 3)], axis=2)
    kp, kn, *_ = ocz.compress_kv(k_all, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v_all, rots, THR)
    for s in range(steps):
        api.iq_append_token(_dev(kn_new[s]), _dev(vn_new[s]), quats_t, cache["k_codes"],
                            cache["k_norms"], cache["v_codes"], cache["v_norms"],
                            cache["seq_lens"])
        out = api.iq_decode_attention(_dev(qs[s]), cache["k_codes"], cache["k_norms"],
                                      cache["v_codes"], cache["v_norms"], cache["seq_lens"],
                                      quats_t, workspace=ws, max_seq_len=cap)
        torch.cuda.synchronize()
        n = t0 + s + 1
        ref = oatt.decode_fused(qs[s], kp, kn, vp, vn, [n], quats, LEVELS)
        check_attention(out.cpu().numpy(), ref, f"step {s}")
    assert int(cache["seq_lens"].item()) == t0 + steps


@pytest.mark.timeout(300)
def test_long_context_needle():
    """Workload 2: 32K context, planted key.  GPU compress + decode; every
    query head checked against the oracle, and the planted head's output
    equals the planted position's value (softmax argmax kept there)."""
    w = synth.WORKLOADS[2]
    seed = 0
    k = synth.kv_tensor(seed, w, "k")
    v = synth.kv_tensor(seed, w, "v")
    q = synth.queries(seed, w)[0]
    pos = synth.plant_needle(seed, w, k, q)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    quats_t = _dev(quats)
    cache = api.alloc_cache(1, w.n_kv_heads, w.context, DEV)
    api.iq_compress_kv(_dev(k), _dev(v), quats_t, cache["k_codes"], cache["k_norms"],
                       cache["v_codes"], cache["v_norms"])
    cache["seq_lens"].fill_(w.context)
    out = api.iq_decode_attention(_dev(q), cache["k_codes"], cache["k_norms"],
                                  cache["v_codes"], cache["v_norms"], cache["seq_lens"],
                                  quats_t).cpu().numpy()
    kp, kn, kc, ky, _ = ocz.compress_kv(k, rots, THR)
    vp, vn, vc, vy, _ = ocz.compress_kv(v, rots, THR)
    check_codes(cache["k_codes"].cpu().numpy(), kc, ky, THR, "w2 k")
    check_codes(cache["v_codes"].cpu().numpy(), vc, vy, THR, "w2 v")
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [w.context], quats, LEVELS)
    check_attention(out, ref, "w2")
    for g in range(w.n_kv_heads):
        h0 = g * w.group
        s = oatt.fused_scores(q[0, h0:h0 + 1], kp[0, g], kn[0, g], rots[g], LEVELS)[0]
        assert int(np.argmax(s)) == int(pos[0, g])
        v_hat = ocz.reconstruct(ocz.unpack(vp[0, g, pos[0, g]]), vn[0, g, pos[0, g]], LEVELS,
                                rots[g])
        assert np.max(np.abs(out[0, h0] - v_hat)) <= 2e-3 * np.max(np.abs(v_hat))


@pytest.mark.timeout(600)
def test_varlen_batched_decode_full_size():
    """Workload 3: 64 sequences, lengths U{2048..32768}, G = 8.  Full GPU
    compress + decode; a seeded sample of sequences checked against the
    oracle (all 16 query heads of each)."""
    w = synth.WORKLOADS[3]
    seed = 0
    lens = synth.context_lengths(seed, w)
    k = synth.kv_tensor(seed, w, "k")
    v = synth.kv_tensor(seed, w, "v")
    q = synth.queries(seed, w)[0]
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    quats_t = _dev(quats)
    cache = api.alloc_cache(w.batch, w.n_kv_heads, w.context, DEV)
    kd, vd = _dev(k), _dev(v)
    api.iq_compress_kv(kd, vd, quats_t, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                       cache["v_norms"])
    del kd, vd
    cache["seq_lens"].copy_(torch.from_numpy(lens))
    out = api.iq_decode_attention(_dev(q), cache["k_codes"], cache["k_norms"],
                                  cache["v_codes"], cache["v_norms"], cache["seq_lens"],
                                  quats_t).cpu().numpy()
    sample = np.random.default_rng(9).choice(w.batch, 5, replace=False)
    for b in sample:
        n = int(lens[b])
        kp, kn, *_ = ocz.compress_kv(k[b:b + 1, :, :n], rots, THR)
        vp, vn, *_ = ocz.compress_kv(v[b:b + 1, :, :n], rots, THR)
        ref = oatt.decode_fused(q[b:b + 1], kp, kn, vp, vn, [n], quats, LEVELS)
        check_attention(out[b:b + 1], ref, f"w3 b{b} len {n}")


@pytest.mark.parametrize("seq", [
    [1], [15, 16, 17], [63, 64, 65], [255, 256, 257], [511, 512, 513], [1000, 0, 2049],
    [4095], [4096], [4097],
])
def test_group8_matrix_core_path(seq):
    """Group-8 decode (matrix-core path: capacity a multiple of 16, 16-byte
    aligned scales) at lengths around every batch/wave/split boundary,
    several sequences per call, one of them empty."""
    w = synth.Workload(8, "g8", len(seq), 8 * 2, 2, max(seq), "f16", rotation_seed=5)
    cap = ((max(max(seq), 1) + 15) // 16) * 16 + 16
    k, v, quats, kp, kn, vp, vn = _oracle_cache(w, 3, max(seq), len(seq), cap)
    q = synth.queries(3, w)[0]
    got = _gpu_decode(q, kp, kn, vp, vn, seq, quats, cap)
    ref = oatt.decode_fused(q, kp, kn, vp, vn, seq, quats, LEVELS)
    check_attention(got, ref, f"g8 {seq}")
    for b, n in enumerate(seq):
        if n == 0:
            assert np.all(got[b] == 0)


def test_group8_workspace_reuse_and_determinism():
    """The split tickets are reset by the call that uses them: repeated calls
    on one workspace, with different shapes, stay correct and bit-identical."""
    w = synth.Workload(8, "g8", 2, 32, 4, 3000, "f16", rotation_seed=6)
    cap = 3008
    k, v, quats, kp, kn, vp, vn = _oracle_cache(w, 5, 3000, 2, cap)
    q = synth.queries(5, w)[0]
    ws = api.alloc_workspace(2, 32, 4, cap, DEV)
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [3000, 1500], quats, LEVELS)
    outs = [_gpu_decode(q, kp, kn, vp, vn, [3000, 1500], quats, cap, ws=ws) for _ in range(3)]
    for o in outs:
        check_attention(o, ref, "reuse")
        assert np.array_equal(o.view(np.uint32), outs[0].view(np.uint32))
    # smaller max_seq_len on the same workspace
    ref2 = oatt.decode_fused(q, kp, kn, vp, vn, [700, 64], quats, LEVELS)
    got2 = _gpu_decode(q, kp, kn, vp, vn, [700, 64], quats, cap, ws=ws)
    check_attention(got2, ref2, "reuse small")


def test_graph_replay_matches_eager():
    """Append + decode captured in a HIP graph: every replay (with eager work
    and synchronizations in between) equals the eager computation on the
    same cache state."""
    w = synth.WORKLOADS[1]
    t0, cap = 1000, 1024
    k = synth.kv_tensor(7, w, "k", n_tokens=t0)
    v = synth.kv_tensor(7, w, "v", n_tokens=t0)
    kn_new, vn_new = synth.appended_tokens(7, w, 1)
    q = _dev(synth.queries(7, w)[0])
    quats = _dev(orot.make_quaternions(w.rotation_seed, w.n_kv_heads))
    caches = []
    for _ in range(2):
        c = api.alloc_cache(1, w.n_kv_heads, cap, DEV)
        api.iq_compress_kv(_dev(k), _dev(v), quats, c["k_codes"], c["k_norms"], c["v_codes"],
                           c["v_norms"])
        c["seq_lens"].fill_(t0)
        caches.append(c)
    ws_g = api.alloc_workspace(1, w.n_q_heads, w.n_kv_heads, cap, DEV)
    ws_e = api.alloc_workspace(1, w.n_q_heads, w.n_kv_heads, cap, DEV)
    kd, vd = _dev(kn_new[0]), _dev(vn_new[0])
    out_g = torch.empty((1, w.n_q_heads, 128), device=DEV)

    def step(c, out, ws):
        api.iq_append_token(kd, vd, quats, c["k_codes"], c["k_norms"], c["v_codes"],
                            c["v_norms"], c["seq_lens"])
        api.iq_decode_attention(q, c["k_codes"], c["k_norms"], c["v_codes"], c["v_norms"],
                                c["seq_lens"], quats, out=out, workspace=ws, max_seq_len=cap)

    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(caches[0], out_g, ws_g)           # warm-up (eager) on the graph cache
    torch.cuda.current_stream().wait_stream(s)
    step(caches[1], torch.empty_like(out_g), ws_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(caches[0], out_g, ws_g)
    for rep in range(4):
        g.replay()
        torch.cuda.synchronize()
        out_e = torch.empty_like(out_g)
        step(caches[1], out_e, ws_e)
        torch.cuda.synchronize()
        assert int(caches[0]["seq_lens"].item()) == int(caches[1]["seq_lens"].item())
        assert torch.equal(out_g, out_e), f"replay {rep}"
        assert torch.equal(caches[0]["k_codes"], caches[1]["k_codes"])
