"""GPU parity of the fused decode step (iq_decode_step: Alg. 1 on the step's
new key and value, then App. A attention over the advanced lengths) against
the oracle, and against the separate append + decode entry points."""

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


def _setup(w, seed, seq0, cap):
    """Oracle-packed cache of cap tokens per sequence; on the GPU only the
    first seq0[b] positions hold records, the rest is poisoned (random codes,
    NaN scales) so that a read of a position that is not attended, or of
    the appended position before it is written, shows up.  The token at
    position seq0[b] is the step's new token."""
    b = len(seq0)
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap, batch=b)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap, batch=b)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, kc, ky, ks = ocz.compress_kv(k, rots, THR)
    vp, vn, vc, vy, vs = ocz.compress_kv(v, rots, THR)
    rng = np.random.default_rng(seed + 100)
    gk, gv = kp.copy(), vp.copy()
    gkn, gvn = kn.copy(), vn.copy()
    for i, n in enumerate(seq0):
        gk[i, :, n:] = rng.integers(0, 256, size=gk[i, :, n:].shape, dtype=np.uint8)
        gv[i, :, n:] = rng.integers(0, 256, size=gv[i, :, n:].shape, dtype=np.uint8)
        gkn[i, :, n:] = np.nan
        gvn[i, :, n:] = np.nan
    cache = dict(k_codes=_dev(gk), k_norms=_dev(gkn), v_codes=_dev(gv), v_norms=_dev(gvn),
                 seq_lens=_dev(np.asarray(seq0, np.int32)))
    idx = np.minimum(np.asarray(seq0), cap - 1)
    k_new = np.stack([k[i, :, idx[i]] for i in range(b)])
    v_new = np.stack([v[i, :, idx[i]] for i in range(b)])
    ora = dict(kp=kp, kn=kn, kc=kc, ky=ky, ks=ks, vp=vp, vn=vn, vc=vc, vy=vy, vs=vs)
    return cache, quats, k_new, v_new, ora


def _step(cache, quats, q, k_new, v_new, cap, max_seq_len=None, status=None, ws=None,
          out=None):
    return api.iq_decode_step(q, k_new, v_new, cache["k_codes"], cache["k_norms"],
                              cache["v_codes"], cache["v_norms"], cache["seq_lens"], quats,
                              max_seq_len=cap if max_seq_len is None else max_seq_len,
                              status=status, workspace=ws, out=out)


def _check_new_records(cache, ora, seq0, cap, label):
    for i, n in enumerate(seq0):
        if n >= cap:
            continue
        for side in ("k", "v"):
            got = cache[f"{side}_codes"][i, :, n].cpu().numpy()
            check_codes(got[None, :, None], ora[f"{side}c"][i:i + 1, :, n:n + 1],
                        ora[f"{side}y"][i:i + 1, :, n:n + 1], THR, f"{label} {side} b{i}")
            check_norms(cache[f"{side}_norms"][i, :, n].cpu().numpy(), ora[f"{side}s"][i, :, n],
                        f"{label} {side} scale b{i}")


@pytest.mark.parametrize("hq,hkv,seq0,cap", [
    # group 8, matrix-core path: the new position at split / wave / batch edges
    (16, 2, [0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 500], 512),
    (32, 4, [2999, 1500], 3008),
    (8, 1, [4095], 4096),
    (8, 1, [4096], 4112),
    (8, 1, [4096], 4100),       # capacity not a multiple of 16: generic path
    (8, 1, [30000], 32768),     # one KV head: more than 64 partials per row
    # a grid of several rounds (64 sequences x 2 KV heads x 4 partials): the
    # instance that reads the length before its loads and skips empty splits
    (16, 2, [0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 223, 224, 225, 447,
             448, 449, 500, 600, 638, 639] + [(97 * i + 13) % 639 for i in range(40)], 640),
    # other group sizes: append kernel, then the generic decode
    (16, 4, [0, 700, 1023], 1024),
    (6, 2, [300], 301),
])
def test_step_matches_oracle(hq, hkv, seq0, cap):
    w = synth.Workload(8, "step", len(seq0), hq, hkv, cap, "f16", rotation_seed=11)
    cache, quats, k_new, v_new, ora = _setup(w, 4, seq0, cap)
    q = synth.queries(4, w)[0]
    out = _step(cache, _dev(quats), _dev(q), _dev(k_new), _dev(v_new), cap)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    seq1 = [n + 1 for n in seq0]
    ref = oatt.decode_fused(q, ora["kp"], ora["kn"], ora["vp"], ora["vn"], seq1, quats, LEVELS)
    check_attention(got, ref, f"step hq{hq} hkv{hkv}")
    assert cache["seq_lens"].cpu().numpy().tolist() == seq1
    _check_new_records(cache, ora, seq0, cap, "step")


@pytest.mark.timeout(300)
def test_step_many_sequences_stale_workspace():
    """A grid of several rounds whose merge has far more workgroups than the
    chip holds at once (384 sequences x 16 query heads = 6144), with lengths
    at exact multiples of the split length (512 here: one position more would
    add a live split) and empty sequences, on a workspace filled with stale
    partials (scores far above any real one).  The merge must count each
    sequence's live splits from the length the step began with, although its
    workgroup of head 0 advances seq_lens[b] during the same launch; a stale
    partial read would dominate the output."""
    cap, n = 2048, 384
    seq0 = [(0, 512, 1024, 1536)[i % 4] if i % 3 else (131 * i) % 2047 for i in range(n)]
    w = synth.Workload(8, "step stale", n, 16, 2, cap, "f16", rotation_seed=12)
    cache, quats, k_new, v_new, ora = _setup(w, 6, seq0, cap)
    q = synth.queries(6, w)[0]
    ws = api.alloc_workspace(n, 16, 2, cap, DEV)
    ws.fill_(0x44)   # every partial m = l = o = 785.07 (0x44444444)
    out = _step(cache, _dev(quats), _dev(q), _dev(k_new), _dev(v_new), cap, ws=ws)
    torch.cuda.synchronize()
    seq1 = [x + 1 for x in seq0]
    assert cache["seq_lens"].cpu().numpy().tolist() == seq1
    _check_new_records(cache, ora, seq0, cap, "stale ws")
    # the decode on the device's own records (the new token's included)
    dev_cache = [cache[nm].cpu().numpy() for nm in ("k_codes", "k_norms", "v_codes", "v_norms")]
    ref = oatt.decode_fused(q, *dev_cache, seq1, quats, LEVELS)
    check_attention(out.cpu().numpy(), ref, "stale ws")


def test_step_f32_inputs_and_custom_scale():
    w = synth.Workload(0, "step32", 2, 16, 2, 777, "f32", rotation_seed=3)
    seq0, cap = [776, 100], 784
    cache, quats, k_new, v_new, ora = _setup(w, 6, seq0, cap)
    q = synth.queries(6, w)[0]
    out = api.iq_decode_step(_dev(q), _dev(k_new), _dev(v_new), cache["k_codes"],
                             cache["k_norms"], cache["v_codes"], cache["v_norms"],
                             cache["seq_lens"], _dev(quats), max_seq_len=cap, softmax_scale=0.05)
    torch.cuda.synchronize()
    ref = oatt.decode_fused(q, ora["kp"], ora["kn"], ora["vp"], ora["vn"], [777, 101], quats,
                            LEVELS, scale=0.05)
    check_attention(out.cpu().numpy(), ref, "step f32 scale 0.05")
    _check_new_records(cache, ora, seq0, cap, "step f32")


@pytest.mark.parametrize("hq,hkv", [(16, 2), (8, 4)])
def test_step_at_capacity(hq, hkv):
    """A sequence already at capacity: its token is dropped, the capacity
    flag is raised, its length stays and its attention covers the full
    cache; the other sequences append as usual."""
    cap = 256
    seq0 = [cap, 40]
    w = synth.Workload(8, "cap", 2, hq, hkv, cap, "f16", rotation_seed=12)
    cache, quats, k_new, v_new, ora = _setup(w, 8, seq0, cap)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    q = synth.queries(8, w)[0]
    out = _step(cache, _dev(quats), _dev(q), _dev(k_new), _dev(v_new), cap, status=status)
    torch.cuda.synchronize()
    ref = oatt.decode_fused(q, ora["kp"], ora["kn"], ora["vp"], ora["vn"], [cap, 41], quats,
                            LEVELS)
    check_attention(out.cpu().numpy(), ref, "at capacity")
    assert cache["seq_lens"].cpu().numpy().tolist() == [cap, 41]
    assert int(status.item()) == 5


def test_step_beyond_max_seq_len():
    """max_seq_len below the advanced length: the token is still written and
    the length advanced, attention is clamped to max_seq_len positions."""
    cap = 512
    seq0 = [300]
    w = synth.Workload(8, "clamp", 1, 16, 2, cap, "f16", rotation_seed=13)
    cache, quats, k_new, v_new, ora = _setup(w, 9, seq0, cap)
    q = synth.queries(9, w)[0]
    out = _step(cache, _dev(quats), _dev(q), _dev(k_new), _dev(v_new), cap, max_seq_len=200)
    torch.cuda.synchronize()
    ref = oatt.decode_fused(q, ora["kp"], ora["kn"], ora["vp"], ora["vn"], [200], quats, LEVELS)
    check_attention(out.cpu().numpy(), ref, "clamped")
    assert cache["seq_lens"].cpu().numpy().tolist() == [301]
    _check_new_records(cache, ora, seq0, cap, "clamped")


@pytest.mark.parametrize("hq,hkv,seq0,cap", [
    (32, 4, [8191], 8208),
    (16, 2, [17, 0, 1000], 1024),
    (32, 4, [8191], 8200),      # capacity not a multiple of 16: generic path
])
def test_step_equals_append_then_decode(hq, hkv, seq0, cap):
    """Fused step and the two separate calls on identical caches: identical
    records and lengths, outputs equal to rounding."""
    w = synth.Workload(8, "sep", len(seq0), hq, hkv, cap, "f16", rotation_seed=14)
    c1, quats, k_new, v_new, _ = _setup(w, 10, seq0, cap)
    c2 = {k: t.clone() for k, t in c1.items()}
    q, qt, kt, vt = synth.queries(10, w)[0], _dev(quats), _dev(k_new), _dev(v_new)
    out1 = _step(c1, qt, _dev(q), kt, vt, cap)
    api.iq_append_token(kt, vt, qt, c2["k_codes"], c2["k_norms"], c2["v_codes"], c2["v_norms"],
                        c2["seq_lens"])
    out2 = api.iq_decode_attention(_dev(q), c2["k_codes"], c2["k_norms"], c2["v_codes"],
                                   c2["v_norms"], c2["seq_lens"], qt, max_seq_len=cap)
    torch.cuda.synchronize()
    assert torch.equal(c1["seq_lens"], c2["seq_lens"])
    for i, n in enumerate(seq0):
        assert torch.equal(c1["k_codes"][i, :, n], c2["k_codes"][i, :, n])
        assert torch.equal(c1["v_codes"][i, :, n], c2["v_codes"][i, :, n])
        assert torch.equal(c1["k_norms"][i, :, n], c2["k_norms"][i, :, n])
    a, b = out1.cpu().numpy(), out2.cpu().numpy()
    err = np.max(np.abs(a - b), axis=-1) / np.max(np.abs(b), axis=-1)
    assert np.all(err < 1e-4), err.max()


def test_step_graph_replay_matches_eager():
    """The fused step captured in a HIP graph: each replay advances the
    length and equals the eager step on a twin cache."""
    w = synth.WORKLOADS[1]
    t0, cap = 1000, 1024
    seq0 = [t0]
    c_g, quats, _, _, _ = _setup(w, 11, seq0, cap)
    c_e = {k: t.clone() for k, t in c_g.items()}
    kn_new, vn_new = synth.appended_tokens(11, w, 1)
    kd, vd = _dev(kn_new[0]), _dev(vn_new[0])
    q = _dev(synth.queries(11, w)[0])
    qt = _dev(quats)
    ws_g = api.alloc_workspace(1, w.n_q_heads, w.n_kv_heads, cap, DEV)
    ws_e = api.alloc_workspace(1, w.n_q_heads, w.n_kv_heads, cap, DEV)
    out_g = torch.empty((1, w.n_q_heads, 128), device=DEV)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        _step(c_g, qt, q, kd, vd, cap, ws=ws_g, out=out_g)     # warm-up (eager)
    torch.cuda.current_stream().wait_stream(s)
    _step(c_e, qt, q, kd, vd, cap, ws=ws_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(c_g, qt, q, kd, vd, cap, ws=ws_g, out=out_g)
    for rep in range(4):
        g.replay()
        torch.cuda.synchronize()
        out_e = _step(c_e, qt, q, kd, vd, cap, ws=ws_e)
        torch.cuda.synchronize()
        assert int(c_g["seq_lens"].item()) == int(c_e["seq_lens"].item()) == t0 + 2 + rep
        assert torch.equal(out_g, out_e), f"replay {rep}"
        assert torch.equal(c_g["k_codes"], c_e["k_codes"])
