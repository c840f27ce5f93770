"""GPU parity of the reconstruct-then-compute baseline (Sec. 1, Fig. 1 top)
through the C ABI: iq_dequantize_kv against the oracle's reconstruction
s R^T C[code], iq_decode_attention_f16 against plain fp64 attention on the
same fp16 cache, and the two chained against the oracle's
reconstruct-then-compute decode."""

import numpy as np
import pytest
import torch

from oracle import attention as oatt
from oracle import codebook as ocb
from oracle import compress as ocz
from oracle import rotation as orot
from paper_2608_08081_amd import api, synth
from tests.parity import check_attention, row_rel_err

pytestmark = pytest.mark.gpu

LEVELS, THR = ocb.isoquant_codebook(128, 3)
DEV = torch.device("cuda:0")

# fp32 reconstruction: every output is s / sqrt(128) times a sum over the
# 128 rotated levels (|C| <= 0.1884) passed through a 4 x 4 block product and
# 5 butterfly stages; with unit roundoff u = 2^-24 the accumulated rounding
# is below ~16 u times sum |terms| <= 16 u * 128 * 0.1884 * 2 s / sqrt(128),
# i.e. about 4e-6 s.  (Typical errors are ~100x smaller.)
DEQ_ATOL_PER_NORM = 4e-6


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _oracle_cache(w, seed, batch, cap):
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap, batch=batch)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap, batch=batch)
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    return quats, rots, kp, kn, vp, vn


def _ulp16(x):
    """Spacing of fp16 values at |x| (subnormal spacing below 2^-14)."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -14)))
    return 2.0 ** (e - 10)


@pytest.mark.parametrize("batch,hkv,cap,n,off,lens", [
    (1, 1, 300, 300, 0, None),          # one chunk plus a ragged tail
    (2, 2, 720, 700, 13, None),         # several chunks, offset window
    (3, 2, 600, 600, 0, [600, 0, 257]),  # lengths: full, empty, ragged
    (1, 3, 40, 9, 31, None),            # tiny window at the end of the cache
])
def test_dequantize_parity(batch, hkv, cap, n, off, lens):
    w = synth.Workload(9, "test", batch, hkv, hkv, cap, "f16", rotation_seed=55)
    quats, rots, kp, kn, vp, vn = _oracle_cache(w, 3, batch, cap)
    ref_k = ocz.reconstruct_kv(kp[:, :, off:off + n], kn[:, :, off:off + n], rots, LEVELS)
    ref_v = ocz.reconstruct_kv(vp[:, :, off:off + n], vn[:, :, off:off + n], rots, LEVELS)
    seq = None if lens is None else _dev(np.asarray(lens, np.int32))
    sentinel = 1234.0   # exact in fp16 and fp32
    for dt in (torch.float32, torch.float16):
        ko = torch.full((batch, hkv, n, 128), sentinel, dtype=dt, device=DEV)
        vo = torch.full((batch, hkv, n, 128), sentinel, dtype=dt, device=DEV)
        api.iq_dequantize_kv(_dev(kp), _dev(kn), _dev(vp), _dev(vn), _dev(quats), n_tokens=n,
                             src_offset=off, seq_lens=seq, out_dtype=dt, k_out=ko, v_out=vo)
        torch.cuda.synchronize()
        for got_t, ref, norms in ((ko, ref_k, kn), (vo, ref_v, vn)):
            got = got_t.float().cpu().numpy().astype(np.float64)
            s = norms[:, :, off:off + n].astype(np.float64)[..., None]
            written = np.ones((batch, hkv, n, 1), bool)
            if lens is not None:
                for b in range(batch):
                    written[b, :, max(lens[b] - off, 0):] = False
            # positions past a sequence's length keep the sentinel
            assert np.all(np.where(written, True, got == sentinel))
            wm = np.broadcast_to(written, got.shape)
            if dt == torch.float32:
                err = np.abs(got - ref)
                assert np.all(err[wm] <= (DEQ_ATOL_PER_NORM * np.broadcast_to(s, got.shape))[wm])
            else:
                ref16 = ref.astype(np.float16).astype(np.float64)
                err = np.abs(got - ref16)
                # rounding is monotone: the fp32 result, within delta of the
                # exact value, rounds to within delta + one fp16 spacing
                delta = DEQ_ATOL_PER_NORM * np.broadcast_to(s, got.shape)
                assert np.all(err[wm] <= (_ulp16(ref) + delta)[wm])
                exact = np.count_nonzero((err == 0) & wm)
                assert exact >= 0.99 * np.count_nonzero(wm)


def test_dequantize_one_side_only():
    w = synth.Workload(9, "test", 1, 2, 2, 64, "f16", rotation_seed=56)
    quats, rots, kp, kn, vp, vn = _oracle_cache(w, 4, 1, 64)
    _, vo = api.iq_dequantize_kv(None, None, _dev(vp), _dev(vn), _dev(quats),
                                 out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = ocz.reconstruct_kv(vp, vn, rots, LEVELS)
    s = vn.astype(np.float64)[..., None]
    assert np.all(np.abs(vo.cpu().numpy() - ref) <= DEQ_ATOL_PER_NORM * s)


def _f16_cache(w, seed, batch, cap):
    k = synth.kv_tensor(seed, w, "k", n_tokens=cap, batch=batch)
    v = synth.kv_tensor(seed, w, "v", n_tokens=cap, batch=batch)
    return k.astype(np.float16), v.astype(np.float16)


@pytest.mark.parametrize("hq,hkv,seq", [
    (1, 1, [1024]),
    (8, 1, [1, 15, 16, 17, 100]),
    (32, 4, [777, 0, 513]),
    (16, 2, [2, 5000]),
    (6, 2, [300]),
    (4, 4, [4096, 33]),
])
def test_decode_f16_parity(hq, hkv, seq):
    """Plain attention on an fp16 cache against fp64 attention on the same
    fp16 values: ragged lengths, an empty sequence, group sizes 1..8, one
    split and many."""
    w = synth.Workload(9, "test", len(seq), hq, hkv, max(seq), "f16", rotation_seed=57)
    cap = max(seq) + 5
    k, v = _f16_cache(w, 5, len(seq), cap)
    q = synth.queries(5, w)[0]
    out = api.iq_decode_attention_f16(_dev(q), _dev(k), _dev(v),
                                      _dev(np.asarray(seq, np.int32)), max_seq_len=cap)
    torch.cuda.synchronize()
    ref = oatt.attention_exact(q, k, v, seq, hkv)
    check_attention(out.cpu().numpy(), ref, f"f16 hq{hq} hkv{hkv}")
    for b, n in enumerate(seq):
        if n == 0:
            assert np.all(out[b].cpu().numpy() == 0)


def test_decode_f16_scale_and_max_len_clamp():
    w = synth.Workload(9, "test", 2, 8, 1, 600, "f16", rotation_seed=58)
    k, v = _f16_cache(w, 6, 2, 640)
    q = synth.queries(6, w)[0]
    seq = [640, 200]           # the first is clamped to max_seq_len = 600
    out = api.iq_decode_attention_f16(_dev(q), _dev(k), _dev(v),
                                      _dev(np.asarray(seq, np.int32)), max_seq_len=600,
                                      softmax_scale=0.05)
    torch.cuda.synchronize()
    ref = oatt.attention_exact(q, k, v, [600, 200], 1, scale=0.05)
    check_attention(out.cpu().numpy(), ref, "f16 scale 0.05")


def test_reconstruct_then_compute_chain():
    """Fig. 1 top end to end on a GQA cache: dequantize to fp16, then fp16
    attention; against fp64 attention on the oracle's fp16-rounded
    reconstruction (the same materialized tensors), and close to the
    oracle's unrounded reconstruct-then-compute decode."""
    w = synth.Workload(9, "test", 2, 16, 2, 3000, "f16", rotation_seed=59)
    seq = [3000, 1234]
    cap = 3008
    quats, rots, kp, kn, vp, vn = _oracle_cache(w, 7, 2, cap)
    q = synth.queries(7, w)[0]
    seq_d = _dev(np.asarray(seq, np.int32))
    ko, vo = api.iq_dequantize_kv(_dev(kp), _dev(kn), _dev(vp), _dev(vn), _dev(quats),
                                  seq_lens=seq_d, out_dtype=torch.float16)
    out = api.iq_decode_attention_f16(_dev(q), ko, vo, seq_d, max_seq_len=cap)
    torch.cuda.synchronize()
    k16 = ocz.reconstruct_kv(kp, kn, rots, LEVELS).astype(np.float16)
    v16 = ocz.reconstruct_kv(vp, vn, rots, LEVELS).astype(np.float16)
    ref = oatt.attention_exact(q, k16, v16, seq, 2)
    check_attention(out.cpu().numpy(), ref, "reconstruct chain")
    # the fp16 materialization itself costs ~2^-12 relative per element
    ref_exact = oatt.decode_reconstruct(q, kp, kn, vp, vn, seq, quats, LEVELS)
    assert np.max(row_rel_err(out.cpu().numpy(), ref_exact)) < 1e-2


def test_full_size_32k_f16_and_dequant_samples():
    """At the 32K shape (32 query heads, 4 KV heads) in the launch
    configuration the benchmark times: every output row of the fp16
    attention against fp64 attention, and sampled tokens of the fp16
    materialization against the oracle."""
    w = synth.WORKLOADS[2]
    t = w.context
    k = synth.kv_tensor(0, w, "k", n_tokens=t)
    v = synth.kv_tensor(0, w, "v", n_tokens=t)
    q = synth.queries(0, w)[0]
    out = api.iq_decode_attention_f16(_dev(q), _dev(k), _dev(v),
                                      _dev(np.full(1, t, np.int32)), max_seq_len=t)
    torch.cuda.synchronize()
    ref = oatt.attention_exact(q, k, v, [t], w.n_kv_heads)
    check_attention(out.cpu().numpy(), ref, "f16 32K")

    # the packed cache comes from the oracle's compression
    quats = orot.make_quaternions(w.rotation_seed, w.n_kv_heads)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, THR)
    vp, vn, *_ = ocz.compress_kv(v, rots, THR)
    ko, vo = api.iq_dequantize_kv(_dev(kp), _dev(kn), _dev(vp), _dev(vn), _dev(quats),
                                  out_dtype=torch.float16)
    torch.cuda.synchronize()
    g = np.random.default_rng(11)
    pos = np.sort(g.choice(t, size=512, replace=False))
    for packed, norms, got in ((kp, kn, ko), (vp, vn, vo)):
        ref = ocz.reconstruct_kv(packed[:, :, pos], norms[:, :, pos], rots, LEVELS)
        gg = got[:, :, pos].float().cpu().numpy().astype(np.float64)
        delta = DEQ_ATOL_PER_NORM * norms[:, :, pos].astype(np.float64)[..., None]
        err = np.abs(gg - ref.astype(np.float16).astype(np.float64))
        assert np.all(err <= _ulp16(ref) + delta)
        assert np.count_nonzero(err == 0) >= 0.99 * err.size
