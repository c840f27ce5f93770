"""CPU tests of the C ABI: the library loads and exports what the header
declares, its host-side functions agree bit-for-bit with the oracle's
independent implementations, and argument validation rejects bad calls
before any HIP call is made (so these run without a GPU)."""

import ctypes

import numpy as np
import pytest

from oracle import codebook as ocb
from oracle import rotation as orot
from paper_2608_08081_amd import _lib

L = None


@pytest.fixture(scope="module", autouse=True)
def loaded():
    global L
    L = _lib.lib()
    return L


def test_exports_every_declared_symbol():
    names = _lib.header_functions()
    assert len(names) >= 9
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    for code, name in _lib.STATUS_NAMES.items():
        assert L.iq_status_string(code).decode() == name
    assert L.iq_status_string(99).decode() == "unknown status"
    assert L.iq_status_string(-1).decode() == "unknown status"
    assert L.iq_version() >= 200


def test_codebook_matches_oracle_bit_for_bit():
    lv = np.zeros(8, np.float32)
    th = np.zeros(7, np.float32)
    assert L.iq_codebook(lv.ctypes.data_as(ctypes.c_void_p), th.ctypes.data_as(ctypes.c_void_p)) == 0
    o_lv, o_th = ocb.isoquant_codebook(128, 3)
    assert np.array_equal(lv.astype(np.float64), o_lv)
    assert np.array_equal(th.astype(np.float64), o_th)


@pytest.mark.parametrize("seed,heads", [(0, 1), (1000, 1), (1002, 4), (2 ** 63 + 12345, 8)])
def test_make_rotation_matches_oracle_bit_for_bit(seed, heads):
    out = np.zeros((heads, 32, 2, 4), np.float32)
    assert L.iq_make_rotation(seed, heads, 128, out.ctypes.data_as(ctypes.c_void_p)) == 0
    want = orot.make_quaternions(seed, heads)
    assert np.array_equal(out.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("variant,name", [(0, "v3_wht_so4"), (1, "wht_so3"), (2, "wht")])
def test_make_rotation_variant_matches_oracle_bit_for_bit(variant, name):
    out = np.zeros((3, 32, 2, 4), np.float32)
    assert L.iq_make_rotation_variant(1002, 3, 128, variant,
                                      out.ctypes.data_as(ctypes.c_void_p)) == 0
    want = orot.variant_quaternions(name, 1002, 3)
    assert np.array_equal(out.view(np.uint32), want.view(np.uint32))


def test_make_rotation_variant_validation():
    out = np.zeros((1, 32, 2, 4), np.float32)
    p = out.ctypes.data_as(ctypes.c_void_p)
    assert L.iq_make_rotation_variant(1, 1, 128, 3, p) == 2
    assert L.iq_make_rotation_variant(1, 1, 128, -1, p) == 2
    for v in (0, 1, 2):
        assert L.iq_make_rotation_variant(1, 1, 64, v, p) == 2
        assert L.iq_make_rotation_variant(1, 0, 128, v, p) == 1
        assert L.iq_make_rotation_variant(1, 1, 128, v, None) == 1


def test_make_rotation_validation():
    out = np.zeros((1, 32, 2, 4), np.float32)
    p = out.ctypes.data_as(ctypes.c_void_p)
    assert L.iq_make_rotation(1, 1, 64, p) == 2
    assert L.iq_make_rotation(1, 0, 128, p) == 1
    assert L.iq_make_rotation(1, 1, 128, None) == 1


# Fake, aligned, never-dereferenced device addresses: validation must reject
# every call below before touching them.
A = ctypes.c_void_p(0x100000)
B = ctypes.c_void_p(0x200000)


def _compress(**kw):
    args = dict(k=A, v=B, dtype=1, batch=1, heads=2, n=10, hd=128, quats=A, kc=A, kn=A, vc=B,
                vn=B, cap=16, off=0)
    args.update(kw)
    return L.iq_compress_kv(args["k"], args["v"], args["dtype"], args["batch"], args["heads"],
                            args["n"], args["hd"], args["quats"], args["kc"], args["kn"],
                            args["vc"], args["vn"], args["cap"], args["off"], None)


def test_compress_validation():
    assert _compress(hd=64) == 2
    assert _compress(dtype=7) == 2
    assert _compress(k=None, v=None) == 1
    assert _compress(k=None, v=None, n=0) == 0   # empty: no-op before pointer checks
    assert _compress(quats=None) == 1
    assert _compress(kc=None) == 1
    assert _compress(n=17) == 1                 # beyond capacity
    assert _compress(off=10) == 1               # 10 + 10 > 16
    assert _compress(off=-1) == 1
    assert _compress(n=-1) == 1
    assert _compress(batch=-1) == 1
    assert _compress(heads=0) == 1
    assert _compress(kc=ctypes.c_void_p(0x100008)) == 1   # codes not 16-byte aligned
    assert _compress(k=ctypes.c_void_p(0x100004)) == 1
    # empty inputs are valid no-ops that launch nothing
    assert _compress(n=0) == 0
    assert _compress(batch=0) == 0


def _append(**kw):
    args = dict(k=A, v=B, dtype=1, batch=2, heads=2, hd=128, quats=A, kc=A, kn=A, vc=B, vn=B,
                cap=16, seq=A, status=None)
    args.update(kw)
    return L.iq_append_token(args["k"], args["v"], args["dtype"], args["batch"], args["heads"],
                             args["hd"], args["quats"], args["kc"], args["kn"], args["vc"],
                             args["vn"], args["cap"], args["seq"], args["status"], None)


def test_append_validation():
    assert _append(hd=96) == 2
    assert _append(dtype=3) == 2
    assert _append(seq=None) == 1
    assert _append(k=None, v=None) == 1
    assert _append(vn=None) == 1
    assert _append(status=ctypes.c_void_p(0x100002)) == 1
    assert _append(batch=0) == 0


def _decode(**kw):
    args = dict(q=A, kc=A, kn=A, vc=B, vn=B, seq=A, cap=1024, maxlen=1024, quats=A, batch=1,
                hq=32, hkv=4, hd=128, scale=0.0, out=B, ws=A, wsb=1 << 30)
    args.update(kw)
    return L.iq_decode_attention(args["q"], args["kc"], args["kn"], args["vc"], args["vn"],
                                 args["seq"], args["cap"], args["maxlen"], args["quats"],
                                 args["batch"], args["hq"], args["hkv"], args["hd"],
                                 args["scale"], args["out"], args["ws"], args["wsb"], None)


def test_decode_validation():
    assert _decode(hd=256) == 2
    assert _decode(hq=30) == 1                  # not a multiple of H_kv
    assert _decode(hq=68) == 2                  # group 17 > 16
    assert _decode(maxlen=2048) == 1            # beyond capacity
    assert _decode(q=None) == 1
    assert _decode(ws=None) == 1
    assert _decode(ws=ctypes.c_void_p(0x100010)) == 1   # workspace not 256-byte aligned
    assert _decode(q=ctypes.c_void_p(0x100004)) == 1
    assert _decode(wsb=16) == 3
    assert _decode(batch=0) == 0


def test_workspace_bytes():
    n = L.iq_decode_workspace_bytes(1, 32, 4, 32768, 128)
    assert n > 0 and n % 256 == 0
    assert L.iq_decode_workspace_bytes(1, 32, 4, 32768, 64) == 0
    assert L.iq_decode_workspace_bytes(1, 30, 4, 32768, 128) == 0
    # monotone in context length
    assert L.iq_decode_workspace_bytes(1, 32, 4, 1024, 128) <= n


def _step(**kw):
    args = dict(q=A, k=A, v=B, dtype=1, kc=A, kn=A, vc=B, vn=B, seq=A, cap=1024, maxlen=1024,
                quats=A, batch=1, hq=32, hkv=4, hd=128, scale=0.0, out=B, ws=A, wsb=1 << 30,
                status=None)
    args.update(kw)
    return L.iq_decode_step(args["q"], args["k"], args["v"], args["dtype"], args["kc"],
                            args["kn"], args["vc"], args["vn"], args["seq"], args["cap"],
                            args["maxlen"], args["quats"], args["batch"], args["hq"],
                            args["hkv"], args["hd"], args["scale"], args["out"], args["ws"],
                            args["wsb"], args["status"], None)


def test_step_validation():
    assert _step(hd=96) == 2
    assert _step(dtype=3) == 2
    assert _step(hq=68) == 2                    # group 17 > 16
    assert _step(k=None) == 1                   # both new vectors are required
    assert _step(v=None) == 1
    assert _step(k=ctypes.c_void_p(0x100004)) == 1   # k_new not 16-byte aligned
    assert _step(maxlen=0) == 1                 # the step always attends the new token
    assert _step(maxlen=2048) == 1              # beyond capacity
    assert _step(seq=None) == 1
    assert _step(status=ctypes.c_void_p(0x100002)) == 1
    assert _step(wsb=16) == 3
    assert _step(batch=0) == 0


def _dequant(**kw):
    args = dict(kc=A, kn=A, vc=B, vn=B, quats=A, seq=None, batch=1, heads=2, n=10, hd=128,
                cap=16, off=0, dtype=1, ko=A, vo=B)
    args.update(kw)
    return L.iq_dequantize_kv(args["kc"], args["kn"], args["vc"], args["vn"], args["quats"],
                              args["seq"], args["batch"], args["heads"], args["n"], args["hd"],
                              args["cap"], args["off"], args["dtype"], args["ko"], args["vo"],
                              None)


def test_dequantize_validation():
    assert _dequant(hd=64) == 2
    assert _dequant(dtype=5) == 2
    assert _dequant(kc=None, vc=None) == 1
    assert _dequant(quats=None) == 1
    assert _dequant(ko=None) == 1
    assert _dequant(vn=None) == 1
    assert _dequant(n=17) == 1                  # beyond capacity
    assert _dequant(off=7) == 1                 # 7 + 10 > 16
    assert _dequant(off=-1) == 1
    assert _dequant(heads=0) == 1
    assert _dequant(ko=ctypes.c_void_p(0x100008)) == 1   # output not 16-byte aligned
    assert _dequant(seq=ctypes.c_void_p(0x100002)) == 1
    assert _dequant(n=0) == 0
    assert _dequant(batch=0) == 0


def _decode_f16(**kw):
    args = dict(q=A, k=A, v=B, seq=A, cap=1024, maxlen=1024, batch=1, hq=32, hkv=4, hd=128,
                scale=0.0, out=B, ws=A, wsb=1 << 30)
    args.update(kw)
    return L.iq_decode_attention_f16(args["q"], args["k"], args["v"], args["seq"], args["cap"],
                                     args["maxlen"], args["batch"], args["hq"], args["hkv"],
                                     args["hd"], args["scale"], args["out"], args["ws"],
                                     args["wsb"], None)


def test_decode_f16_validation():
    assert _decode_f16(hd=64) == 2
    assert _decode_f16(hq=36) == 2              # group 9 > 8
    assert _decode_f16(hq=30) == 1
    assert _decode_f16(maxlen=2048) == 1
    assert _decode_f16(k=None) == 1
    assert _decode_f16(out=ctypes.c_void_p(0x100004)) == 1
    assert _decode_f16(ws=ctypes.c_void_p(0x100040)) == 1
    assert _decode_f16(wsb=16) == 3
    assert _decode_f16(batch=0) == 0
    n = L.iq_decode_f16_workspace_bytes(1, 32, 4, 32768, 128)
    assert n > 0 and n % 256 == 0
    assert L.iq_decode_f16_workspace_bytes(1, 36, 4, 32768, 128) == 0
    assert L.iq_decode_f16_workspace_bytes(1, 32, 4, 32768, 64) == 0


def _paged_decode(**kw):
    args = dict(q=A, kc=A, kn=A, vc=B, vn=B, page=64, n_pages=8, bt=A, max_pages=4, seq=A,
                msl=256, quats=A, batch=1, hq=16, hkv=2, hd=128, scale=0.0, out=A, ws=A,
                wsb=1 << 30)
    args.update(kw)
    return L.iq_decode_attention_paged(args["q"], args["kc"], args["kn"], args["vc"],
                                       args["vn"], args["page"], args["n_pages"], args["bt"],
                                       args["max_pages"], args["seq"], args["msl"],
                                       args["quats"], args["batch"], args["hq"], args["hkv"],
                                       args["hd"], args["scale"], args["out"], args["ws"],
                                       args["wsb"], None)


def test_paged_decode_validation():
    assert _paged_decode(page=48) == 1           # not a power of two
    assert _paged_decode(page=8) == 1
    assert _paged_decode(page=0) == 1
    assert _paged_decode(n_pages=0) == 1
    assert _paged_decode(max_pages=0) == 1
    assert _paged_decode(bt=None) == 1
    assert _paged_decode(msl=257) == 1           # beyond max_pages * page_size
    assert _paged_decode(hq=34) == 2             # group 17 > 16
    assert _paged_decode(hq=7) == 1              # not a multiple of H_kv
    assert _paged_decode(hd=64) == 2
    assert _paged_decode(batch=70000) == 1
    assert _paged_decode(max_pages=1 << 40) == 1
    assert _paged_decode(wsb=16) == 3
    assert _paged_decode(batch=0) == 0           # empty batch: nothing launched


def test_paged_compress_validation():
    def call(**kw):
        a = dict(k=A, v=B, dtype=1, batch=1, hkv=2, n=10, hd=128, quats=A, page=64,
                 n_pages=4, bt=A, max_pages=2, off=0)
        a.update(kw)
        return L.iq_compress_kv_paged(a["k"], a["v"], a["dtype"], a["batch"], a["hkv"], a["n"],
                                      a["hd"], a["quats"], A, A, B, B, a["page"], a["n_pages"],
                                      a["bt"], a["max_pages"], a["off"], None)
    assert call(off=120) == 1                    # 120 + 10 > 2 * 64
    assert call(page=40) == 1
    assert call(page=96) == 1                    # multiple of 16, not a power of two
    assert call(dtype=7) == 2
    assert call(n=0) == 0


def test_codebook_bits_equal_oracle():
    """iq_codebook_bits equals the oracle's stored C_b exactly (b = 2, 3, 4)
    and iq_codebook is C_3; other widths are refused."""
    import numpy as np
    from oracle import codebook as ocb
    for bits in (2, 3, 4):
        n = 1 << bits
        lv = np.zeros(n, np.float32)
        th = np.zeros(n - 1, np.float32)
        assert L.iq_codebook_bits(bits, lv.ctypes.data_as(ctypes.c_void_p),
                                  th.ctypes.data_as(ctypes.c_void_p)) == 0
        s, t = ocb.isoquant_codebook(128, bits)
        assert np.array_equal(lv.astype(np.float64), s)
        assert np.array_equal(th.astype(np.float64), t)
    assert L.iq_codebook_bits(5, None, None) == 2
    assert L.iq_codebook_bits(1, None, None) == 2


def test_bits_entry_point_validation():
    def dec(**kw):
        a = dict(hq=16, hkv=2, cap=256, msl=256, bits=4, b=1)
        a.update(kw)
        return L.iq_decode_attention_bits(A, A, A, B, B, A, a["cap"], a["msl"], A, a["b"],
                                          a["hq"], a["hkv"], 128, 0.0, A, A, 1 << 30, a["bits"],
                                          None)
    assert dec(bits=5) == 2
    assert dec(bits=1) == 2
    assert dec(hq=34) == 2                       # group 17 > 16
    assert dec(cap=250, msl=250) == 2            # capacity not a multiple of 16
    assert dec(msl=300) == 1                     # max_seq_len beyond capacity
    assert dec(b=0) == 0
    assert L.iq_compress_kv_bits(A, B, 1, 1, 2, 10, 128, A, A, A, B, B, 16, 0, 5, None) == 2
    assert L.iq_compress_kv_bits(A, B, 1, 1, 2, 10, 128, A, A, A, B, B, 16, 10, 4, None) == 1
    assert L.iq_compress_kv_bits(A, B, 1, 1, 2, 0, 128, A, A, A, B, B, 16, 0, 2, None) == 0


def test_multi_token_validation():
    def call(**kw):
        a = dict(b=1, t=2, hq=16, hkv=2, cap=256, msl=256, wsb=1 << 30)
        a.update(kw)
        return L.iq_decode_attention_multi(A, A, A, B, B, A, a["cap"], a["msl"], A, a["b"],
                                           a["t"], a["hq"], a["hkv"], 128, 0.0, A, A, a["wsb"],
                                           None)
    assert call(t=5) == 2
    assert call(t=0) == 2
    assert call(hq=8) == 2                       # multi-token: group 8 only
    assert call(cap=250, msl=250) == 2
    assert call(msl=300) == 1
    assert call(wsb=16) == 3
    assert call(b=0) == 0
    ws1 = L.iq_decode_multi_workspace_bytes(1, 1, 16, 2, 256, 128)
    assert ws1 == L.iq_decode_workspace_bytes(1, 16, 2, 256, 128)
    w2 = L.iq_decode_multi_workspace_bytes(1, 2, 16, 2, 256, 128)
    w4 = L.iq_decode_multi_workspace_bytes(1, 4, 16, 2, 256, 128)
    assert w2 > 0 and w4 >= 2 * w2 - 256
    assert L.iq_decode_multi_workspace_bytes(1, 5, 16, 2, 256, 128) == 0
    assert L.iq_decode_multi_workspace_bytes(1, 2, 8, 2, 256, 128) == 0
    # the merge grid takes (sequence, token) as one dimension of <= 65535
    assert L.iq_decode_multi_workspace_bytes(16383, 4, 16, 2, 256, 128) > 0
    assert L.iq_decode_multi_workspace_bytes(16384, 4, 16, 2, 256, 128) == 0
    assert L.iq_decode_multi_workspace_bytes(32767, 2, 16, 2, 256, 128) > 0
    assert L.iq_decode_multi_workspace_bytes(32768, 2, 16, 2, 256, 128) == 0
    assert call(b=16384, t=4) == 2
    assert call(b=32768, t=2) == 2


def test_step_bits_and_multi_paged_validation():
    """Argument checks of iq_decode_step_bits and iq_decode_attention_multi_paged
    (host side only: nothing is launched on a validation error)."""
    def step(**kw):
        a = dict(dtype=1, b=1, hq=16, hkv=2, cap=256, msl=256, bits=4, wsb=1 << 30)
        a.update(kw)
        return L.iq_decode_step_bits(A, A, A, a["dtype"], A, A, B, B, A, a["cap"], a["msl"], A,
                                     a["b"], a["hq"], a["hkv"], 128, 0.0, A, A, a["wsb"], None,
                                     a["bits"], None)
    assert step(bits=5) == 2
    assert step(dtype=7) == 2
    assert step(hq=34) == 2                      # group 17 > 16
    assert step(cap=250, msl=250) == 2           # capacity not a multiple of 16
    assert step(msl=0) == 1                      # the step needs room for a token
    assert step(wsb=16) == 3
    assert step(b=0) == 0

    def mtp(**kw):
        a = dict(page=64, n_pages=8, max_pages=4, msl=256, b=1, t=3, hq=16, hkv=2, wsb=1 << 30)
        a.update(kw)
        return L.iq_decode_attention_multi_paged(A, A, A, B, B, a["page"], a["n_pages"], A,
                                                 a["max_pages"], A, a["msl"], A, a["b"], a["t"],
                                                 a["hq"], a["hkv"], 128, 0.0, A, A, a["wsb"],
                                                 None)
    assert mtp(t=5) == 2
    assert mtp(page=48) == 1                     # not a power of two
    assert mtp(msl=257) == 1                     # beyond max_pages * page_size
    assert mtp(hq=8) == 2                        # multi-token: group 8 only
    assert mtp(wsb=16) == 3
    assert mtp(b=0) == 0
    assert mtp(b=21846, t=3) == 2               # 65538 (sequence, token) rows


def test_multi_bits_and_multi_step_validation():
    """Argument checks of iq_decode_attention_multi_bits and
    iq_decode_step_multi (host side only: nothing is launched on a
    validation error)."""
    def mb(**kw):
        a = dict(b=1, t=2, hq=16, hkv=2, cap=256, msl=256, bits=2, wsb=1 << 30)
        a.update(kw)
        return L.iq_decode_attention_multi_bits(A, A, A, B, B, A, a["cap"], a["msl"], A, a["b"],
                                                a["t"], a["hq"], a["hkv"], 128, 0.0, A, A,
                                                a["wsb"], a["bits"], None)
    assert mb(bits=5) == 2
    assert mb(bits=1) == 2
    assert mb(t=5) == 2
    assert mb(hq=8) == 2                         # multi-token: group 8 only
    assert mb(cap=250, msl=250) == 2
    assert mb(msl=300) == 1
    assert mb(wsb=16) == 3
    assert mb(b=0) == 0

    def st(**kw):
        a = dict(dtype=1, b=1, t=3, hq=16, hkv=2, cap=256, msl=256, bits=4, wsb=1 << 30,
                 kn=A, st=None)
        a.update(kw)
        return L.iq_decode_step_multi(A, a["kn"], A, a["dtype"], A, A, B, B, A, a["cap"],
                                      a["msl"], A, a["b"], a["t"], a["hq"], a["hkv"], 128, 0.0,
                                      A, A, a["wsb"], a["st"], a["bits"], None)
    assert st(bits=5) == 2
    assert st(dtype=7) == 2
    assert st(t=5) == 2
    assert st(hq=8) == 2
    assert st(cap=250, msl=250) == 2
    assert st(msl=0) == 1                        # the step needs room for its tokens
    assert st(kn=None) == 1
    assert st(kn=ctypes.c_void_p(0x100002)) == 1   # k_new not 16-byte aligned
    assert st(st=ctypes.c_void_p(0x100002)) == 1   # status not 4-byte aligned
    assert st(wsb=16) == 3
    assert st(b=0) == 0
    assert st(b=16384, t=4) == 2                 # 65536 (sequence, token) rows
    # the workspace covers the step's new-token rows: one more row per
    # (sequence, KV head) than the splits
    w = L.iq_decode_multi_workspace_bytes(1, 2, 16, 2, 16, 128)
    assert w >= 2 * 2 * 2 * 8 * 130 * 4


def test_stream_read_validation():
    """Argument checks of the streaming-read measurement kernel."""
    def call(nbytes=4096, sink_words=1 << 20, block=256, loads=4, src=A, sink=A):
        return L.iq_stream_read(src, nbytes, sink, sink_words, block, loads, 0, None)
    assert call(block=96) == 1
    assert call(loads=3) == 1
    assert call(nbytes=4097) == 1
    assert call(nbytes=0) == 0
    assert call(src=None) == 1
    assert L.iq_stream_read_sink_words(4096, 256, 4) == 1
    assert L.iq_stream_read_sink_words(16384 * 3 + 16, 256, 4) == 4
    assert call(nbytes=16384 * 3 + 16, sink_words=3) == 1


def test_caller_codebook_validation():
    """The *_cb entry points reject codebooks the kernels cannot take, before
    any HIP call: levels not fp16 values, not symmetric, not ascending,
    thresholds not the midpoints, unknown widths."""
    from paper_2608_08081_amd import api

    lv, _ = api.iq_codebook_bits(3)

    def compress(cb):
        # called only with codebooks that are rejected (nothing is launched)
        return L.iq_compress_kv_cb(A, B, 1, 1, 2, 16, 128, A, ctypes.byref(cb), A, A, B, B, 16,
                                   0, None)

    def decode(cb):
        # head_dim 64: IQ_ERR_UNSUPPORTED once the codebook has been accepted
        return L.iq_decode_attention_cb(A, A, A, B, B, A, 256, 256, A, ctypes.byref(cb), 1, 16,
                                        2, 64, 0.0, A, A, 1 << 30, None)

    good = api.make_codebook(lv)
    assert decode(good) == 2                      # head_dim 64: the codebook was accepted
    bad_half = api.make_codebook(lv)
    bad_half.levels[7] = 0.1883                   # not an fp16 value
    bad_half.levels[0] = -0.1883
    bad_sym = api.make_codebook(lv * np.array([1, 1, 1, 1, 1, 1, 1, 2], np.float32))
    bad_thr = api.make_codebook(lv)
    bad_thr.thresholds[2] = 0.5 * (bad_thr.thresholds[2] + bad_thr.thresholds[3])
    bad_order = api.make_codebook(lv[[0, 2, 1, 3, 4, 6, 5, 7]])
    big = api.make_codebook(lv * 8)               # |level| >= 1
    for cb in (bad_half, bad_sym, bad_thr, bad_order, big):
        assert compress(cb) == 1
        assert decode(cb) == 1
    width = api.make_codebook(lv)
    width.bits = 5
    assert compress(width) == 2
    assert L.iq_compress_kv_cb(A, B, 1, 1, 2, 16, 128, A, None, A, A, B, B, 16, 0, None) == 1
    # dequantization with a codebook: 3-bit codebooks only
    cb2 = api.make_codebook(api.iq_codebook_bits(2)[0])
    assert L.iq_dequantize_kv_cb(A, A, B, B, A, ctypes.byref(cb2), None, 1, 2, 16, 128, 16, 0, 1,
                                 A, B, None) == 2


def test_fit_codebook_validation():
    from paper_2608_08081_amd import api

    x = np.zeros((2, 5, 128), np.float32)        # only zero vectors: nothing to fit
    q = np.zeros((2, 32, 2, 4), np.float32)
    q[..., 0] = 1.0
    cb = _lib.IqCodebook()
    vp = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    assert L.iq_fit_codebook(vp(x), 5, 2, 128, vp(q), 3, ctypes.byref(cb)) == 1
    assert L.iq_fit_codebook(vp(x), 5, 2, 128, vp(q), 5, ctypes.byref(cb)) == 2
    assert L.iq_fit_codebook(vp(x), 5, 2, 64, vp(q), 3, ctypes.byref(cb)) == 2
    assert L.iq_fit_codebook(vp(x), 0, 2, 128, vp(q), 3, ctypes.byref(cb)) == 1
    x[1, 3, 7] = 1.0                             # one usable vector: a codebook comes out
    assert L.iq_fit_codebook(vp(x), 5, 2, 128, vp(q), 3, ctypes.byref(cb)) == 0
    lv, th = api.codebook_arrays(cb)
    assert np.all(np.diff(lv) > 0) and np.array_equal(lv, -lv[::-1])


def test_rope_decode_validation():
    def call(**kw):
        a = dict(hr=1, rd=64, hq=16, hkv=2, cap=256, msl=256, b=1, qr=A, kr=A)
        a.update(kw)
        return L.iq_decode_attention_rope(A, a["qr"], A, A, a["kr"], a["hr"], B, B, A, a["cap"],
                                          a["msl"], A, a["b"], a["hq"], a["hkv"], 128, a["rd"],
                                          0.0, A, A, 1 << 30, None)
    assert call(rd=32) == 2
    assert call(hr=3) == 1                       # neither shared nor one per KV head
    assert call(qr=None) == 1
    assert call(kr=ctypes.c_void_p(0x100008)) == 1   # not 16-byte aligned
    assert call(cap=250, msl=250) == 2           # capacity not a multiple of 16
    assert call(hq=34) == 2                      # group 17
    assert call(b=0) == 0
