"""Thin PyTorch binding of libisoquant (names follow include/isoquant.h).

Argument marshalling only: tensors are checked for device, dtype, shape and
contiguity (the C library cannot see tensor extents), then their device
pointers and the current HIP stream are handed to the C ABI.  All
compression and attention arithmetic runs in the library's HIP kernels.
"""

from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _lib

HEAD_DIM = 128
RECORD_BYTES = 48


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _require(t, name, dtype, shape, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _dtype_code(t):
    if t.dtype == torch.float16:
        return _lib.IQ_DTYPE_F16
    if t.dtype == torch.float32:
        return _lib.IQ_DTYPE_F32
    raise TypeError(f"unsupported K/V dtype {t.dtype} (float16 or float32)")


# ---------------------------------------------------------------------------
# host-side entry points
# ---------------------------------------------------------------------------

def iq_codebook():
    """(levels[8], thresholds[7]) as float32 numpy arrays."""
    lv = np.zeros(8, np.float32)
    th = np.zeros(7, np.float32)
    _lib.check("iq_codebook", _lib.lib().iq_codebook(lv.ctypes.data_as(ctypes.c_void_p),
                                                     th.ctypes.data_as(ctypes.c_void_p)))
    return lv, th


def iq_codebook_bits(bits: int):
    """C_b: (levels[2^b], thresholds[2^b - 1]) as float32 numpy arrays."""
    n = 1 << bits
    lv = np.zeros(n, np.float32)
    th = np.zeros(n - 1, np.float32)
    _lib.check("iq_codebook_bits",
               _lib.lib().iq_codebook_bits(bits, lv.ctypes.data_as(ctypes.c_void_p),
                                           th.ctypes.data_as(ctypes.c_void_p)))
    return lv, th


def make_codebook(levels, thresholds=None):
    """An iq_codebook_t from 2^b levels (thresholds default to the fp32
    midpoints of adjacent levels).  The library validates it on use."""
    lv = np.asarray(levels, dtype=np.float64)
    n = lv.size
    bits = {4: 2, 8: 3, 16: 4}.get(n)
    if bits is None:
        raise ValueError("a codebook has 4, 8 or 16 levels")
    th = (0.5 * (lv[:-1] + lv[1:]) if thresholds is None
          else np.asarray(thresholds, dtype=np.float64))
    cb = _lib.IqCodebook()
    cb.bits = bits
    for i in range(n):
        cb.levels[i] = float(np.float32(lv[i]))
    for i in range(n - 1):
        cb.thresholds[i] = float(np.float32(th[i]))
    return cb


def codebook_arrays(cb):
    """(levels, thresholds) of an iq_codebook_t as float32 numpy arrays."""
    n = 1 << cb.bits
    return (np.array(cb.levels[:n], dtype=np.float32),
            np.array(cb.thresholds[:n - 1], dtype=np.float32))


def iq_fit_codebook(calib, quats, bits: int = 3):
    """Codebook fitted to calibration vectors (host fp32 [n_kv_heads][n][128])
    rotated with the parameters quats ([n_kv_heads][32][2][4])."""
    x = np.ascontiguousarray(np.asarray(calib.cpu() if hasattr(calib, "cpu") else calib,
                                        dtype=np.float32))
    qh = np.ascontiguousarray(np.asarray(quats.cpu() if hasattr(quats, "cpu") else quats,
                                         dtype=np.float32))
    if x.ndim != 3 or x.shape[2] != HEAD_DIM or qh.shape != (x.shape[0], 32, 2, 4):
        raise ValueError("calib must be [n_kv_heads][n_vectors][128], quats [n_kv_heads][32][2][4]")
    cb = _lib.IqCodebook()
    _lib.check("iq_fit_codebook", _lib.lib().iq_fit_codebook(
        x.ctypes.data_as(ctypes.c_void_p), x.shape[1], x.shape[0], HEAD_DIM,
        qh.ctypes.data_as(ctypes.c_void_p), bits, ctypes.byref(cb)))
    return cb


def record_bytes(bits: int = 3) -> int:
    """Bytes of one packed record of 128 b-bit codes."""
    return HEAD_DIM * bits // 8


def iq_make_rotation(seed: int, n_kv_heads: int) -> torch.Tensor:
    """Seeded SO(4) parameters, host float32 tensor [n_kv_heads][32][2][4]."""
    out = np.zeros((n_kv_heads, 32, 2, 4), np.float32)
    _lib.check("iq_make_rotation", _lib.lib().iq_make_rotation(
        seed & ((1 << 64) - 1), n_kv_heads, HEAD_DIM, out.ctypes.data_as(ctypes.c_void_p)))
    return torch.from_numpy(out)


ROTATION_VARIANTS = {"so4": 0, "so3": 1, "wht_only": 2}


def iq_make_rotation_variant(seed: int, n_kv_heads: int, variant: str) -> torch.Tensor:
    """Parameters of one rotation design of the ablation that keeps the
    R_blocks H_128 form ("so4" = the method, "so3" = single-quaternion
    blocks, "wht_only" = identity blocks), host float32 [n_kv_heads][32][2][4]."""
    out = np.zeros((n_kv_heads, 32, 2, 4), np.float32)
    _lib.check("iq_make_rotation_variant", _lib.lib().iq_make_rotation_variant(
        seed & ((1 << 64) - 1), n_kv_heads, HEAD_DIM, ROTATION_VARIANTS[variant],
        out.ctypes.data_as(ctypes.c_void_p)))
    return torch.from_numpy(out)


def iq_fit_rotation(calib, sweeps: int = 4) -> torch.Tensor:
    """Fitted SO(4) block parameters from calibration vectors (host fp32
    [n_kv_heads][n_vectors][128], a tensor or array): host float32
    [n_kv_heads][32][2][4] in the layout of iq_make_rotation."""
    x = np.ascontiguousarray(np.asarray(calib.cpu() if hasattr(calib, "cpu") else calib,
                                        dtype=np.float32))
    if x.ndim != 3 or x.shape[2] != HEAD_DIM:
        raise ValueError("calib must be [n_kv_heads][n_vectors][128]")
    out = np.zeros((x.shape[0], 32, 2, 4), np.float32)
    _lib.check("iq_fit_rotation", _lib.lib().iq_fit_rotation(
        x.ctypes.data_as(ctypes.c_void_p), x.shape[1], x.shape[0], HEAD_DIM, sweeps,
        out.ctypes.data_as(ctypes.c_void_p)))
    return torch.from_numpy(out)


def iq_so4_to_quaternions(m) -> np.ndarray:
    """(q_L, q_R) of a 4 x 4 rotation (fp64): float32 [2][4]."""
    a = np.ascontiguousarray(np.asarray(m, dtype=np.float64))
    if a.shape != (4, 4):
        raise ValueError("m must be 4 x 4")
    out = np.zeros((2, 4), np.float32)
    _lib.check("iq_so4_to_quaternions", _lib.lib().iq_so4_to_quaternions(
        a.ctypes.data_as(ctypes.c_void_p), out.ctypes.data_as(ctypes.c_void_p)))
    return out


def iq_decode_workspace_bytes(batch, n_q_heads, n_kv_heads, max_seq_len) -> int:
    return int(_lib.lib().iq_decode_workspace_bytes(batch, n_q_heads, n_kv_heads,
                                                    max_seq_len, HEAD_DIM))


# ---------------------------------------------------------------------------
# device entry points
# ---------------------------------------------------------------------------

def alloc_cache(batch, n_kv_heads, capacity, device, values=True, bits: int = 3):
    """Zero-filled packed cache buffers for one layer: dict with k_codes,
    k_norms (and v_codes, v_norms), plus seq_lens (int32 zeros); records of
    16 * bits bytes."""
    c = {
        "k_codes": torch.zeros((batch, n_kv_heads, capacity, record_bytes(bits)),
                               dtype=torch.uint8, device=device),
        "k_norms": torch.zeros((batch, n_kv_heads, capacity), dtype=torch.float32, device=device),
        "seq_lens": torch.zeros(batch, dtype=torch.int32, device=device),
    }
    if values:
        c["v_codes"] = torch.zeros_like(c["k_codes"])
        c["v_norms"] = torch.zeros_like(c["k_norms"])
    return c


def iq_compress_kv(k, v, quats, k_codes=None, k_norms=None, v_codes=None, v_norms=None,
                   dst_offset: int = 0):
    """Algorithm 1 over a block of tokens: k, v [B][H][T][128] (f16 or f32,
    either may be None) written into the caches at positions dst_offset.."""
    _compress(k, v, quats, k_codes, k_norms, v_codes, v_norms, dst_offset, 3)


def iq_compress_kv_bits(k, v, quats, k_codes=None, k_norms=None, v_codes=None, v_norms=None,
                        dst_offset: int = 0, bits: int = 3):
    """iq_compress_kv to b-bit records (k_codes / v_codes [B][H][cap][16 b])."""
    _compress(k, v, quats, k_codes, k_norms, v_codes, v_norms, dst_offset, bits)


def iq_compress_kv_cb(k, v, quats, codebook, k_codes=None, k_norms=None, v_codes=None,
                      v_norms=None, dst_offset: int = 0):
    """iq_compress_kv with a caller codebook (records of codebook.bits bits)."""
    _compress(k, v, quats, k_codes, k_norms, v_codes, v_norms, dst_offset, codebook.bits,
              codebook)


def _compress(k, v, quats, k_codes, k_norms, v_codes, v_norms, dst_offset, bits,
              codebook=None):
    src = k if k is not None else v
    if src is None:
        raise ValueError("k and v are both None")
    if src.dim() != 4 or src.shape[-1] != HEAD_DIM:
        raise ValueError("k/v must be [batch][n_kv_heads][n_tokens][128]")
    b, h, t, _ = src.shape
    dev = src.device
    codes_ref = k_codes if k is not None else v_codes
    if codes_ref is None:
        raise ValueError("missing output cache")
    cap = codes_ref.shape[2]
    _require(quats, "quats", torch.float32, (h, 32, 2, 4), dev)
    for name, x, codes, norms in (("k", k, k_codes, k_norms), ("v", v, v_codes, v_norms)):
        if x is None:
            continue
        _require(x, name, src.dtype, (b, h, t, HEAD_DIM), dev)
        _require(codes, f"{name}_codes", torch.uint8, (b, h, cap, record_bytes(bits)), dev)
        _require(norms, f"{name}_norms", torch.float32, (b, h, cap), dev)
    outs = (_ptr(k_codes) if k is not None else None, _ptr(k_norms) if k is not None else None,
            _ptr(v_codes) if v is not None else None, _ptr(v_norms) if v is not None else None,
            cap, dst_offset)
    args = (_ptr(k), _ptr(v), _dtype_code(src), b, h, t, HEAD_DIM, _ptr(quats)) + outs
    if codebook is not None:
        _lib.check("iq_compress_kv_cb", _lib.lib().iq_compress_kv_cb(
            *args[:8], ctypes.byref(codebook), *outs, _stream(dev)))
    elif bits == 3:
        _lib.check("iq_compress_kv", _lib.lib().iq_compress_kv(*args, _stream(dev)))
    else:
        _lib.check("iq_compress_kv_bits",
                   _lib.lib().iq_compress_kv_bits(*args, bits, _stream(dev)))


def iq_append_token(k_new, v_new, quats, k_codes, k_norms, v_codes, v_norms, seq_lens,
                    status=None):
    """Compress one new token per sequence (k_new, v_new: [B][H][128]) into
    position seq_lens[b] and increment seq_lens in place."""
    src = k_new if k_new is not None else v_new
    if src is None:
        raise ValueError("k_new and v_new are both None")
    b, h, _ = src.shape
    dev = src.device
    codes_ref = k_codes if k_new is not None else v_codes
    cap = codes_ref.shape[2]
    _require(quats, "quats", torch.float32, (h, 32, 2, 4), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    if status is not None:
        _require(status, "status", torch.int32, (1,), dev)
    for name, x, codes, norms in (("k_new", k_new, k_codes, k_norms),
                                  ("v_new", v_new, v_codes, v_norms)):
        if x is None:
            continue
        _require(x, name, src.dtype, (b, h, HEAD_DIM), dev)
        _require(codes, f"{name}_codes", torch.uint8, (b, h, cap, RECORD_BYTES), dev)
        _require(norms, f"{name}_norms", torch.float32, (b, h, cap), dev)
    st = _lib.lib().iq_append_token(
        _ptr(k_new), _ptr(v_new), _dtype_code(src), b, h, HEAD_DIM, _ptr(quats),
        _ptr(k_codes) if k_new is not None else None,
        _ptr(k_norms) if k_new is not None else None,
        _ptr(v_codes) if v_new is not None else None,
        _ptr(v_norms) if v_new is not None else None,
        cap, _ptr(seq_lens), _ptr(status), _stream(dev))
    _lib.check("iq_append_token", st)


def iq_decode_workspace_init(workspace):
    st = _lib.lib().iq_decode_workspace_init(_ptr(workspace), workspace.numel() *
                                             workspace.element_size(), _stream(workspace.device))
    _lib.check("iq_decode_workspace_init", st)


def alloc_workspace(batch, n_q_heads, n_kv_heads, max_seq_len, device):
    nbytes = iq_decode_workspace_bytes(batch, n_q_heads, n_kv_heads, max_seq_len)
    if nbytes <= 0:
        raise ValueError("unsupported decode shape")
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    iq_decode_workspace_init(ws)
    return ws


def iq_decode_attention(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out=None,
                        workspace=None, max_seq_len=None, softmax_scale: float = 0.0):
    """Decode attention on the packed cache.  q: [B][H_q][128] fp32 (original
    space); returns out [B][H_q][128] fp32 (original space)."""
    return _decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out, workspace,
                   max_seq_len, softmax_scale, 3)


def iq_decode_attention_bits(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out=None,
                             workspace=None, max_seq_len=None, softmax_scale: float = 0.0,
                             bits: int = 3):
    """iq_decode_attention on b-bit records ([B][H_kv][cap][16 b])."""
    return _decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out, workspace,
                   max_seq_len, softmax_scale, bits)


def iq_decode_attention_cb(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, codebook,
                           out=None, workspace=None, max_seq_len=None,
                           softmax_scale: float = 0.0):
    """iq_decode_attention on records written with a caller codebook."""
    return _decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out, workspace,
                   max_seq_len, softmax_scale, codebook.bits, codebook)


def _decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out, workspace,
            max_seq_len, softmax_scale, bits, codebook=None):
    if q.dim() != 3 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_q_heads][128]")
    b, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, hq, HEAD_DIM), dev)
    if k_codes.dim() != 4:
        raise ValueError("k_codes must be [batch][n_kv_heads][capacity][16 * bits]")
    _, hkv, cap, _ = k_codes.shape
    _require(k_codes, "k_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(v_codes, "v_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(k_norms, "k_norms", torch.float32, (b, hkv, cap), dev)
    _require(v_norms, "v_norms", torch.float32, (b, hkv, cap), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if max_seq_len is None:
        max_seq_len = cap
    if out is None:
        out = torch.empty((b, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    if workspace is None:
        workspace = alloc_workspace(b, hq, hkv, max_seq_len, dev)
    if workspace.dtype != torch.uint8 or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    args = (_ptr(q), _ptr(k_codes), _ptr(k_norms), _ptr(v_codes), _ptr(v_norms), _ptr(seq_lens),
            cap, max_seq_len, _ptr(quats), b, hq, hkv, HEAD_DIM, float(softmax_scale), _ptr(out),
            _ptr(workspace), workspace.numel())
    if codebook is not None:
        _lib.check("iq_decode_attention_cb", _lib.lib().iq_decode_attention_cb(
            *args[:9], ctypes.byref(codebook), *args[9:], _stream(dev)))
    elif bits == 3:
        _lib.check("iq_decode_attention", _lib.lib().iq_decode_attention(*args, _stream(dev)))
    else:
        _lib.check("iq_decode_attention_bits",
                   _lib.lib().iq_decode_attention_bits(*args, bits, _stream(dev)))
    return out


def iq_decode_attention_rope(q, q_rope, k_codes, k_norms, k_rope, v_codes, v_norms, seq_lens,
                             quats, out=None, workspace=None, max_seq_len=None,
                             softmax_scale: float = 0.0):
    """Decode with the content / RoPE sub-block split: q [B][H_q][128] and
    q_rope [B][H_q][64] fp32; the compressed content cache; k_rope fp16
    [B][1 or H_kv][cap][64] (stored as given).  Returns out [B][H_q][128]."""
    if q.dim() != 3 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_q_heads][128]")
    b, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, hq, HEAD_DIM), dev)
    _require(q_rope, "q_rope", torch.float32, (b, hq, 64), dev)
    if k_codes.dim() != 4 or k_rope.dim() != 4:
        raise ValueError("k_codes must be [batch][n_kv_heads][capacity][48], "
                         "k_rope [batch][n_rope_heads][capacity][64]")
    _, hkv, cap, _ = k_codes.shape
    hr = k_rope.shape[1]
    _require(k_codes, "k_codes", torch.uint8, (b, hkv, cap, RECORD_BYTES), dev)
    _require(v_codes, "v_codes", torch.uint8, (b, hkv, cap, RECORD_BYTES), dev)
    _require(k_norms, "k_norms", torch.float32, (b, hkv, cap), dev)
    _require(v_norms, "v_norms", torch.float32, (b, hkv, cap), dev)
    _require(k_rope, "k_rope", torch.float16, (b, hr, cap, 64), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if max_seq_len is None:
        max_seq_len = cap
    if out is None:
        out = torch.empty((b, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    if workspace is None:
        workspace = alloc_workspace(b, hq, hkv, max_seq_len, dev)
    st = _lib.lib().iq_decode_attention_rope(
        _ptr(q), _ptr(q_rope), _ptr(k_codes), _ptr(k_norms), _ptr(k_rope), hr, _ptr(v_codes),
        _ptr(v_norms), _ptr(seq_lens), cap, max_seq_len, _ptr(quats), b, hq, hkv, HEAD_DIM, 64,
        float(softmax_scale), _ptr(out), _ptr(workspace), workspace.numel(), _stream(dev))
    _lib.check("iq_decode_attention_rope", st)
    return out


def iq_decode_multi_workspace_bytes(batch, n_tokens, n_q_heads, n_kv_heads, max_seq_len) -> int:
    return int(_lib.lib().iq_decode_multi_workspace_bytes(batch, n_tokens, n_q_heads, n_kv_heads,
                                                          max_seq_len, HEAD_DIM))


def iq_decode_attention_multi(q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out=None,
                              workspace=None, max_seq_len=None, softmax_scale: float = 0.0,
                              bits: int = 3):
    """Multi-token decode: q [B][T][H_q][128] fp32 (T = 1..4 query tokens per
    sequence, the last T of its seq_lens[b] cached positions; token t attends
    positions before seq_lens[b] - T + 1 + t) on b-bit records
    ([B][H_kv][cap][16 b]).  Returns out [B][T][H_q][128]."""
    if q.dim() != 4 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_tokens][n_q_heads][128]")
    b, t, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, t, hq, HEAD_DIM), dev)
    if k_codes.dim() != 4:
        raise ValueError("k_codes must be [batch][n_kv_heads][capacity][16 bits]")
    _, hkv, cap, _ = k_codes.shape
    _require(k_codes, "k_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(v_codes, "v_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(k_norms, "k_norms", torch.float32, (b, hkv, cap), dev)
    _require(v_norms, "v_norms", torch.float32, (b, hkv, cap), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if max_seq_len is None:
        max_seq_len = cap
    if out is None:
        out = torch.empty((b, t, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, t, hq, HEAD_DIM), dev)
    if workspace is None:
        nbytes = iq_decode_multi_workspace_bytes(b, t, hq, hkv, max_seq_len)
        if nbytes <= 0:
            raise ValueError("unsupported multi-token decode shape")
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    if workspace.dtype != torch.uint8 or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    args = (_ptr(q), _ptr(k_codes), _ptr(k_norms), _ptr(v_codes), _ptr(v_norms), _ptr(seq_lens),
            cap, max_seq_len, _ptr(quats), b, t, hq, hkv, HEAD_DIM, float(softmax_scale))
    tail = (_ptr(out), _ptr(workspace), workspace.numel(), _stream(dev))
    if bits == 3:
        _lib.check("iq_decode_attention_multi",
                   _lib.lib().iq_decode_attention_multi(*args, *tail))
    else:
        _lib.check("iq_decode_attention_multi_bits",
                   _lib.lib().iq_decode_attention_multi_bits(*args, *tail[:3], bits, tail[3]))
    return out


def iq_decode_step_multi(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats,
                         out=None, workspace=None, max_seq_len=None, softmax_scale: float = 0.0,
                         status=None, bits: int = 3):
    """Fused multi-token step: append the T new tokens (k_new, v_new
    [B][T][H_kv][128], fp16 or fp32) at positions seq_lens[b] .. + T - 1 as
    b-bit records, attend q [B][T][H_q][128] (token t: the cached positions
    and new positions 0 .. t) and advance seq_lens by T in place.  Returns
    out [B][T][H_q][128] fp32 (original space)."""
    if q.dim() != 4 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_tokens][n_q_heads][128]")
    b, t, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, t, hq, HEAD_DIM), dev)
    if k_codes.dim() != 4:
        raise ValueError("k_codes must be [batch][n_kv_heads][capacity][16 bits]")
    _, hkv, cap, _ = k_codes.shape
    _require(k_new, "k_new", k_new.dtype, (b, t, hkv, HEAD_DIM), dev)
    _require(v_new, "v_new", k_new.dtype, (b, t, hkv, HEAD_DIM), dev)
    _require(k_codes, "k_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(v_codes, "v_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(k_norms, "k_norms", torch.float32, (b, hkv, cap), dev)
    _require(v_norms, "v_norms", torch.float32, (b, hkv, cap), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if status is not None:
        _require(status, "status", torch.int32, (1,), dev)
    if max_seq_len is None:
        max_seq_len = cap
    if out is None:
        out = torch.empty((b, t, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, t, hq, HEAD_DIM), dev)
    if workspace is None:
        nbytes = iq_decode_multi_workspace_bytes(b, t, hq, hkv, max_seq_len)
        if nbytes <= 0:
            raise ValueError("unsupported multi-token step shape")
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    if workspace.dtype != torch.uint8 or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    st = _lib.lib().iq_decode_step_multi(
        _ptr(q), _ptr(k_new), _ptr(v_new), _dtype_code(k_new), _ptr(k_codes), _ptr(k_norms),
        _ptr(v_codes), _ptr(v_norms), _ptr(seq_lens), cap, max_seq_len, _ptr(quats), b, t, hq,
        hkv, HEAD_DIM, float(softmax_scale), _ptr(out), _ptr(workspace), workspace.numel(),
        _ptr(status), bits, _stream(dev))
    _lib.check("iq_decode_step_multi", st)
    return out


def iq_decode_step(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats,
                   out=None, workspace=None, max_seq_len=None, softmax_scale: float = 0.0,
                   status=None):
    """Fused decode step: append (k_new, v_new) [B][H_kv][128] at position
    seq_lens[b], attend q [B][H_q][128] over the advanced lengths and advance
    seq_lens in place.  Returns out [B][H_q][128] fp32 (original space)."""
    return _step(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out,
                 workspace, max_seq_len, softmax_scale, status, 3)


def iq_decode_step_noalloc(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens,
                           quats, out, max_seq_len=None, softmax_scale: float = 0.0,
                           status=None):
    """iq_decode_step with its split partials in the library's static device
    scratch (no workspace; nothing allocated by the call, `out` is the
    caller's).  Shapes whose workspace exceeds the scratch raise."""
    b, hq, hkv, cap = _step_shapes(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms,
                                   seq_lens, quats, status, 3)
    dev = q.device
    if max_seq_len is None:
        max_seq_len = cap
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    st = _lib.lib().iq_decode_step_noalloc(
        _ptr(q), _ptr(k_new), _ptr(v_new), _dtype_code(k_new), _ptr(k_codes), _ptr(k_norms),
        _ptr(v_codes), _ptr(v_norms), _ptr(seq_lens), cap, max_seq_len, _ptr(quats), b, hq, hkv,
        HEAD_DIM, float(softmax_scale), _ptr(out), _ptr(status), _stream(dev))
    _lib.check("iq_decode_step_noalloc", st)
    return out


def iq_decode_step_bits(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats,
                        out=None, workspace=None, max_seq_len=None, softmax_scale: float = 0.0,
                        status=None, bits: int = 3):
    """iq_decode_step on b-bit records ([B][H_kv][cap][16 b])."""
    return _step(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out,
                 workspace, max_seq_len, softmax_scale, status, bits)


def _step_shapes(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, status,
                 bits):
    """Checks of a fused step's tensors; returns (batch, n_q_heads,
    n_kv_heads, capacity)."""
    if q.dim() != 3 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_q_heads][128]")
    b, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, hq, HEAD_DIM), dev)
    if k_codes.dim() != 4:
        raise ValueError("k_codes must be [batch][n_kv_heads][capacity][48]")
    _, hkv, cap, _ = k_codes.shape
    _require(k_new, "k_new", k_new.dtype, (b, hkv, HEAD_DIM), dev)
    _require(v_new, "v_new", k_new.dtype, (b, hkv, HEAD_DIM), dev)
    _require(k_codes, "k_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(v_codes, "v_codes", torch.uint8, (b, hkv, cap, record_bytes(bits)), dev)
    _require(k_norms, "k_norms", torch.float32, (b, hkv, cap), dev)
    _require(v_norms, "v_norms", torch.float32, (b, hkv, cap), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if status is not None:
        _require(status, "status", torch.int32, (1,), dev)
    return b, hq, hkv, cap


def iq_decode_step_cb(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats,
                      codebook, out=None, workspace=None, max_seq_len=None,
                      softmax_scale: float = 0.0, status=None):
    """iq_decode_step with a caller codebook for the new records and the
    attention."""
    return _step(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out,
                 workspace, max_seq_len, softmax_scale, status, codebook.bits, codebook)


def _step(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, out, workspace,
          max_seq_len, softmax_scale, status, bits, codebook=None):
    b, hq, hkv, cap = _step_shapes(q, k_new, v_new, k_codes, k_norms, v_codes, v_norms,
                                   seq_lens, quats, status, bits)
    dev = q.device
    if max_seq_len is None:
        max_seq_len = cap
    if out is None:
        out = torch.empty((b, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    if workspace is None:
        workspace = alloc_workspace(b, hq, hkv, max_seq_len, dev)
    if workspace.dtype != torch.uint8 or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    args = (_ptr(q), _ptr(k_new), _ptr(v_new), _dtype_code(k_new), _ptr(k_codes), _ptr(k_norms),
            _ptr(v_codes), _ptr(v_norms), _ptr(seq_lens), cap, max_seq_len, _ptr(quats), b, hq,
            hkv, HEAD_DIM, float(softmax_scale), _ptr(out), _ptr(workspace), workspace.numel(),
            _ptr(status))
    if codebook is not None:
        _lib.check("iq_decode_step_cb", _lib.lib().iq_decode_step_cb(
            *args[:12], ctypes.byref(codebook), *args[12:], _stream(dev)))
    elif bits == 3:
        _lib.check("iq_decode_step", _lib.lib().iq_decode_step(*args, _stream(dev)))
    else:
        _lib.check("iq_decode_step_bits",
                   _lib.lib().iq_decode_step_bits(*args, bits, _stream(dev)))
    return out


# ---------------------------------------------------------------------------
# paged cache (page pools shared by all sequences + per-sequence page tables)
# ---------------------------------------------------------------------------

def alloc_paged_cache(n_pages, n_kv_heads, page_size, device):
    """Zero-filled page pools: dict with k_codes / v_codes
    [n_pages][n_kv_heads][page_size][48] uint8 and k_norms / v_norms
    [n_pages][n_kv_heads][page_size] fp32."""
    c = {}
    for side in ("k", "v"):
        c[f"{side}_codes"] = torch.zeros((n_pages, n_kv_heads, page_size, RECORD_BYTES),
                                         dtype=torch.uint8, device=device)
        c[f"{side}_norms"] = torch.zeros((n_pages, n_kv_heads, page_size), dtype=torch.float32,
                                         device=device)
    return c


def _paged_pools(pool, block_tables, dev):
    if pool["k_codes"].dim() != 4:
        raise ValueError("k_codes must be [n_pages][n_kv_heads][page_size][48]")
    n_pages, hkv, page, _ = pool["k_codes"].shape
    for side in ("k", "v"):
        if pool.get(f"{side}_codes") is None:
            continue
        _require(pool[f"{side}_codes"], f"{side}_codes", torch.uint8,
                 (n_pages, hkv, page, RECORD_BYTES), dev)
        _require(pool[f"{side}_norms"], f"{side}_norms", torch.float32, (n_pages, hkv, page),
                 dev)
    if block_tables.dim() != 2:
        raise ValueError("block_tables must be [batch][max_pages]")
    _require(block_tables, "block_tables", torch.int32, tuple(block_tables.shape), dev)
    return n_pages, hkv, page, block_tables.shape[1]


def iq_compress_kv_paged(k, v, quats, pool, block_tables, dst_offset: int = 0):
    """iq_compress_kv into page pools (dict from alloc_paged_cache): k / v
    [B][H_kv][T][128] (fp16 or fp32; either may be None) to logical positions
    dst_offset .. dst_offset + T - 1 of every sequence."""
    src = k if k is not None else v
    if src is None:
        raise ValueError("k and v are both None")
    b, hkv, t, _ = src.shape
    dev = src.device
    n_pages, phkv, page, max_pages = _paged_pools(pool, block_tables, dev)
    if phkv != hkv or block_tables.shape[0] != b:
        raise ValueError("pools / block_tables do not match the inputs")
    for x, name in ((k, "k"), (v, "v")):
        if x is not None:
            _require(x, name, src.dtype, (b, hkv, t, HEAD_DIM), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    st = _lib.lib().iq_compress_kv_paged(
        _ptr(k), _ptr(v), _dtype_code(src), b, hkv, t, HEAD_DIM, _ptr(quats),
        _ptr(pool["k_codes"]) if k is not None else None,
        _ptr(pool["k_norms"]) if k is not None else None,
        _ptr(pool["v_codes"]) if v is not None else None,
        _ptr(pool["v_norms"]) if v is not None else None,
        page, n_pages, _ptr(block_tables), max_pages, dst_offset, _stream(dev))
    _lib.check("iq_compress_kv_paged", st)


def iq_decode_attention_paged(q, pool, block_tables, seq_lens, quats, out=None,
                              workspace=None, max_seq_len=None, softmax_scale: float = 0.0):
    """iq_decode_attention on page pools; q [B][8 H_kv][128]."""
    b, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, hq, HEAD_DIM), dev)
    n_pages, hkv, page, max_pages = _paged_pools(pool, block_tables, dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if max_seq_len is None:
        max_seq_len = max_pages * page
    if out is None:
        out = torch.empty((b, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    if workspace is None:
        workspace = alloc_workspace(b, hq, hkv, max_seq_len, dev)
    st = _lib.lib().iq_decode_attention_paged(
        _ptr(q), _ptr(pool["k_codes"]), _ptr(pool["k_norms"]), _ptr(pool["v_codes"]),
        _ptr(pool["v_norms"]), page, n_pages, _ptr(block_tables), max_pages, _ptr(seq_lens),
        max_seq_len, _ptr(quats), b, hq, hkv, HEAD_DIM, float(softmax_scale), _ptr(out),
        _ptr(workspace), workspace.numel(), _stream(dev))
    _lib.check("iq_decode_attention_paged", st)
    return out


def iq_decode_step_paged(q, k_new, v_new, pool, block_tables, seq_lens, quats, out=None,
                         workspace=None, max_seq_len=None, softmax_scale: float = 0.0,
                         status=None):
    """iq_decode_step on page pools: the new token goes to logical position
    seq_lens[b] (its page must be mapped in block_tables)."""
    b, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, hq, HEAD_DIM), dev)
    n_pages, hkv, page, max_pages = _paged_pools(pool, block_tables, dev)
    _require(k_new, "k_new", k_new.dtype, (b, hkv, HEAD_DIM), dev)
    _require(v_new, "v_new", k_new.dtype, (b, hkv, HEAD_DIM), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if status is not None:
        _require(status, "status", torch.int32, (1,), dev)
    if max_seq_len is None:
        max_seq_len = max_pages * page
    if out is None:
        out = torch.empty((b, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    if workspace is None:
        workspace = alloc_workspace(b, hq, hkv, max_seq_len, dev)
    st = _lib.lib().iq_decode_step_paged(
        _ptr(q), _ptr(k_new), _ptr(v_new), _dtype_code(k_new), _ptr(pool["k_codes"]),
        _ptr(pool["k_norms"]), _ptr(pool["v_codes"]), _ptr(pool["v_norms"]), page, n_pages,
        _ptr(block_tables), max_pages, _ptr(seq_lens), max_seq_len, _ptr(quats), b, hq, hkv,
        HEAD_DIM, float(softmax_scale), _ptr(out), _ptr(workspace), workspace.numel(),
        _ptr(status), _stream(dev))
    _lib.check("iq_decode_step_paged", st)
    return out


def iq_decode_attention_multi_paged(q, pool, block_tables, seq_lens, quats, out=None,
                                    workspace=None, max_seq_len=None,
                                    softmax_scale: float = 0.0):
    """iq_decode_attention_multi on page pools; q [B][T][8 H_kv][128]."""
    if q.dim() != 4 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_tokens][n_q_heads][128]")
    b, t, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, t, hq, HEAD_DIM), dev)
    n_pages, hkv, page, max_pages = _paged_pools(pool, block_tables, dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if max_seq_len is None:
        max_seq_len = max_pages * page
    if out is None:
        out = torch.empty((b, t, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, t, hq, HEAD_DIM), dev)
    if workspace is None:
        nbytes = iq_decode_multi_workspace_bytes(b, t, hq, hkv, max_seq_len)
        if nbytes <= 0:
            raise ValueError("unsupported multi-token decode shape")
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    st = _lib.lib().iq_decode_attention_multi_paged(
        _ptr(q), _ptr(pool["k_codes"]), _ptr(pool["k_norms"]), _ptr(pool["v_codes"]),
        _ptr(pool["v_norms"]), page, n_pages, _ptr(block_tables), max_pages, _ptr(seq_lens),
        max_seq_len, _ptr(quats), b, t, hq, hkv, HEAD_DIM, float(softmax_scale), _ptr(out),
        _ptr(workspace), workspace.numel(), _stream(dev))
    _lib.check("iq_decode_attention_multi_paged", st)
    return out


# ---------------------------------------------------------------------------
# reconstruct-then-compute baseline (materialized fp16 cache)
# ---------------------------------------------------------------------------

def iq_dequantize_kv_cb(k_codes, k_norms, v_codes, v_norms, quats, codebook, n_tokens=None,
                        src_offset: int = 0, seq_lens=None, out_dtype=torch.float16,
                        k_out=None, v_out=None):
    """iq_dequantize_kv of records written with a caller (3-bit) codebook."""
    return iq_dequantize_kv(k_codes, k_norms, v_codes, v_norms, quats, n_tokens, src_offset,
                            seq_lens, out_dtype, k_out, v_out, codebook=codebook)


def iq_dequantize_kv(k_codes, k_norms, v_codes, v_norms, quats, n_tokens=None,
                     src_offset: int = 0, seq_lens=None, out_dtype=torch.float16,
                     k_out=None, v_out=None, codebook=None):
    """Materialize cache positions src_offset .. src_offset + n_tokens - 1 as
    original-space vectors [B][H_kv][n_tokens][128] of out_dtype (fp16 or
    fp32).  Either side may be None.  With seq_lens, tokens at or past a
    sequence's length are not written.  Returns (k_out, v_out)."""
    ref = k_codes if k_codes is not None else v_codes
    if ref is None or ref.dim() != 4:
        raise ValueError("codes must be [batch][n_kv_heads][capacity][48]")
    b, hkv, cap, _ = ref.shape
    dev = ref.device
    if n_tokens is None:
        n_tokens = cap - src_offset
    if out_dtype not in (torch.float16, torch.float32):
        raise TypeError("out_dtype must be torch.float16 or torch.float32")
    shape = (b, hkv, n_tokens, HEAD_DIM)
    outs = []
    for codes, norms, out, name in ((k_codes, k_norms, k_out, "k"), (v_codes, v_norms, v_out, "v")):
        if codes is None:
            outs.append(None)
            continue
        _require(codes, f"{name}_codes", torch.uint8, (b, hkv, cap, RECORD_BYTES), dev)
        _require(norms, f"{name}_norms", torch.float32, (b, hkv, cap), dev)
        if out is None:
            out = torch.empty(shape, dtype=out_dtype, device=dev)
        _require(out, f"{name}_out", out_dtype, shape, dev)
        outs.append(out)
    _require(quats, "quats", torch.float32, (hkv, 32, 2, 4), dev)
    if seq_lens is not None:
        _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    code = _lib.IQ_DTYPE_F16 if out_dtype == torch.float16 else _lib.IQ_DTYPE_F32
    if codebook is not None:
        st = _lib.lib().iq_dequantize_kv_cb(
            _ptr(k_codes), _ptr(k_norms), _ptr(v_codes), _ptr(v_norms), _ptr(quats),
            ctypes.byref(codebook), _ptr(seq_lens), b, hkv, n_tokens, HEAD_DIM, cap, src_offset,
            code, _ptr(outs[0]), _ptr(outs[1]), _stream(dev))
        _lib.check("iq_dequantize_kv_cb", st)
        return outs[0], outs[1]
    st = _lib.lib().iq_dequantize_kv(
        _ptr(k_codes), _ptr(k_norms), _ptr(v_codes), _ptr(v_norms), _ptr(quats), _ptr(seq_lens),
        b, hkv, n_tokens, HEAD_DIM, cap, src_offset, code, _ptr(outs[0]), _ptr(outs[1]),
        _stream(dev))
    _lib.check("iq_dequantize_kv", st)
    return outs[0], outs[1]


def iq_decode_f16_workspace_bytes(batch, n_q_heads, n_kv_heads, max_seq_len) -> int:
    return int(_lib.lib().iq_decode_f16_workspace_bytes(batch, n_q_heads, n_kv_heads,
                                                        max_seq_len, HEAD_DIM))


def alloc_f16_workspace(batch, n_q_heads, n_kv_heads, max_seq_len, device):
    nbytes = iq_decode_f16_workspace_bytes(batch, n_q_heads, n_kv_heads, max_seq_len)
    if nbytes <= 0:
        raise ValueError("unsupported decode shape")
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def iq_decode_attention_f16(q, k, v, seq_lens, out=None, workspace=None, max_seq_len=None,
                            softmax_scale: float = 0.0):
    """Decode attention on an fp16 cache k, v [B][H_kv][capacity][128]; q
    [B][H_q][128] fp32.  Returns out [B][H_q][128] fp32."""
    if q.dim() != 3 or q.shape[-1] != HEAD_DIM:
        raise ValueError("q must be [batch][n_q_heads][128]")
    b, hq, _ = q.shape
    dev = q.device
    _require(q, "q", torch.float32, (b, hq, HEAD_DIM), dev)
    if k.dim() != 4:
        raise ValueError("k must be [batch][n_kv_heads][capacity][128]")
    _, hkv, cap, _ = k.shape
    _require(k, "k", torch.float16, (b, hkv, cap, HEAD_DIM), dev)
    _require(v, "v", torch.float16, (b, hkv, cap, HEAD_DIM), dev)
    _require(seq_lens, "seq_lens", torch.int32, (b,), dev)
    if max_seq_len is None:
        max_seq_len = cap
    if out is None:
        out = torch.empty((b, hq, HEAD_DIM), dtype=torch.float32, device=dev)
    _require(out, "out", torch.float32, (b, hq, HEAD_DIM), dev)
    if workspace is None:
        workspace = alloc_f16_workspace(b, hq, hkv, max_seq_len, dev)
    if workspace.dtype != torch.uint8 or workspace.device != dev or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 device tensor")
    st = _lib.lib().iq_decode_attention_f16(
        _ptr(q), _ptr(k), _ptr(v), _ptr(seq_lens), cap, max_seq_len, b, hq, hkv, HEAD_DIM,
        float(softmax_scale), _ptr(out), _ptr(workspace), workspace.numel(), _stream(dev))
    _lib.check("iq_decode_attention_f16", st)
    return out


# ---------------------------------------------------------------------------
# measurement support
# ---------------------------------------------------------------------------

def iq_stream_read_sink_words(nbytes: int, block_threads: int, loads_per_thread: int) -> int:
    return int(_lib.lib().iq_stream_read_sink_words(nbytes, block_threads, loads_per_thread))


def iq_stream_read(src, sink, block_threads: int = 256, loads_per_thread: int = 4,
                   sentinel: int = 0x9E3779B9):
    """Streaming read of the whole of `src` (a contiguous device tensor of a
    multiple of 16 bytes); `sink` is a uint32 device tensor of at least
    iq_stream_read_sink_words(...) words."""
    if not isinstance(src, torch.Tensor) or src.device.type != "cuda" or not src.is_contiguous():
        raise ValueError("src must be a contiguous device tensor")
    if sink.dtype != torch.int32 or sink.device != src.device or not sink.is_contiguous():
        raise ValueError("sink must be a contiguous int32 device tensor on src's device")
    nbytes = src.numel() * src.element_size()
    st = _lib.lib().iq_stream_read(_ptr(src), nbytes, _ptr(sink), sink.numel(), block_threads,
                                   loads_per_thread, sentinel, _stream(src.device))
    _lib.check("iq_stream_read", st)
