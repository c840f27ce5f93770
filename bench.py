"""Benchmark: IsoQuant decode attention on the packed 3-bit cache, 32K context.

One step = one attention layer's decode step on the hot path: append the new
token's key and value to the packed cache (compression, Alg. 1) and decode
attention over the whole cache (App. A), issued as one fused call
(iq_decode_step).  Shape: batch 1, 32 query heads,
4 KV heads, head_dim 128, ~32K cached positions.  Steps cycle through NL
distinct layer caches (default 48 x 13.6 MB = 654 MB, more than twice the
256 MB last-level cache), as a model's layer sweep does, so the cache bytes
are streamed from HBM.  Exactly --steps steps are timed, replayed from HIP
graphs of consecutive distinct layers (whole sweeps over the layers, then one
graph for the remainder).

Prints one JSON line.  ``value`` is the achieved algorithmic HBM bandwidth of
a step (bytes the method must move / step time); ``us_per_step`` is the
decode-attention step time.

``--workload`` selects the other measured shapes (each prints its own line;
the default is the one above):
  varlen    batch 64, 16 query heads, 2 KV heads, per-sequence contexts drawn
            uniform in [2048, 32768]: one fused decode step per sequence;
  compress  iq_compress_kv over 4 sequences x 32768 tokens x 8 KV heads, K and
            V, fp16 Student-t(4) entries times log-normal channel scales;
  append8k  batch 1, 32 query heads, 4 KV heads, 8192 compressed tokens, then
            fused steps that each append one token (48 layer caches cycled);
  rotation_fit  SO(4) block parameters fitted on the host (iq_fit_rotation)
            to 4 x 4096 anisotropic calibration keys, then the 3-bit distortion
            of 4 x 32768 held-out keys with the same channel scales, compressed
            and materialized by the library's kernels, for the fitted, random,
            single-quaternion and Hadamard-only parameters;
  paged     the varlen shape on a paged cache (iq_decode_step_paged; pages of
            --page-size positions, physical pages randomly permuted), then
            on contiguous caches with the same lengths for comparison;
  bits32k   decode attention (and the fused step) at the 32K shape on 2-, 3-
            and 4-bit records (Algorithm 1 with C_b; --bits picks the one
            reported as value);
  multi32k  decode of 1-4 query tokens per call at the 32K shape
            (iq_decode_attention_multi, speculative verification; --tokens picks
            the one reported as value), against single-token calls;
  baseline32k  the 32K shape above through the reconstruct-then-compute
            pipeline the packed path replaces (Fig. 1 top): decode attention
            on an fp16 cache, materialization of the packed cache as fp16
            (iq_dequantize_kv) and the two chained, next to the packed decode
            attention on the same caches (48 layers cycled).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode-attention µs/step + achieved HBM GB/s on packed 3-bit KV, 32K ctx"
HBM_PEAK_GBS = 8000.0
RECORD = 48
BYTES_PER_TOKEN_HEAD = 2 * (RECORD + 4)      # K and V: 48-byte record + fp32 scale


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--workload", choices=("step32k", "varlen", "compress", "append8k",
                                          "baseline32k", "rotation_fit", "paged", "bits32k",
                                          "multi32k", "tiny1k", "shard"),
                   default="step32k")
    p.add_argument("--steps", type=int, default=None,
                   help="timed steps (default: 4800; varlen 240; compress 20; append8k 1000)")
    p.add_argument("--warmup", type=int, default=None,
                   help="untimed steps (default: steps / 10)")
    p.add_argument("--layers", type=int, default=None,
                   help="distinct layer caches cycled (default: 48; varlen 3)")
    p.add_argument("--context", type=int, default=32768)
    p.add_argument("--bits", type=int, choices=(2, 3, 4), default=4,
                   help="code width reported as value by the bits32k workload")
    p.add_argument("--tokens", type=int, choices=(1, 2, 3, 4), default=4,
                   help="query tokens per call reported as value by the multi32k workload")
    p.add_argument("--page-size", type=int, default=16,
                   help="positions per page of the paged workload (a power of two, >= 16)")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--calibrate-copy-mib", type=int, default=0,
                   help="also run one plain device copy of this many MiB (counter calibration)")
    a = p.parse_args()
    defaults = {"step32k": (4800, 48), "varlen": (240, 3), "compress": (20, 1),
                "append8k": (1000, 48), "baseline32k": (960, 48),
                "rotation_fit": (1, 1), "paged": (240, 3), "bits32k": (960, 48),
                "multi32k": (960, 48), "tiny1k": (960, 48), "shard": (4800, 0)}[a.workload]
    if a.steps is None:
        a.steps = defaults[0]
    if a.warmup is None:
        a.warmup = max(1, a.steps // 10)
    if a.layers is None:
        a.layers = defaults[1]
    if a.page_size < 16 or a.page_size & (a.page_size - 1):
        p.error("--page-size must be a power of two, at least 16")
    return a


# sources of the decode step's kernels and their launch path: the counter
# figures in profiles/ hold only while these are unchanged
DECODE_SOURCES = ("iq_api.cpp", "iq_decode.hip", "iq_decode_g8.hip", "iq_g8_device.h",
                  "iq_device.h", "iq_internal.h")


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_08081_amd", "csrc")
    for name in DECODE_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def make_layers(api, synth, w, n_layers, context, capacity, seed, dev, bits=3):
    """Per layer: packed caches filled with `context` compressed tokens of
    fresh synthetic keys/values (seeded, drawn on the device with the same
    recipe as synth.kv_tensor), the token to append, and the query."""
    import numpy as np
    import torch

    layers = []
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(dev)
    for li in range(n_layers):
        g = torch.Generator(device=dev)
        g.manual_seed(seed * 100003 + li)
        cache = api.alloc_cache(w.batch, w.n_kv_heads, capacity, dev, bits=bits)
        scales = []
        for which, stream in (("k", 0), ("v", 1)):
            sc = synth.channel_scales(synth.rng(seed + li, w.wid, stream), w.n_kv_heads)
            scales.append(torch.from_numpy(sc).to(dev))
        k = torch.randn((w.batch, w.n_kv_heads, context, 128), generator=g, device=dev)
        k = (k * scales[0][None, :, None, :]).half()
        v = torch.randn((w.batch, w.n_kv_heads, context, 128), generator=g, device=dev)
        v = (v * scales[1][None, :, None, :]).half()
        api.iq_compress_kv_bits(k, v, quats, cache["k_codes"], cache["k_norms"],
                                cache["v_codes"], cache["v_norms"], bits=bits)
        del k, v
        cache["seq_lens"].fill_(context)
        k_new = (torch.randn((w.batch, w.n_kv_heads, 128), generator=g, device=dev)
                 * scales[0][None]).half()
        v_new = (torch.randn((w.batch, w.n_kv_heads, 128), generator=g, device=dev)
                 * scales[1][None]).half()
        q = torch.randn((w.batch, w.n_q_heads, 128), generator=g, device=dev)
        out = torch.empty((w.batch, w.n_q_heads, 128), device=dev)
        layers.append(dict(cache=cache, k_new=k_new, v_new=v_new, q=q, out=out))
    torch.cuda.synchronize()
    return quats, layers


def cpu_baseline(w, context, seconds):
    """Time the CPU oracle's compressed-space decode on a bounded sample: one
    KV head (its 8 query heads) of one 32K decode step, repeated until about
    `seconds` have passed.  Reported in the same unit as `value`."""
    import numpy as np

    from oracle import attention as oatt
    from oracle import codebook as ocb
    from oracle import compress as ocz
    from oracle import rotation as orot
    from paper_2608_08081_amd import synth

    levels, thr = ocb.isoquant_codebook()
    one = synth.Workload(90, "cpu_sample", 1, w.group, 1, context, "f16", rotation_seed=7)
    k = synth.kv_tensor(1, one, "k")
    v = synth.kv_tensor(1, one, "v")
    q = synth.queries(1, one)[0]
    quats = orot.make_quaternions(7, 1)
    rots = orot.rotation_matrices(quats)
    kp, kn, *_ = ocz.compress_kv(k, rots, thr)
    vp, vn, *_ = ocz.compress_kv(v, rots, thr)
    reps, t0 = 0, time.perf_counter()
    while True:
        oatt.decode_fused(q, kp, kn, vp, vn, [context], quats, levels)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds or reps >= 1000:
            break
    per = el / reps
    bytes_sample = context * BYTES_PER_TOKEN_HEAD
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads") or 1) for i in threadpool_info()) if threadpool_info() else 1
    except Exception:
        threads = os.cpu_count()
    return {"value": bytes_sample / per / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"oracle fp64 decode_fused, 1 KV head x {w.group} query heads x {context} "
                      f"positions, {reps} reps in {el:.1f}s ({per * 1e3:.1f} ms each); "
                      f"scaled: algorithmic bytes of the sample / time"}


def read_traffic(digest: str):
    path = os.path.join(ROOT, "profiles", "decode_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            t = json.load(f)
    except Exception:
        return None
    if t.get("source_digest") != digest:
        return None
    return t.get("hbm_bytes_per_launch")


def make_varlen_layers(api, synth, w, n_layers, lengths, capacity, seed, dev, slice_b=8):
    """Per layer: batch caches where sequence b holds lengths[b] compressed
    tokens (compressed in slices of `slice_b` sequences, each slice up to its
    longest sequence; positions past a sequence's length are never read)."""
    import torch

    layers = []
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(dev)
    for li in range(n_layers):
        g = torch.Generator(device=dev)
        g.manual_seed(seed * 100003 + 7919 * li + 1)
        cache = api.alloc_cache(w.batch, w.n_kv_heads, capacity, dev)
        scales = []
        for stream in (0, 1):
            sc = synth.channel_scales(synth.rng(seed + li, w.wid, stream), w.n_kv_heads)
            scales.append(torch.from_numpy(sc).to(dev))
        for b0 in range(0, w.batch, slice_b):
            b1 = min(w.batch, b0 + slice_b)
            t = int(lengths[b0:b1].max())
            kv = []
            for which in (0, 1):
                x = torch.randn((b1 - b0, w.n_kv_heads, t, 128), generator=g, device=dev)
                kv.append((x * scales[which][None, :, None, :]).half())
            api.iq_compress_kv(kv[0], kv[1], quats, cache["k_codes"][b0:b1],
                               cache["k_norms"][b0:b1], cache["v_codes"][b0:b1],
                               cache["v_norms"][b0:b1])
            del kv
        cache["seq_lens"].copy_(torch.from_numpy(lengths).to(dev))
        k_new = (torch.randn((w.batch, w.n_kv_heads, 128), generator=g, device=dev)
                 * scales[0][None]).half()
        v_new = (torch.randn((w.batch, w.n_kv_heads, 128), generator=g, device=dev)
                 * scales[1][None]).half()
        q = torch.randn((w.batch, w.n_q_heads, 128), generator=g, device=dev)
        out = torch.empty((w.batch, w.n_q_heads, 128), device=dev)
        layers.append(dict(cache=cache, k_new=k_new, v_new=v_new, q=q, out=out))
    torch.cuda.synchronize()
    return quats, layers


def make_paged_layers(api, synth, w, n_layers, lengths, capacity, page, seed, dev,
                      slice_b=8):
    """Per layer: page pools for the varlen shape, located through one page
    table shared by all layers (as a serving engine keeps one page list per
    sequence).  Sequence b maps ceil((its length + growth) / page) logical
    pages; the physical pages of all sequences are one random permutation of
    the pool (no two neighbours in a sequence are adjacent in memory, as in
    a long-running server).  Tokens are compressed straight into the pages
    (iq_compress_kv_paged)."""
    import numpy as np
    import torch

    layers = []
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(dev)
    max_pages = capacity // page
    need = [min(max_pages, -(-(int(n) + capacity - int(lengths.max())) // page))
            for n in lengths]
    n_pages = int(sum(need))
    perm = np.random.default_rng([seed, 11]).permutation(n_pages).astype(np.int32)
    tables = np.full((w.batch, max_pages), -1, np.int32)
    k0 = 0
    for b, m in enumerate(need):
        tables[b, :m] = perm[k0:k0 + m]
        k0 += m
    bt = torch.from_numpy(tables).to(dev)
    for li in range(n_layers):
        g = torch.Generator(device=dev)
        g.manual_seed(seed * 100003 + 7919 * li + 1)
        pool = api.alloc_paged_cache(n_pages, w.n_kv_heads, page, dev)
        scales = []
        for stream in (0, 1):
            sc = synth.channel_scales(synth.rng(seed + li, w.wid, stream), w.n_kv_heads)
            scales.append(torch.from_numpy(sc).to(dev))
        for b0 in range(0, w.batch, slice_b):
            b1 = min(w.batch, b0 + slice_b)
            t = int(lengths[b0:b1].max())
            kv = []
            for which in (0, 1):
                x = torch.randn((b1 - b0, w.n_kv_heads, t, 128), generator=g, device=dev)
                kv.append((x * scales[which][None, :, None, :]).half())
            api.iq_compress_kv_paged(kv[0], kv[1], quats, pool, bt[b0:b1])
            del kv
        pool["seq_lens"] = torch.from_numpy(lengths).to(dev)
        k_new = (torch.randn((w.batch, w.n_kv_heads, 128), generator=g, device=dev)
                 * scales[0][None]).half()
        v_new = (torch.randn((w.batch, w.n_kv_heads, 128), generator=g, device=dev)
                 * scales[1][None]).half()
        q = torch.randn((w.batch, w.n_q_heads, 128), generator=g, device=dev)
        out = torch.empty((w.batch, w.n_q_heads, 128), device=dev)
        layers.append(dict(cache=pool, tables=bt, k_new=k_new, v_new=v_new, q=q, out=out))
    torch.cuda.synchronize()
    return quats, layers


def visits_per_layer(warmup, steps, n_layers):
    """Upper bound of the calls one layer receives from time_graph_calls:
    the eager pass, the set-up replays of the captured graphs (four at most)
    and the warm-up and timed calls."""
    return 1 + 4 + math.ceil(warmup / n_layers) + math.ceil(steps / n_layers) + 1


def cache_capacity(longest, warmup, steps, n_layers):
    """Capacity of the cycled layer caches: the longest sequence, one
    appended token per visit of the layer (visits_per_layer), rounded up
    to a multiple of 64 with at least 64 spare positions."""
    return (longest + visits_per_layer(warmup, steps, n_layers) + 64 + 63) // 64 * 64


def time_graph_calls(torch, fn, n_layers, steps, warmup):
    """fn(li) issues one call for layer li.  Times exactly `steps` calls that
    cycle the layers, replayed from HIP graphs of consecutive distinct layers
    (whole sweeps of n_layers calls, then one graph for the remainder), with
    HIP events on the replay stream.  Before that, untimed: one eager call
    per layer (loads the code objects), one replay of every captured graph,
    one whole sweep (so each layer's data was last touched n_layers - 1
    layers ago), then `warmup` calls continuing the cycle from layer 0; the
    timed calls go on from there.  Returns (us per call, wall seconds)."""
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        for li in range(n_layers):
            fn(li)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()

    graphs = {}

    def graph(start, count):
        key = (start, count)
        if key not in graphs:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(count):
                    fn((start + i) % n_layers)
            graphs[key] = g
        return graphs[key]

    def plan(start, count):
        full, tail = divmod(count, n_layers)
        seq = [graph(start, n_layers)] * full
        if tail:
            seq.append(graph(start, tail))
        return seq

    sweep0 = graph(0, n_layers)
    warm = plan(0, warmup)
    timed = plan(warmup % n_layers, steps)
    torch.cuda.synchronize()
    # set-up replays: every graph once (its first launch), then a whole sweep
    for g in list(graphs.values()) + [sweep0]:
        g.replay()
    for g in warm:
        g.replay()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for g in timed:
        g.replay()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    us = ev0.elapsed_time(ev1) * 1e3 / steps
    del graphs, warm, timed, sweep0
    return us, wall


def time_steps(api, layers, quats, ws, capacity, args):
    """`args.steps` fused steps (append + attention) cycling the layers after
    `args.warmup` untimed ones (time_graph_calls), then as many calls of the
    attention alone (iq_decode_attention, at most 2400) the same way.
    Returns (us per fused step, us per decode-only call, wall seconds of the
    timed steps)."""
    import torch

    nl = len(layers)

    def step(li, append=True):
        L = layers[li]
        c = L["cache"]
        if "tables" in L:
            if append:
                api.iq_decode_step_paged(L["q"], L["k_new"], L["v_new"], c, L["tables"],
                                         c["seq_lens"], quats, out=L["out"], workspace=ws,
                                         max_seq_len=capacity)
            else:
                api.iq_decode_attention_paged(L["q"], c, L["tables"], c["seq_lens"], quats,
                                              out=L["out"], workspace=ws, max_seq_len=capacity)
        elif append:
            api.iq_decode_step(L["q"], L["k_new"], L["v_new"], c["k_codes"], c["k_norms"],
                               c["v_codes"], c["v_norms"], c["seq_lens"], quats, out=L["out"],
                               workspace=ws, max_seq_len=capacity)
        else:
            api.iq_decode_attention(L["q"], c["k_codes"], c["k_norms"], c["v_codes"],
                                    c["v_norms"], c["seq_lens"], quats, out=L["out"],
                                    workspace=ws, max_seq_len=capacity)

    us_per_step, wall = time_graph_calls(torch, step, nl, args.steps, args.warmup)
    decode_us, _ = time_graph_calls(torch, lambda li: step(li, append=False), nl,
                                    min(args.steps, 2400), args.warmup)
    return us_per_step, decode_us, wall


def achievable_read(torch, api, dev, nbytes, n_buffers, steps, warmup):
    """The achievable single-launch read bandwidth at the step's size: a
    plain streaming read (iq_stream_read) of `nbytes`, cycled over n_buffers
    distinct buffers and timed exactly as the steps are (time_graph_calls),
    for several workgroup sizes and loads per thread; the fastest is
    reported."""
    n16 = -(-nbytes // 16)
    bufs = [torch.full((4 * n16,), i + 1, dtype=torch.int32, device=dev)
            for i in range(n_buffers)]
    best = None
    for block, loads in ((256, 1), (256, 2), (256, 4), (256, 8), (512, 1), (512, 2), (512, 4),
                         (1024, 1), (1024, 2), (1024, 4)):
        sink = torch.zeros(api.iq_stream_read_sink_words(16 * n16, block, loads),
                           dtype=torch.int32, device=dev)

        def read(li, block=block, loads=loads, sink=sink):
            api.iq_stream_read(bufs[li], sink, block_threads=block, loads_per_thread=loads)

        us, _ = time_graph_calls(torch, read, n_buffers, max(steps, 2 * n_buffers), warmup)
        if best is None or us < best[0]:
            best = (us, block, loads)
    del bufs
    torch.cuda.empty_cache()
    us, block, loads = best
    return {"value": round(16 * n16 / (us * 1e-6) / 1e9, 2), "unit": "GB/s",
            "us_per_launch": round(us, 3), "bytes": int(16 * n16),
            "kernel": f"stream_read_kernel<{loads}>, {block}-thread workgroups (fastest of 10 "
                      f"shapes), {n_buffers} buffers cycled (cold)"}


def step_result(metric, workload, w, layers, nl, us_per_step, decode_us, wall, args, kernel,
                extra_config=None):
    """JSON line of a fused-step workload: algorithmic bytes of the attended
    positions (per KV head and position: K and V records + scales) plus the
    appended tokens' inputs and records, over the measured step time."""
    seq_sum = sum(float(L["cache"]["seq_lens"].sum()) for L in layers) / nl
    decode_bytes = w.n_kv_heads * seq_sum * BYTES_PER_TOKEN_HEAD
    append_bytes = w.batch * w.n_kv_heads * 2 * (128 * 2 + RECORD + 4)
    step_bytes = decode_bytes + append_bytes
    value = step_bytes / (us_per_step * 1e-6) / 1e9
    config = {"workload": workload, "batch": w.batch, "n_q_heads": w.n_q_heads,
              "n_kv_heads": w.n_kv_heads, "mean_context": int(round(seq_sum / w.batch)),
              "layers_cycled": nl, "step": "iq_decode_step (fused append + attention), one layer"}
    config.update(extra_config or {})
    return {
        "metric": metric,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us_per_step / 1e3, 6),
        "us_per_step": round(us_per_step, 3),
        "decode_us": round(decode_us, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u3 codes, f32 accumulate",
        "data": "synthetic (seeded anisotropic fp16 K/V, compressed on device)",
        "config": config,
        "roofline": {
            "bound": "hbm",
            "achieved": round(value, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(value / HBM_PEAK_GBS, 4),
            "traffic": None,
            "kernel": kernel,
            "bytes_per_launch": int(step_bytes),
            "launch_us": round(us_per_step, 3),
            "decode_only_us": round(decode_us, 3),
        },
        "wall_s": round(wall, 3),
    }


def run_step32k(args, torch, api, synth, dev):
    w = synth.WORKLOADS[2]
    nl = args.layers
    capacity = cache_capacity(args.context, args.warmup, args.steps, nl)
    print(f"# building {nl} layer caches ({args.context} positions each)", file=sys.stderr,
          flush=True)
    quats, layers = make_layers(api, synth, w, nl, args.context, capacity, args.seed, dev)
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    us_per_step, decode_us, wall = time_steps(api, layers, quats, ws, capacity, args)
    digest = source_digest()
    result = step_result(
        METRIC,
        f"32K-context GQA decode step (append + attention), batch 1, 32 query heads, 4 KV "
        f"heads, head_dim 128, 3-bit packed KV; {nl} distinct layer caches cycled (cold HBM)",
        w, layers, nl, us_per_step, decode_us, wall, args,
        "iq_decode_step per call = decode_g8_kernel<NB, append> + merge_g8_kernel<append>, back "
        f"to back in one graph; algorithmic bytes = {BYTES_PER_TOKEN_HEAD} B x positions x KV "
        "heads + the appended token's inputs and records")
    result["config"]["context"] = result["config"].pop("mean_context")
    result["roofline"]["traffic"] = read_traffic(digest)
    ach = achievable_read(torch, api, dev, result["roofline"]["bytes_per_launch"], nl,
                          args.steps, args.warmup)
    result["roofline"]["achievable"] = ach["value"]
    result["roofline"]["frac_of_achievable"] = round(result["roofline"]["achieved"] /
                                                     ach["value"], 4)
    result["roofline"]["achievable_read"] = ach
    result["source_digest"] = digest
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.context, args.cpu_seconds)
    return result


def run_shard(args, torch, api, synth, dev):
    """The 32K step at one GPU's share of it: by KV heads (tensor parallel over
    2 and 4 GPUs: 2 or 1 KV heads with their 8 query heads each) and by
    positions (context parallel over 2, 4 and 8 GPUs: 16K, 8K and 4K of the
    positions, all heads).  Each share cycles enough layer caches to span
    twice the 256 MB cache on the memory side (so every step reads cold
    data); value = the full step's share measured on this GPU."""
    import dataclasses

    w2 = synth.WORKLOADS[2]
    shares = [("whole step", 4, 32768), ("TP=2", 2, 32768), ("TP=4", 1, 32768),
              ("CP=2", 4, 16384), ("CP=4", 4, 8192), ("CP=8", 4, 4096)]
    rows = []
    for name, hkv, ctx in shares:
        w = dataclasses.replace(w2, n_kv_heads=hkv, n_q_heads=8 * hkv)
        layer_bytes = hkv * ctx * BYTES_PER_TOKEN_HEAD
        nl = args.layers if args.layers else max(48, -(-(512 << 20) // layer_bytes))
        capacity = cache_capacity(ctx, args.warmup, args.steps, nl)
        print(f"# {name}: {nl} layer caches, {hkv} KV heads, {ctx} positions", file=sys.stderr,
              flush=True)
        quats, layers = make_layers(api, synth, w, nl, ctx, capacity, args.seed, dev)
        ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
        us, dec, wall = time_steps(api, layers, quats, ws, capacity, args)
        r = step_result(METRIC, name, w, layers, nl, us, dec, wall, args, "")
        rows.append({"share": name, "n_kv_heads": hkv, "n_q_heads": 8 * hkv, "context": ctx,
                     "layers_cycled": nl, "us_per_step": r["us_per_step"],
                     "decode_us": r["decode_us"], "GB/s": r["value"],
                     "frac": r["roofline"]["frac"]})
        del layers, ws
        torch.cuda.empty_cache()
    whole = rows[0]
    return {
        "metric": "32K decode step at one GPU's share (µs/step)",
        "value": rows[2]["us_per_step"],
        "unit": "µs/step (TP=4 share)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "higher_is_better": False,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "u3 codes, f32 accumulate",
        "data": "synthetic (seeded anisotropic fp16 K/V, compressed on device)",
        "config": {"workload": "the 32K GQA fused step (batch 1, 32 query heads, 4 KV heads, "
                               "32768 positions) at one GPU's share, one GPU",
                   "shares": rows,
                   "note": "a share's time plus the exchange of partials (context parallel) is "
                           "the sharded step; the exchange is not measured here; "
                           f"whole step {whole['us_per_step']} us"},
    }


def run_varlen(args, torch, api, synth, dev):
    w = synth.WORKLOADS[3]
    nl = args.layers
    lengths = synth.context_lengths(args.seed, w)
    capacity = cache_capacity(int(lengths.max()), args.warmup, args.steps, nl)
    print(f"# building {nl} varlen layer caches (batch {w.batch}, mean context "
          f"{lengths.mean():.0f})", file=sys.stderr, flush=True)
    quats, layers = make_varlen_layers(api, synth, w, nl, lengths, capacity, args.seed, dev)
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    us_per_step, decode_us, wall = time_steps(api, layers, quats, ws, capacity, args)
    return step_result(
        "batched varlen decode µs/step + achieved HBM GB/s on packed 3-bit KV",
        f"batched serving decode step (append + attention), batch {w.batch}, {w.n_q_heads} "
        f"query heads, {w.n_kv_heads} KV heads, head_dim 128, contexts uniform in "
        f"[{w.varlen[0]}, {w.varlen[1]}] (seeded); {nl} distinct layer caches cycled",
        w, layers, nl, us_per_step, decode_us, wall, args,
        "iq_decode_step per call = decode_g8_kernel<NB, append> + merge_g8_kernel<append>; "
        f"algorithmic bytes = {BYTES_PER_TOKEN_HEAD} B x attended positions x KV heads + the "
        "appended tokens' inputs and records",
        {"lengths_min": int(lengths.min()), "lengths_max": int(lengths.max())})


def run_paged(args, torch, api, synth, dev):
    """The varlen shape on page pools (iq_decode_step_paged), then the same
    lengths on contiguous caches (iq_decode_step) for comparison."""
    w = synth.WORKLOADS[3]
    nl = args.layers
    page = args.page_size
    lengths = synth.context_lengths(args.seed, w)
    total_visits = visits_per_layer(args.warmup, args.steps, nl)
    capacity = (int(lengths.max()) + total_visits + page + page - 1) // page * page
    print(f"# building {nl} paged layer caches (batch {w.batch}, page {page})",
          file=sys.stderr, flush=True)
    quats, layers = make_paged_layers(api, synth, w, nl, lengths, capacity, page, args.seed,
                                      dev)
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    us_per_step, decode_us, wall = time_steps(api, layers, quats, ws, capacity, args)
    result = step_result(
        "paged batched varlen decode µs/step + achieved HBM GB/s on packed 3-bit KV",
        f"batched serving decode step (append + attention) on a paged cache ({page}-position "
        f"pages, randomly permuted pool, one page table for all layers), batch {w.batch}, {w.n_q_heads} query heads, "
        f"{w.n_kv_heads} KV heads, head_dim 128, contexts uniform in [{w.varlen[0]}, "
        f"{w.varlen[1]}] (seeded); {nl} distinct layer pools cycled",
        w, layers, nl, us_per_step, decode_us, wall, args,
        "iq_decode_step_paged per call = decode_g8_kernel<NB, append, wide, paged> + "
        f"merge_g8_kernel; algorithmic bytes = {BYTES_PER_TOKEN_HEAD} B x attended positions x "
        "KV heads + the appended tokens' inputs and records",
        {"page_size": page, "lengths_min": int(lengths.min()),
         "lengths_max": int(lengths.max())})
    del layers, ws
    torch.cuda.empty_cache()
    print("# contiguous caches, same lengths", file=sys.stderr, flush=True)
    quats, layers = make_varlen_layers(api, synth, w, nl, lengths, capacity, args.seed, dev)
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    c_us, c_dec, _ = time_steps(api, layers, quats, ws, capacity, args)
    result["contiguous"] = {"us_per_step": round(c_us, 3), "decode_us": round(c_dec, 3),
                            "paged_over_contiguous": round(us_per_step / c_us, 4)}
    return result


def run_append8k(args, torch, api, synth, dev):
    w = synth.WORKLOADS[1]
    nl = args.layers
    capacity = cache_capacity(w.context, args.warmup, args.steps, nl)
    print(f"# building {nl} layer caches ({w.context} positions each)", file=sys.stderr,
          flush=True)
    quats, layers = make_layers(api, synth, w, nl, w.context, capacity, args.seed, dev)
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    us_per_step, decode_us, wall = time_steps(api, layers, quats, ws, capacity, args)
    return step_result(
        "8K-context decode step (append one token + attention) µs/step + achieved HBM GB/s",
        f"GQA decode steps that each append one token, batch 1, 32 query heads, 4 KV heads, "
        f"head_dim 128, {w.context} compressed tokens to start; {nl} distinct layer caches "
        "cycled",
        w, layers, nl, us_per_step, decode_us, wall, args,
        "iq_decode_step per call = decode_g8_kernel<NB, append> + merge_g8_kernel<append>; "
        f"algorithmic bytes = {BYTES_PER_TOKEN_HEAD} B x attended positions x KV heads + the "
        "appended tokens' inputs and records")


def run_tiny1k(args, torch, api, synth, dev):
    """The single-head workload: batch 1, one query and one KV head (group 1:
    the matrix-core kernel with one query row of eight in use), 1024 fp32 keys and values
    compressed (iq_compress_kv), then one decode-attention call over them
    (iq_decode_attention), each timed over --layers distinct layers cycled
    (time_graph_calls).  Both are latency-bound at this size."""
    w = synth.WORKLOADS[0]
    nl = args.layers
    t = w.context
    quats = api.iq_make_rotation(w.rotation_seed, 1).to(dev)
    layers = []
    for li in range(nl):
        g = torch.Generator(device=dev)
        g.manual_seed(args.seed * 100003 + li)
        sc = [torch.from_numpy(synth.channel_scales(synth.rng(args.seed + li, w.wid, s), 1))
              .to(dev) for s in (0, 1)]
        k = torch.randn((1, 1, t, 128), generator=g, device=dev) * sc[0][None, :, None, :]
        v = torch.randn((1, 1, t, 128), generator=g, device=dev) * sc[1][None, :, None, :]
        cache = api.alloc_cache(1, 1, t, dev)
        cache["seq_lens"].fill_(t)
        q = torch.randn((1, 1, 128), generator=g, device=dev)
        layers.append(dict(k=k, v=v, cache=cache, q=q, out=torch.empty((1, 1, 128), device=dev)))
    ws = api.alloc_workspace(1, 1, 1, t, dev)

    def compress(li):
        L = layers[li]
        c = L["cache"]
        api.iq_compress_kv(L["k"], L["v"], quats, c["k_codes"], c["k_norms"], c["v_codes"],
                           c["v_norms"])

    def decode(li):
        L = layers[li]
        c = L["cache"]
        api.iq_decode_attention(L["q"], c["k_codes"], c["k_norms"], c["v_codes"], c["v_norms"],
                                c["seq_lens"], quats, out=L["out"], workspace=ws,
                                max_seq_len=t)

    us_c, _ = time_graph_calls(torch, compress, nl, args.steps, args.warmup)
    us_d, _ = time_graph_calls(torch, decode, nl, args.steps, args.warmup)
    dec_bytes = t * BYTES_PER_TOKEN_HEAD
    comp_bytes = 2 * t * (128 * 4 + RECORD + 4)
    value = dec_bytes / (us_d * 1e-6) / 1e9
    return {
        "metric": "single-head decode-attention µs/call + achieved HBM GB/s on packed 3-bit KV, "
                  "1K ctx",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us_d / 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u3 codes, f32 accumulate",
        "data": "synthetic (seeded anisotropic fp32 K/V, compressed on device)",
        "config": {"workload": f"batch 1, 1 query head, 1 KV head (group 1), "
                               f"head_dim 128, {t} fp32 keys and values; {nl} distinct layers "
                               "cycled", "context": t},
        "roofline": {"bound": "hbm", "achieved": round(value, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(value / HBM_PEAK_GBS, 5), "traffic": None,
                     "kernel": "decode_g8_kernel<NB, false, false, false, 3, false, true> + "
                               "merge_g8_kernel<false, 1, true, false>",
                     "bytes_per_launch": dec_bytes, "launch_us": round(us_d, 3)},
        "compress": {"us_per_call": round(us_c, 3), "bytes": comp_bytes,
                     "gbs": round(comp_bytes / (us_c * 1e-6) / 1e9, 2),
                     "kernel": "compress_kernel<float, false, 3>"},
    }


def run_bits32k(args, torch, api, synth, dev):
    """Decode attention at the 32K shape on caches of b-bit records (Algorithm
    1 with C_b; b = 2, 3, 4, each its own set of layer caches compressed from
    the same seeded fp16 K/V recipe), iq_decode_attention_bits replayed from
    HIP graphs over the cycled layers.  Algorithmic bytes per position and
    KV head: K and V records of 16 b bytes plus their fp32 scales."""
    w = synth.WORKLOADS[2]
    nl = args.layers
    cap = args.context
    per = {}
    for bits in (2, 3, 4):
        print(f"# building {nl} layer caches of {bits}-bit records", file=sys.stderr, flush=True)
        quats, layers = make_layers(api, synth, w, nl, cap, cap, args.seed, dev, bits=bits)
        ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, cap, dev)

        def call(li, layers=layers, quats=quats, ws=ws, bits=bits):
            L = layers[li]
            c = L["cache"]
            api.iq_decode_attention_bits(L["q"], c["k_codes"], c["k_norms"], c["v_codes"],
                                         c["v_norms"], c["seq_lens"], quats, out=L["out"],
                                         workspace=ws, max_seq_len=cap, bits=bits)

        us = time_graph_calls(torch, call, nl, args.steps, args.warmup)[0]
        nbytes = w.batch * w.n_kv_heads * cap * 2 * (16 * bits + 4)
        per[bits] = {"us_per_call": round(us, 3), "bytes": int(nbytes),
                     "gbs": round(nbytes / (us * 1e-6) / 1e9, 2)}
        # the fused step (append + attention) on the same caches: the lengths
        # advance by one per visit, so the caches are filled to cap - visits
        for L in layers:
            L["cache"]["seq_lens"].fill_(cap - visits_per_layer(args.warmup, args.steps, nl))

        def step(li, layers=layers, quats=quats, ws=ws, bits=bits):
            L = layers[li]
            c = L["cache"]
            api.iq_decode_step_bits(L["q"], L["k_new"], L["v_new"], c["k_codes"], c["k_norms"],
                                    c["v_codes"], c["v_norms"], c["seq_lens"], quats,
                                    out=L["out"], workspace=ws, max_seq_len=cap, bits=bits)

        us_step = time_graph_calls(torch, step, nl, args.steps, args.warmup)[0]
        per[bits]["step_us"] = round(us_step, 3)
        del layers, ws
        torch.cuda.empty_cache()
    b = args.bits
    value = per[b]["gbs"]
    return {
        "metric": f"{b}-bit decode-attention µs/call + achieved HBM GB/s, 32K ctx",
        "value": value,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(per[b]["us_per_call"] / 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": f"u{b} codes, f32 accumulate",
        "data": "synthetic (seeded anisotropic fp16 K/V, compressed on device)",
        "config": {"workload": f"32K-context GQA decode attention on {b}-bit records, batch 1, "
                               f"32 query heads, 4 KV heads, head_dim 128; {nl} distinct layer "
                               "caches cycled (cold HBM)",
                   "context": cap, "bits": b},
        "roofline": {"bound": "hbm", "achieved": value, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(value / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": f"decode_g8_kernel<NB, false, false, false, {b}> + "
                               "merge_g8_kernel<false>",
                     "bytes_per_launch": per[b]["bytes"], "launch_us": per[b]["us_per_call"]},
        "per_bits": {str(k): v for k, v in per.items()},
    }


def run_multi32k(args, torch, api, synth, dev):
    """Multi-token decode at the 32K shape: T = 1..4 query tokens per call
    over the same 48 cycled layer caches (iq_decode_attention_multi), against
    T single-token calls.  Algorithmic bytes per call: the cache read once
    (104 B per position and KV head) plus the T tokens' queries and outputs.
    Then the fused multi-token step (iq_decode_step_multi, T = 2 and 4: the T
    new tokens compressed, appended and attended causally in the same call)
    on the same caches, whose capacity leaves room for the appended tokens;
    its bytes add the new fp16 keys and values read and their records
    written."""
    import numpy as np

    w = synth.WORKLOADS[2]
    nl = args.layers
    cap = args.context
    capacity = (cap + 4 * visits_per_layer(args.warmup, args.steps, nl) + 64 + 63) // 64 * 64
    print(f"# building {nl} layer caches", file=sys.stderr, flush=True)
    quats, layers = make_layers(api, synth, w, nl, cap, capacity, args.seed, dev)
    per = {}
    for n_tok in (1, 2, 3, 4):
        g = torch.Generator(device=dev)
        g.manual_seed(args.seed * 7 + n_tok)
        qs = [torch.randn((w.batch, n_tok, w.n_q_heads, 128), generator=g, device=dev)
              for _ in range(nl)]
        outs = [torch.empty_like(x) for x in qs]
        ws = torch.empty(api.iq_decode_multi_workspace_bytes(w.batch, n_tok, w.n_q_heads,
                                                             w.n_kv_heads, cap),
                         dtype=torch.uint8, device=dev)

        def call(li, n_tok=n_tok, qs=qs, outs=outs, ws=ws):
            c = layers[li]["cache"]
            api.iq_decode_attention_multi(qs[li], c["k_codes"], c["k_norms"], c["v_codes"],
                                          c["v_norms"], c["seq_lens"], quats, out=outs[li],
                                          workspace=ws, max_seq_len=cap)

        us = time_graph_calls(torch, call, nl, args.steps, args.warmup)[0]
        nbytes = w.n_kv_heads * cap * BYTES_PER_TOKEN_HEAD + 2 * n_tok * w.n_q_heads * 128 * 4
        per[n_tok] = {"us_per_call": round(us, 3), "bytes": int(nbytes),
                      "gbs": round(nbytes / (us * 1e-6) / 1e9, 2),
                      "tokens_per_s": round(n_tok / (us * 1e-6), 1)}
        del qs, outs, ws
    t = args.tokens
    single = per[1]["us_per_call"]
    for n_tok, d in per.items():
        d["vs_single_calls"] = round(n_tok * single / d["us_per_call"], 3)
    fused = {}
    for n_tok in (2, 4):
        for layer in layers:
            layer["cache"]["seq_lens"].fill_(cap)
        g = torch.Generator(device=dev)
        g.manual_seed(args.seed * 11 + n_tok)
        qs = [torch.randn((w.batch, n_tok, w.n_q_heads, 128), generator=g, device=dev)
              for _ in range(nl)]
        kv = [[torch.randn((w.batch, n_tok, w.n_kv_heads, 128), generator=g, device=dev).half()
               for _ in range(2)] for _ in range(nl)]
        outs = [torch.empty_like(x) for x in qs]
        ws = torch.empty(api.iq_decode_multi_workspace_bytes(w.batch, n_tok, w.n_q_heads,
                                                             w.n_kv_heads, capacity),
                         dtype=torch.uint8, device=dev)

        def step(li, qs=qs, kv=kv, outs=outs, ws=ws):
            c = layers[li]["cache"]
            api.iq_decode_step_multi(qs[li], kv[li][0], kv[li][1], c["k_codes"], c["k_norms"],
                                     c["v_codes"], c["v_norms"], c["seq_lens"], quats,
                                     out=outs[li], workspace=ws, max_seq_len=capacity)

        us = time_graph_calls(torch, step, nl, args.steps, args.warmup)[0]
        grown = int(layers[0]["cache"]["seq_lens"][0].item())
        assert cap < grown <= capacity, (cap, grown, capacity)
        nbytes = (w.n_kv_heads * cap * BYTES_PER_TOKEN_HEAD + 2 * n_tok * w.n_q_heads * 128 * 4
                  + n_tok * w.n_kv_heads * (2 * 128 * 2 + BYTES_PER_TOKEN_HEAD))
        fused[n_tok] = {"us_per_call": round(us, 3), "bytes": int(nbytes),
                        "gbs": round(nbytes / (us * 1e-6) / 1e9, 2),
                        "vs_multi_decode": round(us / per[n_tok]["us_per_call"], 3),
                        "length_after": grown}
        del qs, kv, outs, ws
    for layer in layers:
        layer["cache"]["seq_lens"].fill_(cap)
    value = per[t]["gbs"]
    return {
        "metric": f"{t}-token decode-attention µs/call + achieved HBM GB/s, 32K ctx",
        "value": value,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(per[t]["us_per_call"] / 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u3 codes, f32 accumulate",
        "data": "synthetic (seeded anisotropic fp16 K/V, compressed on device)",
        "config": {"workload": f"32K-context GQA decode of {t} query tokens per sequence "
                               "(speculative verification, causal among them), batch 1, 32 query "
                               f"heads, 4 KV heads, head_dim 128; {nl} distinct layer caches "
                               "cycled (cold HBM)",
                   "context": cap, "tokens": t},
        "roofline": {"bound": "hbm", "achieved": value, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(value / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": f"decode_g8_multi_kernel<NB, false, {t}> + merge_g8_kernel<false, "
                               f"{t}>" if t > 1 else "decode_g8_kernel + merge_g8_kernel",
                     "bytes_per_launch": per[t]["bytes"], "launch_us": per[t]["us_per_call"]},
        "per_tokens": {str(k): v for k, v in per.items()},
        "fused_step": {str(k): v for k, v in fused.items()},
    }


def run_baseline32k(args, torch, api, synth, dev):
    """Reconstruct-then-compute (Fig. 1 top) against compressed-space decode
    (Fig. 1 bottom) at the 32K shape.  Per layer the same seeded fp16 K/V
    are kept as an fp16 cache and compressed into a packed cache.  Paths:
      packed       iq_decode_attention on the packed cache;
      fp16         iq_decode_attention_f16 on the fp16 cache;
      dequantize   iq_dequantize_kv of the packed cache into one fp16
                   scratch cache shared by all layers (as a pipeline that
                   materializes per layer would);
      reconstruct  dequantize, then iq_decode_attention_f16 on the scratch."""
    w = synth.WORKLOADS[2]
    nl = args.layers
    t = args.context
    capacity = t
    print(f"# building {nl} layer caches, packed and fp16 ({t} positions each)",
          file=sys.stderr, flush=True)
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(dev)
    layers = []
    for li in range(nl):
        g = torch.Generator(device=dev)
        g.manual_seed(args.seed * 100003 + li)
        scales = [torch.from_numpy(synth.channel_scales(synth.rng(args.seed + li, w.wid, st),
                                                        w.n_kv_heads)).to(dev)
                  for st in (0, 1)]
        k = (torch.randn((w.batch, w.n_kv_heads, t, 128), generator=g, device=dev)
             * scales[0][None, :, None, :]).half()
        v = (torch.randn((w.batch, w.n_kv_heads, t, 128), generator=g, device=dev)
             * scales[1][None, :, None, :]).half()
        cache = api.alloc_cache(w.batch, w.n_kv_heads, capacity, dev)
        api.iq_compress_kv(k, v, quats, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                           cache["v_norms"])
        cache["seq_lens"].fill_(t)
        q = torch.randn((w.batch, w.n_q_heads, 128), generator=g, device=dev)
        layers.append(dict(cache=cache, k=k, v=v, q=q,
                           out=torch.empty((w.batch, w.n_q_heads, 128), device=dev)))
    torch.cuda.synchronize()
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    ws16 = api.alloc_f16_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)
    k_s = torch.empty((w.batch, w.n_kv_heads, t, 128), dtype=torch.float16, device=dev)
    v_s = torch.empty_like(k_s)

    def packed(li):
        L = layers[li]
        c = L["cache"]
        api.iq_decode_attention(L["q"], c["k_codes"], c["k_norms"], c["v_codes"], c["v_norms"],
                                c["seq_lens"], quats, out=L["out"], workspace=ws,
                                max_seq_len=capacity)

    def fp16(li):
        L = layers[li]
        api.iq_decode_attention_f16(L["q"], L["k"], L["v"], L["cache"]["seq_lens"],
                                    out=L["out"], workspace=ws16, max_seq_len=capacity)

    def dequantize(li):
        c = layers[li]["cache"]
        api.iq_dequantize_kv(c["k_codes"], c["k_norms"], c["v_codes"], c["v_norms"], quats,
                             n_tokens=t, seq_lens=c["seq_lens"], out_dtype=torch.float16,
                             k_out=k_s, v_out=v_s)

    def reconstruct(li):
        dequantize(li)
        L = layers[li]
        api.iq_decode_attention_f16(L["q"], k_s, v_s, L["cache"]["seq_lens"], out=L["out"],
                                    workspace=ws16, max_seq_len=capacity)

    t0 = time.perf_counter()
    us = {name: time_graph_calls(torch, fn, nl, args.steps, args.warmup)[0]
          for name, fn in (("packed", packed), ("fp16", fp16), ("dequantize", dequantize),
                           ("reconstruct", reconstruct))}
    wall = time.perf_counter() - t0
    pos = w.n_kv_heads * t
    fp16_bytes = pos * 2 * 128 * 2
    byts = {"packed": pos * BYTES_PER_TOKEN_HEAD,
            "fp16": fp16_bytes,
            "dequantize": pos * BYTES_PER_TOKEN_HEAD + fp16_bytes,
            "reconstruct": pos * BYTES_PER_TOKEN_HEAD + 2 * fp16_bytes}
    paths = {}
    for name in us:
        gbs = byts[name] / (us[name] * 1e-6) / 1e9
        paths[name] = {"us_per_call": round(us[name], 3), "algorithmic_bytes": int(byts[name]),
                       "GB/s": round(gbs, 2), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}
    f16_gbs = paths["fp16"]["GB/s"]
    return {
        "metric": "32K decode attention µs/call: packed 3-bit (compressed-space) vs fp16 cache "
                  "vs reconstruct-then-compute",
        "value": round(us["packed"], 3),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us["packed"] / 1e3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u3 codes / f16 cache, f32 accumulate",
        "data": "synthetic (seeded anisotropic fp16 K/V; packed caches compressed on device)",
        "config": {"workload": f"decode attention, batch 1, 32 query heads, 4 KV heads, "
                               f"head_dim 128, context {t}; {nl} distinct layer caches cycled",
                   "context": t, "layers_cycled": nl},
        "paths": paths,
        "speedup_vs_fp16": round(us["fp16"] / us["packed"], 3),
        "speedup_vs_reconstruct": round(us["reconstruct"] / us["packed"], 3),
        "roofline": {
            "bound": "hbm",
            "achieved": f16_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(f16_gbs / HBM_PEAK_GBS, 4),
            "traffic": None,
            "kernel": "iq_decode_attention_f16 = decode_f16_kernel<4> + merge_f16_kernel; "
                      "algorithmic bytes = 512 B (fp16 K + V) x positions x KV heads",
            "bytes_per_launch": int(fp16_bytes),
            "launch_us": round(us["fp16"], 3),
        },
        "wall_s": round(wall, 3),
    }

def cpu_compress_baseline(seconds):
    """The oracle's fp64 compression on a bounded sample of vectors."""
    import numpy as np

    from oracle import codebook as ocb
    from oracle import compress as ocz
    from oracle import rotation as orot
    from paper_2608_08081_amd import synth

    _, thr = ocb.isoquant_codebook()
    w = synth.WORKLOADS[4]
    k = synth.kv_tensor(3, w, "k", n_tokens=1024, batch=1)[:, :1]
    rots = orot.rotation_matrices(orot.make_quaternions(w.rotation_seed, 1))
    n_vec = k.shape[2]
    reps, t0 = 0, time.perf_counter()
    while True:
        ocz.compress_kv(k, rots, thr)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds or reps >= 1000:
            break
    per = el / reps
    return {"value": n_vec * (256 + 52) / per / 1e9, "unit": "GB/s", "cores": os.cpu_count(),
            "kind": "oracle",
            "sample": f"oracle fp64 compress_kv of {n_vec} fp16 vectors, {reps} reps in "
                      f"{el:.1f}s ({per * 1e3:.1f} ms each); algorithmic bytes / time"}


def run_compress(args, torch, api, synth, dev):
    w = synth.WORKLOADS[4]
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed * 100003 + 4)
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(dev)
    kv = []
    for stream in (0, 1):
        sc = torch.from_numpy(synth.channel_scales(synth.rng(args.seed, w.wid, stream),
                                                   w.n_kv_heads, n_outliers=0)).to(dev)
        shape = (w.batch, w.n_kv_heads, w.context, 128)
        # Student-t(4) = N(0,1) / sqrt(chi2_4 / 4)
        z = torch.randn(shape, generator=g, device=dev)
        chi = sum(torch.randn(shape, generator=g, device=dev) ** 2 for _ in range(4))
        kv.append((z * torch.rsqrt(chi / 4.0) * sc[None, :, None, :]).half())
        del z, chi
    cache = api.alloc_cache(w.batch, w.n_kv_heads, w.context, dev)

    def call():
        api.iq_compress_kv(kv[0], kv[1], quats, cache["k_codes"], cache["k_norms"],
                           cache["v_codes"], cache["v_norms"])

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        call()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    us = ev0.elapsed_time(ev1) * 1e3 / args.steps
    n_vec = 2 * w.batch * w.n_kv_heads * w.context
    byts = n_vec * (128 * 2 + RECORD + 4)
    value = byts / (us * 1e-6) / 1e9
    result = {
        "metric": "compression GB/s (read + written) and vectors/s, prefill-scale",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(us / 1e3, 6),
        "us_per_call": round(us, 3),
        "vectors_per_s": round(n_vec / (us * 1e-6), 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 in, u3 codes + f32 scales out, f32/f64 arithmetic",
        "data": "synthetic (seeded Student-t(4) x log-normal channel scales, fp16)",
        "config": {"workload": f"iq_compress_kv of K and V, {w.batch} sequences x {w.context} "
                               f"tokens x {w.n_kv_heads} KV heads, head_dim 128",
                   "vectors": n_vec},
        "roofline": {
            "bound": "hbm",
            "achieved": round(value, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(value / HBM_PEAK_GBS, 4),
            "traffic": None,
            "kernel": "compress_kernel<__half>: 256 B read + 52 B written per vector",
            "bytes_per_launch": int(byts),
            "launch_us": round(us, 3),
        },
        "wall_s": round(wall, 3),
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_compress_baseline(min(args.cpu_seconds, 10.0))
    return result


def run_rotation_fit(args, torch, api, synth, dev):
    """Fit the SO(4) blocks on calibration keys (host), then measure the
    held-out relative squared error ||x - x_hat||^2 / ||x||^2 of keys
    compressed (iq_compress_kv) and materialized (iq_dequantize_kv) on the
    GPU with each parameter set, and with codebooks fitted to the same
    calibration keys (iq_fit_codebook, iq_compress_kv_cb,
    iq_dequantize_kv_cb).  A quality figure, not a throughput."""
    n_heads, n_cal, n_held = 4, 4096, 32768
    w = synth.Workload(96, "rotation_fit", 1, 8 * n_heads, n_heads, n_cal + n_held, "f16")
    k = synth.kv_tensor(args.seed, w, "k")                      # [1][H][T][d] fp16
    cal = k[0, :, :n_cal].astype("float32")
    t0 = time.perf_counter()
    fitted = api.iq_fit_rotation(cal, sweeps=4)
    fit_s = time.perf_counter() - t0
    held = torch.from_numpy(k[:, :, n_cal:].copy()).to(dev)
    params = {"fitted": fitted,
              "random_so4": api.iq_make_rotation(w.rotation_seed, n_heads),
              "single_quaternion": api.iq_make_rotation_variant(w.rotation_seed, n_heads, "so3"),
              "wht_only": api.iq_make_rotation_variant(w.rotation_seed, n_heads, "wht_only")}
    x = held.float()
    x2 = (x * x).sum(-1)
    res = {}

    def distortion(q, codebook=None):
        qd = q.to(dev)
        cache = api.alloc_cache(1, n_heads, n_held, dev, values=False)
        if codebook is None:
            api.iq_compress_kv(held, None, qd, cache["k_codes"], cache["k_norms"], None, None)
        else:
            api.iq_compress_kv_cb(held, None, qd, codebook, cache["k_codes"], cache["k_norms"],
                                  None, None)
        xh, _ = api.iq_dequantize_kv(cache["k_codes"], cache["k_norms"], None, None, qd,
                                     out_dtype=torch.float32, codebook=codebook)
        err = ((x - xh) ** 2).sum(-1) / x2
        return round(float(err.mean()), 6)

    for name, q in params.items():
        res[name] = distortion(q)
    # codebooks fitted (iq_fit_codebook) on the same calibration keys, under
    # the fitted and the random block parameters
    t0 = time.perf_counter()
    cb_fitted = api.iq_fit_codebook(cal, fitted, bits=3)
    cb_fit_s = time.perf_counter() - t0
    cb_random = api.iq_fit_codebook(cal, params["random_so4"], bits=3)
    res["fitted+fitted_codebook"] = distortion(fitted, cb_fitted)
    res["random_so4+fitted_codebook"] = distortion(params["random_so4"], cb_random)
    torch.cuda.synchronize()
    return {
        "metric": "held-out 3-bit relative squared error of keys, fitted vs random SO(4) blocks",
        "value": res["fitted"],
        "unit": "mean ||x - x_hat||^2 / ||x||^2",
        "n_gpus": 1,
        "steps": 1,
        "warmup": 0,
        "higher_is_better": False,
        "vs_baseline": None,
        "dtype": "f16 in, u3 codes, f32 out",
        "data": "synthetic (seeded anisotropic fp16 keys: N(0,1) x log-normal channel scales, "
                "4 outlier channels x20)",
        "config": {"workload": f"{n_heads} KV heads, {n_cal} calibration + {n_held} held-out "
                               f"keys per head, head_dim 128, 4 fitting sweeps"},
        "distortion": res,
        "fit_seconds_host": round(fit_s, 3),
        "codebook_fit_seconds_host": round(cb_fit_s, 3),
        "fitted_codebook_levels": [round(float(x), 7) for x in api.codebook_arrays(cb_fitted)[0]],
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2608_08081_amd import api, synth

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    if args.calibrate_copy_mib > 0:
        # a plain copy kernel of known size, for scaling FETCH_SIZE/WRITE_SIZE
        src = torch.ones(args.calibrate_copy_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    run = {"step32k": run_step32k, "varlen": run_varlen, "compress": run_compress,
           "shard": run_shard,
           "append8k": run_append8k, "baseline32k": run_baseline32k,
           "rotation_fit": run_rotation_fit, "paged": run_paged,
           "bits32k": run_bits32k, "multi32k": run_multi32k, "tiny1k": run_tiny1k}[args.workload]
    print(json.dumps(run(args, torch, api, synth, dev)), flush=True)


if __name__ == "__main__":
    main()
