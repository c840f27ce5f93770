"""Benchmark: IsoQuant decode attention on the packed 3-bit cache, 32K context.

One step = one attention layer's decode step on the hot path: append the new
token's key and value to the packed cache (compression, Alg. 1) and decode
attention over the whole cache (App. A), issued as one fused call
(iq_decode_step).  Shape: batch 1, 32 query heads,
4 KV heads, head_dim 128, ~32K cached positions.  Steps cycle through NL
distinct layer caches (default 48 x 13.6 MB = 654 MB, more than twice the
256 MB last-level cache), as a model's layer sweep does, so the cache bytes
are streamed from HBM.  Steps are replayed from HIP graphs (one graph per
sweep over the layers).

Prints one JSON line.  ``value`` is the achieved algorithmic HBM bandwidth of
a step (bytes the method must move / step time); ``us_per_step`` is the
decode-attention step time.
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
    p.add_argument("--steps", type=int, default=4800)
    p.add_argument("--warmup", type=int, default=480)
    p.add_argument("--layers", type=int, default=48)
    p.add_argument("--context", type=int, default=32768)
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--calibrate-copy-mib", type=int, default=0,
                   help="also run one plain device copy of this many MiB (counter calibration)")
    return p.parse_args()


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_08081_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def make_layers(api, synth, w, n_layers, context, capacity, seed, dev):
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
        cache = api.alloc_cache(w.batch, w.n_kv_heads, capacity, dev)
        scales = []
        for which, stream in (("k", 0), ("v", 1)):
            sc = synth.channel_scales(synth.rng(seed + li, w.wid, stream), w.n_kv_heads)
            scales.append(torch.from_numpy(sc).to(dev))
        k = torch.randn((w.batch, w.n_kv_heads, context, 128), generator=g, device=dev)
        k = (k * scales[0][None, :, None, :]).half()
        v = torch.randn((w.batch, w.n_kv_heads, context, 128), generator=g, device=dev)
        v = (v * scales[1][None, :, None, :]).half()
        api.iq_compress_kv(k, v, quats, cache["k_codes"], cache["k_norms"], cache["v_codes"],
                           cache["v_norms"])
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
    w = synth.WORKLOADS[2]
    nl = args.layers
    total_visits = math.ceil((args.warmup + args.steps) / nl) + 2
    capacity = (args.context + total_visits + 64 + 63) // 64 * 64
    print(f"# building {nl} layer caches ({args.context} positions each)", file=sys.stderr,
          flush=True)
    quats, layers = make_layers(api, synth, w, nl, args.context, capacity, args.seed, dev)
    ws = api.alloc_workspace(w.batch, w.n_q_heads, w.n_kv_heads, capacity, dev)

    def step(li, append=True):
        L = layers[li]
        c = L["cache"]
        if append:
            api.iq_decode_step(L["q"], L["k_new"], L["v_new"], c["k_codes"], c["k_norms"],
                               c["v_codes"], c["v_norms"], c["seq_lens"], quats, out=L["out"],
                               workspace=ws, max_seq_len=capacity)
        else:
            api.iq_decode_attention(L["q"], c["k_codes"], c["k_norms"], c["v_codes"],
                                    c["v_norms"], c["seq_lens"], quats, out=L["out"],
                                    workspace=ws, max_seq_len=capacity)

    if args.calibrate_copy_mib > 0:
        # a plain copy kernel of known size, for scaling FETCH_SIZE/WRITE_SIZE
        src = torch.ones(args.calibrate_copy_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # eager warm-up of every layer once (loads the code object), then capture
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        for li in range(nl):
            step(li)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()

    def capture(fn):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        return g

    sweep = capture(lambda: [step(li) for li in range(nl)])
    singles = [capture(lambda li=li: step(li)) for li in range(nl)]
    decode_sweep = capture(lambda: [step(li, append=False) for li in range(nl)])
    torch.cuda.synchronize()

    def run_steps(n, start):
        done = 0
        li = start % nl
        while done < n:
            if li == 0 and n - done >= nl:
                sweep.replay()
                done += nl
            else:
                singles[li].replay()
                done += 1
                li = (li + 1) % nl
        return (start + n) % nl

    pos = run_steps(args.warmup, 0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    pos = run_steps(args.steps, pos)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = ev0.elapsed_time(ev1)
    us_per_step = ms_total * 1e3 / args.steps

    # decode-only: HIP events around graph replays of decode launches on the
    # replay stream (the graph launches onto torch's current stream)
    reps = max(1, 2400 // nl)
    d0, d1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    d0.record()
    for _ in range(reps):
        decode_sweep.replay()
    d1.record()
    torch.cuda.synchronize()
    decode_us = d0.elapsed_time(d1) * 1e3 / (reps * nl)

    seq_now = float(sum(int(L["cache"]["seq_lens"][0]) for L in layers)) / nl
    decode_bytes = w.batch * w.n_kv_heads * seq_now * BYTES_PER_TOKEN_HEAD
    append_bytes = w.batch * w.n_kv_heads * 2 * (128 * 2 + RECORD + 4)
    step_bytes = decode_bytes + append_bytes
    value = step_bytes / (us_per_step * 1e-6) / 1e9
    digest = source_digest()

    result = {
        "metric": METRIC,
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
        "config": {
            "workload": f"32K-context GQA decode step (append + attention), batch 1, 32 query "
                        f"heads, 4 KV heads, head_dim 128, 3-bit packed KV; {nl} distinct layer "
                        f"caches cycled (cold HBM)",
            "batch": w.batch, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
            "context": int(round(seq_now)), "layers_cycled": nl,
            "step": "iq_decode_step (fused append + attention), one layer",
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(value, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(value / HBM_PEAK_GBS, 4),
            "traffic": read_traffic(digest),
            "kernel": "iq_decode_step per call = decode_g8_kernel<NB, append> + "
                      "merge_g8_kernel<append>, back to back in one graph; algorithmic bytes = "
                      f"{BYTES_PER_TOKEN_HEAD} B x positions x KV heads + the appended token's "
                      "inputs and records",
            "bytes_per_launch": int(step_bytes),
            "launch_us": round(us_per_step, 3),
            "decode_only_us": round(decode_us, 3),
        },
        "wall_s": round(wall, 3),
        "source_digest": digest,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.context, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
