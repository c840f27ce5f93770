"""HIP graph capture of the multi-token, code-width and paged decode entry
points: one graph holding all three is replayed several times, with eager
work and synchronizations between the replays, and every replay must equal
the eager outputs bit for bit (the calls record kernel launches only)."""

import numpy as np
import pytest
import torch

from paper_2608_08081_amd import api, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def test_graph_replays_equal_eager():
    seq, hkv, cap = [1500, 200, 17], 2, 1536
    w = synth.Workload(88, "graphs", len(seq), 16, hkv, cap, "f16", rotation_seed=1088)
    k = torch.from_numpy(synth.kv_tensor(11, w, "k")).to(DEV)
    v = torch.from_numpy(synth.kv_tensor(11, w, "v")).to(DEV)
    quats = api.iq_make_rotation(w.rotation_seed, hkv).to(DEV)
    lens = torch.tensor(seq, dtype=torch.int32, device=DEV)
    c3 = api.alloc_cache(len(seq), hkv, cap, DEV)
    c4 = api.alloc_cache(len(seq), hkv, cap, DEV, bits=4)
    api.iq_compress_kv(k, v, quats, c3["k_codes"], c3["k_norms"], c3["v_codes"], c3["v_norms"])
    api.iq_compress_kv_bits(k, v, quats, c4["k_codes"], c4["k_norms"], c4["v_codes"],
                            c4["v_norms"], bits=4)
    page, max_pages = 128, cap // 128
    perm = np.random.default_rng(5).permutation(len(seq) * max_pages).astype(np.int32)
    tables = torch.from_numpy(perm.reshape(len(seq), max_pages)).to(DEV)
    pool = api.alloc_paged_cache(len(seq) * max_pages, hkv, page, DEV)
    api.iq_compress_kv_paged(k, v, quats, pool, tables)
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    q1 = torch.randn((len(seq), 16, 128), generator=g, device=DEV)
    q3 = torch.randn((len(seq), 3, 16, 128), generator=g, device=DEV)
    outs = {"multi": torch.empty_like(q3), "bits": torch.empty_like(q1),
            "paged": torch.empty_like(q1)}
    ws_m = torch.empty(api.iq_decode_multi_workspace_bytes(len(seq), 3, 16, hkv, cap),
                       dtype=torch.uint8, device=DEV)
    ws_b = api.alloc_workspace(len(seq), 16, hkv, cap, DEV)
    ws_p = api.alloc_workspace(len(seq), 16, hkv, cap, DEV)

    def calls():
        api.iq_decode_attention_multi(q3, c3["k_codes"], c3["k_norms"], c3["v_codes"],
                                      c3["v_norms"], lens, quats, out=outs["multi"],
                                      workspace=ws_m)
        api.iq_decode_attention_bits(q1, c4["k_codes"], c4["k_norms"], c4["v_codes"],
                                     c4["v_norms"], lens, quats, out=outs["bits"],
                                     workspace=ws_b, bits=4)
        api.iq_decode_attention_paged(q1, pool, tables, lens, quats, out=outs["paged"],
                                      workspace=ws_p, max_seq_len=cap)

    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        calls()
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    eager = {n: t.clone() for n, t in outs.items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        calls()
    for rep in range(4):
        for t in outs.values():
            t.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for n, t in outs.items():
            assert torch.equal(t, eager[n]), f"replay {rep}: {n} differs from eager"
        # eager work between replays (the same calls, then other kernels)
        calls()
        torch.randn((1 << 20,), device=DEV).sum().item()
        torch.cuda.synchronize()
