"""iq_decode_step_noalloc (the fused step with its partials in the library's
static device scratch) against iq_decode_step with a caller workspace, on
twin caches: identical outputs, records and lengths.  Two calls in a row on
one GPU, the second on a smaller input (the scratch keeps the first call's
contents), then a group size that takes the generic path, a grid of several
rounds, and a shape whose workspace exceeds the scratch (rejected on the
host)."""

import numpy as np
import pytest
import torch

from paper_2608_08081_amd import _lib, api, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _twins(w, lens, cap, seed):
    quats = api.iq_make_rotation(w.rotation_seed, w.n_kv_heads).to(DEV)
    k = torch.from_numpy(synth.kv_tensor(seed, w, "k", n_tokens=cap)).to(DEV)
    v = torch.from_numpy(synth.kv_tensor(seed, w, "v", n_tokens=cap)).to(DEV)
    c = api.alloc_cache(w.batch, w.n_kv_heads, cap, DEV)
    api.iq_compress_kv(k, v, quats, c["k_codes"], c["k_norms"], c["v_codes"], c["v_norms"])
    c["seq_lens"].copy_(torch.tensor(lens, dtype=torch.int32))
    kn, vn = synth.appended_tokens(seed, w, 1)
    return (c, {n: t.clone() for n, t in c.items()}, quats,
            torch.from_numpy(kn[0]).to(DEV), torch.from_numpy(vn[0]).to(DEV),
            torch.from_numpy(synth.queries(seed, w)[0]).to(DEV))


def _compare(w, lens, cap, seed, label):
    a, b, quats, k_new, v_new, q = _twins(w, lens, cap, seed)
    out_a = torch.full((w.batch, w.n_q_heads, 128), float("nan"), device=DEV)
    st_a = torch.zeros(1, dtype=torch.int32, device=DEV)
    st_b = torch.zeros(1, dtype=torch.int32, device=DEV)
    api.iq_decode_step_noalloc(q, k_new, v_new, a["k_codes"], a["k_norms"], a["v_codes"],
                               a["v_norms"], a["seq_lens"], quats, out_a, max_seq_len=cap,
                               status=st_a)
    out_b = api.iq_decode_step(q, k_new, v_new, b["k_codes"], b["k_norms"], b["v_codes"],
                               b["v_norms"], b["seq_lens"], quats, max_seq_len=cap, status=st_b)
    torch.cuda.synchronize()
    print(f"[noalloc] {label}: batch {w.batch}, {w.n_q_heads}/{w.n_kv_heads} heads, "
          f"lens {lens[:4]}..., cap {cap}", flush=True)
    assert torch.equal(out_a, out_b), label
    for n in a:
        assert torch.equal(a[n], b[n]), (label, n)
    assert torch.equal(st_a, st_b)


def test_noalloc_step_equals_workspace_step_twice():
    w1 = synth.Workload(2, "noalloc_32k", 1, 32, 4, 32896, "f16", rotation_seed=1002)
    _compare(w1, [32768], 32896, 3, "32K step")
    # second call, smaller input: the scratch holds the first call's partials
    w2 = synth.Workload(8, "noalloc_small", 3, 16, 2, 1024, "f16", rotation_seed=1008)
    _compare(w2, [1000, 37, 1024], 1024, 4, "small step, one sequence at capacity")
    # group 4 (generic path: append kernel, split kernel, combine kernel)
    w3 = synth.Workload(9, "noalloc_g4", 2, 16, 4, 700, "f16", rotation_seed=1009)
    _compare(w3, [699, 5], 704, 5, "group 4")


def test_noalloc_grid_of_several_rounds():
    """A fused step whose grid takes several rounds (24 sequences x 2 KV heads
    x 10 partials), with lengths at multiples of the split length (352) and an
    empty sequence: the merge counts each sequence's live splits from the
    lengths the step records in the scratch after the partials."""
    from tests.test_gpu_bench_shapes import g8_instance

    w = synth.Workload(10, "noalloc_wide", 24, 16, 2, 3072, "f16", rotation_seed=1010)
    assert g8_instance(w.batch, w.n_kv_heads, 3072)[2]
    lens = [0, 352, 704, 3071] + [(131 * i) % 3000 for i in range(20)]
    _compare(w, lens, 3072, 6, "grid of several rounds")


def test_noalloc_rejects_shapes_beyond_the_scratch():
    w = synth.Workload(3, "noalloc_big", 128, 16, 2, 64, "f16", rotation_seed=1003)
    cap = 33024
    need = api.iq_decode_workspace_bytes(128, 16, 2, cap)
    assert need > 64 << 20
    q = torch.zeros((128, 16, 128), device=DEV)
    kn = torch.zeros((128, 2, 128), dtype=torch.float16, device=DEV)
    codes = torch.zeros((128, 2, cap, 48), dtype=torch.uint8, device=DEV)
    norms = torch.zeros((128, 2, cap), device=DEV)
    lens = torch.zeros(128, dtype=torch.int32, device=DEV)
    quats = api.iq_make_rotation(1, 2).to(DEV)
    out = torch.zeros((128, 16, 128), device=DEV)
    with pytest.raises(_lib.IsoQuantError) as e:
        api.iq_decode_step_noalloc(q, kn, kn, codes, norms, codes, norms, lens, quats, out)
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert int(lens.abs().sum()) == 0 and int(out.abs().sum()) == 0
