"""GPU parity for the rotation designs of the ablation (Sec. 4.6) that the
kernels run unchanged (R = R_blocks H_128): single-quaternion SO(3) blocks
and the Hadamard transform alone, through compression (Alg. 1) and decode
(App. A), against the oracle built from the same parameters."""

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


@pytest.mark.parametrize("variant,name", [("so3", "wht_so3"), ("wht_only", "wht"),
                                          ("so4", "v3_wht_so4")])
@pytest.mark.parametrize("t", [1000, 4100])
def test_variant_compress_and_decode_match_oracle(variant, name, t):
    w = synth.Workload(93, "rotvar", 1, 32, 4, t, "f16", rotation_seed=1093)
    k = synth.kv_tensor(3, w, "k")
    v = synth.kv_tensor(3, w, "v")
    q = synth.queries(3, w)[0]
    quats = api.iq_make_rotation_variant(w.rotation_seed, w.n_kv_heads, variant)
    oq = orot.variant_quaternions(name, w.rotation_seed, w.n_kv_heads)
    assert np.array_equal(quats.numpy().view(np.uint32), oq.view(np.uint32))
    cap = (t + 15) // 16 * 16
    cache = api.alloc_cache(1, w.n_kv_heads, cap, DEV)
    qd = quats.to(DEV)
    api.iq_compress_kv(torch.from_numpy(k).to(DEV), torch.from_numpy(v).to(DEV), qd,
                       cache["k_codes"], cache["k_norms"], cache["v_codes"], cache["v_norms"])
    cache["seq_lens"].fill_(t)
    out = api.iq_decode_attention(torch.from_numpy(q).to(DEV), cache["k_codes"],
                                  cache["k_norms"], cache["v_codes"], cache["v_norms"],
                                  cache["seq_lens"], qd, max_seq_len=cap)
    torch.cuda.synchronize()
    rots = orot.rotation_matrices(oq)
    kp, kn, kc, ky, ks = ocz.compress_kv(k, rots, THR)
    vp, vn, vc, vy, vs = ocz.compress_kv(v, rots, THR)
    check_codes(cache["k_codes"][:, :, :t].cpu().numpy(), kc, ky, THR, f"{name} K")
    check_codes(cache["v_codes"][:, :, :t].cpu().numpy(), vc, vy, THR, f"{name} V")
    check_norms(cache["k_norms"][:, :, :t].cpu().numpy(), ks, f"{name} K scale")
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [t], oq, LEVELS)
    check_attention(out.cpu().numpy(), ref, f"{name} decode")


def test_fitted_parameters_compress_and_decode_match_oracle():
    """Parameters from the host fitter (iq_fit_rotation) drive the same
    kernels: codes, scales and attention against the oracle built from the
    fitted quaternions."""
    w = synth.Workload(94, "rotfit", 1, 32, 4, 2048, "f16", rotation_seed=1094)
    k = synth.kv_tensor(5, w, "k")
    v = synth.kv_tensor(5, w, "v")
    q = synth.queries(5, w)[0]
    quats = api.iq_fit_rotation(k[0].astype(np.float32), sweeps=2)
    oq = quats.numpy()
    t = 2048
    cache = api.alloc_cache(1, w.n_kv_heads, t, DEV)
    qd = quats.to(DEV)
    api.iq_compress_kv(torch.from_numpy(k).to(DEV), torch.from_numpy(v).to(DEV), qd,
                       cache["k_codes"], cache["k_norms"], cache["v_codes"], cache["v_norms"])
    cache["seq_lens"].fill_(t)
    out = api.iq_decode_attention(torch.from_numpy(q).to(DEV), cache["k_codes"],
                                  cache["k_norms"], cache["v_codes"], cache["v_norms"],
                                  cache["seq_lens"], qd, max_seq_len=t)
    torch.cuda.synchronize()
    rots = orot.rotation_matrices(oq)
    kp, kn, kc, ky, ks = ocz.compress_kv(k, rots, THR)
    vp, vn, vc, vy, vs = ocz.compress_kv(v, rots, THR)
    check_codes(cache["k_codes"].cpu().numpy(), kc, ky, THR, "fitted K")
    check_codes(cache["v_codes"].cpu().numpy(), vc, vy, THR, "fitted V")
    check_norms(cache["k_norms"].cpu().numpy(), ks, "fitted K scale")
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [t], oq, LEVELS)
    check_attention(out.cpu().numpy(), ref, "fitted decode")
