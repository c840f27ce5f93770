"""GPU parity of the fused decode step on 2- and 4-bit records
(iq_decode_step_bits: Algorithm 1 with C_b on the step's new key and value,
then App. A attention over the advanced lengths) against the oracle."""

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

DEV = torch.device("cuda:0")
BOOKS = {b: ocb.isoquant_codebook(128, b) for b in (2, 4)}


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("hq,hkv,seq0,cap", [
    (16, 2, [0, 1, 15, 16, 17, 63, 64, 65, 127, 128, 129, 500], 512),
    (32, 4, [2999, 1500], 3008),
    (16, 2, [int(x) for x in np.linspace(0, 2046, 40)], 2048),   # several rounds
])
def test_step_bits_parity(bits, hq, hkv, seq0, cap):
    """Cache tails past each length hold random codes and NaN scales, so a
    read of a position that is not attended shows up; the new records, the
    advanced lengths and the outputs are checked against the oracle."""
    levels, thr = BOOKS[bits]
    w = synth.Workload(90, "step_bits", len(seq0), hq, hkv, cap, "f16", rotation_seed=1090)
    b = len(seq0)
    k = synth.kv_tensor(7, w, "k", n_tokens=cap)
    v = synth.kv_tensor(7, w, "v", n_tokens=cap)
    quats = orot.make_quaternions(w.rotation_seed, hkv)
    rots = orot.rotation_matrices(quats)
    kp, kn, kc, ky, ks = ocz.compress_kv(k, rots, thr)
    vp, vn, vc, vy, vs = ocz.compress_kv(v, rots, thr)
    rng = np.random.default_rng(8)
    gk, gv, gkn, gvn = kp.copy(), vp.copy(), kn.copy(), vn.copy()
    for i, n in enumerate(seq0):
        gk[i, :, n:] = rng.integers(0, 256, size=gk[i, :, n:].shape, dtype=np.uint8)
        gv[i, :, n:] = rng.integers(0, 256, size=gv[i, :, n:].shape, dtype=np.uint8)
        gkn[i, :, n:] = np.nan
        gvn[i, :, n:] = np.nan
    k_new = np.stack([k[i, :, n] for i, n in enumerate(seq0)])
    v_new = np.stack([v[i, :, n] for i, n in enumerate(seq0)])
    q = synth.queries(7, w)[0]
    caches = [_dev(gk), _dev(gkn), _dev(gv), _dev(gvn)]
    lens = _dev(np.asarray(seq0, np.int32))
    print(f"[step bits] b={bits} hkv={hkv} batch={b} cap={cap}", flush=True)
    got = api.iq_decode_step_bits(_dev(q), _dev(k_new), _dev(v_new), *caches, lens,
                                  _dev(quats), max_seq_len=cap, bits=bits).cpu().numpy()
    assert lens.cpu().numpy().tolist() == [n + 1 for n in seq0]
    for i, n in enumerate(seq0):
        for side, cc, yy, ss, g in (("k", kc, ky, ks, 0), ("v", vc, vy, vs, 2)):
            rec = caches[g][i, :, n].cpu().numpy()
            check_codes(rec[None, :, None], cc[i:i + 1, :, n:n + 1], yy[i:i + 1, :, n:n + 1],
                        thr, f"{side} b{bits} seq{i}")
            check_norms(caches[g + 1][i, :, n].cpu().numpy(), ss[i, :, n], f"{side} scale")
    ref = oatt.decode_fused(q, kp, kn, vp, vn, [n + 1 for n in seq0], quats, levels)
    check_attention(got, ref, f"step b{bits} hkv{hkv} n{b}")
