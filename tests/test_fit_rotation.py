"""The host-side SO(4) fitting and quaternion extraction of the library
(iq_fit_rotation, iq_so4_to_quaternions; Sec. 3.2 "Why structured rotation
works", App. B) checked with the oracle: pure host functions, no GPU."""

import ctypes

import numpy as np
import pytest

from oracle import codebook as ocb
from oracle import rotation as orot
from oracle import rotation_study as ors
from paper_2608_08081_amd import _lib, api, synth

L = _lib.lib()
LEVELS, THR = ocb.isoquant_codebook(128, 3)


def test_so4_to_quaternions_round_trip():
    """For seeded pairs: the extracted pair rebuilds the same 4 x 4 block
    (oracle construction) and equals the input up to the common sign."""
    q = orot.make_quaternions(77, 1)[0]
    for blk in range(32):
        ql, qr = q[blk, 0].astype(np.float64), q[blk, 1].astype(np.float64)
        m = orot.so4_block(ql, qr)
        got = api.iq_so4_to_quaternions(m).astype(np.float64)
        assert np.allclose(orot.so4_block(got[0], got[1]), m, atol=1e-6)
        sgn = 1.0 if np.dot(got[0], ql) > 0 else -1.0
        assert np.allclose(sgn * got[0], ql / np.linalg.norm(ql), atol=2e-7)
        assert np.allclose(sgn * got[1], qr / np.linalg.norm(qr), atol=2e-7)


@pytest.mark.parametrize("ql", [(1, 0, 0, 0), (0, 1, 0, 0), (0, 0, 0, 1), (0.5, -0.5, 0.5, -0.5)])
def test_so4_to_quaternions_special_rotations(ql):
    """Rotations whose stable branch is each of the four cases of the
    extraction (largest of w, x, y, z), paired with the SO(3) case q_R = q_L
    (App. B: the real axis is fixed)."""
    ql = np.asarray(ql, np.float64)
    for qr in (ql, np.array([0.0, 0.0, 1.0, 0.0])):
        m = orot.so4_block(ql, qr)
        got = api.iq_so4_to_quaternions(m).astype(np.float64)
        assert np.allclose(orot.so4_block(got[0], got[1]), m, atol=1e-6)


def test_so4_to_quaternions_rejects_non_rotations():
    out = np.zeros(8, np.float32)
    refl = np.diag([1.0, 1.0, 1.0, -1.0])
    skew = np.eye(4)
    skew[0, 1] = 0.1
    for m in (refl, skew, 2 * np.eye(4)):
        a = np.ascontiguousarray(m)
        assert L.iq_so4_to_quaternions(a.ctypes.data_as(ctypes.c_void_p),
                                       out.ctypes.data_as(ctypes.c_void_p)) == 1
    assert L.iq_so4_to_quaternions(None, out.ctypes.data_as(ctypes.c_void_p)) == 1


def _calib(seed, heads, n, dist="anisotropic"):
    w = synth.Workload(95, "fit", 1, 8 * heads, heads, 2 * n, "f32", kv_dist=dist)
    k = synth.kv_tensor(seed, w, "k")[0].astype(np.float32)      # [H][2n][d]
    return k[:, :n], k[:, n:]                                      # calibration, held out


def _dist(x, quats):
    return ors.distortion(x[None], orot.rotation_matrices(quats), THR, LEVELS)


def test_fit_with_zero_sweeps_is_the_identity():
    cal, _ = _calib(1, 1, 64)
    q = api.iq_fit_rotation(cal, sweeps=0).numpy()
    assert np.array_equal(q, orot.identity_quaternions(1))


def test_fit_is_deterministic_and_unit():
    cal, _ = _calib(2, 2, 256)
    a = api.iq_fit_rotation(cal, sweeps=2).numpy()
    b = api.iq_fit_rotation(cal, sweeps=2).numpy()
    assert np.array_equal(a, b)
    n = np.linalg.norm(a.astype(np.float64), axis=-1)
    assert np.max(np.abs(n - 1)) < 4e-7


def test_fit_never_raises_calibration_distortion():
    """The fitter starts at the identity blocks and keeps only improving
    plane rotations, so on its own calibration set the oracle's distortion
    is at most that of H_128 alone (slack: fp32 rounding of the stored
    quaternions)."""
    for dist in ("anisotropic", "heavy_tailed"):
        cal, _ = _calib(3, 2, 512, dist)
        fitted = api.iq_fit_rotation(cal, sweeps=3).numpy()
        d_fit = _dist(cal, fitted)
        d_wht = _dist(cal, orot.identity_quaternions(2))
        assert d_fit <= d_wht + 1e-6, (dist, d_fit, d_wht)


def test_fit_generalizes_to_held_out_vectors():
    """Fitted on 2048 anisotropic vectors per head, evaluated on 2048 other
    vectors with the same channel scales: lower distortion than H_128 alone
    and than random SO(4) blocks (Sec. 3.2: the blocks fine-tune the
    rotation)."""
    cal, held = _calib(4, 2, 2048)
    fitted = api.iq_fit_rotation(cal, sweeps=4).numpy()
    d_fit = _dist(held, fitted)
    d_wht = _dist(held, orot.identity_quaternions(2))
    d_rand = _dist(held, orot.make_quaternions(5, 2))
    print(f"held-out distortion: fitted {d_fit:.5f}, WHT only {d_wht:.5f}, random SO(4) {d_rand:.5f}")
    assert d_fit < d_wht and d_fit < d_rand


def test_fit_validation():
    x = np.zeros((1, 4, 128), np.float32)
    out = np.zeros((1, 32, 2, 4), np.float32)
    xp, op = x.ctypes.data_as(ctypes.c_void_p), out.ctypes.data_as(ctypes.c_void_p)
    assert L.iq_fit_rotation(xp, 4, 1, 64, 1, op) == 2
    assert L.iq_fit_rotation(xp, 0, 1, 128, 1, op) == 1
    assert L.iq_fit_rotation(xp, 4, 0, 128, 1, op) == 1
    assert L.iq_fit_rotation(xp, 4, 1, 128, -1, op) == 1
    assert L.iq_fit_rotation(None, 4, 1, 128, 1, op) == 1
    # all-zero calibration vectors are skipped: identity blocks
    assert L.iq_fit_rotation(xp, 4, 1, 128, 2, op) == 0
    assert np.array_equal(out, orot.identity_quaternions(1))
