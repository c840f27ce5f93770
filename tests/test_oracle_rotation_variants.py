"""Pins for the designs of the rotation ablation (Sec. 4.6, "Rotation
Design Ablation" and its table of designs; the rotation comparison table of
Sec. 2; App. B) and for the study built on them (oracle.rotation_study)."""

import numpy as np
import pytest

from oracle import codebook as ocb
from oracle import rotation as rot
from oracle import rotation_study as rs
from paper_2608_08081_amd import synth

D = 128
Q = rot.make_quaternions(31, 2)


def _orthogonal(r, tol=1e-12):
    return np.max(np.abs(r @ r.T - np.eye(r.shape[0]))) < tol


@pytest.mark.parametrize("variant", [v for v in rot.VARIANTS if v != "dense"])
def test_every_design_is_a_rotation(variant):
    r = rot.variant_rotation(variant, Q[0])
    assert r.shape == (D, D)
    assert _orthogonal(r)
    # proper rotations (det +1): every design but the dense one is built from
    # SO(4) blocks and H_128, whose determinant is +1 for d = 128
    assert abs(np.linalg.det(r) - 1.0) < 1e-9


def test_v1_fixes_the_real_axis_of_every_block():
    """Single-quaternion conjugation fixes Re(v) (App. B): design v1 leaves
    coordinate 4i of every block untouched, a quarter of all coordinates
    (the table's "25% dims unmixed")."""
    r = rot.variant_rotation("v1_so3", Q[0])
    for i in range(D // 4):
        e = np.zeros(D)
        e[4 * i] = 1.0
        assert np.allclose(r @ e, e, atol=1e-14)
        assert np.allclose(e @ r, e, atol=1e-14)
    x = np.random.default_rng(0).standard_normal((5, D))
    y = x @ r.T
    assert np.allclose(y[:, ::4], x[:, ::4], atol=1e-13)
    # while v2 (paired quaternions) moves those axes
    r2 = rot.variant_rotation("v2_so4", Q[0])
    assert not np.allclose(r2[::4, ::4], np.eye(D // 4), atol=1e-3)


def test_designs_relate_through_the_hadamard_factor():
    """v3 = v2 H_d (Eq. 2: the SO(4) blocks after the WHT); wht_so3 = v1 H_d;
    the Hadamard-only design is H_d, an involution."""
    h = rot.hadamard(D)
    assert np.allclose(rot.variant_rotation("v3_wht_so4", Q[1]),
                       rot.variant_rotation("v2_so4", Q[1]) @ h, atol=1e-14)
    assert np.allclose(rot.variant_rotation("wht_so3", Q[1]),
                       rot.variant_rotation("v1_so3", Q[1]) @ h, atol=1e-14)
    w = rot.variant_rotation("wht", Q[1])
    assert np.allclose(w @ w, np.eye(D), atol=1e-13)
    assert np.array_equal(rot.variant_rotation("none", Q[1]), np.eye(D))
    assert np.array_equal(rot.variant_rotation("v3_wht_so4", Q[1]), rot.rotation_matrix(Q[1]))


def test_v2_is_block_diagonal():
    r = rot.variant_rotation("v2_so4", Q[0])
    mask = np.kron(np.eye(D // 4), np.ones((4, 4))) > 0
    assert np.all(r[~mask] == 0.0)


def test_dense_design_is_the_sign_fixed_qr_factor():
    """Q of G = Q R with diag(R) > 0: Q^T G is upper triangular with a
    positive diagonal, and Q is orthogonal."""
    g = synth.gaussian_matrices(3, 2)
    for h in range(2):
        q = rot.dense_orthogonal(g[h])
        assert _orthogonal(q)
        t = q.T @ g[h]
        assert np.max(np.abs(np.tril(t, -1))) < 1e-10
        assert np.all(np.diag(t) > 0)


def test_dense_design_is_haar_on_average():
    """Each entry of a Haar orthogonal matrix has E[Q_ij^2] = 1/d: over 64
    draws the mean of d * Q_00^2 and of d * Q_{d-1,3}^2 lies within 4
    standard errors of 1 (Var(d Q_ij^2) ~ 2 for large d)."""
    g = synth.gaussian_matrices(5, 64)
    a = np.array([D * rot.dense_orthogonal(m)[0, 0] ** 2 for m in g])
    b = np.array([D * rot.dense_orthogonal(m)[D - 1, 3] ** 2 for m in g])
    se = np.sqrt(2.0 / len(g))
    assert abs(a.mean() - 1) < 4 * se and abs(b.mean() - 1) < 4 * se


def test_variant_quaternions():
    q3 = rot.variant_quaternions("v3_wht_so4", 7, 2)
    assert np.array_equal(q3, rot.make_quaternions(7, 2))
    q1 = rot.variant_quaternions("wht_so3", 7, 2)
    assert np.array_equal(q1[:, :, 0], q3[:, :, 0]) and np.array_equal(q1[:, :, 1], q3[:, :, 0])
    assert np.allclose(rot.rotation_matrix(q1[0]), rot.variant_rotation("wht_so3", q3[0]),
                       atol=1e-14)
    qw = rot.variant_quaternions("wht", 7, 2)
    assert np.allclose(rot.rotation_matrix(qw[0]), rot.hadamard(D), atol=1e-15)
    with pytest.raises(ValueError):
        rot.variant_quaternions("v1_so3", 7, 1)


def test_energy_of_every_design_averages_to_one():
    """sum_i (R u)_i^2 = ||u||^2 = 1 for a unit u and any orthogonal R, so
    the coordinate energies d * E[(R u)_i^2] average to exactly 1."""
    w = synth.WORKLOADS[0]
    x = synth.kv_tensor(2, w, "k", n_tokens=64).astype(np.float64)
    g = synth.gaussian_matrices(2, 1)
    for v in rot.VARIANTS:
        e = rs.coordinate_energy(x, rs.rotations(v, 9, 1, g))
        assert abs(e.mean() - 1.0) < 1e-12


def test_fixed_coordinate_share():
    w = synth.WORKLOADS[0]
    x = synth.kv_tensor(2, w, "k", n_tokens=8).astype(np.float64)
    assert rs.unmixed_share(x, rs.rotations("v1_so3", 9, 1)) == 0.25
    assert rs.unmixed_share(x, rs.rotations("none", 9, 1)) == 1.0
    assert rs.unmixed_share(x, rs.rotations("v3_wht_so4", 9, 1)) == 0.0


def test_isotropic_input_has_the_same_distortion_under_every_design():
    """For isotropic Gaussian vectors x / ||x|| is uniform on S^127 whatever
    the rotation, so every design sees the codebook's own sphere distortion
    (d * MSE per coordinate of the 8-level sphere quantizer, Sec. 3.2
    Step 3): the same mean up to sampling noise, near that value."""
    levels, thr = ocb.isoquant_codebook(D, 3)
    # expected ||u - C[q(u)]||^2 for u uniform on the sphere: d times the
    # per-coordinate MSE under the sphere marginal
    want = D * ocb.distortion(ocb.SphereMarginalModel(D), levels, thr)
    x = synth.rng(4, 92, 0).standard_normal((1, 2, 1024, D))
    g = synth.gaussian_matrices(4, 2)
    vals = [rs.distortion(x, rs.rotations(v, 9, 2, g), thr, levels) for v in rot.VARIANTS]
    assert max(vals) - min(vals) < 0.004, vals
    assert all(abs(v - want) < 0.003 for v in vals), (vals, want)


def test_study_separates_designs_with_and_without_the_global_mix():
    """On the anisotropic workload (outlier channels) the designs without
    H_d keep most of the outlier energy in few coordinates and distort far
    more than those with it (the ablation's "no global correlations" and
    "dims unmixed" failures)."""
    res = rs.study(seed=1, n_heads=1, n_tokens=256, group=2)
    with_h = [res[v]["distortion_k"] for v in ("v3_wht_so4", "wht", "wht_so3", "dense")]
    without = [res[v]["distortion_k"] for v in ("v1_so3", "v2_so4", "none")]
    assert max(with_h) * 4 < min(without)
    assert res["v1_so3"]["unmixed"] == 0.25
    assert res["v3_wht_so4"]["score_err"] < res["v2_so4"]["score_err"]
