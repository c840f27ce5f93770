"""Pins for the oracle's structured rotation (Sec. 3.2 Step 2, Eq. 2;
Sec. 3.3; App. A; App. B)."""

import itertools
import os

import numpy as np
import pytest

from oracle import rotation as rot


# SplitMix64 reference outputs for seed 0 (the values that accompany the
# generator's published description; first three outputs).
SPLITMIX64_SEED0 = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_splitmix64_reference_outputs():
    s = rot.splitmix64_stream(0)
    assert [next(s) for _ in range(3)] == SPLITMIX64_SEED0


def test_quaternions_unit_and_deterministic():
    q = rot.make_quaternions(42, 4)
    assert q.shape == (4, 32, 2, 4) and q.dtype == np.float32
    n = np.linalg.norm(q.astype(np.float64), axis=-1)
    assert np.max(np.abs(n - 1.0)) < 4 * 2.0 ** -24
    assert np.array_equal(q, rot.make_quaternions(42, 4))
    assert not np.array_equal(q, rot.make_quaternions(43, 4))
    # heads are a prefix-stable stream: head 0 does not depend on n_heads
    assert np.array_equal(rot.make_quaternions(42, 1)[0], q[0])


def test_quaternions_uniform_on_s3():
    """Rejection sampling from the cube gives uniform directions on S^3:
    zero mean and E[q_i^2] = 1/4 per component."""
    q = rot.make_quaternions(5, 64).reshape(-1, 4).astype(np.float64)
    assert q.shape[0] == 4096
    assert np.all(np.abs(q.mean(axis=0)) < 4 * 0.5 / np.sqrt(q.shape[0]))
    assert np.all(np.abs((q ** 2).mean(axis=0) - 0.25) < 0.02)


# --------------------------------------------------------------------------
# Hamilton product, brute force from the unit multiplication table
# --------------------------------------------------------------------------

# products of basis units 1, i, j, k: (index, sign) of e_a * e_b
_UNIT = {
    (0, 0): (0, 1), (0, 1): (1, 1), (0, 2): (2, 1), (0, 3): (3, 1),
    (1, 0): (1, 1), (1, 1): (0, -1), (1, 2): (3, 1), (1, 3): (2, -1),
    (2, 0): (2, 1), (2, 1): (3, -1), (2, 2): (0, -1), (2, 3): (1, 1),
    (3, 0): (3, 1), (3, 1): (2, 1), (3, 2): (1, -1), (3, 3): (0, -1),
}


def _brute_mul(p, q):
    out = np.zeros(4)
    for a, b in itertools.product(range(4), range(4)):
        idx, sgn = _UNIT[(a, b)]
        out[idx] += sgn * p[a] * q[b]
    return out


def test_unit_table_defines_hamilton_algebra():
    """The table obeys i^2 = j^2 = k^2 = ijk = -1."""
    e = np.eye(4)
    minus_one = -e[0]
    for u in (1, 2, 3):
        assert np.array_equal(_brute_mul(e[u], e[u]), minus_one)
    assert np.array_equal(_brute_mul(_brute_mul(e[1], e[2]), e[3]), minus_one)


def test_quat_mul_matches_brute_force():
    g = np.random.default_rng(0)
    for _ in range(50):
        p, q = g.standard_normal(4), g.standard_normal(4)
        np.testing.assert_allclose(rot.quat_mul(p, q), _brute_mul(p, q), atol=1e-14)
        # norm is multiplicative
        assert abs(np.linalg.norm(rot.quat_mul(p, q)) - np.linalg.norm(p) * np.linalg.norm(q)) < 1e-12


# --------------------------------------------------------------------------
# SO(4) blocks
# --------------------------------------------------------------------------

def test_so4_block_orthogonal_det_one():
    q = rot.make_quaternions(11, 2).reshape(-1, 2, 4)
    for ql, qr in q:
        m = rot.so4_block(ql, qr)
        np.testing.assert_allclose(m.T @ m, np.eye(4), atol=1e-15)
        assert abs(np.linalg.det(m) - 1.0) < 1e-14


def test_so4_block_is_the_quaternion_map():
    """M v equals q_L v conj(q_R) computed with the brute-force product."""
    g = np.random.default_rng(1)
    for _ in range(20):
        ql, qr = g.standard_normal(4), g.standard_normal(4)
        ql /= np.linalg.norm(ql)
        qr /= np.linalg.norm(qr)
        v = g.standard_normal(4)
        want = _brute_mul(_brute_mul(ql, v), qr * np.array([1, -1, -1, -1]))
        np.testing.assert_allclose(rot.so4_block(ql, qr) @ v, want, atol=1e-14)


def test_so4_special_cases():
    one = np.array([1.0, 0, 0, 0])
    np.testing.assert_allclose(rot.so4_block(one, one), np.eye(4), atol=0)
    # single-quaternion conjugation fixes the real axis and acts on the rest
    # as SO(3) (App. B; rotation design v1)
    g = np.random.default_rng(2)
    q = g.standard_normal(4)
    m = rot.so3_block(q)
    np.testing.assert_allclose(m[:, 0], [1, 0, 0, 0], atol=1e-15)
    np.testing.assert_allclose(m[0, :], [1, 0, 0, 0], atol=1e-15)
    assert abs(np.linalg.det(m[1:, 1:]) - 1.0) < 1e-14
    # double cover: (-q_L, -q_R) is the same rotation
    ql, qr = g.standard_normal(4), g.standard_normal(4)
    np.testing.assert_allclose(rot.so4_block(-ql, -qr), rot.so4_block(ql, qr), atol=1e-15)


def test_so4_pair_has_six_degrees_of_freedom():
    """The map (q_L, q_R) -> M has rank-6 differential (dim SO(4) = 6), while
    single-quaternion conjugation only reaches a 3-dim family (App. B)."""
    g = np.random.default_rng(3)
    ql, qr = g.standard_normal(4), g.standard_normal(4)
    ql /= np.linalg.norm(ql)
    qr /= np.linalg.norm(qr)
    eps = 1e-6

    def tangent(fun, base):
        cols = []
        for k in range(base.size):
            d = np.zeros(base.size)
            d[k] = eps
            cols.append(((fun(base + d) - fun(base - d)) / (2 * eps)).ravel())
        return np.stack(cols, axis=1)

    j6 = tangent(lambda z: rot.so4_block(z[:4], z[4:]), np.concatenate([ql, qr]))
    s = np.linalg.svd(j6, compute_uv=False)
    assert np.sum(s > 1e-6) == 6
    j3 = tangent(lambda z: rot.so3_block(z), ql)
    s3 = np.linalg.svd(j3, compute_uv=False)
    assert np.sum(s3 > 1e-6) == 3


# --------------------------------------------------------------------------
# Walsh-Hadamard and the composed rotation
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d", [1, 2, 4, 32, 128])
def test_hadamard_definition_and_orthogonality(d):
    h = rot.hadamard(d)
    brute = np.array([[(-1) ** bin(i & j).count("1") for j in range(d)] for i in range(d)]) / np.sqrt(d)
    np.testing.assert_allclose(h, brute, atol=1e-16)
    np.testing.assert_allclose(h @ h.T, np.eye(d), atol=1e-15)
    np.testing.assert_allclose(h @ h, np.eye(d), atol=1e-15)
    e0 = np.zeros(d)
    e0[0] = 1
    np.testing.assert_allclose(h @ e0, np.full(d, 1 / np.sqrt(d)), atol=1e-16)


def test_rotation_orthogonal_and_round_trip():
    q = rot.make_quaternions(1002, 4)
    g = np.random.default_rng(4)
    for h in range(4):
        r = rot.rotation_matrix(q[h])
        np.testing.assert_allclose(r @ r.T, np.eye(128), atol=1e-13)
        x = g.standard_normal((16, 128)) * g.lognormal(0, 0.5, 128)
        back = (x @ r.T) @ r                       # R^T (R x) row-wise
        assert np.max(np.abs(back - x)) / np.max(np.abs(x)) < 1e-12


def test_rotation_structure():
    """Identity parameters give R = H_d; otherwise R = blockdiag(M_i) H_d with
    each diagonal 4 x 4 block of R H_d equal to M_i."""
    np.testing.assert_allclose(rot.rotation_matrix(rot.identity_quaternions(1)[0]),
                               rot.hadamard(128), atol=0)
    q = rot.make_quaternions(9, 1)[0]
    r = rot.rotation_matrix(q)
    rh = r @ rot.hadamard(128)                     # H is an involution
    for i in range(32):
        blk = rh[4 * i:4 * i + 4, 4 * i:4 * i + 4]
        np.testing.assert_allclose(blk, rot.so4_block(q[i, 0], q[i, 1]), atol=1e-15)
        off = rh[4 * i:4 * i + 4].copy()
        off[:, 4 * i:4 * i + 4] = 0
        assert np.max(np.abs(off)) < 1e-15


def test_post_wht_isotropy():
    """Sec. 3.2: after the WHT every coordinate carries the same share of the
    energy.  For a diagonal covariance Sigma, diag(H Sigma H) = tr(Sigma)/d
    exactly; checked on anisotropic samples with outlier channels."""
    d = 128
    g = np.random.default_rng(5)
    scale = g.lognormal(0, 0.5, d)
    scale[g.choice(d, 4, replace=False)] *= 20
    x = g.standard_normal((20000, d)) * scale
    y = x @ rot.hadamard(d).T
    per_coord = (y ** 2).mean(axis=0)
    target = np.sum(scale ** 2) / d
    assert np.max(np.abs(per_coord / target - 1)) < 0.06
    # without the WHT the outlier channels carry hundreds of times the mean
    assert np.max((x ** 2).mean(axis=0)) / target > 50
