"""Structured rotation R = R_SO(4) o H_d (Sec. 3.2 Step 2, Eq. 2; Sec. 3.3
"SO(4) parameterization"; App. B).  Test infrastructure only.

* H_d is the d x d normalized Walsh-Hadamard matrix.  Reading (the paper does
  not state an ordering or random signs): Sylvester (natural) ordering,
  H_1 = [1], H_2n = [[H_n, H_n], [H_n, -H_n]], scaled by 1/sqrt(d), with no
  random sign diagonal.  H_d is symmetric and orthogonal.
* R_SO(4) acts independently on each contiguous 4-dimensional block
  (0-based blocks i = 0 .. d/4 - 1 covering dims 4i .. 4i+3) by the
  quaternion map v -> q_L v conj(q_R).  Reading of the embedding: block
  component 0 is the real part, components 1..3 the i, j, k parts; Hamilton
  product convention i^2 = j^2 = k^2 = ijk = -1.
* The stored parameters are one (q_L, q_R) pair per block, 8 floats per block,
  256 floats per head at d = 128 (App. B).  Reading of "seeded random unit
  quaternions": a SplitMix64 stream (Steele, Lea & Flood, OOPSLA 2014, with
  the 64-bit finalizer published alongside it) seeded with the user seed,
  drawn in the order head -> block -> q_L then q_R; each quaternion takes
  four 53-bit uniforms mapped to [-1, 1), rejects draws whose squared norm is
  not in (1e-6, 1] (uniform on the ball, hence uniform direction on S^3) and
  divides by the norm in fp64; the result is rounded to fp32.  The rotation
  is defined by the directions of the stored fp32 quaternions: the oracle
  renormalizes them in fp64 before building the 4 x 4 blocks, so R is
  orthogonal to fp64 precision.
"""

from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15


# --------------------------------------------------------------------------
# Seeded parameters
# --------------------------------------------------------------------------

def splitmix64_stream(seed: int):
    """Yield the SplitMix64 sequence for ``seed``: the state advances by the
    golden gamma and each output is the state passed through the
    xor-shift-multiply finalizer."""
    state = seed & MASK64
    while True:
        state = (state + GOLDEN_GAMMA) & MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        yield z ^ (z >> 31)


def _uniform_pm1(stream) -> float:
    """One draw mapped to [-1, 1): top 53 bits scaled by 2^-53, then 2u - 1
    (both steps exact in fp64)."""
    u = float(next(stream) >> 11) * (2.0 ** -53)
    return 2.0 * u - 1.0


def _random_unit_quaternion(stream) -> np.ndarray:
    while True:
        u = [_uniform_pm1(stream) for _ in range(4)]
        n2 = u[0] * u[0]
        n2 = n2 + u[1] * u[1]
        n2 = n2 + u[2] * u[2]
        n2 = n2 + u[3] * u[3]
        if 1e-6 < n2 <= 1.0:
            n = np.sqrt(n2)
            return np.array([np.float32(c / n) for c in u], dtype=np.float32)


def make_quaternions(seed: int, n_heads: int, d: int = 128) -> np.ndarray:
    """Seeded SO(4) parameters: float32 array [n_heads][d/4][2][4] holding
    (q_L, q_R) per block, components (w, x, y, z)."""
    if d % 4:
        raise ValueError("d must be a multiple of 4")
    stream = splitmix64_stream(seed)
    out = np.empty((n_heads, d // 4, 2, 4), dtype=np.float32)
    for h in range(n_heads):
        for b in range(d // 4):
            out[h, b, 0] = _random_unit_quaternion(stream)
            out[h, b, 1] = _random_unit_quaternion(stream)
    return out


def identity_quaternions(n_heads: int, d: int = 128) -> np.ndarray:
    q = np.zeros((n_heads, d // 4, 2, 4), dtype=np.float32)
    q[..., 0] = 1.0
    return q


# --------------------------------------------------------------------------
# Building blocks
# --------------------------------------------------------------------------

def hadamard(d: int) -> np.ndarray:
    """Normalized Sylvester Walsh-Hadamard matrix H_d (fp64)."""
    if d < 1 or d & (d - 1):
        raise ValueError("d must be a power of two")
    h = np.ones((1, 1))
    while h.shape[0] < d:
        h = np.block([[h, h], [h, -h]])
    return h / np.sqrt(d)


def quat_mul(p, q) -> np.ndarray:
    """Hamilton product p q of quaternions given as (w, x, y, z)."""
    p0, p1, p2, p3 = (float(v) for v in p)
    q0, q1, q2, q3 = (float(v) for v in q)
    return np.array([
        p0 * q0 - p1 * q1 - p2 * q2 - p3 * q3,
        p0 * q1 + p1 * q0 + p2 * q3 - p3 * q2,
        p0 * q2 - p1 * q3 + p2 * q0 + p3 * q1,
        p0 * q3 + p1 * q2 - p2 * q1 + p3 * q0,
    ])


def quat_conj(q) -> np.ndarray:
    q = np.asarray(q, dtype=np.float64)
    return np.array([q[0], -q[1], -q[2], -q[3]])


def _unit(q) -> np.ndarray:
    q = np.asarray(q, dtype=np.float64)
    return q / np.sqrt(np.dot(q, q))


def so4_block(q_left, q_right) -> np.ndarray:
    """4 x 4 matrix of v -> q_L v conj(q_R) (Sec. 3.3, App. B), built column
    by column from the images of the basis quaternions 1, i, j, k."""
    ql, qr = _unit(q_left), _unit(q_right)
    cols = []
    for c in range(4):
        e = np.zeros(4)
        e[c] = 1.0
        cols.append(quat_mul(quat_mul(ql, e), quat_conj(qr)))
    return np.stack(cols, axis=1)


def so3_block(q) -> np.ndarray:
    """Single-quaternion conjugation v -> q v conj(q) (rotation design v1 of
    the ablation in Sec. 4.6 / App. B): an SO(3) action fixing the real axis."""
    return so4_block(q, q)


def block_diag_so4(quats_head) -> np.ndarray:
    """d x d block-diagonal R_SO(4) for one head's [d/4][2][4] parameters."""
    nb = quats_head.shape[0]
    r = np.zeros((4 * nb, 4 * nb))
    for i in range(nb):
        r[4 * i:4 * i + 4, 4 * i:4 * i + 4] = so4_block(quats_head[i, 0], quats_head[i, 1])
    return r


def rotation_matrix(quats_head) -> np.ndarray:
    """R = R_SO(4) H_d for one head (Eq. 2): first the WHT global mix, then
    the per-block SO(4) maps.  Orthogonal, so R^{-1} = R^T (Sec. 3.4)."""
    d = 4 * quats_head.shape[0]
    return block_diag_so4(quats_head) @ hadamard(d)


def rotation_matrices(quats) -> np.ndarray:
    """Stack of R for every head: [n_heads][d][d]."""
    return np.stack([rotation_matrix(quats[h]) for h in range(quats.shape[0])])


# --------------------------------------------------------------------------
# Designs of the rotation ablation (Sec. 4.6, "Rotation Design Ablation", and
# its table of designs; the rotation comparison table of Sec. 2)
# --------------------------------------------------------------------------

# v1: one quaternion per block, v -> q v conj(q) (an SO(3) action), no WHT;
# v2: the paired SO(4) blocks without the WHT pre-mix;
# v3: the method, R_SO(4) H_d (Eq. 2);
# wht: H_d alone (the Hadamard row of the comparison table);
# wht_so3: H_d followed by v1's single-quaternion blocks (the variant of v1
#   that the GPU kernels can run unchanged: q_R = q_L);
# dense: a Haar-random dense orthogonal matrix (the dense-random row);
# none: no rotation.
VARIANTS = ("v1_so3", "v2_so4", "v3_wht_so4", "wht", "wht_so3", "dense", "none")


def dense_orthogonal(gaussian) -> np.ndarray:
    """Haar-distributed orthogonal matrix from a d x d matrix of independent
    standard normal entries: the Q factor of its QR factorization with the
    column signs chosen so that the triangular factor has a positive
    diagonal (the sign fix that makes Q Haar distributed; Mezzadri, Notices
    of the AMS 54(5), 2007).  The entries are passed in (drawn by the seeded
    input generator)."""
    g = np.asarray(gaussian, dtype=np.float64)
    q, r = np.linalg.qr(g)
    return q * np.sign(np.diag(r))[None, :]


def block_diag_so3(quats_head) -> np.ndarray:
    """d x d block diagonal of v -> q v conj(q) with q = each block's q_L."""
    nb = quats_head.shape[0]
    r = np.zeros((4 * nb, 4 * nb))
    for i in range(nb):
        r[4 * i:4 * i + 4, 4 * i:4 * i + 4] = so3_block(quats_head[i, 0])
    return r


def variant_rotation(variant: str, quats_head, gaussian=None) -> np.ndarray:
    """d x d orthogonal rotation of one head for a design of the ablation
    (names in VARIANTS).  quats_head: [d/4][2][4]; ``gaussian`` (d x d
    standard normal entries) only for "dense"."""
    d = 4 * quats_head.shape[0]
    if variant == "v1_so3":
        return block_diag_so3(quats_head)
    if variant == "v2_so4":
        return block_diag_so4(quats_head)
    if variant == "v3_wht_so4":
        return rotation_matrix(quats_head)
    if variant == "wht":
        return hadamard(d)
    if variant == "wht_so3":
        return block_diag_so3(quats_head) @ hadamard(d)
    if variant == "dense":
        if gaussian is None:
            raise ValueError("the dense design needs its Gaussian entries")
        return dense_orthogonal(gaussian)
    if variant == "none":
        return np.eye(d)
    raise ValueError(f"unknown rotation design {variant!r}")


def variant_quaternions(variant: str, seed: int, n_heads: int, d: int = 128) -> np.ndarray:
    """Stored parameters of the designs the structured kernels run as they
    are (R = R_blocks H_d): "v3_wht_so4" the seeded pairs, "wht_so3" the
    same draws with q_R replaced by q_L, "wht" identity quaternions."""
    if variant == "v3_wht_so4":
        return make_quaternions(seed, n_heads, d)
    if variant == "wht_so3":
        q = make_quaternions(seed, n_heads, d)
        q[:, :, 1] = q[:, :, 0]
        return q
    if variant == "wht":
        return identity_quaternions(n_heads, d)
    raise ValueError(f"design {variant!r} is not of the form R_blocks H_d")
