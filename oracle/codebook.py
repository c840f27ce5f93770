"""Lloyd-Max scalar codebooks (Sec. 3.2, Step 3).  Test infrastructure only.

Step 3 of the compression pipeline quantizes every coordinate of the rotated
unit vector to ``b`` bits with a Lloyd-Max codebook, i.e. the set of levels
that minimizes the expected squared error under the marginal distribution of
one coordinate after the rotation.  Two facts fix the codebook:

* Lloyd-Max optimality: each decision threshold is the midpoint of its two
  neighbouring levels, and each level is the conditional mean of its cell.
  The alternating fixed-point iteration below (Lloyd's "Method I") is the
  textbook way to reach that point.
* The marginal: the rotation spreads a unit vector isotropically (the
  "Why structured rotation works" paragraph of Sec. 3.2), so one coordinate
  of a uniform point on the sphere S^(d-1) is the distribution quantized.
  Its density is proportional to (1 - t^2)^((d-3)/2) on [-1, 1].

Reading (the paper ships its codebook files only in its code archive): the
levels are the analytic sphere-marginal Lloyd-Max levels at d = 128, b = 3,
stored rounded to the nearest IEEE half-precision value, and the thresholds
are the exact midpoints of those stored levels, so "nearest stored level" and
"count of thresholds at or below the value" agree exactly.
"""

from __future__ import annotations

import numpy as np
from scipy import special


# --------------------------------------------------------------------------
# Distribution models: partial moments  M_m(a, b) = integral_a^b t^m f(t) dt
# for m = 0, 1, 2.  Lloyd's iteration needs m = 0, 1; the distortion needs 2.
# --------------------------------------------------------------------------

class GaussianModel:
    """Standard normal N(0, 1).  Used to pin the Lloyd machinery to the
    textbook Gaussian table (Max 1960) and as the d -> infinity limit of the
    sphere marginal."""

    support = (-np.inf, np.inf)

    @staticmethod
    def _anti(m: int, t):
        t = np.asarray(t, dtype=np.float64)
        phi = np.exp(-0.5 * t * t) / np.sqrt(2.0 * np.pi)
        phi = np.where(np.isfinite(t), phi, 0.0)
        big_phi = special.ndtr(t)
        if m == 0:
            return big_phi
        if m == 1:
            return -phi
        if m == 2:
            with np.errstate(invalid="ignore"):
                tphi = np.where(np.isfinite(t), t * phi, 0.0)
            return big_phi - tphi
        raise ValueError(m)

    def moment(self, m: int, a, b):
        return self._anti(m, b) - self._anti(m, a)


class SphereMarginalModel:
    """One coordinate of a uniform point on S^(d-1): density
    f(t) = (1 - t^2)^k / B(1/2, k + 1) on [-1, 1] with k = (d - 3) / 2.

    Partial moments use the substitution u = t^2:
    integral_0^x t^m (1 - t^2)^k dt = 1/2 * B(x^2; (m + 1)/2, k + 1),
    with B(x; p, q) the (unregularized) incomplete beta function, extended to
    negative x by the parity of the integrand."""

    support = (-1.0, 1.0)

    def __init__(self, d: int):
        if d < 3:
            raise ValueError("sphere marginal needs d >= 3")
        self.d = d
        self.k = (d - 3) / 2.0
        self.norm = special.beta(0.5, self.k + 1.0)

    def _anti(self, m: int, t):
        t = np.asarray(t, dtype=np.float64)
        p = (m + 1) / 2.0
        q = self.k + 1.0
        x = np.minimum(t * t, 1.0)
        half = 0.5 * special.betainc(p, q, x) * special.beta(p, q)
        # t^m (1-t^2)^k is odd in t for even m (antiderivative odd), even for
        # odd m (antiderivative even).
        sign = np.sign(t) if m % 2 == 0 else 1.0
        return sign * half / self.norm

    def moment(self, m: int, a, b):
        return self._anti(m, b) - self._anti(m, a)


# --------------------------------------------------------------------------
# Lloyd-Max iteration
# --------------------------------------------------------------------------

def lloyd_max(model, n_levels: int, init=None, tol: float = 1e-15,
              max_iter: int = 200000):
    """Lloyd's alternating optimization for a scalar quantizer.

    thresholds <- midpoints of adjacent levels (nearest-neighbour condition);
    levels     <- conditional mean of each cell (centroid condition);
    repeated until no level moves by more than ``tol``.

    Returns (levels, thresholds), both ascending fp64 arrays.
    """
    lo, hi = model.support
    if init is None:
        # start from levels spread over the bulk of the distribution
        spread = 2.0 if not np.isfinite(hi) else 2.0 / np.sqrt(getattr(model, "d", 4))
        init = np.linspace(-spread, spread, n_levels)
    c = np.array(init, dtype=np.float64)
    for _ in range(max_iter):
        t = 0.5 * (c[:-1] + c[1:])
        edges = np.concatenate([[lo], t, [hi]])
        mass = model.moment(0, edges[:-1], edges[1:])
        first = model.moment(1, edges[:-1], edges[1:])
        c_new = first / mass
        moved = np.max(np.abs(c_new - c))
        c = c_new
        if moved < tol:
            break
    else:
        raise RuntimeError("Lloyd-Max iteration did not converge")
    return c, 0.5 * (c[:-1] + c[1:])


def distortion(model, levels, thresholds) -> float:
    """Expected squared error E[(T - Q(T))^2] of the quantizer that maps each
    cell [t_{j-1}, t_j) to levels[j], computed from partial moments."""
    lo, hi = model.support
    edges = np.concatenate([[lo], np.asarray(thresholds, float), [hi]])
    a, b = edges[:-1], edges[1:]
    c = np.asarray(levels, dtype=np.float64)
    m0 = model.moment(0, a, b)
    m1 = model.moment(1, a, b)
    m2 = model.moment(2, a, b)
    return float(np.sum(m2 - 2.0 * c * m1 + c * c * m0))


def sphere_codebook(d: int = 128, bits: int = 3):
    """Unrounded Lloyd-Max levels/thresholds for one coordinate of a uniform
    point on S^(d-1) (Sec. 3.2 Step 3, marginal read analytically)."""
    return lloyd_max(SphereMarginalModel(d), 2 ** bits)


def isoquant_codebook(d: int = 128, bits: int = 3):
    """The codebook C_b used by the compression pipeline (Alg. 1 input).

    Levels: sphere-marginal Lloyd-Max levels rounded to the nearest IEEE
    half-precision value (reading of the silent storage format).
    Thresholds: exact midpoints of the stored levels (nearest-level rule).
    Both returned as fp64 arrays whose values are exact in fp16 (levels) and
    fp32 (thresholds).
    """
    levels, _ = sphere_codebook(d, bits)
    stored = levels.astype(np.float16).astype(np.float64)
    if not np.array_equal(stored, -stored[::-1]):
        raise AssertionError("stored codebook is not symmetric")
    thresholds = 0.5 * (stored[:-1] + stored[1:])
    return stored, thresholds


# --------------------------------------------------------------------------
# Empirical codebook (Sec. 3.2 Step 3 on calibration data)
# --------------------------------------------------------------------------

def rotated_coordinates(x, rot):
    """Post-rotation coordinates of calibration vectors: R x / ||x|| in fp64
    for every non-zero finite row of x ([n][d]); rot is the d x d matrix R of
    Eq. 2 (rotation.rotation_matrix).  Returns [m][d]."""
    x = np.asarray(x, dtype=np.float64)
    n2 = np.einsum("nd,nd->n", x, x)
    keep = np.isfinite(n2) & (n2 > 0)
    x = x[keep]
    return (x / np.sqrt(n2[keep])[:, None]) @ np.asarray(rot, np.float64).T


def empirical_lloyd_max(samples, n_levels: int, init, max_iter: int = 10000):
    """Lloyd's iteration on the empirical distribution of `samples` made
    symmetric (the sample and its negation), the fixed point the paper's
    Step 3 asks for when the marginal is measured instead of derived.

    Cells follow the coding rule of the pipeline: cell j holds the values y
    with t_(j-1) <= y < t_j.  thresholds <- midpoints of adjacent levels;
    levels <- mean of the sample values in each cell (an empty cell keeps
    its level).  On a finite sample the cells stop changing after finitely
    many steps and the levels are then exact fixed points.
    Returns (levels, thresholds), unrounded fp64."""
    y = np.asarray(samples, dtype=np.float64).ravel()
    y = np.sort(np.concatenate([y, -y]))
    c = np.array(init, dtype=np.float64)
    for _ in range(max_iter):
        t = 0.5 * (c[:-1] + c[1:])
        cells = np.split(y, np.searchsorted(y, t, side="left"))
        c_new = np.array([cell.mean() if cell.size else c[j] for j, cell in enumerate(cells)])
        if np.array_equal(c_new, c):
            break
        c = c_new
    else:
        raise RuntimeError("empirical Lloyd-Max did not reach a fixed point")
    return c, 0.5 * (c[:-1] + c[1:])


def empirical_isoquant_codebook(samples, bits: int = 3, d: int = 128):
    """A fitted codebook in the library's storage format: empirical
    Lloyd-Max levels (started from the sphere-marginal levels) rounded to
    the nearest half-precision value, made exactly symmetric, thresholds the
    midpoints of the stored levels.  Also returns the unrounded levels."""
    init, _ = sphere_codebook(d, bits)
    levels, _ = empirical_lloyd_max(samples, 2 ** bits, init)
    stored = levels.astype(np.float16).astype(np.float64)
    n = stored.size
    stored[: n // 2] = -stored[::-1][: n // 2]
    return stored, 0.5 * (stored[:-1] + stored[1:]), levels
