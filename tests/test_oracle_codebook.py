"""Pins for the oracle's Lloyd-Max codebook (Sec. 3.2 Step 3)."""

import os

import numpy as np
import pytest
from scipy import integrate, special

from oracle import codebook as cb


def _read_max_table(golden_dir):
    rows = {"threshold": [], "level": [], "mse": []}
    with open(os.path.join(golden_dir, "max1960_gaussian_8level.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            kind, val = line.split()
            rows[kind].append(float(val))
    return rows


def test_gaussian_lloyd_reproduces_max_table(golden_dir):
    """The generic Lloyd iteration on N(0,1) reproduces Max's printed table
    to within one unit of its last printed digit (the 1960 values were
    computed by hand-era numerics; 0.50055 prints there as 0.5006)."""
    table = _read_max_table(golden_dir)
    levels, thr = cb.lloyd_max(cb.GaussianModel(), 8)
    pos_levels = levels[4:]
    pos_thr = thr[4:]
    for got, want in zip(pos_levels, table["level"]):
        assert abs(got - want) <= 10 ** (np.floor(np.log10(want)) - 3)
    for got, want in zip(pos_thr, table["threshold"]):
        assert abs(got - want) <= 10 ** (np.floor(np.log10(want)) - 3)
    mse = cb.distortion(cb.GaussianModel(), levels, thr)
    assert abs(mse - table["mse"][0]) < 2e-5
    assert abs(thr[3]) < 1e-14


@pytest.mark.parametrize("d", [3, 8, 64, 128, 1024])
def test_sphere_two_level_closed_form(d):
    """1-bit Lloyd-Max on the sphere marginal: threshold 0, levels
    +-E|T| = +-Gamma(d/2) / (sqrt(pi) Gamma((d+1)/2))."""
    levels, thr = cb.lloyd_max(cb.SphereMarginalModel(d), 2, init=[-0.3, 0.2])
    want = np.exp(special.gammaln(d / 2) - special.gammaln((d + 1) / 2)) / np.sqrt(np.pi)
    assert abs(thr[0]) < 1e-14
    np.testing.assert_allclose(levels, [-want, want], rtol=1e-12)


def test_sphere_marginal_moments():
    """Density integrates to 1 and E[T^2] = 1/d (a coordinate of a unit
    vector uniform on the sphere)."""
    for d in (3, 16, 128):
        m = cb.SphereMarginalModel(d)
        assert abs(m.moment(0, -1.0, 1.0) - 1.0) < 1e-13
        assert abs(m.moment(1, -1.0, 1.0)) < 1e-15
        assert abs(m.moment(2, -1.0, 1.0) - 1.0 / d) < 1e-14


def test_sphere_partial_moments_match_quadrature():
    """The incomplete-beta partial moments agree with direct quadrature of
    (1 - t^2)^((d-3)/2), normalized by quadrature too."""
    d = 128
    m = cb.SphereMarginalModel(d)
    f = lambda t: (1.0 - t * t) ** ((d - 3) / 2)
    z = integrate.quad(f, -1, 1, epsabs=0, epsrel=1e-13)[0]
    for a, b in [(-1.0, -0.15), (-0.15, -0.04), (-0.04, 0.0), (0.0, 0.09), (0.09, 1.0)]:
        for k in range(3):
            want = integrate.quad(lambda t: t ** k * f(t), a, b, epsabs=1e-17, epsrel=1e-13)[0] / z
            assert abs(m.moment(k, a, b) - want) < 1e-13


def test_sphere_codebook_optimality_conditions():
    """Centroid condition (by quadrature) and midpoint condition hold."""
    d = 128
    levels, thr = cb.sphere_codebook(d, 3)
    f = lambda t: (1.0 - t * t) ** ((d - 3) / 2)
    edges = np.concatenate([[-1.0], thr, [1.0]])
    for j in range(8):
        num = integrate.quad(lambda t: t * f(t), edges[j], edges[j + 1], epsabs=0, epsrel=1e-13)[0]
        den = integrate.quad(f, edges[j], edges[j + 1], epsabs=0, epsrel=1e-13)[0]
        assert abs(num / den - levels[j]) < 1e-12
    np.testing.assert_allclose(thr, 0.5 * (levels[:-1] + levels[1:]), atol=1e-16)
    np.testing.assert_allclose(levels, -levels[::-1], atol=1e-15)


def test_sphere_codebook_tends_to_gaussian():
    """sqrt(d) * sphere levels -> Max's Gaussian levels as d grows (the
    coordinate of a uniform unit vector, times sqrt(d), tends to N(0,1))."""
    g_levels, _ = cb.lloyd_max(cb.GaussianModel(), 8)
    errs = []
    for d in (128, 2048, 32768):
        levels, _ = cb.sphere_codebook(d, 3)
        errs.append(np.max(np.abs(levels * np.sqrt(d) - g_levels)))
    assert errs[0] > errs[1] > errs[2]
    assert errs[2] < 1e-3


def test_sphere_codebook_monte_carlo():
    """Empirical check on sampled unit vectors: the conditional means of a
    coordinate within the oracle's cells equal the oracle's levels."""
    d = 128
    g = np.random.default_rng(7)
    x = g.standard_normal((200000, d))
    t = (x / np.linalg.norm(x, axis=1, keepdims=True)).ravel()
    levels, thr = cb.sphere_codebook(d, 3)
    cell = np.searchsorted(thr, t, side="right")
    for j in range(8):
        sel = t[cell == j]
        se = sel.std() / np.sqrt(sel.size)
        assert abs(sel.mean() - levels[j]) < 5 * se
    mse = np.mean((t - levels[cell]) ** 2)
    want = cb.distortion(cb.SphereMarginalModel(d), levels, thr)
    assert abs(mse - want) / want < 0.01


def test_stored_codebook_format():
    """Stored levels are fp16-exact and symmetric; thresholds are their exact
    midpoints, representable in fp32; distortion barely moves."""
    stored, thr = cb.isoquant_codebook(128, 3)
    raw, _ = cb.sphere_codebook(128, 3)
    assert np.array_equal(stored.astype(np.float16).astype(np.float64), stored)
    assert np.array_equal(stored, -stored[::-1])
    assert np.array_equal(thr, 0.5 * (stored[:-1] + stored[1:]))
    assert np.array_equal(thr.astype(np.float32).astype(np.float64), thr)
    assert thr[3] == 0.0
    assert np.all(np.abs(stored - raw) <= np.abs(raw) * 2.0 ** -11)
    model = cb.SphereMarginalModel(128)
    d_raw = cb.distortion(model, raw, 0.5 * (raw[:-1] + raw[1:]))
    d_st = cb.distortion(model, stored, thr)
    assert d_raw <= d_st < d_raw * (1 + 1e-5)
    # MSE per coordinate times d: close to the Gaussian 0.0345 (sphere is a
    # bit lighter-tailed)
    assert 0.0335 < 128 * d_st < 0.0346
    # margin from fp16 rounding boundaries, so an independent implementation
    # with ~1e-12 error rounds to the same stored values
    for v in raw[4:]:
        h = np.float16(v)
        up = float(np.nextafter(h, np.float16(1)))
        dn = float(np.nextafter(h, np.float16(0)))
        assert min(abs(v - 0.5 * (float(h) + up)), abs(v - 0.5 * (float(h) + dn))) > 1e-9
