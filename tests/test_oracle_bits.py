"""Pins for the oracle at the other bit widths of Algorithm 1 (b = 2 and
b = 4; Sec. 3.2 Steps 3-4 are stated for a general b with codebook C_b):
Max's 1960 Gaussian tables for 4 and 16 levels, the centroid and midpoint
conditions by quadrature, Monte Carlo, the stored format, bit positions by
brute force, the nearest-level rule in exact arithmetic, attention by
explicit loops, and the distortion of the whole pipeline."""

import math
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import integrate

from oracle import attention as att
from oracle import codebook as cb
from oracle import compress as cz
from oracle import rotation as rot

BOOKS = {b: cb.isoquant_codebook(128, b) for b in (2, 3, 4)}


def test_bits_of():
    for b, (levels, thr) in BOOKS.items():
        assert cz.bits_of(levels) == b and cz.bits_of(thr) == b
    with pytest.raises(ValueError):
        cz.bits_of(np.zeros(6))


def _read_table(path):
    rows = {"threshold": [], "level": [], "mse": []}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                kind, val = line.split()
                rows[kind].append(float(val))
    return rows


@pytest.mark.parametrize("n", [4, 16])
def test_gaussian_lloyd_reproduces_max_table(golden_dir, n):
    """The generic Lloyd iteration on N(0,1) reproduces Max's printed N = 4
    and N = 16 columns to within one unit of the last printed digit."""
    table = _read_table(os.path.join(golden_dir, f"max1960_gaussian_{n}level.txt"))
    levels, thr = cb.lloyd_max(cb.GaussianModel(), n)
    assert len(table["level"]) == n // 2 and len(table["threshold"]) == n // 2 - 1
    for got, want in zip(levels[n // 2:], table["level"]):
        assert abs(got - want) <= 10 ** (np.floor(np.log10(want)) - 3)
    for got, want in zip(thr[n // 2:], table["threshold"]):
        assert abs(got - want) <= 10 ** (np.floor(np.log10(want)) - 3)
    assert abs(thr[n // 2 - 1]) < 1e-14
    mse = cb.distortion(cb.GaussianModel(), levels, thr)
    # the printed MSE column carries the hand-era numerics' error in its
    # last digit (0.009497 at N = 16 against 0.009501)
    assert abs(mse - table["mse"][0]) < 1e-3 * table["mse"][0]


@pytest.mark.parametrize("bits", [2, 4])
def test_sphere_codebook_optimality_conditions(bits):
    """Centroid condition (by quadrature of (1 - t^2)^((d-3)/2)) and midpoint
    condition hold for the 4- and 16-level sphere codebooks."""
    d = 128
    levels, thr = cb.sphere_codebook(d, bits)
    f = lambda t: (1.0 - t * t) ** ((d - 3) / 2)
    edges = np.concatenate([[-1.0], thr, [1.0]])
    for j in range(2 ** bits):
        num = integrate.quad(lambda t: t * f(t), edges[j], edges[j + 1], epsabs=0,
                             epsrel=1e-13)[0]
        den = integrate.quad(f, edges[j], edges[j + 1], epsabs=0, epsrel=1e-13)[0]
        assert abs(num / den - levels[j]) < 1e-12
    np.testing.assert_allclose(thr, 0.5 * (levels[:-1] + levels[1:]), atol=1e-16)
    np.testing.assert_allclose(levels, -levels[::-1], atol=1e-15)


@pytest.mark.parametrize("bits", [2, 4])
def test_sphere_codebook_monte_carlo(bits):
    """Conditional means of a coordinate of sampled unit vectors within the
    oracle's cells equal its levels; the empirical MSE equals its
    distortion."""
    d = 128
    g = np.random.default_rng(11 + bits)
    x = g.standard_normal((100000, d))
    t = (x / np.linalg.norm(x, axis=1, keepdims=True)).ravel()
    levels, thr = cb.sphere_codebook(d, bits)
    cell = np.searchsorted(thr, t, side="right")
    for j in range(2 ** bits):
        sel = t[cell == j]
        se = sel.std() / np.sqrt(sel.size)
        assert abs(sel.mean() - levels[j]) < 5 * se
    mse = np.mean((t - levels[cell]) ** 2)
    want = cb.distortion(cb.SphereMarginalModel(d), levels, thr)
    assert abs(mse - want) / want < 0.01


@pytest.mark.parametrize("bits,lo,hi", [(2, 0.113, 0.1175), (4, 0.0091, 0.0095)])
def test_stored_codebook_format(bits, lo, hi):
    """Stored levels fp16-exact and symmetric, thresholds their exact fp32
    midpoints with 0 in the middle; d times the per-coordinate MSE just
    below the Gaussian value (0.1175 at 4 levels, 0.009497 at 16); the
    unrounded levels keep a margin from fp16 rounding boundaries."""
    stored, thr = BOOKS[bits]
    raw, _ = cb.sphere_codebook(128, bits)
    n = 2 ** bits
    assert stored.shape == (n,) and thr.shape == (n - 1,)
    assert np.array_equal(stored.astype(np.float16).astype(np.float64), stored)
    assert np.array_equal(stored, -stored[::-1])
    assert np.array_equal(thr, 0.5 * (stored[:-1] + stored[1:]))
    assert np.array_equal(thr.astype(np.float32).astype(np.float64), thr)
    assert thr[n // 2 - 1] == 0.0
    assert np.all(np.abs(stored - raw) <= np.abs(raw) * 2.0 ** -11)
    d_st = cb.distortion(cb.SphereMarginalModel(128), stored, thr)
    assert lo < 128 * d_st < hi
    for v in raw[n // 2:]:
        h = np.float16(v)
        up = float(np.nextafter(h, np.float16(1)))
        dn = float(np.nextafter(h, np.float16(0)))
        assert min(abs(v - 0.5 * (float(h) + up)), abs(v - 0.5 * (float(h) + dn))) > 1e-9


@pytest.mark.parametrize("bits", [2, 4])
def test_pack_bit_positions_brute_force(bits):
    """Setting bit j of code i sets exactly bit b*i + j of the d*b/8-byte
    record; packing round-trips."""
    nbytes = 16 * bits
    for i in range(128):
        for j in range(bits):
            codes = np.zeros(128, np.uint8)
            codes[i] = 1 << j
            rec = cz.pack(codes, bits)
            assert rec.shape == (nbytes,)
            bitlist = [(int(rec[n // 8]) >> (n % 8)) & 1 for n in range(8 * nbytes)]
            assert sum(bitlist) == 1 and bitlist[bits * i + j] == 1
    g = np.random.default_rng(bits)
    codes = g.integers(0, 2 ** bits, size=(17, 128), dtype=np.uint8)
    assert np.array_equal(cz.unpack(cz.pack(codes, bits), 128, bits), codes)


@pytest.mark.parametrize("bits", [2, 4])
def test_quantizer_matches_brute_force_nearest_level(bits):
    """Code = index of the nearest stored level in exact rational arithmetic,
    ties to the higher index, at every threshold, its neighbours and every
    level."""
    levels, thr = BOOKS[bits]
    pts = [0.0, -0.0, 1.0, -1.0, 0.3, -0.3]
    for t in thr:
        up = dn = float(t)
        pts.append(up)
        for _ in range(2):
            up, dn = np.nextafter(up, np.inf), np.nextafter(dn, -np.inf)
            pts += [up, dn]
    pts += [float(c) for c in levels] + list(np.linspace(-0.35, 0.35, 2001))

    def nearest(y):
        yf = Fraction(float(y))
        best, best_d = 0, None
        for k, c in enumerate(levels):
            dist = abs(yf - Fraction(float(c)))
            if best_d is None or dist <= best_d:
                best, best_d = k, dist
        return best

    got = cz.quantize(np.array(pts), thr)
    assert list(got) == [nearest(y) for y in pts]


def _cache(seed, bits, hkv, t, hq):
    g = np.random.default_rng(seed)
    levels, thr = BOOKS[bits]
    quats = rot.make_quaternions(seed, hkv)
    rots = rot.rotation_matrices(quats)
    k = (g.standard_normal((1, hkv, t, 128)) * g.lognormal(0, 0.5, 128)).astype(np.float32)
    v = (g.standard_normal((1, hkv, t, 128)) * g.lognormal(0, 0.5, 128)).astype(np.float32)
    kp, kn, *_ = cz.compress_kv(k, rots, thr)
    vp, vn, *_ = cz.compress_kv(v, rots, thr)
    q = g.standard_normal((1, hq, 128)).astype(np.float32)
    return q, kp, kn, vp, vn, quats, rots, levels


@pytest.mark.parametrize("bits", [2, 4])
def test_fused_brute_force_loops(bits):
    """App. A decode at b bits recomputed with explicit Python loops (codes
    read bit by bit from the records), so a wrong record size or bit order
    in the oracle's vectorized unpacking would show."""
    q, kp, kn, vp, vn, quats, rots, levels = _cache(3, bits, 1, 4, 2)
    assert kp.shape[-1] == 16 * bits
    d = 128
    r = rots[0]

    def code(rec, i):
        return sum(((int(rec[(bits * i + j) // 8]) >> ((bits * i + j) % 8)) & 1) << j
                   for j in range(bits))

    got = att.decode_fused(q, kp, kn, vp, vn, [4], quats, levels)
    for h in range(2):
        qt = [sum(r[i][j] * float(q[0, h, j]) for j in range(d)) for i in range(d)]
        scores = []
        for t in range(4):
            dot = sum(qt[i] * float(levels[code(kp[0, 0, t], i)]) for i in range(d))
            scores.append(float(kn[0, 0, t]) * dot / math.sqrt(d))
        m = max(scores)
        e = [math.exp(s - m) for s in scores]
        z = sum(e)
        ot = [sum(e[t] / z * float(vn[0, 0, t]) * float(levels[code(vp[0, 0, t], i)])
                  for t in range(4)) for i in range(d)]
        o = [sum(r[i][j] * ot[i] for i in range(d)) for j in range(d)]
        np.testing.assert_allclose(got[0, h], o, rtol=0, atol=1e-12 * max(map(abs, o)))


@pytest.mark.parametrize("bits", [2, 4])
def test_fused_equals_reconstruct(bits):
    """q . R^T k_hat = (R q) . k_hat at b bits too (orthogonality)."""
    q, kp, kn, vp, vn, quats, _, levels = _cache(5, bits, 2, 23, 8)
    a = att.decode_fused(q, kp, kn, vp, vn, [23], quats, levels)
    b = att.decode_reconstruct(q, kp, kn, vp, vn, [23], quats, levels)
    assert np.max(np.abs(a - b)) <= 1e-12 * np.max(np.abs(b))


def test_pipeline_distortion_by_bits():
    """Relative squared reconstruction error of Algorithm 1 on isotropic
    inputs equals d times the codebook's per-coordinate MSE at every b
    (0.116, 0.034, 0.0093), so it falls by ~3.4x per added bit."""
    g = np.random.default_rng(4)
    x = g.standard_normal((4000, 128))
    r = rot.rotation_matrix(rot.make_quaternions(9, 1)[0])
    errs = {}
    for bits, (levels, thr) in BOOKS.items():
        _, norm, codes, _, _ = cz.compress(x, r, thr)
        xr = cz.reconstruct(codes, norm, levels, r)
        errs[bits] = np.mean(np.sum((xr - x) ** 2, axis=1) / np.sum(x ** 2, axis=1))
        want = 128 * cb.distortion(cb.SphereMarginalModel(128), levels, thr)
        assert abs(errs[bits] - want) < 0.03 * want
    assert errs[2] > 3 * errs[3] > 9 * errs[4]
