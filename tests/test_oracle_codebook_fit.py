"""Pins for the oracle's empirical codebook (Sec. 3.2 Step 3 measured on
calibration data: Lloyd-Max on the sample of rotated coordinates), and the
library's host fitter (iq_fit_codebook) against it bit for bit."""

import os

import numpy as np
import pytest

from oracle import codebook as cb
from oracle import compress as ocz
from oracle import rotation as orot
from paper_2608_08081_amd import api, synth


def _max_table(golden_dir, name):
    rows = {"threshold": [], "level": []}
    with open(os.path.join(golden_dir, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            kind, val = line.split()
            if kind in rows:
                rows[kind].append(float(val))
    return rows


@pytest.mark.parametrize("name,n", [("max1960_gaussian_8level.txt", 8),
                                    ("max1960_gaussian_4level.txt", 4)])
def test_large_gaussian_sample_gives_max_table(golden_dir, name, n):
    """On 2M standard normal draws the empirical iteration lands on Max's
    printed Gaussian quantizer within the sampling error of the cell means
    (about 1e-3; 5e-3 allowed)."""
    table = _max_table(golden_dir, name)
    x = np.random.default_rng(1).standard_normal(2_000_000)
    levels, thr = cb.empirical_lloyd_max(x, n, np.linspace(-2.0, 2.0, n))
    np.testing.assert_allclose(levels[n // 2:], table["level"], atol=5e-3)
    np.testing.assert_allclose(thr[n // 2:], table["threshold"], atol=5e-3)


def test_fixed_point_conditions_on_the_sample():
    """At the returned point every level is the mean of the (symmetrized)
    sample values of its cell, recomputed here cell by cell with explicit
    masks, and every threshold the midpoint of its neighbours."""
    rng = np.random.default_rng(2)
    x = rng.standard_t(4.0, size=50_000) * 0.05
    init, _ = cb.sphere_codebook(128, 3)
    levels, thr = cb.empirical_lloyd_max(x, 8, init)
    y = np.concatenate([x, -x])
    edges = np.concatenate([[-np.inf], thr, [np.inf]])
    for j in range(8):
        cell = y[(y >= edges[j]) & (y < edges[j + 1])]
        assert cell.size > 0
        assert abs(cell.mean() - levels[j]) <= 1e-12 * abs(levels[j])
    np.testing.assert_array_equal(thr, 0.5 * (levels[:-1] + levels[1:]))
    np.testing.assert_allclose(levels, -levels[::-1], rtol=0, atol=1e-15)


def test_iteration_does_not_increase_the_sample_error():
    """Lloyd's steps never increase the mean squared error on the sample,
    so the fitted levels quantize it at least as well as the starting
    (sphere-marginal) levels."""
    rng = np.random.default_rng(3)
    x = rng.standard_t(4.0, size=40_000) * 0.04
    y = np.concatenate([x, -x])
    init, init_thr = cb.sphere_codebook(128, 3)
    levels, thr = cb.empirical_lloyd_max(x, 8, init)

    def mse(lv, th):
        code = np.searchsorted(th, y, side="right")
        return np.mean((y - lv[code]) ** 2)

    assert mse(levels, thr) <= mse(init, init_thr)
    assert mse(levels, thr) < 0.9 * mse(init, init_thr)   # a heavy-tailed sample moves it


def test_isotropic_input_gives_the_sphere_codebook():
    """Rotated coordinates of isotropic Gaussian vectors are samples of the
    sphere marginal; the fitted levels approach the analytic codebook
    (2.56M coordinates: relative error a few 1e-3)."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((20_000, 128))
    rot = orot.rotation_matrices(orot.make_quaternions(5, 1))[0]
    y = cb.rotated_coordinates(x, rot)
    levels, _ = cb.empirical_lloyd_max(y, 8, cb.sphere_codebook(128, 3)[0])
    want, _ = cb.sphere_codebook(128, 3)
    np.testing.assert_allclose(levels, want, rtol=5e-3)


def test_rotated_coordinates_match_the_compression_path():
    """rotated_coordinates = the y of compress_kv (R x / ||x||), rows of
    unit norm; zero and non-finite rows are dropped."""
    w = synth.Workload(91, "cbfit", 1, 8, 2, 64, "f32")
    k = synth.kv_tensor(0, w, "k")
    quats = orot.make_quaternions(9, 2)
    rots = orot.rotation_matrices(quats)
    _, _, _, y, _ = ocz.compress_kv(k, rots, cb.isoquant_codebook(128, 3)[1])
    for h in range(2):
        got = cb.rotated_coordinates(k[0, h], rots[h])
        np.testing.assert_allclose(got, y[0, h], rtol=0, atol=1e-14)
        np.testing.assert_allclose(np.sum(got * got, axis=1), 1.0, atol=1e-13)
    x = np.vstack([np.zeros((1, 128)), np.full((1, 128), np.nan), k[0, 0, :3]])
    assert cb.rotated_coordinates(x, rots[0]).shape == (3, 128)


def test_storage_format():
    """Stored levels are fp16 values, exactly symmetric, thresholds their
    midpoints (the format the kernels take)."""
    x = np.random.default_rng(6).standard_normal((4000, 128))
    y = cb.rotated_coordinates(x * np.linspace(0.1, 3.0, 128), np.eye(128))
    for bits in (2, 3, 4):
        lv, th, raw = cb.empirical_isoquant_codebook(y, bits)
        assert lv.size == 2 ** bits and th.size == 2 ** bits - 1
        np.testing.assert_array_equal(lv.astype(np.float16).astype(np.float64), lv)
        np.testing.assert_array_equal(lv, -lv[::-1])
        np.testing.assert_array_equal(th, 0.5 * (lv[:-1] + lv[1:]))
        assert np.all(np.diff(lv) > 0)
        assert np.max(np.abs(lv - raw)) <= np.max(np.abs(raw)) * 2.0 ** -11


@pytest.mark.parametrize("dist,bits,seed", [("anisotropic", 3, 0), ("heavy_tailed", 3, 1),
                                            ("anisotropic", 2, 2), ("heavy_tailed", 4, 3)])
def test_library_fitter_equals_oracle(dist, bits, seed):
    """iq_fit_codebook (host C++, own WHT, quaternion products and prefix
    sums) returns the oracle's stored codebook bit for bit."""
    w = synth.Workload(92, "cbfit", 1, 16, 2, 3000, "f16", kv_dist=dist)
    k = synth.kv_tensor(seed, w, "k")[0].astype(np.float32)
    k[0, 5] = 0.0                           # a zero vector is skipped
    quats = orot.make_quaternions(40 + seed, 2)
    rots = orot.rotation_matrices(quats)
    y = np.concatenate([cb.rotated_coordinates(k[h], rots[h]) for h in range(2)])
    want_lv, want_th, _ = cb.empirical_isoquant_codebook(y, bits)
    got = api.iq_fit_codebook(k, quats, bits)
    lv, th = api.codebook_arrays(got)
    assert got.bits == bits
    np.testing.assert_array_equal(lv.astype(np.float64), want_lv)
    np.testing.assert_array_equal(th.astype(np.float64), want_th)
