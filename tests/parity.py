"""Shared helpers for the GPU parity tests (compare the HIP path with the
oracle on identical seeded inputs)."""

from __future__ import annotations

import numpy as np

from oracle import compress as ocz

# Tolerances (fixed by the benchmark spec of the hot path):
#  * packed codes and norms bit-exact, except elements within 1e-6 of a
#    decision boundary (measured on the oracle's fp64 rotated coordinate);
#    those may differ by one level and must be <= 1e-5 of all elements;
#  * attention outputs within 2e-3 relative error per output row
#    (max-abs error / max-abs oracle value), fp32 GPU vs fp64 oracle.
BOUNDARY_WINDOW = 1e-6
MISMATCH_FRACTION = 1e-5
ATTN_RTOL = 2e-3


def check_codes(gpu_packed, oracle_codes, oracle_y, thresholds, label=""):
    """Compare GPU records with the oracle's codes (code width b read off the
    thresholds of C_b).  Returns the number of (allowed) boundary
    mismatches."""
    g = ocz.unpack(np.asarray(gpu_packed), 128, ocz.bits_of(thresholds))
    o = np.asarray(oracle_codes)
    assert g.shape == o.shape, (g.shape, o.shape)
    bad = g != o
    n = int(np.count_nonzero(bad))
    if n:
        gi = g[bad].astype(np.int64)
        oi = o[bad].astype(np.int64)
        assert np.all(np.abs(gi - oi) == 1), f"{label}: code off by more than one level"
        y = np.asarray(oracle_y)[bad]
        t = np.asarray(thresholds)[np.minimum(gi, oi)]
        dist = np.abs(y - t)
        assert np.all(dist < BOUNDARY_WINDOW), (
            f"{label}: {n} mismatches, farthest {dist.max():.3e} from its boundary")
    assert n <= MISMATCH_FRACTION * o.size, f"{label}: {n} mismatches of {o.size}"
    return n


def check_norms(gpu_norms, oracle_s64, label=""):
    """Stored scale = fp32 rounding of the fp64 norm; a mismatch is allowed
    only where the fp64 norm lies within 1e-12 (relative) of an fp32
    rounding midpoint.  Returns the mismatch count."""
    gn = np.asarray(gpu_norms, dtype=np.float32)
    s = np.asarray(oracle_s64, dtype=np.float64)
    want = s.astype(np.float32)
    bad = gn.view(np.uint32) != want.view(np.uint32)
    n = int(np.count_nonzero(bad))
    if n:
        sb = s[bad]
        lo = np.minimum(gn[bad], want[bad]).astype(np.float64)
        hi = np.maximum(gn[bad], want[bad]).astype(np.float64)
        assert np.all(np.nextafter(lo.astype(np.float32), np.float32(np.inf)) == hi.astype(np.float32))
        mid = 0.5 * (lo + hi)
        assert np.all(np.abs(sb - mid) <= 1e-12 * sb), f"{label}: norm off an fp32 midpoint"
    assert n <= MISMATCH_FRACTION * s.size, f"{label}: {n} norm mismatches of {s.size}"
    return n


def row_rel_err(got, ref):
    """Per output row: max|got - ref| / max|ref| (rows of zeros compare
    absolutely)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.max(np.abs(got - ref), axis=-1)
    den = np.max(np.abs(ref), axis=-1)
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), num)


def check_attention(got, ref, label=""):
    err = row_rel_err(got, ref)
    assert np.all(np.isfinite(got)), f"{label}: non-finite output"
    print(f"[attn] {label}: max row rel err {err.max():.3e}")
    assert np.all(err <= ATTN_RTOL), f"{label}: max row rel err {err.max():.3e}"
    return float(err.max())
