"""Synthetic study of the rotation designs of the ablation (Sec. 4.6,
"Rotation Design Ablation", and its table of designs; the rotation
comparison table of Sec. 2).  Test infrastructure only.

For each design (oracle.rotation.VARIANTS) and seeded anisotropic K/V shaped
like the paper's MoE attention layers (oracle-independent generator
paper_2608_08081_amd.synth), three quantities:

* distortion: mean over vectors of ||x - x_hat||^2 / ||x||^2, x_hat the
  3-bit reconstruction s R^T C[code] (Alg. 1, Steps 1-4);
* coordinate energy: d * mean over vectors of (R x / ||x||)_i^2 for each
  coordinate i (1 everywhere is the isotropy the WHT is meant to give,
  Sec. 3.3 and Eq. 4); reported as its minimum and maximum over i and the
  share of coordinates whose energy the rotation leaves exactly as it was
  (the "dims unmixed" failure of design v1);
* attention error of the compressed-space decode (App. A) against fp64
  attention on the unquantized K/V (context, not a target): the relative l2
  error of the output rows, and the RMS error of the scores relative to the
  spread of the exact scores.

The paper's quality gate (five prompts on the real models) is not
reproduced: it needs the models.  Run ``python -m oracle.rotation_study``
for the table.
"""

from __future__ import annotations

import numpy as np

from . import attention as _att
from . import codebook as _cb
from . import compress as _cz
from . import rotation as _rot


def rotations(variant: str, seed: int, n_heads: int, gaussian=None, d: int = 128):
    """[n_heads][d][d] rotation matrices of one design (seeded quaternion
    pairs, shared by all designs that use quaternions)."""
    quats = _rot.make_quaternions(seed, n_heads, d)
    return np.stack([_rot.variant_rotation(variant, quats[h],
                                           None if gaussian is None else gaussian[h])
                     for h in range(n_heads)])


def distortion(x, rots, thresholds, levels):
    """Mean relative squared reconstruction error of x ([B][H][T][d])."""
    packed, norms, *_ = _cz.compress_kv(x, rots, thresholds)
    xh = _cz.reconstruct_kv(packed, norms, rots, levels)
    x = np.asarray(x, dtype=np.float64)
    num = np.sum((x - xh) ** 2, axis=-1)
    den = np.sum(x * x, axis=-1)
    ok = den > 0
    return float(np.mean(num[ok] / den[ok]))


def coordinate_energy(x, rots):
    """d * mean over vectors of the squared rotated unit-vector coordinates,
    per (head, coordinate): [H][d]."""
    x = np.asarray(x, dtype=np.float64)
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    u = np.where(n > 0, x / np.where(n > 0, n, 1.0), 0.0)          # [B][H][T][d]
    y = np.einsum("hij,bhtj->bhti", rots, u)
    d = x.shape[-1]
    return d * np.mean(y * y, axis=(0, 2))


def unmixed_share(x, rots, tol=1e-12):
    """Share of coordinates (over heads) whose energy the rotation leaves
    unchanged for every vector: (R x)_i = x_i exactly, i.e. R fixes e_i."""
    d = rots.shape[-1]
    eye = np.eye(d)
    fixed = np.all(np.abs(rots - eye[None]) <= tol, axis=1) & (np.abs(np.diagonal(rots, axis1=1, axis2=2) - 1) <= tol)
    return float(np.mean(fixed))


def attention_error(q, k, v, seq_lens, rots, thresholds, levels, scale=None):
    """Errors of compressed-space decode (App. A) against fp64 attention on
    the unquantized K/V: (mean over rows of ||o - o_exact||_2 /
    ||o_exact||_2, RMS score error / RMS spread of the exact scores).  The
    second isolates the key side: score_j = s^K_j (R q . C[code_j]) * scale
    against q . k_j * scale."""
    q = np.asarray(q, dtype=np.float64)
    kp, kn, *_ = _cz.compress_kv(k, rots, thresholds)
    vp, vn, *_ = _cz.compress_kv(v, rots, thresholds)
    got = _att.decode_fused_rotations(q, kp, kn, vp, vn, seq_lens, rots, levels, scale)
    ref = _att.attention_exact(q, k, v, seq_lens, k.shape[1], scale)
    out_err = np.linalg.norm(got - ref, axis=-1) / np.linalg.norm(ref, axis=-1)
    d = q.shape[-1]
    sc = 1.0 / np.sqrt(d) if scale is None else scale
    group = q.shape[1] // k.shape[1]
    num = den = 0.0
    for b in range(q.shape[0]):
        n = int(seq_lens[b])
        for g in range(k.shape[1]):
            heads = q[b, g * group:(g + 1) * group]
            s_c = _att.fused_scores(heads, kp[b, g, :n], kn[b, g, :n], rots[g], levels, sc)
            s_e = heads @ np.asarray(k[b, g, :n], dtype=np.float64).T * sc
            num += np.sum((s_c - s_e) ** 2)
            den += np.sum((s_e - s_e.mean(axis=-1, keepdims=True)) ** 2)
    return float(np.mean(out_err)), float(np.sqrt(num / den))


def study(seed: int = 0, n_heads: int = 4, n_tokens: int = 2048, group: int = 8,
          variants=_rot.VARIANTS, kv_dist: str = "anisotropic"):
    """The three quantities for each design on one seeded workload."""
    from paper_2608_08081_amd import synth   # seeded inputs only

    levels, thr = _cb.isoquant_codebook(128, 3)
    w = synth.Workload(91, "rotation_study", 1, n_heads * group, n_heads, n_tokens, "f32",
                       kv_dist=kv_dist, rotation_seed=seed + 17)
    k = synth.kv_tensor(seed, w, "k")
    v = synth.kv_tensor(seed, w, "v")
    q = synth.queries(seed, w)[0]
    gauss = synth.gaussian_matrices(seed, n_heads)
    lens = np.full(1, n_tokens)
    out = {}
    for var in variants:
        r = rotations(var, w.rotation_seed, n_heads, gauss)
        e = coordinate_energy(k, r)
        oe, se = attention_error(q, k, v, lens, r, thr, levels)
        out[var] = {"distortion_k": distortion(k, r, thr, levels),
                    "distortion_v": distortion(v, r, thr, levels),
                    "energy_min": float(e.min()), "energy_max": float(e.max()),
                    "unmixed": unmixed_share(k, r),
                    "out_err": oe, "score_err": se}
    return out


def main():
    import argparse
    p = argparse.ArgumentParser()
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--heads", type=int, default=4)
    p.add_argument("--tokens", type=int, default=2048)
    p.add_argument("--dist", default="anisotropic")
    a = p.parse_args()
    res = study(a.seed, a.heads, a.tokens, kv_dist=a.dist)
    print("| design | distortion K | distortion V | coord. energy min..max | fixed coords | "
          "output l2 err | score err |")
    print("|---|---|---|---|---|---|---|")
    for var, r in res.items():
        print(f"| {var} | {r['distortion_k']:.4f} | {r['distortion_v']:.4f} | "
              f"{r['energy_min']:.3f}..{r['energy_max']:.3f} | {100 * r['unmixed']:.0f} % | "
              f"{r['out_err']:.3f} | {r['score_err']:.3f} |")


if __name__ == "__main__":
    main()
