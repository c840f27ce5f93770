// Host-side fitting of the SO(4) block parameters (Sec. 3.2, "Why
// structured rotation works": the blocks fine-tune the rotation after the
// WHT, 6 degrees of freedom each, 192 per head) on calibration vectors, and
// the conversion of a 4 x 4 rotation into its quaternion pair (App. B).
//
// The paper names the parameters learnable but gives no procedure.  Reading
// used here: the objective is the one Step 3 states for the quantizer, the
// expected squared quantization error of the block's four coordinates,
// measured on the calibration set; it is separable over blocks (each
// coordinate's error depends only on its own block), so the 32 blocks are
// fitted independently.  Each block starts at the identity (the WHT alone)
// and runs Jacobi sweeps over its six coordinate planes: per plane a grid
// of angles, then a golden-section refinement around the best, accepting a
// plane rotation only if it lowers the error, so the fitted error never
// exceeds the WHT-only error on the calibration set.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <thread>
#include <vector>

#include "iq_internal.h"

namespace iq {
namespace {

constexpr int kPlanes[6][2] = {{0, 1}, {2, 3}, {0, 2}, {1, 3}, {0, 3}, {1, 2}};
constexpr int kGrid = 24;          // angles per plane in (-pi/4, pi/4]
constexpr int kGoldenSteps = 24;

struct Quantizer {
  double thr[7];
  double level[8];
  double err(double y) const {
    int c = 0;
    for (int j = 0; j < 7; ++j) c += (thr[j] <= y) ? 1 : 0;
    const double e = y - level[c];
    return e * e;
  }
};

// In-place normalized Walsh-Hadamard transform (Sylvester order) of 128
// values: the butterfly (a, b) -> (a + b, a - b) over every index bit.
void wht128(double* x) {
  for (int h = 1; h < kDim; h <<= 1)
    for (int i = 0; i < kDim; i += 2 * h)
      for (int j = i; j < i + h; ++j) {
        const double a = x[j], b = x[j + h];
        x[j] = a + b;
        x[j + h] = a - b;
      }
  const double s = 1.0 / sqrt(static_cast<double>(kDim));
  for (int i = 0; i < kDim; ++i) x[i] *= s;
}

// Hamilton product (w, x, y, z).
void qmul(const double* a, const double* b, double* o) {
  o[0] = a[0] * b[0] - a[1] * b[1] - a[2] * b[2] - a[3] * b[3];
  o[1] = a[0] * b[1] + a[1] * b[0] + a[2] * b[3] - a[3] * b[2];
  o[2] = a[0] * b[2] - a[1] * b[3] + a[2] * b[0] + a[3] * b[1];
  o[3] = a[0] * b[3] + a[1] * b[2] - a[2] * b[1] + a[3] * b[0];
}

// Fits the 4 x 4 rotation m (row-major, starts as identity) of one block.
// z: the block's post-WHT coordinates, n x 4.
void fit_block(const std::vector<double>& z, int64_t n, const Quantizer& qz, int sweeps,
               double* m) {
  for (int i = 0; i < 16; ++i) m[i] = (i % 5 == 0) ? 1.0 : 0.0;
  std::vector<double> y(z);                 // current rotated coordinates
  std::vector<double> col_err(4, 0.0);
  for (int64_t t = 0; t < n; ++t)
    for (int i = 0; i < 4; ++i) col_err[i] += qz.err(y[4 * t + i]);
  auto plane_err = [&](int a, int b, double th) {
    const double c = cos(th), s = sin(th);
    double e = 0.0;
    for (int64_t t = 0; t < n; ++t) {
      const double ya = y[4 * t + a], yb = y[4 * t + b];
      e += qz.err(c * ya - s * yb) + qz.err(s * ya + c * yb);
    }
    return e;
  };
  const double quarter = 0.78539816339744830962;   // pi / 4
  for (int sw = 0; sw < sweeps; ++sw) {
    bool moved = false;
    for (const auto& pl : kPlanes) {
      const int a = pl[0], b = pl[1];
      const double base = col_err[a] + col_err[b];
      double best = base, best_th = 0.0;
      for (int k = -kGrid / 2 + 1; k <= kGrid / 2; ++k) {
        const double th = quarter * 2.0 * k / kGrid;
        const double e = plane_err(a, b, th);
        if (e < best) best = e, best_th = th;
      }
      // golden-section refinement within one grid step of the best angle
      double lo = best_th - quarter * 2.0 / kGrid, hi = best_th + quarter * 2.0 / kGrid;
      const double gr = 0.61803398874989484820;
      double x1 = hi - gr * (hi - lo), x2 = lo + gr * (hi - lo);
      double f1 = plane_err(a, b, x1), f2 = plane_err(a, b, x2);
      for (int it = 0; it < kGoldenSteps; ++it) {
        if (f1 < f2) {
          hi = x2, x2 = x1, f2 = f1;
          x1 = hi - gr * (hi - lo), f1 = plane_err(a, b, x1);
        } else {
          lo = x1, x1 = x2, f1 = f2;
          x2 = lo + gr * (hi - lo), f2 = plane_err(a, b, x2);
        }
      }
      if (f1 < best) best = f1, best_th = x1;
      if (f2 < best) best = f2, best_th = x2;
      if (!(best < base) || best_th == 0.0) continue;
      // apply G(theta) in plane (a, b): rows a, b of m and the coordinates
      const double c = cos(best_th), s = sin(best_th);
      for (int j = 0; j < 4; ++j) {
        const double ra = m[4 * a + j], rb = m[4 * b + j];
        m[4 * a + j] = c * ra - s * rb;
        m[4 * b + j] = s * ra + c * rb;
      }
      double ea = 0.0, eb = 0.0;
      for (int64_t t = 0; t < n; ++t) {
        const double ya = y[4 * t + a], yb = y[4 * t + b];
        y[4 * t + a] = c * ya - s * yb;
        y[4 * t + b] = s * ya + c * yb;
        ea += qz.err(y[4 * t + a]);
        eb += qz.err(y[4 * t + b]);
      }
      col_err[a] = ea;
      col_err[b] = eb;
      moved = true;
    }
    if (!moved) break;
  }
}

}  // namespace

// (q_L, q_R) of a rotation m of R^4 (row-major 4 x 4, block component 0 the
// real part) with m v = q_L v conj(q_R): p = m(1) = q_L conj(q_R); the map
// v -> m(v) conj(p) = q_L v conj(q_L) fixes 1 and rotates the imaginary
// part; q_L is read from that 3 x 3 rotation (the largest of 1 + trace and
// the 1 + 2 R_ii - trace picks the stable formula), then q_R = conj(p) q_L.
// Returns false if m is not a rotation to within 1e-6.
bool so4_to_quaternions(const double* m, double* ql, double* qr) {
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) {
      double dot = 0.0;
      for (int k = 0; k < 4; ++k) dot += m[4 * i + k] * m[4 * j + k];
      if (fabs(dot - (i == j ? 1.0 : 0.0)) > 1e-6) return false;
    }
  const double p[4] = {m[0], m[4], m[8], m[12]};
  const double pc[4] = {p[0], -p[1], -p[2], -p[3]};
  double n[4][4];   // n[:, c] = m(e_c) conj(p)
  for (int c = 0; c < 4; ++c) {
    const double col[4] = {m[c], m[4 + c], m[8 + c], m[12 + c]};
    double o[4];
    qmul(col, pc, o);
    for (int r = 0; r < 4; ++r) n[r][c] = o[r];
  }
  // n fixes 1 (n(1) = p conj(p) = 1), so its imaginary block r carries the
  // determinant of m: -1 means a reflection, not in SO(4)
  double r[3][3];
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) r[i][j] = n[1 + i][1 + j];
  const double det = r[0][0] * (r[1][1] * r[2][2] - r[1][2] * r[2][1]) -
                     r[0][1] * (r[1][0] * r[2][2] - r[1][2] * r[2][0]) +
                     r[0][2] * (r[1][0] * r[2][1] - r[1][1] * r[2][0]);
  if (!(det > 0.0)) return false;
  const double tr = r[0][0] + r[1][1] + r[2][2];
  double q[4];
  const double c0 = 1.0 + tr, c1 = 1.0 + 2 * r[0][0] - tr, c2 = 1.0 + 2 * r[1][1] - tr,
               c3 = 1.0 + 2 * r[2][2] - tr;
  if (c0 >= c1 && c0 >= c2 && c0 >= c3) {
    const double s = 2.0 * sqrt(c0);
    q[0] = 0.25 * s;
    q[1] = (r[2][1] - r[1][2]) / s;
    q[2] = (r[0][2] - r[2][0]) / s;
    q[3] = (r[1][0] - r[0][1]) / s;
  } else if (c1 >= c2 && c1 >= c3) {
    const double s = 2.0 * sqrt(c1);
    q[0] = (r[2][1] - r[1][2]) / s;
    q[1] = 0.25 * s;
    q[2] = (r[0][1] + r[1][0]) / s;
    q[3] = (r[0][2] + r[2][0]) / s;
  } else if (c2 >= c3) {
    const double s = 2.0 * sqrt(c2);
    q[0] = (r[0][2] - r[2][0]) / s;
    q[1] = (r[0][1] + r[1][0]) / s;
    q[2] = 0.25 * s;
    q[3] = (r[1][2] + r[2][1]) / s;
  } else {
    const double s = 2.0 * sqrt(c3);
    q[0] = (r[1][0] - r[0][1]) / s;
    q[1] = (r[0][2] + r[2][0]) / s;
    q[2] = (r[1][2] + r[2][1]) / s;
    q[3] = 0.25 * s;
  }
  double nq = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3]);
  for (int i = 0; i < 4; ++i) ql[i] = q[i] / nq;
  qmul(pc, ql, qr);   // q_R = conj(p) q_L
  nq = sqrt(qr[0] * qr[0] + qr[1] * qr[1] + qr[2] * qr[2] + qr[3] * qr[3]);
  for (int i = 0; i < 4; ++i) qr[i] /= nq;
  return true;
}

}  // namespace iq

iq_status iq_so4_to_quaternions(const double* m, float* q_pair) {
  if (m == nullptr || q_pair == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  double ql[4], qr[4];
  if (!iq::so4_to_quaternions(m, ql, qr)) return IQ_ERR_INVALID_ARGUMENT;
  for (int i = 0; i < 4; ++i) {
    q_pair[i] = static_cast<float>(ql[i]);
    q_pair[4 + i] = static_cast<float>(qr[i]);
  }
  return IQ_OK;
}

iq_status iq_fit_rotation(const float* calib, int64_t n_vectors, int64_t n_kv_heads,
                          int64_t head_dim, int32_t sweeps, float* quats_host) {
  if (head_dim != iq::kDim) return IQ_ERR_UNSUPPORTED;
  if (calib == nullptr || quats_host == nullptr || n_vectors <= 0 || n_kv_heads <= 0 ||
      sweeps < 0 || n_vectors > (int64_t(1) << 24))
    return IQ_ERR_INVALID_ARGUMENT;
  const iq::Codebook& cb = iq::codebook();
  iq::Quantizer qz;
  for (int i = 0; i < 7; ++i) qz.thr[i] = cb.thr[i];
  for (int i = 0; i < 8; ++i) qz.level[i] = cb.level[i];
  constexpr int kBlocks = iq::kNumBlocks;
  iq_status status = IQ_OK;
  for (int64_t h = 0; h < n_kv_heads && status == IQ_OK; ++h) {
    // post-WHT unit vectors of the head, split into the 32 blocks
    std::vector<std::vector<double>> z(kBlocks);
    for (auto& v : z) v.reserve(static_cast<size_t>(n_vectors) * 4);
    int64_t n = 0;
    std::vector<double> x(iq::kDim);
    for (int64_t t = 0; t < n_vectors; ++t) {
      const float* src = calib + (h * n_vectors + t) * iq::kDim;
      double ss = 0.0;
      for (int i = 0; i < iq::kDim; ++i) ss += static_cast<double>(src[i]) * src[i];
      if (!(ss > 0.0) || !std::isfinite(ss)) continue;
      const double inv = 1.0 / sqrt(ss);
      for (int i = 0; i < iq::kDim; ++i) x[i] = src[i] * inv;
      iq::wht128(x.data());
      for (int b = 0; b < kBlocks; ++b)
        for (int i = 0; i < 4; ++i) z[b].push_back(x[4 * b + i]);
      ++n;
    }
    std::vector<double> mats(kBlocks * 16);
    if (n > 0) {
      // the 32 blocks are independent problems
      const unsigned hw = std::max(1u, std::min(8u, std::thread::hardware_concurrency()));
      std::vector<std::thread> pool;
      for (unsigned w = 0; w < hw; ++w)
        pool.emplace_back([&, w] {
          for (int b = static_cast<int>(w); b < kBlocks; b += static_cast<int>(hw))
            iq::fit_block(z[b], n, qz, sweeps, &mats[16 * b]);
        });
      for (auto& th : pool) th.join();
    } else {
      for (int b = 0; b < kBlocks; ++b)
        for (int i = 0; i < 16; ++i) mats[16 * b + i] = (i % 5 == 0) ? 1.0 : 0.0;
    }
    for (int b = 0; b < kBlocks; ++b) {
      double ql[4], qr[4];
      if (!iq::so4_to_quaternions(&mats[16 * b], ql, qr)) {
        // products of plane rotations stay in SO(4); only a numerical
        // breakdown could land here
        status = IQ_ERR_INVALID_ARGUMENT;
        break;
      }
      float* dst = quats_host + (h * kBlocks + b) * 8;
      for (int i = 0; i < 4; ++i) {
        dst[i] = static_cast<float>(ql[i]);
        dst[4 + i] = static_cast<float>(qr[i]);
      }
    }
  }
  return status;
}

// ---------------------------------------------------------------------------
// Empirical codebook (Sec. 3.2 Step 3 measured on calibration data): the
// Lloyd-Max levels of the distribution of the rotated, normalized
// coordinates of calibration vectors, instead of the analytic sphere
// marginal.  Reading: one codebook for all heads (as the library's), fitted
// to the sample made symmetric (each coordinate and its negation: the
// marginal of an isotropic rotation is symmetric, and the kernels' quantizer
// relies on it), started from the library's C_b, iterated until the cells
// stop changing; then stored like C_b (levels rounded to fp16, made exactly
// symmetric, thresholds their midpoints).
// ---------------------------------------------------------------------------
namespace iq {
namespace {

// Nearest binary16 value (ties to even) of v, for |v| in the normal range
// or zero.
double nearest_half(double v) {
  if (v == 0.0) return 0.0;
  int e = 0;
  frexp(fabs(v), &e);
  const double ulp = ldexp(1.0, e - 11);
  return nearbyint(v / ulp) * ulp;
}

// y = R x / ||x|| (Eq. 2) of one calibration vector in fp64; false for a
// zero or non-finite vector.  quats: the head's 32 (q_L, q_R) pairs.
bool rotate_normalized(const float* src, const float* quats, double* y) {
  double ss = 0.0;
  for (int i = 0; i < kDim; ++i) ss += static_cast<double>(src[i]) * src[i];
  if (!(ss > 0.0) || !std::isfinite(ss)) return false;
  const double inv = 1.0 / sqrt(ss);
  for (int i = 0; i < kDim; ++i) y[i] = src[i] * inv;
  wht128(y);
  for (int b = 0; b < kNumBlocks; ++b) {
    double ql[4], qr[4];
    for (int i = 0; i < 4; ++i) {
      ql[i] = quats[8 * b + i];
      qr[i] = quats[8 * b + 4 + i];
    }
    // the stored pair, made unit in fp64, acting as v -> q_L v conj(q_R)
    const double nl = sqrt(ql[0] * ql[0] + ql[1] * ql[1] + ql[2] * ql[2] + ql[3] * ql[3]);
    const double nr = sqrt(qr[0] * qr[0] + qr[1] * qr[1] + qr[2] * qr[2] + qr[3] * qr[3]);
    for (int i = 0; i < 4; ++i) ql[i] /= nl;
    const double qrc[4] = {qr[0] / nr, -qr[1] / nr, -qr[2] / nr, -qr[3] / nr};
    double t[4];
    qmul(ql, &y[4 * b], t);
    qmul(t, qrc, &y[4 * b]);
  }
  return true;
}

}  // namespace
}  // namespace iq

iq_status iq_fit_codebook(const float* calib, int64_t n_vectors, int64_t n_kv_heads,
                          int64_t head_dim, const float* quats_host, int32_t bits,
                          iq_codebook_t* out) {
  if (head_dim != iq::kDim || (bits != 2 && bits != 3 && bits != 4)) return IQ_ERR_UNSUPPORTED;
  if (calib == nullptr || quats_host == nullptr || out == nullptr || n_vectors <= 0 ||
      n_kv_heads <= 0 || n_vectors > (int64_t(1) << 24) || n_kv_heads > (int64_t(1) << 16) ||
      n_vectors * n_kv_heads > (int64_t(1) << 24))
    return IQ_ERR_INVALID_ARGUMENT;
  const int n = 1 << bits;
  float init_levels[16], init_thr[15];
  iq_codebook_bits(bits, init_levels, init_thr);
  // the symmetrized sample, sorted
  std::vector<double> ys;
  ys.reserve(static_cast<size_t>(2 * iq::kDim * n_vectors * n_kv_heads));
  std::vector<double> y(iq::kDim);
  for (int64_t h = 0; h < n_kv_heads; ++h)
    for (int64_t t = 0; t < n_vectors; ++t) {
      if (!iq::rotate_normalized(calib + (h * n_vectors + t) * iq::kDim,
                                 quats_host + h * iq::kQuatFloats, y.data()))
        continue;
      for (int i = 0; i < iq::kDim; ++i) {
        ys.push_back(y[i]);
        ys.push_back(-y[i]);
      }
    }
  if (ys.empty()) return IQ_ERR_INVALID_ARGUMENT;
  std::sort(ys.begin(), ys.end());
  // prefix sums: the mean of a cell [lo, hi) of the sorted sample is
  // (P[hi] - P[lo]) / (hi - lo)
  std::vector<double> prefix(ys.size() + 1, 0.0);
  for (size_t i = 0; i < ys.size(); ++i) prefix[i + 1] = prefix[i] + ys[i];
  double c[16];
  for (int i = 0; i < n; ++i) c[i] = init_levels[i];
  bool fixed = false;
  for (int it = 0; it < 10000 && !fixed; ++it) {
    // cell j: t_(j-1) <= y < t_j, t_j the midpoints (the coding rule)
    size_t edge[17];
    edge[0] = 0;
    edge[n] = ys.size();
    for (int j = 1; j < n; ++j)
      edge[j] = static_cast<size_t>(
          std::lower_bound(ys.begin(), ys.end(), 0.5 * (c[j - 1] + c[j])) - ys.begin());
    fixed = true;
    for (int j = 0; j < n; ++j) {
      if (edge[j + 1] <= edge[j]) continue;   // an empty cell keeps its level
      const double m = (prefix[edge[j + 1]] - prefix[edge[j]]) /
                       static_cast<double>(edge[j + 1] - edge[j]);
      if (m != c[j]) fixed = false;
      c[j] = m;
    }
  }
  if (!fixed) return IQ_ERR_INVALID_ARGUMENT;
  iq_codebook_t cb{};
  cb.bits = bits;
  for (int i = 0; i < n; ++i) cb.levels[i] = static_cast<float>(iq::nearest_half(c[i]));
  for (int i = 0; i < n / 2; ++i) cb.levels[i] = -cb.levels[n - 1 - i];
  for (int i = 0; i < n - 1; ++i)
    cb.thresholds[i] =
        static_cast<float>(0.5 * (static_cast<double>(cb.levels[i]) + cb.levels[i + 1]));
  for (int i = 1; i < n; ++i)
    if (!(cb.levels[i] > cb.levels[i - 1])) return IQ_ERR_INVALID_ARGUMENT;
  *out = cb;
  return IQ_OK;
}
