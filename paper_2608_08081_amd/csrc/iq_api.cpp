// Host side of libisoquant: the C ABI declared in isoquant.h.
//
// Validation happens here, before any HIP call; the kernels live in
// iq_compress.hip and iq_decode.hip.  The codebook (Sec. 3.2 Step 3) is
// derived here on first use with a Lloyd-Max iteration in double precision,
// and the seeded rotation parameters (App. B) with SplitMix64.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "iq_internal.h"

// IEEE-exact host arithmetic for the parameter generator: no contraction of
// a*b + c into fused multiply-adds in this translation unit.
#pragma clang fp contract(off)

namespace iq {
namespace {

// ---------------------------------------------------------------------------
// Codebook: Lloyd-Max levels for one coordinate of a uniform point on the
// sphere S^(d-1), density proportional to (1 - t^2)^k with k = (d - 3) / 2.
// Level of a cell [a, b] = conditional mean
//   integral t (1-t^2)^k dt / integral (1-t^2)^k dt,
// numerator in closed form  ((1-a^2)^(k+1) - (1-b^2)^(k+1)) / (2(k+1)),
// denominator by composite Simpson quadrature.
// ---------------------------------------------------------------------------
double sphere_density(double t, double k) {
  const double u = 1.0 - t * t;
  return u > 0.0 ? exp(k * log(u)) : 0.0;
}

double simpson_mass(double a, double b, double k) {
  const int n = 4096;  // even
  const double h = (b - a) / n;
  double s = sphere_density(a, k) + sphere_density(b, k);
  for (int i = 1; i < n; ++i) s += sphere_density(a + i * h, k) * ((i & 1) ? 4.0 : 2.0);
  return s * h / 3.0;
}

double first_moment(double a, double b, double k) {
  const double ua = 1.0 - a * a, ub = 1.0 - b * b;
  const double pa = ua > 0.0 ? exp((k + 1.0) * log(ua)) : 0.0;
  const double pb = ub > 0.0 ? exp((k + 1.0) * log(ub)) : 0.0;
  return (pa - pb) / (2.0 * (k + 1.0));
}

// Round to the nearest IEEE binary16 value (ties to even) for values in the
// normal binary16 range.
double round_to_half(double v) {
  if (v == 0.0) return 0.0;
  int e = 0;
  frexp(fabs(v), &e);                   // |v| = f * 2^e, f in [0.5, 1)
  const double ulp = ldexp(1.0, e - 11);  // 11 significant bits
  return nearbyint(v / ulp) * ulp;
}

template <int kBits>
CodebookB<kBits> build_codebook() {
  constexpr int d = kDim, n = 1 << kBits;
  const double k = (d - 3) / 2.0;
  double c[n];
  for (int i = 0; i < n; ++i) c[i] = -2.0 / sqrt(static_cast<double>(d)) + i * (4.0 / sqrt(static_cast<double>(d))) / (n - 1);
  for (int it = 0; it < 20000; ++it) {
    double edges[n + 1];
    edges[0] = -1.0;
    edges[n] = 1.0;
    for (int i = 1; i < n; ++i) edges[i] = 0.5 * (c[i - 1] + c[i]);
    double moved = 0.0;
    for (int i = 0; i < n; ++i) {
      const double nc = first_moment(edges[i], edges[i + 1], k) / simpson_mass(edges[i], edges[i + 1], k);
      moved = fmax(moved, fabs(nc - c[i]));
      c[i] = nc;
    }
    if (moved < 1e-13) break;
  }
  CodebookB<kBits> cb{};
  for (int i = 0; i < n; ++i) cb.level[i] = static_cast<float>(round_to_half(c[i]));
  // enforce the symmetry of the symmetric density exactly
  for (int i = 0; i < n / 2; ++i) cb.level[i] = -cb.level[n - 1 - i];
  for (int i = 0; i < n - 1; ++i)
    cb.thr[i] = static_cast<float>(0.5 * (static_cast<double>(cb.level[i]) + cb.level[i + 1]));
  return cb;
}

// ---------------------------------------------------------------------------
// SplitMix64 (Steele, Lea & Flood 2014) and the unit-quaternion sampler.
// ---------------------------------------------------------------------------
struct SplitMix64 {
  uint64_t state;
  uint64_t next() {
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform_pm1() {
    const double u = static_cast<double>(next() >> 11) * 0x1.0p-53;
    return 2.0 * u - 1.0;
  }
};

void random_unit_quaternion(SplitMix64& g, float* out) {
  for (;;) {
    double u[4];
    for (int i = 0; i < 4; ++i) u[i] = g.uniform_pm1();
    double n2 = u[0] * u[0];
    n2 = n2 + u[1] * u[1];
    n2 = n2 + u[2] * u[2];
    n2 = n2 + u[3] * u[3];
    if (n2 > 1e-6 && n2 <= 1.0) {
      const double n = sqrt(n2);
      for (int i = 0; i < 4; ++i) out[i] = static_cast<float>(u[i] / n);
      return;
    }
  }
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Largest element index touched must fit: all sizes here are products of
// validated non-negative int64 values below 2^62.
bool mul_ok(int64_t a, int64_t b) { return a == 0 || b <= (int64_t(1) << 62) / a; }

}  // namespace

template <int kBits>
const CodebookB<kBits>& codebook_b() {
  static CodebookB<kBits> cb;
  static std::once_flag once;
  std::call_once(once, [] { cb = build_codebook<kBits>(); });
  return cb;
}
template const CodebookB<2>& codebook_b<2>();
template const CodebookB<3>& codebook_b<3>();
template const CodebookB<4>& codebook_b<4>();

const Codebook& codebook() { return codebook_b<3>(); }

}  // namespace iq

using iq::kDim;

extern "C" {

const char* iq_status_string(int32_t s) {
  switch (s) {
    case IQ_OK: return "IQ_OK";
    case IQ_ERR_INVALID_ARGUMENT: return "IQ_ERR_INVALID_ARGUMENT";
    case IQ_ERR_UNSUPPORTED: return "IQ_ERR_UNSUPPORTED";
    case IQ_ERR_WORKSPACE_TOO_SMALL: return "IQ_ERR_WORKSPACE_TOO_SMALL";
    case IQ_ERR_HIP: return "IQ_ERR_HIP";
    case IQ_ERR_CAPACITY: return "IQ_ERR_CAPACITY";
  }
  return "unknown status";
}

int iq_version(void) { return 200; }

iq_status iq_codebook(float* levels, float* thresholds) { return iq_codebook_bits(3, levels, thresholds); }

iq_status iq_codebook_bits(int bits, float* levels, float* thresholds) {
  auto copy = [&](const auto& cb) {
    if (levels) memcpy(levels, cb.level, sizeof(cb.level));
    if (thresholds) memcpy(thresholds, cb.thr, sizeof(cb.thr));
    return IQ_OK;
  };
  switch (bits) {
    case 2: return copy(iq::codebook_b<2>());
    case 3: return copy(iq::codebook_b<3>());
    case 4: return copy(iq::codebook_b<4>());
    default: return IQ_ERR_UNSUPPORTED;
  }
}

iq_status iq_make_rotation(uint64_t seed, int64_t n_kv_heads, int64_t head_dim,
                           float* quats_host) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (n_kv_heads <= 0 || quats_host == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  iq::SplitMix64 g{seed};
  for (int64_t h = 0; h < n_kv_heads; ++h)
    for (int blk = 0; blk < iq::kNumBlocks; ++blk) {
      float* dst = quats_host + (h * iq::kNumBlocks + blk) * 8;
      iq::random_unit_quaternion(g, dst);
      iq::random_unit_quaternion(g, dst + 4);
    }
  return IQ_OK;
}

iq_status iq_make_rotation_variant(uint64_t seed, int64_t n_kv_heads, int64_t head_dim,
                                   int32_t variant, float* quats_host) {
  if (variant != IQ_ROTATION_SO4 && variant != IQ_ROTATION_SO3 &&
      variant != IQ_ROTATION_WHT_ONLY)
    return IQ_ERR_UNSUPPORTED;
  if (variant == IQ_ROTATION_WHT_ONLY) {
    if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
    if (n_kv_heads <= 0 || quats_host == nullptr) return IQ_ERR_INVALID_ARGUMENT;
    for (int64_t i = 0; i < n_kv_heads * iq::kNumBlocks * 2; ++i) {
      float* q = quats_host + 4 * i;
      q[0] = 1.0f;
      q[1] = q[2] = q[3] = 0.0f;
    }
    return IQ_OK;
  }
  const iq_status st = iq_make_rotation(seed, n_kv_heads, head_dim, quats_host);
  if (st != IQ_OK || variant == IQ_ROTATION_SO4) return st;
  // single quaternion per block: q_R = q_L
  for (int64_t i = 0; i < n_kv_heads * iq::kNumBlocks; ++i)
    for (int c = 0; c < 4; ++c) quats_host[8 * i + 4 + c] = quats_host[8 * i + c];
  return IQ_OK;
}

iq_status iq_compress_kv(const void* k, const void* v, int32_t dtype, int64_t batch,
                         int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                         const float* quats, uint8_t* k_codes, float* k_norms,
                         uint8_t* v_codes, float* v_norms, int64_t capacity,
                         int64_t dst_offset, hipStream_t stream) {
  return iq_compress_kv_bits(k, v, dtype, batch, n_kv_heads, n_tokens, head_dim, quats, k_codes,
                             k_norms, v_codes, v_norms, capacity, dst_offset, 3, stream);
}

namespace {

// A caller codebook the kernels can take: b in {2, 3, 4}; 2^b finite levels,
// strictly ascending, fp16-exact, below 1 in magnitude and symmetric
// (level[i] = -level[2^b - 1 - i], the compression quantizer's sign rule);
// thresholds exactly the fp32 midpoints of adjacent levels.
iq_status check_codebook(const iq_codebook_t* cb) {
  if (cb == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  if (cb->bits != 2 && cb->bits != 3 && cb->bits != 4) return IQ_ERR_UNSUPPORTED;
  const int n = 1 << cb->bits;
  for (int i = 0; i < n; ++i) {
    const double l = cb->levels[i];
    if (!(fabs(l) < 1.0) || iq::round_to_half(l) != l) return IQ_ERR_INVALID_ARGUMENT;
    if (cb->levels[i] != -cb->levels[n - 1 - i]) return IQ_ERR_INVALID_ARGUMENT;
    if (i > 0 && !(cb->levels[i] > cb->levels[i - 1])) return IQ_ERR_INVALID_ARGUMENT;
  }
  for (int i = 0; i < n - 1; ++i)
    if (cb->thresholds[i] !=
        static_cast<float>(0.5 * (static_cast<double>(cb->levels[i]) + cb->levels[i + 1])))
      return IQ_ERR_INVALID_ARGUMENT;
  return IQ_OK;
}

iq_status compress_common(const void* k, const void* v, int32_t dtype, int64_t batch,
                          int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                          const float* quats, uint8_t* k_codes, float* k_norms,
                          uint8_t* v_codes, float* v_norms, int64_t capacity,
                          int64_t dst_offset, int bits, const iq_codebook_t* cb,
                          hipStream_t stream) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (bits < 2 || bits > 4) return IQ_ERR_UNSUPPORTED;
  if (dtype != IQ_DTYPE_F32 && dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || n_kv_heads <= 0 || n_tokens < 0 || capacity < 0 || dst_offset < 0)
    return IQ_ERR_INVALID_ARGUMENT;
  if (dst_offset > capacity || n_tokens > capacity - dst_offset) return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::mul_ok(batch, n_kv_heads) || !iq::mul_ok(batch * n_kv_heads, capacity + 1) ||
      !iq::mul_ok(batch * n_kv_heads * (capacity + 1), kDim))
    return IQ_ERR_INVALID_ARGUMENT;
  // an empty block is a no-op (empty tensors may carry null data pointers)
  if (batch == 0 || n_tokens == 0) return IQ_OK;
  if (k == nullptr && v == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  if (quats == nullptr || !iq::aligned(quats, 16)) return IQ_ERR_INVALID_ARGUMENT;
  if (k && (!k_codes || !k_norms || !iq::aligned(k, 16) || !iq::aligned(k_codes, 16) ||
            !iq::aligned(k_norms, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (v && (!v_codes || !v_norms || !iq::aligned(v, 16) || !iq::aligned(v_codes, 16) ||
            !iq::aligned(v_norms, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  const hipError_t e = iq::launch_compress(k, v, dtype, batch, n_kv_heads, n_tokens, quats,
                                           k_codes, k_norms, v_codes, v_norms, capacity,
                                           dst_offset, bits, stream, cb);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // namespace

iq_status iq_compress_kv_bits(const void* k, const void* v, int32_t dtype, int64_t batch,
                              int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                              const float* quats, uint8_t* k_codes, float* k_norms,
                              uint8_t* v_codes, float* v_norms, int64_t capacity,
                              int64_t dst_offset, int bits, hipStream_t stream) {
  return compress_common(k, v, dtype, batch, n_kv_heads, n_tokens, head_dim, quats, k_codes,
                         k_norms, v_codes, v_norms, capacity, dst_offset, bits, nullptr, stream);
}

iq_status iq_compress_kv_cb(const void* k, const void* v, int32_t dtype, int64_t batch,
                            int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                            const float* quats, const iq_codebook_t* cb, uint8_t* k_codes,
                            float* k_norms, uint8_t* v_codes, float* v_norms, int64_t capacity,
                            int64_t dst_offset, hipStream_t stream) {
  const iq_status st = check_codebook(cb);
  if (st != IQ_OK) return st;
  return compress_common(k, v, dtype, batch, n_kv_heads, n_tokens, head_dim, quats, k_codes,
                         k_norms, v_codes, v_norms, capacity, dst_offset, cb->bits, cb, stream);
}

iq_status iq_append_token(const void* k_new, const void* v_new, int32_t dtype, int64_t batch,
                          int64_t n_kv_heads, int64_t head_dim, const float* quats,
                          uint8_t* k_codes, float* k_norms, uint8_t* v_codes, float* v_norms,
                          int64_t capacity, int32_t* seq_lens, int32_t* status_dev,
                          hipStream_t stream) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (dtype != IQ_DTYPE_F32 && dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || batch > 0x7fffffff || n_kv_heads <= 0 || n_kv_heads > 512 || capacity < 0 ||
      capacity > 0x7fffffff)
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::mul_ok(batch, n_kv_heads) || !iq::mul_ok(batch * n_kv_heads, capacity + 1) ||
      !iq::mul_ok(batch * n_kv_heads * (capacity + 1), kDim))
    return IQ_ERR_INVALID_ARGUMENT;
  if (k_new == nullptr && v_new == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  if (quats == nullptr || seq_lens == nullptr || !iq::aligned(seq_lens, 4) ||
      !iq::aligned(quats, 16) || (status_dev && !iq::aligned(status_dev, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (k_new && (!k_codes || !k_norms || !iq::aligned(k_new, 16) || !iq::aligned(k_codes, 16) ||
                !iq::aligned(k_norms, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (v_new && (!v_codes || !v_norms || !iq::aligned(v_new, 16) || !iq::aligned(v_codes, 16) ||
                !iq::aligned(v_norms, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (batch == 0) return IQ_OK;
  const hipError_t e = iq::launch_append(k_new, v_new, dtype, batch, n_kv_heads, quats, k_codes,
                                         k_norms, v_codes, v_norms, capacity, seq_lens,
                                         status_dev, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

size_t iq_decode_workspace_bytes(int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                 int64_t max_seq_len, int64_t head_dim) {
  if (head_dim != kDim) return 0;
  iq::DecodePlan plan;
  if (!iq::plan_decode(batch, n_q_heads, n_kv_heads, max_seq_len, &plan)) return 0;
  return plan.total_bytes;
}

iq_status iq_decode_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (workspace == nullptr || !iq::aligned(workspace, 256)) return IQ_ERR_INVALID_ARGUMENT;
  const hipError_t e = iq::launch_fill_zero(workspace, workspace_bytes, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

namespace {

// Shared argument checks of iq_decode_attention and iq_decode_step; fills
// the split plan.
iq_status check_decode_args(const float* q, const void* k_codes, const float* k_norms,
                            const void* v_codes, const float* v_norms, const int32_t* seq_lens,
                            int64_t capacity, int64_t max_seq_len, const float* quats,
                            int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                            int64_t head_dim, const float* out, const void* workspace,
                            size_t workspace_bytes, iq::DecodePlan* plan) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || capacity < 0 || max_seq_len < 0 ||
      max_seq_len > capacity || capacity > 0x7fffffff || batch > 0xffffff)
    return IQ_ERR_INVALID_ARGUMENT;
  if (n_q_heads % n_kv_heads) return IQ_ERR_INVALID_ARGUMENT;
  if (n_q_heads / n_kv_heads > iq::kMaxGroup) return IQ_ERR_UNSUPPORTED;
  if (!iq::mul_ok(batch, n_kv_heads) || !iq::mul_ok(batch * n_kv_heads, capacity + 1) ||
      !iq::mul_ok(batch * n_kv_heads * (capacity + 1), kDim))
    return IQ_ERR_INVALID_ARGUMENT;
  if (!q || !k_codes || !k_norms || !v_codes || !v_norms || !seq_lens || !quats || !out ||
      !workspace)
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::aligned(q, 16) || !iq::aligned(k_codes, 16) || !iq::aligned(v_codes, 16) ||
      !iq::aligned(k_norms, 4) || !iq::aligned(v_norms, 4) || !iq::aligned(out, 16) ||
      !iq::aligned(seq_lens, 4) || !iq::aligned(quats, 16) || !iq::aligned(workspace, 256))
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::plan_decode(batch, n_q_heads, n_kv_heads, max_seq_len, plan))
    return IQ_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < plan->total_bytes) return IQ_ERR_WORKSPACE_TOO_SMALL;
  return IQ_OK;
}

float resolve_scale(float softmax_scale) {
  return softmax_scale > 0.f ? softmax_scale : 1.0f / sqrtf(static_cast<float>(kDim));
}

// Shapes the matrix-core path takes (after check_decode_args, which bounds
// the group by 16): rows of whole 16-position batches addressed with 32-bit
// byte offsets (records of record_bytes bytes), 16-byte aligned scale
// arrays, and sequences and (KV head, head group of 8) rows as grid
// dimensions.
iq_status check_g8_shape(int64_t n_q_heads, int64_t n_kv_heads, int64_t batch, int64_t capacity,
                         int64_t record_bytes, const float* k_norms, const float* v_norms,
                         const iq::DecodePlan& plan) {
  if (plan.g8_batches <= 0) return IQ_ERR_UNSUPPORTED;
  const int64_t rows = n_kv_heads * ((n_q_heads / n_kv_heads + 7) / 8);
  if (capacity % 16 || capacity < 16 || capacity * record_bytes > 0x7fffffff ||
      !iq::aligned(k_norms, 16) || !iq::aligned(v_norms, 16) || batch > 65535 || rows > 65535)
    return IQ_ERR_UNSUPPORTED;
  // work items of a grid of several rounds (32-bit indices)
  if (batch * rows * (plan.g8_splits + 1) > (int64_t{1} << 30)) return IQ_ERR_UNSUPPORTED;
  return IQ_OK;
}

}  // namespace

namespace {

// Decode attention on records of `bits` bits with codebook cb (null: the
// library's C_b).  3-bit records take the group-8 matrix-core path where the
// shapes allow it and the generic path otherwise; 2- and 4-bit records the
// matrix-core path only.
iq_status decode_common(const float* q, const uint8_t* k_codes, const float* k_norms,
                        const uint8_t* v_codes, const float* v_norms, const int32_t* seq_lens,
                        int64_t capacity, int64_t max_seq_len, const float* quats, int64_t batch,
                        int64_t n_q_heads, int64_t n_kv_heads, int64_t head_dim,
                        float softmax_scale, float* out, void* workspace,
                        size_t workspace_bytes, int bits, const iq_codebook_t* cb,
                        hipStream_t stream) {
  if (bits != 2 && bits != 3 && bits != 4) return IQ_ERR_UNSUPPORTED;
  iq::DecodePlan plan;
  const iq_status st = check_decode_args(q, k_codes, k_norms, v_codes, v_norms, seq_lens,
                                         capacity, max_seq_len, quats, batch, n_q_heads,
                                         n_kv_heads, head_dim, out, workspace, workspace_bytes,
                                         &plan);
  if (st != IQ_OK) return st;
  if (bits != 3) {
    const iq_status shape = check_g8_shape(n_q_heads, n_kv_heads, batch, capacity, 16 * bits,
                                           k_norms, v_norms, plan);
    if (shape != IQ_OK) return shape;
  }
  if (batch == 0) return IQ_OK;
  hipError_t e;
  if (bits == 3) {
    // without an append the launch only reads the cache and the lengths
    e = iq::launch_decode(plan, q, const_cast<uint8_t*>(k_codes), const_cast<float*>(k_norms),
                          const_cast<uint8_t*>(v_codes), const_cast<float*>(v_norms),
                          const_cast<int32_t*>(seq_lens), capacity, max_seq_len, quats, batch,
                          n_q_heads, n_kv_heads, resolve_scale(softmax_scale), out, workspace,
                          nullptr, stream, cb);
  } else {
    float* parts = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
    e = iq::launch_decode_g8(plan.g8_batches, plan.g8_splits, plan.g8_split_len, q,
                             const_cast<uint8_t*>(k_codes), const_cast<float*>(k_norms),
                             const_cast<uint8_t*>(v_codes), const_cast<float*>(v_norms),
                             const_cast<int32_t*>(seq_lens), capacity, max_seq_len, quats, batch,
                             n_kv_heads, n_q_heads / n_kv_heads, resolve_scale(softmax_scale),
                             out, parts, nullptr, nullptr, bits, stream, cb);
  }
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // namespace

iq_status iq_decode_attention(const float* q, const uint8_t* k_codes, const float* k_norms,
                              const uint8_t* v_codes, const float* v_norms,
                              const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                              const float* quats, int64_t batch, int64_t n_q_heads,
                              int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                              float* out, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  return decode_common(q, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity, max_seq_len,
                       quats, batch, n_q_heads, n_kv_heads, head_dim, softmax_scale, out,
                       workspace, workspace_bytes, 3, nullptr, stream);
}

iq_status iq_decode_attention_bits(const float* q, const uint8_t* k_codes, const float* k_norms,
                                   const uint8_t* v_codes, const float* v_norms,
                                   const int32_t* seq_lens, int64_t capacity,
                                   int64_t max_seq_len, const float* quats, int64_t batch,
                                   int64_t n_q_heads, int64_t n_kv_heads, int64_t head_dim,
                                   float softmax_scale, float* out, void* workspace,
                                   size_t workspace_bytes, int bits, hipStream_t stream) {
  return decode_common(q, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity, max_seq_len,
                       quats, batch, n_q_heads, n_kv_heads, head_dim, softmax_scale, out,
                       workspace, workspace_bytes, bits, nullptr, stream);
}

iq_status iq_decode_attention_cb(const float* q, const uint8_t* k_codes, const float* k_norms,
                                 const uint8_t* v_codes, const float* v_norms,
                                 const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                                 const float* quats, const iq_codebook_t* cb, int64_t batch,
                                 int64_t n_q_heads, int64_t n_kv_heads, int64_t head_dim,
                                 float softmax_scale, float* out, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  const iq_status st = check_codebook(cb);
  if (st != IQ_OK) return st;
  return decode_common(q, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity, max_seq_len,
                       quats, batch, n_q_heads, n_kv_heads, head_dim, softmax_scale, out,
                       workspace, workspace_bytes, cb->bits, cb, stream);
}

iq_status iq_decode_attention_rope(const float* q, const float* q_rope, const uint8_t* k_codes,
                                   const float* k_norms, const void* k_rope,
                                   int64_t n_rope_heads, const uint8_t* v_codes,
                                   const float* v_norms, const int32_t* seq_lens,
                                   int64_t capacity, int64_t max_seq_len, const float* quats,
                                   int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                   int64_t head_dim, int64_t rope_dim, float softmax_scale,
                                   float* out, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  if (rope_dim != 64) return IQ_ERR_UNSUPPORTED;
  iq::DecodePlan plan;
  const iq_status st = check_decode_args(q, k_codes, k_norms, v_codes, v_norms, seq_lens,
                                         capacity, max_seq_len, quats, batch, n_q_heads,
                                         n_kv_heads, head_dim, out, workspace, workspace_bytes,
                                         &plan);
  if (st != IQ_OK) return st;
  if (n_rope_heads != 1 && n_rope_heads != n_kv_heads) return IQ_ERR_INVALID_ARGUMENT;
  if (!q_rope || !k_rope || !iq::aligned(q_rope, 16) || !iq::aligned(k_rope, 16))
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::mul_ok(batch * n_rope_heads, capacity + 1) ||
      !iq::mul_ok(batch * n_rope_heads * (capacity + 1), rope_dim))
    return IQ_ERR_INVALID_ARGUMENT;
  // the matrix-core path only
  const iq_status shape = check_g8_shape(n_q_heads, n_kv_heads, batch, capacity,
                                         iq::kRecordBytes, k_norms, v_norms, plan);
  if (shape != IQ_OK) return shape;
  if (batch == 0) return IQ_OK;
  const float scale = softmax_scale > 0.f
                          ? softmax_scale
                          : 1.0f / sqrtf(static_cast<float>(kDim + rope_dim));
  const iq::RopeKeys rope{static_cast<const uint16_t*>(k_rope), q_rope,
                          n_rope_heads == 1 && n_kv_heads > 1 ? 1 : 0};
  float* parts = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
  const hipError_t e = iq::launch_decode_g8(
      plan.g8_batches, plan.g8_splits, plan.g8_split_len, q, const_cast<uint8_t*>(k_codes),
      const_cast<float*>(k_norms), const_cast<uint8_t*>(v_codes), const_cast<float*>(v_norms),
      const_cast<int32_t*>(seq_lens), capacity, max_seq_len, quats, batch, n_kv_heads,
      n_q_heads / n_kv_heads, scale, out, parts, nullptr, nullptr, 3, stream, nullptr, &rope);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

size_t iq_decode_multi_workspace_bytes(int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                                       int64_t n_kv_heads, int64_t max_seq_len,
                                       int64_t head_dim) {
  if (n_tokens == 1)
    return iq_decode_workspace_bytes(batch, n_q_heads, n_kv_heads, max_seq_len, head_dim);
  if (head_dim != kDim || batch < 0 || n_tokens < 2 || n_tokens > 4 || n_kv_heads <= 0 ||
      n_q_heads != 8 * n_kv_heads || max_seq_len < 0 || batch > 65535 || n_kv_heads > 65535 ||
      batch * n_tokens > 65535)   // the merge's grid takes (sequence, token) as one dimension
    return 0;
  int nb = 0;
  int64_t splits = 0, len = 0;
  iq::g8_plan(batch, n_kv_heads, max_seq_len, &nb, &splits, &len);
  // the splits' partial rows and the fused step's new-token rows
  const size_t bytes = static_cast<size_t>(batch) * n_kv_heads * (splits + 1) * n_tokens * 8 *
                       (2 + kDim) * sizeof(float);
  return bytes > 0 ? (bytes + 255) / 256 * 256 : 256;
}

namespace {

// Multi-token decode and the fused multi-token step (append != null) on
// contiguous caches of `bits`-bit records.
iq_status multi_common(const float* q, const iq::StepAppend* append, uint8_t* k_codes,
                       float* k_norms, uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                       int64_t capacity, int64_t max_seq_len, const float* quats, int64_t batch,
                       int64_t n_tokens, int64_t n_q_heads, int64_t n_kv_heads,
                       int64_t head_dim, float softmax_scale, int bits, float* out,
                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (n_tokens < 2 || n_tokens > 4) return IQ_ERR_UNSUPPORTED;
  if (bits != 2 && bits != 3 && bits != 4) return IQ_ERR_UNSUPPORTED;
  iq::DecodePlan plan;
  // the single-token checks cover the cache, pointers and alignment; the
  // workspace is checked against the multi-token size below
  const iq_status st = check_decode_args(q, k_codes, k_norms, v_codes, v_norms, seq_lens,
                                         capacity, max_seq_len, quats, batch, n_q_heads,
                                         n_kv_heads, head_dim, out, workspace, SIZE_MAX, &plan);
  if (st != IQ_OK) return st;
  // multi-token decode runs 8 query heads per KV head
  if (n_q_heads != 8 * n_kv_heads) return IQ_ERR_UNSUPPORTED;
  const iq_status shape = check_g8_shape(n_q_heads, n_kv_heads, batch, capacity, 16 * bits,
                                         k_norms, v_norms, plan);
  if (shape != IQ_OK) return shape;
  if (!iq::mul_ok(batch, n_tokens) || !iq::mul_ok(batch * n_tokens, n_q_heads))
    return IQ_ERR_INVALID_ARGUMENT;
  // the merge kernel's grid takes (sequence, token) as one dimension
  if (batch * n_tokens > 65535) return IQ_ERR_UNSUPPORTED;
  const size_t need = iq_decode_multi_workspace_bytes(batch, n_tokens, n_q_heads, n_kv_heads,
                                                      max_seq_len, head_dim);
  if (need == 0) return IQ_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < need) return IQ_ERR_WORKSPACE_TOO_SMALL;
  if (batch == 0) return IQ_OK;
  const hipError_t e = iq::launch_decode_g8_multi(
      plan.g8_batches, plan.g8_splits, plan.g8_split_len, static_cast<int>(n_tokens), q,
      k_codes, k_norms, v_codes, v_norms, seq_lens, capacity, max_seq_len, quats, batch,
      n_kv_heads, resolve_scale(softmax_scale), out, static_cast<float*>(workspace), nullptr,
      bits, append, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // namespace

iq_status iq_decode_attention_multi(const float* q, const uint8_t* k_codes,
                                    const float* k_norms, const uint8_t* v_codes,
                                    const float* v_norms, const int32_t* seq_lens,
                                    int64_t capacity, int64_t max_seq_len, const float* quats,
                                    int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                                    int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                                    float* out, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
  if (n_tokens == 1)
    return iq_decode_attention(q, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity,
                               max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                               softmax_scale, out, workspace, workspace_bytes, stream);
  // without an append the launch only reads the cache and the lengths
  return multi_common(q, nullptr, const_cast<uint8_t*>(k_codes), const_cast<float*>(k_norms),
                      const_cast<uint8_t*>(v_codes), const_cast<float*>(v_norms),
                      const_cast<int32_t*>(seq_lens), capacity, max_seq_len, quats, batch,
                      n_tokens, n_q_heads, n_kv_heads, head_dim, softmax_scale, 3, out,
                      workspace, workspace_bytes, stream);
}

iq_status iq_decode_attention_multi_bits(const float* q, const uint8_t* k_codes,
                                         const float* k_norms, const uint8_t* v_codes,
                                         const float* v_norms, const int32_t* seq_lens,
                                         int64_t capacity, int64_t max_seq_len,
                                         const float* quats, int64_t batch, int64_t n_tokens,
                                         int64_t n_q_heads, int64_t n_kv_heads,
                                         int64_t head_dim, float softmax_scale, float* out,
                                         void* workspace, size_t workspace_bytes, int bits,
                                         hipStream_t stream) {
  if (n_tokens == 1)
    return iq_decode_attention_bits(q, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity,
                                    max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                                    softmax_scale, out, workspace, workspace_bytes, bits,
                                    stream);
  return multi_common(q, nullptr, const_cast<uint8_t*>(k_codes), const_cast<float*>(k_norms),
                      const_cast<uint8_t*>(v_codes), const_cast<float*>(v_norms),
                      const_cast<int32_t*>(seq_lens), capacity, max_seq_len, quats, batch,
                      n_tokens, n_q_heads, n_kv_heads, head_dim, softmax_scale, bits, out,
                      workspace, workspace_bytes, stream);
}

namespace {

// The fused step on records of `bits` bits with codebook cb (null: C_b); the
// paths as in decode_common.
iq_status step_common(const float* q, const void* k_new, const void* v_new, int32_t dtype,
                      uint8_t* k_codes, float* k_norms, uint8_t* v_codes, float* v_norms,
                      int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                      const float* quats, int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                      int64_t head_dim, float softmax_scale, float* out, void* workspace,
                      size_t workspace_bytes, int32_t* status_dev, int bits,
                      const iq_codebook_t* cb, hipStream_t stream) {
  if (bits != 2 && bits != 3 && bits != 4) return IQ_ERR_UNSUPPORTED;
  if (dtype != IQ_DTYPE_F32 && dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  iq::DecodePlan plan;
  const iq_status st = check_decode_args(q, k_codes, k_norms, v_codes, v_norms, seq_lens,
                                         capacity, max_seq_len, quats, batch, n_q_heads,
                                         n_kv_heads, head_dim, out, workspace, workspace_bytes,
                                         &plan);
  if (st != IQ_OK) return st;
  if (max_seq_len < 1 || n_kv_heads > 512) return IQ_ERR_INVALID_ARGUMENT;
  if (!k_new || !v_new || !iq::aligned(k_new, 16) || !iq::aligned(v_new, 16) ||
      (status_dev && !iq::aligned(status_dev, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (bits != 3) {
    // the matrix-core path only, as for iq_decode_attention_bits
    const iq_status shape = check_g8_shape(n_q_heads, n_kv_heads, batch, capacity, 16 * bits,
                                           k_norms, v_norms, plan);
    if (shape != IQ_OK) return shape;
  }
  if (batch == 0) return IQ_OK;
  const iq::StepAppend append{k_new, v_new, dtype == IQ_DTYPE_F16 ? 1 : 0, status_dev};
  hipError_t e;
  if (bits == 3) {
    e = iq::launch_decode(plan, q, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity,
                          max_seq_len, quats, batch, n_q_heads, n_kv_heads,
                          resolve_scale(softmax_scale), out, workspace, &append, stream, cb);
  } else {
    float* parts = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
    e = iq::launch_decode_g8(plan.g8_batches, plan.g8_splits, plan.g8_split_len, q, k_codes,
                             k_norms, v_codes, v_norms, seq_lens, capacity, max_seq_len, quats,
                             batch, n_kv_heads, n_q_heads / n_kv_heads,
                             resolve_scale(softmax_scale), out, parts, &append, nullptr, bits,
                             stream, cb);
  }
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // namespace

iq_status iq_decode_step(const float* q, const void* k_new, const void* v_new, int32_t dtype,
                         uint8_t* k_codes, float* k_norms, uint8_t* v_codes, float* v_norms,
                         int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                         const float* quats, int64_t batch, int64_t n_q_heads,
                         int64_t n_kv_heads, int64_t head_dim, float softmax_scale, float* out,
                         void* workspace, size_t workspace_bytes, int32_t* status_dev,
                         hipStream_t stream) {
  return step_common(q, k_new, v_new, dtype, k_codes, k_norms, v_codes, v_norms, seq_lens,
                     capacity, max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                     softmax_scale, out, workspace, workspace_bytes, status_dev, 3, nullptr,
                     stream);
}

iq_status iq_decode_step_bits(const float* q, const void* k_new, const void* v_new,
                              int32_t dtype, uint8_t* k_codes, float* k_norms,
                              uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                              int64_t capacity, int64_t max_seq_len, const float* quats,
                              int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                              int64_t head_dim, float softmax_scale, float* out, void* workspace,
                              size_t workspace_bytes, int32_t* status_dev, int bits,
                              hipStream_t stream) {
  return step_common(q, k_new, v_new, dtype, k_codes, k_norms, v_codes, v_norms, seq_lens,
                     capacity, max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                     softmax_scale, out, workspace, workspace_bytes, status_dev, bits, nullptr,
                     stream);
}

iq_status iq_decode_step_cb(const float* q, const void* k_new, const void* v_new,
                            int32_t dtype, uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                            float* v_norms, int32_t* seq_lens, int64_t capacity,
                            int64_t max_seq_len, const float* quats, const iq_codebook_t* cb,
                            int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                            int64_t head_dim, float softmax_scale, float* out, void* workspace,
                            size_t workspace_bytes, int32_t* status_dev, hipStream_t stream) {
  const iq_status st = check_codebook(cb);
  if (st != IQ_OK) return st;
  return step_common(q, k_new, v_new, dtype, k_codes, k_norms, v_codes, v_norms, seq_lens,
                     capacity, max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                     softmax_scale, out, workspace, workspace_bytes, status_dev, cb->bits, cb,
                     stream);
}

iq_status iq_decode_step_multi(const float* q, const void* k_new, const void* v_new,
                               int32_t dtype, uint8_t* k_codes, float* k_norms,
                               uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                               int64_t capacity, int64_t max_seq_len, const float* quats,
                               int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                               int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                               float* out, void* workspace, size_t workspace_bytes,
                               int32_t* status_dev, int bits, hipStream_t stream) {
  if (n_tokens == 1)
    return step_common(q, k_new, v_new, dtype, k_codes, k_norms, v_codes, v_norms, seq_lens,
                       capacity, max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                       softmax_scale, out, workspace, workspace_bytes, status_dev, bits, nullptr,
                       stream);
  if (dtype != IQ_DTYPE_F32 && dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  if (max_seq_len < 1) return IQ_ERR_INVALID_ARGUMENT;
  if (!k_new || !v_new || !iq::aligned(k_new, 16) || !iq::aligned(v_new, 16) ||
      (status_dev && !iq::aligned(status_dev, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  const iq::StepAppend append{k_new, v_new, dtype == IQ_DTYPE_F16 ? 1 : 0, status_dev};
  return multi_common(q, &append, k_codes, k_norms, v_codes, v_norms, seq_lens, capacity,
                      max_seq_len, quats, batch, n_tokens, n_q_heads, n_kv_heads, head_dim,
                      softmax_scale, bits, out, workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// Paged cache (page pools + per-sequence page tables)
// ---------------------------------------------------------------------------
namespace {

// Checks shared by the paged entry points; fills the page table.
iq_status check_pages(int64_t n_kv_heads, int64_t page_size, int64_t n_pages,
                      const int32_t* block_tables, int64_t max_pages, iq::PageTable* pt) {
  if (page_size < 16 || page_size > (int64_t(1) << 20) || (page_size & (page_size - 1)))
    return IQ_ERR_INVALID_ARGUMENT;
  int32_t shift = 0;
  while ((int64_t(1) << shift) < page_size) ++shift;
  if (n_pages < 1 || n_pages > 0x7fffffff || max_pages < 1 || block_tables == nullptr ||
      !iq::aligned(block_tables, 4))
    return IQ_ERR_INVALID_ARGUMENT;
  // the decode kernel addresses positions with 32-bit byte offsets
  if (!iq::mul_ok(max_pages, page_size) || max_pages * page_size * iq::kRecordBytes > 0x7fffffff)
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::mul_ok(n_pages, n_kv_heads) || !iq::mul_ok(n_pages * n_kv_heads, page_size) ||
      !iq::mul_ok(n_pages * n_kv_heads * page_size, iq::kRecordBytes))
    return IQ_ERR_INVALID_ARGUMENT;
  *pt = iq::PageTable{block_tables, max_pages, shift, static_cast<int32_t>(n_pages)};
  return IQ_OK;
}

iq_status check_paged_decode(const float* q, const void* k_codes, const float* k_norms,
                             const void* v_codes, const float* v_norms,
                             const int32_t* seq_lens, int64_t max_seq_len, const float* quats,
                             int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                             int64_t head_dim, const float* out, const void* workspace,
                             size_t workspace_bytes, const iq::PageTable& pt,
                             iq::DecodePlan* plan) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || n_kv_heads <= 0 || n_q_heads <= 0 || max_seq_len < 0 ||
      max_seq_len > (pt.max_pages << pt.page_shift) || batch > 65535 || n_kv_heads > 65535)
    return IQ_ERR_INVALID_ARGUMENT;
  // paged caches run on the matrix-core path: up to 16 query heads per KV
  // head, (KV head, head group of 8) rows as a grid dimension
  if (n_q_heads % n_kv_heads) return IQ_ERR_INVALID_ARGUMENT;
  if (n_q_heads / n_kv_heads > iq::kMaxGroup ||
      n_kv_heads * ((n_q_heads / n_kv_heads + 7) / 8) > 65535)
    return IQ_ERR_UNSUPPORTED;
  if (!q || !k_codes || !k_norms || !v_codes || !v_norms || !seq_lens || !quats || !out ||
      !workspace)
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::aligned(q, 16) || !iq::aligned(k_codes, 16) || !iq::aligned(v_codes, 16) ||
      !iq::aligned(k_norms, 16) || !iq::aligned(v_norms, 16) || !iq::aligned(out, 16) ||
      !iq::aligned(seq_lens, 4) || !iq::aligned(quats, 16) || !iq::aligned(workspace, 256))
    return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::plan_decode(batch, n_q_heads, n_kv_heads, max_seq_len, plan))
    return IQ_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < plan->total_bytes) return IQ_ERR_WORKSPACE_TOO_SMALL;
  return IQ_OK;
}

}  // namespace

iq_status iq_compress_kv_paged(const void* k, const void* v, int32_t dtype, int64_t batch,
                               int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                               const float* quats, uint8_t* k_codes, float* k_norms,
                               uint8_t* v_codes, float* v_norms, int64_t page_size,
                               int64_t n_pages, const int32_t* block_tables, int64_t max_pages,
                               int64_t dst_offset, hipStream_t stream) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (dtype != IQ_DTYPE_F32 && dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || n_kv_heads <= 0 || n_tokens < 0 || dst_offset < 0)
    return IQ_ERR_INVALID_ARGUMENT;
  iq::PageTable pt;
  const iq_status ps = check_pages(n_kv_heads, page_size, n_pages, block_tables, max_pages, &pt);
  if (ps != IQ_OK) return ps;
  const int64_t capacity = max_pages * page_size;
  if (dst_offset > capacity || n_tokens > capacity - dst_offset) return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::mul_ok(batch, n_kv_heads) || !iq::mul_ok(batch * n_kv_heads, n_tokens + 1) ||
      !iq::mul_ok(batch * n_kv_heads * (n_tokens + 1), kDim))
    return IQ_ERR_INVALID_ARGUMENT;
  if (batch == 0 || n_tokens == 0) return IQ_OK;
  if (k == nullptr && v == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  if (quats == nullptr || !iq::aligned(quats, 16)) return IQ_ERR_INVALID_ARGUMENT;
  if (k && (!k_codes || !k_norms || !iq::aligned(k, 16) || !iq::aligned(k_codes, 16) ||
            !iq::aligned(k_norms, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (v && (!v_codes || !v_norms || !iq::aligned(v, 16) || !iq::aligned(v_codes, 16) ||
            !iq::aligned(v_norms, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  const hipError_t e = iq::launch_compress_paged(k, v, dtype, batch, n_kv_heads, n_tokens, quats,
                                                 k_codes, k_norms, v_codes, v_norms, pt,
                                                 dst_offset, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

iq_status iq_decode_attention_paged(const float* q, const uint8_t* k_codes,
                                    const float* k_norms, const uint8_t* v_codes,
                                    const float* v_norms, int64_t page_size, int64_t n_pages,
                                    const int32_t* block_tables, int64_t max_pages,
                                    const int32_t* seq_lens, int64_t max_seq_len,
                                    const float* quats, int64_t batch, int64_t n_q_heads,
                                    int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                                    float* out, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
  iq::PageTable pt;
  iq_status st = check_pages(n_kv_heads, page_size, n_pages, block_tables, max_pages, &pt);
  if (st != IQ_OK) return st;
  iq::DecodePlan plan;
  st = check_paged_decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, max_seq_len, quats,
                          batch, n_q_heads, n_kv_heads, head_dim, out, workspace,
                          workspace_bytes, pt, &plan);
  if (st != IQ_OK) return st;
  if (batch == 0) return IQ_OK;
  float* parts = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
  const hipError_t e = iq::launch_decode_g8(
      plan.g8_batches, plan.g8_splits, plan.g8_split_len, q, const_cast<uint8_t*>(k_codes),
      const_cast<float*>(k_norms), const_cast<uint8_t*>(v_codes), const_cast<float*>(v_norms),
      const_cast<int32_t*>(seq_lens), max_pages * page_size, max_seq_len, quats, batch,
      n_kv_heads, n_q_heads / n_kv_heads, resolve_scale(softmax_scale), out, parts, nullptr, &pt,
      3, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

iq_status iq_decode_step_paged(const float* q, const void* k_new, const void* v_new,
                               int32_t dtype, uint8_t* k_codes, float* k_norms,
                               uint8_t* v_codes, float* v_norms, int64_t page_size,
                               int64_t n_pages, const int32_t* block_tables, int64_t max_pages,
                               int32_t* seq_lens, int64_t max_seq_len, const float* quats,
                               int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                               int64_t head_dim, float softmax_scale, float* out,
                               void* workspace, size_t workspace_bytes, int32_t* status_dev,
                               hipStream_t stream) {
  if (dtype != IQ_DTYPE_F32 && dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  iq::PageTable pt;
  iq_status st = check_pages(n_kv_heads, page_size, n_pages, block_tables, max_pages, &pt);
  if (st != IQ_OK) return st;
  iq::DecodePlan plan;
  st = check_paged_decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, max_seq_len, quats,
                          batch, n_q_heads, n_kv_heads, head_dim, out, workspace,
                          workspace_bytes, pt, &plan);
  if (st != IQ_OK) return st;
  if (max_seq_len < 1) return IQ_ERR_INVALID_ARGUMENT;
  if (!k_new || !v_new || !iq::aligned(k_new, 16) || !iq::aligned(v_new, 16) ||
      (status_dev && !iq::aligned(status_dev, 4)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (batch == 0) return IQ_OK;
  const iq::StepAppend append{k_new, v_new, dtype == IQ_DTYPE_F16 ? 1 : 0, status_dev};
  float* parts = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
  const hipError_t e = iq::launch_decode_g8(
      plan.g8_batches, plan.g8_splits, plan.g8_split_len, q, k_codes, k_norms, v_codes, v_norms,
      seq_lens, max_pages * page_size, max_seq_len, quats, batch, n_kv_heads,
      n_q_heads / n_kv_heads, resolve_scale(softmax_scale), out, parts, &append, &pt, 3, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

iq_status iq_decode_attention_multi_paged(
    const float* q, const uint8_t* k_codes, const float* k_norms, const uint8_t* v_codes,
    const float* v_norms, int64_t page_size, int64_t n_pages, const int32_t* block_tables,
    int64_t max_pages, const int32_t* seq_lens, int64_t max_seq_len, const float* quats,
    int64_t batch, int64_t n_tokens, int64_t n_q_heads, int64_t n_kv_heads, int64_t head_dim,
    float softmax_scale, float* out, void* workspace, size_t workspace_bytes,
    hipStream_t stream) {
  if (n_tokens == 1)
    return iq_decode_attention_paged(q, k_codes, k_norms, v_codes, v_norms, page_size, n_pages,
                                     block_tables, max_pages, seq_lens, max_seq_len, quats,
                                     batch, n_q_heads, n_kv_heads, head_dim, softmax_scale, out,
                                     workspace, workspace_bytes, stream);
  if (n_tokens < 2 || n_tokens > 4) return IQ_ERR_UNSUPPORTED;
  iq::PageTable pt;
  iq_status st = check_pages(n_kv_heads, page_size, n_pages, block_tables, max_pages, &pt);
  if (st != IQ_OK) return st;
  iq::DecodePlan plan;
  st = check_paged_decode(q, k_codes, k_norms, v_codes, v_norms, seq_lens, max_seq_len, quats,
                          batch, n_q_heads, n_kv_heads, head_dim, out, workspace, SIZE_MAX, pt,
                          &plan);
  if (st != IQ_OK) return st;
  // multi-token decode runs 8 query heads per KV head
  if (n_q_heads != 8 * n_kv_heads) return IQ_ERR_UNSUPPORTED;
  if (!iq::mul_ok(batch, n_tokens) || !iq::mul_ok(batch * n_tokens, n_q_heads))
    return IQ_ERR_INVALID_ARGUMENT;
  // the merge kernel's grid takes (sequence, token) as one dimension
  if (batch * n_tokens > 65535) return IQ_ERR_UNSUPPORTED;
  const size_t need = iq_decode_multi_workspace_bytes(batch, n_tokens, n_q_heads, n_kv_heads,
                                                      max_seq_len, head_dim);
  if (need == 0) return IQ_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < need) return IQ_ERR_WORKSPACE_TOO_SMALL;
  if (batch == 0) return IQ_OK;
  const hipError_t e = iq::launch_decode_g8_multi(
      plan.g8_batches, plan.g8_splits, plan.g8_split_len, static_cast<int>(n_tokens), q,
      const_cast<uint8_t*>(k_codes), const_cast<float*>(k_norms), const_cast<uint8_t*>(v_codes),
      const_cast<float*>(v_norms), const_cast<int32_t*>(seq_lens), max_pages << pt.page_shift,
      max_seq_len, quats, batch, n_kv_heads, resolve_scale(softmax_scale), out,
      static_cast<float*>(workspace), &pt, 3, nullptr, stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

namespace {

iq_status dequant_common(const uint8_t* k_codes, const float* k_norms, const uint8_t* v_codes,
                         const float* v_norms, const float* quats, const int32_t* seq_lens,
                         int64_t batch, int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                         int64_t capacity, int64_t src_offset, int32_t out_dtype, void* k_out,
                         void* v_out, const iq_codebook_t* cb, hipStream_t stream) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (out_dtype != IQ_DTYPE_F32 && out_dtype != IQ_DTYPE_F16) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || n_kv_heads <= 0 || n_tokens < 0 || capacity < 0 || src_offset < 0)
    return IQ_ERR_INVALID_ARGUMENT;
  if (src_offset > capacity || n_tokens > capacity - src_offset) return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::mul_ok(batch, n_kv_heads) || !iq::mul_ok(batch * n_kv_heads, capacity + 1) ||
      !iq::mul_ok(batch * n_kv_heads * (capacity + 1), kDim))
    return IQ_ERR_INVALID_ARGUMENT;
  if (batch == 0 || n_tokens == 0) return IQ_OK;
  if (k_codes == nullptr && v_codes == nullptr) return IQ_ERR_INVALID_ARGUMENT;
  if (quats == nullptr || !iq::aligned(quats, 16)) return IQ_ERR_INVALID_ARGUMENT;
  if (seq_lens && !iq::aligned(seq_lens, 4)) return IQ_ERR_INVALID_ARGUMENT;
  if (k_codes && (!k_norms || !k_out || !iq::aligned(k_codes, 4) || !iq::aligned(k_norms, 4) ||
                  !iq::aligned(k_out, 16)))
    return IQ_ERR_INVALID_ARGUMENT;
  if (v_codes && (!v_norms || !v_out || !iq::aligned(v_codes, 4) || !iq::aligned(v_norms, 4) ||
                  !iq::aligned(v_out, 16)))
    return IQ_ERR_INVALID_ARGUMENT;
  const hipError_t e = iq::launch_dequant(k_codes, k_norms, v_codes, v_norms, quats, seq_lens,
                                          batch, n_kv_heads, n_tokens, capacity, src_offset,
                                          out_dtype == IQ_DTYPE_F16 ? 1 : 0, k_out, v_out,
                                          stream, cb);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // namespace

iq_status iq_dequantize_kv(const uint8_t* k_codes, const float* k_norms,
                           const uint8_t* v_codes, const float* v_norms, const float* quats,
                           const int32_t* seq_lens, int64_t batch, int64_t n_kv_heads,
                           int64_t n_tokens, int64_t head_dim, int64_t capacity,
                           int64_t src_offset, int32_t out_dtype, void* k_out, void* v_out,
                           hipStream_t stream) {
  return dequant_common(k_codes, k_norms, v_codes, v_norms, quats, seq_lens, batch, n_kv_heads,
                        n_tokens, head_dim, capacity, src_offset, out_dtype, k_out, v_out,
                        nullptr, stream);
}

iq_status iq_dequantize_kv_cb(const uint8_t* k_codes, const float* k_norms,
                              const uint8_t* v_codes, const float* v_norms, const float* quats,
                              const iq_codebook_t* cb, const int32_t* seq_lens, int64_t batch,
                              int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                              int64_t capacity, int64_t src_offset, int32_t out_dtype,
                              void* k_out, void* v_out, hipStream_t stream) {
  const iq_status st = check_codebook(cb);
  if (st != IQ_OK) return st;
  // the materialization kernel decodes 3-bit records
  if (cb->bits != 3) return IQ_ERR_UNSUPPORTED;
  return dequant_common(k_codes, k_norms, v_codes, v_norms, quats, seq_lens, batch, n_kv_heads,
                        n_tokens, head_dim, capacity, src_offset, out_dtype, k_out, v_out, cb,
                        stream);
}

size_t iq_decode_f16_workspace_bytes(int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                     int64_t max_seq_len, int64_t head_dim) {
  if (head_dim != kDim || batch < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || max_seq_len < 0)
    return 0;
  if (n_q_heads % n_kv_heads || n_q_heads / n_kv_heads > 8) return 0;
  return iq::f16_workspace_bytes(batch, n_kv_heads, max_seq_len);
}

iq_status iq_decode_attention_f16(const float* q, const void* k, const void* v,
                                  const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                                  int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                  int64_t head_dim, float softmax_scale, float* out,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (head_dim != kDim) return IQ_ERR_UNSUPPORTED;
  if (batch < 0 || n_q_heads <= 0 || n_kv_heads <= 0 || capacity < 0 || max_seq_len < 0 ||
      max_seq_len > capacity || capacity > 0x7fffffff || batch > 0xffffff)
    return IQ_ERR_INVALID_ARGUMENT;
  if (n_q_heads % n_kv_heads) return IQ_ERR_INVALID_ARGUMENT;
  if (n_q_heads / n_kv_heads > 8) return IQ_ERR_UNSUPPORTED;
  if (!iq::mul_ok(batch, n_kv_heads) || !iq::mul_ok(batch * n_kv_heads, capacity + 1) ||
      !iq::mul_ok(batch * n_kv_heads * (capacity + 1), kDim) ||
      !iq::mul_ok(batch, n_q_heads) || batch * n_q_heads > 0x7fffffff)
    return IQ_ERR_INVALID_ARGUMENT;
  if (!q || !k || !v || !seq_lens || !out || !workspace) return IQ_ERR_INVALID_ARGUMENT;
  if (!iq::aligned(q, 16) || !iq::aligned(k, 16) || !iq::aligned(v, 16) ||
      !iq::aligned(out, 16) || !iq::aligned(seq_lens, 4) || !iq::aligned(workspace, 256))
    return IQ_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < iq::f16_workspace_bytes(batch, n_kv_heads, max_seq_len))
    return IQ_ERR_WORKSPACE_TOO_SMALL;
  if (batch == 0) return IQ_OK;
  const hipError_t e = iq::launch_decode_f16(
      q, static_cast<const __half*>(k), static_cast<const __half*>(v), seq_lens, capacity,
      max_seq_len, batch, n_kv_heads, n_q_heads / n_kv_heads, resolve_scale(softmax_scale), out,
      static_cast<float*>(workspace), stream);
  return e == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // extern "C"
