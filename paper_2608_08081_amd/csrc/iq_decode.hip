// Decode attention on the packed 3-bit cache (App. A; Table 2; Sec. 3.4)
// for gfx950, generic path (any group size G <= 16).
//
// Two launches:
//  1. split kernel, one workgroup per (sequence, KV head, split of positions):
//     rotates the G query heads of the group into the compressed space once
//     (q_tilde = R q, Eq. 2 applied to the query, App. A), scores every
//     position of the split against the packed keys (fused QK, Table 2 A),
//     takes a numerically safe softmax over the split (Table 2 B) and
//     accumulates the value records weighted by it (fused V, Table 2 C).
//     Output per (query head, split): running max m, sum l and the
//     unnormalized rotated-space output o_tilde[128].
//  2. combine kernel, one workgroup per (sequence, query head): merges the
//     splits (flash-decoding rescale by exp(m_s - max m)), divides by the
//     total sum and applies the single inverse rotation R^T = H_128 M^T
//     (Table 2 D; Sec. 3.4).
// Neither kernel ever forms a full-precision key or value vector.
#include <hip/hip_runtime.h>
#include <math.h>

#include "iq_device.h"
#include "iq_internal.h"

namespace iq {
namespace {

constexpr int kSplitThreads = 256;
constexpr int kMaxSplitLen = 512;
constexpr int kPartialFloats = 2 + kDim;   // m, l, o_tilde[128]
constexpr float kInvSqrtDim = 0.08838834764831845f;

// In-LDS rotation of nvec 128-vectors (row-major in buf): forward
// y = diag(M_i) H_128 x  (WHT first, then the SO(4) blocks).
__device__ void rotate_forward_lds(float* buf, int nvec, const float* __restrict__ quats_head,
                                   int tid, int nthreads) {
  const int n = nvec * kDim;
  for (int st = 1; st < kDim; st <<= 1) {
    for (int e = tid; e < n; e += nthreads) {
      const int i = e & (kDim - 1);
      if (!(i & st)) {
        const float a = buf[e], b = buf[e + st];
        buf[e] = a + b;
        buf[e + st] = a - b;
      }
    }
    __syncthreads();
  }
  // SO(4) blocks: thread per (vector, block)
  for (int e = tid; e < nvec * kNumBlocks; e += nthreads) {
    const int v = e / kNumBlocks, blk = e % kNumBlocks;
    float m[4][4];
    so4_matrix(quats_head + 8 * blk, m);
    float* z = buf + v * kDim + 4 * blk;
    const float z0 = z[0] * kInvSqrtDim, z1 = z[1] * kInvSqrtDim;
    const float z2 = z[2] * kInvSqrtDim, z3 = z[3] * kInvSqrtDim;
#pragma unroll
    for (int r = 0; r < 4; ++r) z[r] = m[r][0] * z0 + m[r][1] * z1 + m[r][2] * z2 + m[r][3] * z3;
  }
  __syncthreads();
}

// Decode the 128 levels of one packed record (12 words) into registers.
__device__ __forceinline__ void unpack_record(const uint32_t (&w)[kRecordWords],
                                              const float* __restrict__ lut, float (&val)[kDim]) {
#pragma unroll
  for (int i = 0; i < kDim; ++i) {
    const int bit = 3 * i, word = bit >> 5, off = bit & 31;
    uint32_t c = w[word] >> off;
    if (off > 29) c |= w[word + 1] << (32 - off);
    val[i] = lut[c & 7u];
  }
}

__global__ __launch_bounds__(kSplitThreads) void decode_split_kernel(
    const float* __restrict__ q, const uint8_t* __restrict__ k_codes,
    const float* __restrict__ k_norms, const uint8_t* __restrict__ v_codes,
    const float* __restrict__ v_norms, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ quats, float* __restrict__ partials, int64_t capacity,
    int64_t max_seq_len, int n_q_heads, int n_kv_heads, int group, int split_len, int n_splits,
    float scale, Codebook cb) {
  __shared__ float qt[kMaxGroup * kDim];
  __shared__ float wts[kMaxGroup * kMaxSplitLen];
  __shared__ float lut[8];
  __shared__ float stat_m[kMaxGroup], stat_l[kMaxGroup];

  const int tid = threadIdx.x;
  const int split = blockIdx.x % n_splits;
  const int bg = blockIdx.x / n_splits;
  const int g = bg % n_kv_heads;
  const int b = bg / n_kv_heads;

  int64_t seq = seq_lens[b];
  if (seq > max_seq_len) seq = max_seq_len;
  const int64_t start = static_cast<int64_t>(split) * split_len;
  int64_t end = start + split_len;
  if (end > seq) end = seq;
  const int n = end > start ? static_cast<int>(end - start) : 0;

  float* part_base = partials;
  auto part = [&](int hh) -> float* {
    const int64_t h = static_cast<int64_t>(g) * group + hh;
    return part_base + ((static_cast<int64_t>(b) * n_q_heads + h) * n_splits + split) * kPartialFloats;
  };

  if (n == 0) {
    for (int e = tid; e < group * kPartialFloats; e += kSplitThreads) {
      const int hh = e / kPartialFloats, k = e % kPartialFloats;
      part(hh)[k] = (k == 0) ? -INFINITY : 0.0f;
    }
    return;
  }

  if (tid < 8) lut[tid] = codebook_level(cb, tid);
  const float* qsrc = q + (static_cast<int64_t>(b) * n_q_heads + static_cast<int64_t>(g) * group) * kDim;
  for (int e = tid; e < group * kDim; e += kSplitThreads) qt[e] = qsrc[e];
  __syncthreads();
  rotate_forward_lds(qt, group, quats + g * kQuatFloats, tid, kSplitThreads);
  for (int e = tid; e < group * kDim; e += kSplitThreads) qt[e] *= scale;
  __syncthreads();

  const int64_t cache_row = (static_cast<int64_t>(b) * n_kv_heads + g) * capacity;

  // Phase A: scores.  One thread per position; the record is unpacked into
  // registers and dotted with each query head read from LDS (broadcast).
  for (int j = tid; j < n; j += kSplitThreads) {
    const int64_t pos = cache_row + start + j;
    const uint4* rec = reinterpret_cast<const uint4*>(k_codes + pos * kRecordBytes);
    const uint4 u0 = rec[0], u1 = rec[1], u2 = rec[2];
    const uint32_t w[kRecordWords] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y,
                                      u1.z, u1.w, u2.x, u2.y, u2.z, u2.w};
    float val[kDim];
    unpack_record(w, lut, val);
    const float sk = k_norms[pos];
    for (int hh = 0; hh < group; ++hh) {
      const float* qh = qt + hh * kDim;
      float acc0 = 0.f, acc1 = 0.f, acc2 = 0.f, acc3 = 0.f;
#pragma unroll
      for (int i = 0; i < kDim; i += 4) {
        acc0 += val[i] * qh[i];
        acc1 += val[i + 1] * qh[i + 1];
        acc2 += val[i + 2] * qh[i + 2];
        acc3 += val[i + 3] * qh[i + 3];
      }
      wts[hh * kMaxSplitLen + j] = ((acc0 + acc1) + (acc2 + acc3)) * sk;
    }
  }
  __syncthreads();

  // Phase B: per head, max and exp-sum over the split; weights *= s^V.
  const int wave = tid >> 6, lane = tid & 63;
  for (int hh = wave; hh < group; hh += kSplitThreads / 64) {
    float* wrow = wts + hh * kMaxSplitLen;
    float mx = -INFINITY;
    for (int j = lane; j < n; j += 64) mx = fmaxf(mx, wrow[j]);
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    float sum = 0.f;
    for (int j = lane; j < n; j += 64) {
      const float e = __expf(wrow[j] - mx);
      sum += e;
      wrow[j] = e * v_norms[cache_row + start + j];
    }
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) {
      stat_m[hh] = mx;
      stat_l[hh] = sum;
    }
  }
  __syncthreads();

  // Phase C: thread per (head, dim pair f); field f = bits 6f..6f+5 of each
  // value record holds the codes of dims 2f and 2f+1.
  for (int p = tid; p < group * 64; p += kSplitThreads) {
    const int hh = p >> 6, f = p & 63;
    const int bit = 6 * f, word = bit >> 5, off = bit & 31;
    const float* wrow = wts + hh * kMaxSplitLen;
    float acc0 = 0.f, acc1 = 0.f;
    for (int j = 0; j < n; ++j) {
      const uint32_t* rec =
          reinterpret_cast<const uint32_t*>(v_codes + (cache_row + start + j) * kRecordBytes);
      uint32_t field = rec[word] >> off;
      if (off > 26) field |= rec[word + 1] << (32 - off);
      const float wj = wrow[j];
      acc0 += wj * lut[field & 7u];
      acc1 += wj * lut[(field >> 3) & 7u];
    }
    float* dst = part(hh);
    dst[2 + 2 * f] = acc0;
    dst[2 + 2 * f + 1] = acc1;
    if (f == 0) {
      dst[0] = stat_m[hh];
      dst[1] = stat_l[hh];
    }
  }
}

__global__ __launch_bounds__(kDim) void decode_combine_kernel(
    const float* __restrict__ partials, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ quats, float* __restrict__ out, int64_t max_seq_len, int n_q_heads,
    int group, int split_len, int n_splits) {
  __shared__ float buf[kDim];
  const int d = threadIdx.x;
  const int h = blockIdx.x % n_q_heads;
  const int b = blockIdx.x / n_q_heads;
  const int g = h / group;
  int64_t seq = seq_lens[b];
  if (seq > max_seq_len) seq = max_seq_len;
  int used = static_cast<int>((seq + split_len - 1) / split_len);
  if (used > n_splits) used = n_splits;
  float* dst = out + (static_cast<int64_t>(b) * n_q_heads + h) * kDim;
  if (used <= 0) {
    dst[d] = 0.f;
    return;
  }
  const float* base = partials + (static_cast<int64_t>(b) * n_q_heads + h) * n_splits * kPartialFloats;
  float mx = -INFINITY;
  for (int s = 0; s < used; ++s) mx = fmaxf(mx, base[s * kPartialFloats]);
  float l = 0.f, o = 0.f;
  for (int s = 0; s < used; ++s) {
    const float* p = base + s * kPartialFloats;
    const float c = __expf(p[0] - mx);
    l += c * p[1];
    o += c * p[2 + d];
  }
  buf[d] = o / l;
  __syncthreads();
  // inverse rotation: z = M_blk^T o_blk, then H_128 z / sqrt(128)
  const int blk = d >> 2, r = d & 3;
  float m[4][4];
  so4_matrix(quats + g * kQuatFloats + 8 * blk, m);
  const float* ob = buf + 4 * blk;
  const float z = m[0][r] * ob[0] + m[1][r] * ob[1] + m[2][r] * ob[2] + m[3][r] * ob[3];
  __syncthreads();
  buf[d] = z;
  __syncthreads();
  for (int st = 1; st < kDim; st <<= 1) {
    const float a = buf[d], bb = buf[d ^ st];
    const float y = (d & st) ? (bb - a) : (a + bb);
    __syncthreads();
    buf[d] = y;
    __syncthreads();
  }
  dst[d] = buf[d] * kInvSqrtDim;
}

}  // namespace

// Splits of the generic path: aim at >= 1024 workgroups; 64..512 positions.
static void plan_generic(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len,
                         int64_t* split_len, int64_t* n_splits) {
  const int64_t work = batch * n_kv_heads * (max_seq_len > 0 ? max_seq_len : 1);
  int64_t len = (work + 1023) / 1024;
  len = ((len + 63) / 64) * 64;
  if (len < 64) len = 64;
  if (len > kMaxSplitLen) len = kMaxSplitLen;
  *split_len = len;
  *n_splits = max_seq_len > 0 ? (max_seq_len + len - 1) / len : 1;
}

static size_t round256(size_t x) { return (x + 255) / 256 * 256; }

bool plan_decode(int64_t batch, int64_t n_q_heads, int64_t n_kv_heads, int64_t max_seq_len,
                 DecodePlan* plan) {
  if (batch < 0 || n_kv_heads <= 0 || n_q_heads <= 0 || max_seq_len < 0) return false;
  if (n_q_heads % n_kv_heads) return false;
  const int64_t group = n_q_heads / n_kv_heads;
  if (group > kMaxGroup) return false;
  DecodePlan p{};
  p.kernel = 0;
  plan_generic(batch, n_kv_heads, max_seq_len, &p.split_len, &p.n_splits);
  // workspace = split partials of whichever path runs (no other state)
  p.ticket_bytes = 0;
  p.partial_bytes =
      round256(static_cast<size_t>(batch) * n_q_heads * p.n_splits * kPartialFloats * 4);
  size_t need = p.partial_bytes;
  {
    // the matrix-core path: KV heads in head groups of 8 query heads
    const int64_t rows = n_kv_heads * ((group + 7) / 8);
    int nb = 0;
    int64_t splits = 0, len = 0;
    g8_plan(batch, rows, max_seq_len, &nb, &splits, &len);
    p.g8_batches = nb;
    p.g8_splits = splits;
    p.g8_split_len = len;
    // one partial per split, and one for the fused step's new token
    p.g8_partial_bytes = g8_partial_region_bytes(batch, rows, splits) +
                         round256(static_cast<size_t>(batch) * 4);
    if (p.g8_partial_bytes > need) need = p.g8_partial_bytes;
  }
  size_t generic_bytes = p.ticket_bytes + need;
  p.total_bytes = generic_bytes > 0 ? generic_bytes : 256;
  *plan = p;
  return true;
}

hipError_t launch_decode(const DecodePlan& plan, const float* q, uint8_t* k_codes,
                         float* k_norms, uint8_t* v_codes, float* v_norms,
                         int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                         const float* quats, int64_t batch, int64_t n_q_heads,
                         int64_t n_kv_heads, float scale, float* out, void* workspace,
                         const StepAppend* append, hipStream_t stream, const iq_codebook_t* cb) {
  if (batch == 0) return hipSuccess;
  const int group = static_cast<int>(n_q_heads / n_kv_heads);
  const bool aligned16 = (reinterpret_cast<uintptr_t>(k_norms) % 16 == 0) &&
                         (reinterpret_cast<uintptr_t>(v_norms) % 16 == 0);
  // the matrix-core kernel addresses one (sequence, KV head) row with
  // 32-bit byte offsets, loads whole batches of 16 positions below
  // max_seq_len (clamped to the row: capacity a multiple of 16, at least
  // 16), and takes (KV head, head group) rows and sequences as grid
  // dimensions (at most 65535 each)
  const bool row32 = capacity * kRecordBytes <= 0x7fffffff;
  const bool grid_ok = batch <= 65535 && n_kv_heads * ((group + 7) / 8) <= 65535;
  if (plan.g8_batches > 0 && capacity % 16 == 0 && capacity >= 16 && aligned16 && row32 &&
      grid_ok) {
    float* parts = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
    return launch_decode_g8(plan.g8_batches, plan.g8_splits, plan.g8_split_len, q, k_codes,
                            k_norms, v_codes, v_norms, seq_lens, capacity, max_seq_len, quats,
                            batch, n_kv_heads, group, scale, out, parts, append, nullptr, 3,
                            stream, cb);
  }
  if (append) {
    // generic path of the fused step: the append kernel, then attention
    // over the advanced lengths
    const hipError_t e =
        launch_append(append->k_new, append->v_new, append->f16 ? IQ_DTYPE_F16 : IQ_DTYPE_F32,
                      batch, n_kv_heads, quats, k_codes, k_norms, v_codes, v_norms, capacity,
                      seq_lens, append->status, stream, cb);
    if (e != hipSuccess) return e;
  }
  float* partials = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.ticket_bytes);
  const int64_t split_blocks = batch * n_kv_heads * plan.n_splits;
  hipLaunchKernelGGL(decode_split_kernel, dim3(static_cast<unsigned>(split_blocks)),
                     dim3(kSplitThreads), 0, stream, q, k_codes, k_norms, v_codes, v_norms,
                     seq_lens, quats, partials, capacity, max_seq_len,
                     static_cast<int>(n_q_heads), static_cast<int>(n_kv_heads), group,
                     static_cast<int>(plan.split_len), static_cast<int>(plan.n_splits), scale,
                     codebook_for<3>(cb));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(static_cast<unsigned>(batch * n_q_heads)),
                     dim3(kDim), 0, stream, partials, seq_lens, quats, out, max_seq_len,
                     static_cast<int>(n_q_heads), group, static_cast<int>(plan.split_len),
                     static_cast<int>(plan.n_splits));
  return hipGetLastError();
}

}  // namespace iq
