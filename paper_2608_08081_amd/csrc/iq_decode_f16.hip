// Decode attention on an uncompressed fp16 KV cache: the "FP16 tensors ->
// GEMM Q K^T -> softmax, . V" half of the reconstruct-then-compute pipeline
// (Sec. 1, Fig. 1 top), and the uncompressed-cache baseline the packed path
// is measured against.  Split-K (flash-decoding), gfx950.
//
// Work decomposition: one 512-thread workgroup (8 waves) per (sequence b,
// KV head g, split); the split's 16-position batches are dealt to the waves
// in contiguous runs.  All of a wave's loads (query, then keys, then values)
// are issued before any arithmetic.
//
// Both contractions run on the matrix cores:
//   QK: v_mfma_f32_16x16x32_f16, rows = 16 positions, columns = 16 query
//       columns, 32 dims per instruction.  The fp32 query (pre-scaled by
//       scale * log2 e) is split into fp16 hi + lo parts: columns 0..7 carry
//       the group's (up to 8) heads' hi parts, columns 8..15 their lo parts;
//       lanes n and n ^ 8 add their products (DPP row rotation by 8), so the
//       scores carry ~22 bits.  A lane (t, gk) supplies dims 32kb+8gk..+7
//       of position t for instruction kb, read straight from the cache.
//   PV: v_mfma_f32_16x16x16_f16, O[row][n] += sum_k P[row][k] V[k][8n + j]
//       for the 8 instructions j = 0..7.  Row h < 8 carries head h's fp16
//       weights, row 8 + h the fp16 remainder of the same fp32 weights, so
//       the weights also carry ~22 bits.  Lane group gk holds positions
//       4gk..4gk+3 in both operands, exactly the rows the QK accumulator left
//       in that lane group, so the weights never leave their lanes.  A lane
//       loads dims 8n..8n+7 of its 4 positions (16 bytes each) and builds
//       the B operand of instruction j by pairing element j of the four
//       loads (byte permutes).
// Softmax is two-phase per wave (all scores, one max per head, then the
// weights), in log2 units so exp2 is one instruction.  The 8 waves merge in
// LDS; with several splits each workgroup writes its partial (m, l, O) per
// head and a second kernel merges them and divides by the sum.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "iq_device.h"
#include "iq_internal.h"

namespace iq {
namespace {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxBatches = 4;     // 16-position batches per wave (register budget)
constexpr int kCols = 8;           // query heads per KV head carried by the MFMA columns
constexpr int kPart = 2 + kDim;    // m, l, o[128] per head
constexpr int kMergeThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f32x4_t mfma_qk(u32x4_t a, u32x4_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a),
                                                __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma_pv(u32x2_t a, u32x2_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(half4_t, a),
                                               __builtin_bit_cast(half4_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_half2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __floats2half2_rn(lo, hi));
}

__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Fixed position range of one split and the wave's run of batches in it.
struct WaveRange {
  int p0;      // first position of the wave's first batch
  int nb;      // batches of the wave (0 = nothing to attend)
  int end;     // first position not attended
};

__device__ __forceinline__ WaveRange wave_range(int split, int split_len, int len, int wave) {
  const int s0 = split * split_len;
  int s1 = s0 + split_len;
  s1 = s1 < len ? s1 : len;
  const int n = s1 > s0 ? s1 - s0 : 0;
  const int nbat = (n + 15) >> 4;
  const int per = nbat / kWaves, extra = nbat % kWaves;
  const int b0 = wave * per + (wave < extra ? wave : extra);
  return WaveRange{s0 + 16 * b0, per + (wave < extra ? 1 : 0), s1};
}

// Workgroup (b, g, split).  Partials layout: [b][g][split][8][kPart].
template <int NB>
__global__ __launch_bounds__(kThreads) void decode_f16_kernel(
    const float* __restrict__ q, const __half* __restrict__ kc, const __half* __restrict__ vc,
    const int32_t* __restrict__ seq_lens, float* __restrict__ partials, float* __restrict__ out,
    int64_t capacity, int max_len, int n_kv_heads, int group, int n_splits, int split_len,
    float qscale) {
  __shared__ __attribute__((aligned(16))) f32x4_t wave_o[kWaves][8][64];   // [w][j][lane]
  __shared__ float wave_ml[kWaves][2][kCols];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x % n_splits;
  const int bg = blockIdx.x / n_splits;
  const int b = bg / n_kv_heads, g = bg % n_kv_heads;
  int len = seq_lens[b];
  len = len < max_len ? len : max_len;
  len = len > 0 ? len : 0;
  const WaveRange wr = wave_range(split, split_len, len, wave);
  const int n = lane & 15, gk = lane >> 4;
  const int head = n & 7;

  float m_w = -INFINITY, l_w = 0.f;
  f32x4_t o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (wr.nb > 0) {   // uniform over the wave
    // ---- loads: query slice, then keys, then values of every batch ----------
    const bool live = head < group;
    const float* qh = q + (static_cast<int64_t>(b) * n_kv_heads * group +
                           static_cast<int64_t>(g) * group + (live ? head : 0)) * kDim;
    f32x4_t qv[4][2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const f32x4_t* src = reinterpret_cast<const f32x4_t*>(qh + 32 * kb + 8 * gk);
      qv[kb][0] = src[0];
      qv[kb][1] = src[1];
    }
    const int64_t row0 = static_cast<int64_t>(bg) * capacity;
    const int last = len - 1;
    u32x4_t kop[NB][4], vop[NB][4];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int ib = i < wr.nb ? i : wr.nb - 1;   // repeated batches are masked
      int t = wr.p0 + 16 * ib + n;
      t = t < last ? t : last;
      const u32x4_t* src = reinterpret_cast<const u32x4_t*>(kc + (row0 + t) * kDim + 8 * gk);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kop[i][kb] = src[4 * kb];   // dims 32kb + 8gk
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int ib = i < wr.nb ? i : wr.nb - 1;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        int t = wr.p0 + 16 * ib + 4 * gk + e;
        t = t < last ? t : last;
        vop[i][e] = *reinterpret_cast<const u32x4_t*>(vc + (row0 + t) * kDim + 8 * n);
      }
    }
    // every load is in flight before the first use
    __builtin_amdgcn_sched_barrier(0);

    // query columns: hi parts in columns 0..7, lo parts in 8..15
    u32x4_t qb[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float x0 = qv[kb][e >> 1][2 * (e & 1)] * qscale;
        float x1 = qv[kb][e >> 1][2 * (e & 1) + 1] * qscale;
        if (n >= 8) {   // lo part: what the fp16 hi part leaves
          x0 -= __half2float(__float2half_rn(x0));
          x1 -= __half2float(__float2half_rn(x1));
        }
        w[e] = live ? pack_half2(x0, x1) : 0u;
      }
      qb[kb] = u32x4_t{w[0], w[1], w[2], w[3]};
    }

    // ---- phase 1: scores of every batch, running max ----------------------
    float sc[NB][4];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) acc = mfma_qk(kop[i][kb], qb[kb], acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float s = acc[r] + xor_lane<8>(acc[r]);   // hi + lo columns
        const int t = wr.p0 + 16 * i + 4 * gk + r;
        const bool ok = i < wr.nb && t < wr.end;
        sc[i][r] = ok ? s : -INFINITY;
        m_w = fmaxf(m_w, sc[i][r]);
      }
    }
    m_w = fmaxf(m_w, __shfl_xor(m_w, 16));
    m_w = fmaxf(m_w, __shfl_xor(m_w, 32));

    // ---- phase 2: weights and the PV products -----------------------------
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      float p[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[r] = __builtin_amdgcn_exp2f(sc[i][r] - m_w);   // exp2(-inf) = 0
        l_w += p[r];
      }
      uint32_t aw[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        float x0 = p[2 * e], x1 = p[2 * e + 1];
        if (n >= 8) {
          x0 -= __half2float(__float2half_rn(x0));
          x1 -= __half2float(__float2half_rn(x1));
        }
        aw[e] = pack_half2(x0, x1);
      }
      const u32x2_t a = u32x2_t{aw[0], aw[1]};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int w = j >> 1;
        const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
        const u32x2_t bv = u32x2_t{__builtin_amdgcn_perm(vop[i][1][w], vop[i][0][w], sel),
                                   __builtin_amdgcn_perm(vop[i][3][w], vop[i][2][w], sel)};
        o[j] = mfma_pv(a, bv, o[j]);
      }
    }
    // lanes n and n ^ 8 hold the same weights: sum the hi-column lanes only
    l_w = n < 8 ? l_w : 0.f;
    l_w += __shfl_xor(l_w, 16);
    l_w += __shfl_xor(l_w, 32);
  }

  // ---- merge of the 8 waves in LDS --------------------------------------------
#pragma unroll
  for (int j = 0; j < 8; ++j) wave_o[wave][j][lane] = o[j];
  if (lane < kCols) {
    wave_ml[wave][0][lane] = m_w;   // lane h: head h (lanes 0..7 hold heads 0..7)
    wave_ml[wave][1][lane] = l_w;
  }
  lds_barrier();
  // thread (h, dims 2dp, 2dp + 1); head h >= group is idle
  const int h = tid >> 6, dp = tid & 63;
  if (h >= group) return;
  const int d0 = 2 * dp;
  const int j0 = d0 & 7, cn = d0 >> 3;
  const int lane_hi = 16 * (h >> 2) + cn, lane_lo = lane_hi + 32, r = h & 3;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wave_ml[w][0][h]);
  float L = 0.f, O0 = 0.f, O1 = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const float mw = wave_ml[w][0][h];
    const float c = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - M);
    L += c * wave_ml[w][1][h];
    O0 += c * (wave_o[w][j0][lane_hi][r] + wave_o[w][j0][lane_lo][r]);
    O1 += c * (wave_o[w][j0 + 1][lane_hi][r] + wave_o[w][j0 + 1][lane_lo][r]);
  }
  const int64_t hq = static_cast<int64_t>(b) * n_kv_heads * group +
                     static_cast<int64_t>(g) * group + h;
  if (n_splits == 1) {
    const float inv = L > 0.f ? 1.0f / L : 0.f;   // an empty sequence gives zeros
    *reinterpret_cast<float2*>(out + hq * kDim + d0) = float2{O0 * inv, O1 * inv};
    return;
  }
  float* pp = partials + (static_cast<int64_t>(bg) * n_splits + split) * (kCols * kPart) +
              h * kPart;
  if (dp == 0) {
    pp[0] = M;
    pp[1] = L;
  }
  *reinterpret_cast<float2*>(pp + 2 + d0) = float2{O0, O1};
}

// Merge of the split partials of one (sequence b, query head h): thread
// (sg, dq) takes splits sg, sg + 8, ... and dims 4dq .. 4dq + 3.  Splits with
// nothing to attend carry m = -inf and are skipped.
__global__ __launch_bounds__(kMergeThreads) void merge_f16_kernel(
    const float* __restrict__ partials, float* __restrict__ out, int n_kv_heads, int group,
    int n_splits) {
  constexpr int kUnroll = 8;
  __shared__ __attribute__((aligned(16))) float red_o[8][kDim];
  __shared__ float red_m[8], red_l[8];
  const int tid = threadIdx.x;
  const int n_q_heads = n_kv_heads * group;
  const int hq = blockIdx.x % n_q_heads;
  const int b = blockIdx.x / n_q_heads;
  const int g = hq / group, h = hq % group;
  const int sg = tid >> 5, dq = tid & 31;
  const float* base = partials +
                      static_cast<int64_t>(b * n_kv_heads + g) * n_splits * (kCols * kPart) +
                      h * kPart;
  float M = -INFINITY, L = 0.f;
  f32x4_t O = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int s0 = sg; s0 < n_splits; s0 += 8 * kUnroll) {
    float mv[kUnroll], lv[kUnroll];
    f32x4_t ov[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int s = s0 + 8 * u;
      const int sc = s < n_splits ? s : s0;
      const float* p = base + static_cast<int64_t>(sc) * (kCols * kPart);
      mv[u] = s < n_splits ? p[0] : -INFINITY;
      lv[u] = p[1];
      ov[u] = *reinterpret_cast<const f32x4_t*>(p + 2 + 4 * dq);
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) Mn = fmaxf(Mn, mv[u]);
    const float cM = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    L *= cM;
    O *= cM;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const bool live = mv[u] != -INFINITY;
      const float c = live ? __builtin_amdgcn_exp2f(mv[u] - Mn) : 0.f;
      L += live ? c * lv[u] : 0.f;
      O[0] += live ? c * ov[u][0] : 0.f;
      O[1] += live ? c * ov[u][1] : 0.f;
      O[2] += live ? c * ov[u][2] : 0.f;
      O[3] += live ? c * ov[u][3] : 0.f;
    }
    M = Mn;
  }
  if (dq == 0) red_m[sg] = M;
  lds_barrier();
  float Mt = red_m[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) Mt = fmaxf(Mt, red_m[j]);
  const float c = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mt);
  *reinterpret_cast<f32x4_t*>(&red_o[sg][4 * dq]) = c * O;
  if (dq == 0) red_l[sg] = c * L;
  lds_barrier();
  if (tid < 32) {
    f32x4_t o = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      o += *reinterpret_cast<const f32x4_t*>(&red_o[j][4 * tid]);
      l += red_l[j];
    }
    const f32x4_t r = l > 0.f ? o * (1.0f / l) : f32x4_t{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4_t*>(out + (static_cast<int64_t>(b) * n_q_heads + hq) * kDim +
                                4 * tid) = r;
  }
}

}  // namespace

// Split plan: a split holds at most 8 waves x 4 batches x 16 = 512 positions;
// while the grid is small (<= 4 rounds of one workgroup per CU) the split
// count is raised so the grid fills whole rounds, keeping at least one batch
// per wave.
void f16_plan(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len, int* nb,
              int64_t* n_splits, int64_t* split_len) {
  constexpr int64_t kCus = 256;
  constexpr int64_t kMaxLen = 16 * kWaves * kMaxBatches;
  const int64_t t = max_seq_len > 0 ? max_seq_len : 1;
  const int64_t bg = batch * n_kv_heads > 0 ? batch * n_kv_heads : 1;
  int64_t s = (t + kMaxLen - 1) / kMaxLen;
  const int64_t wgs = bg * s;
  if (wgs <= 4 * kCus) {
    const int64_t rounds = (wgs + kCus - 1) / kCus;
    int64_t s_fill = (rounds * kCus) / bg;
    const int64_t s_min_len = (t + 16 * kWaves - 1) / (16 * kWaves);
    if (s_fill > s_min_len) s_fill = s_min_len;
    if (s_fill > s) s = s_fill;
  }
  int64_t len = (t + s - 1) / s;
  len = (len + 15) / 16 * 16;
  s = (t + len - 1) / len;
  *split_len = len;
  *n_splits = s;
  *nb = static_cast<int>((len / 16 + kWaves - 1) / kWaves);
}

size_t f16_workspace_bytes(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len) {
  int nb = 0;
  int64_t splits = 0, len = 0;
  f16_plan(batch, n_kv_heads, max_seq_len, &nb, &splits, &len);
  const size_t bytes = static_cast<size_t>(batch) * n_kv_heads * splits * kCols * kPart * 4;
  return bytes > 0 ? (bytes + 255) / 256 * 256 : 256;
}

hipError_t launch_decode_f16(const float* q, const __half* k, const __half* v,
                             const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                             int64_t batch, int64_t n_kv_heads, int64_t group, float scale,
                             float* out, float* partials, hipStream_t stream) {
  int nb = 0;
  int64_t n_splits = 0, split_len = 0;
  f16_plan(batch, n_kv_heads, max_seq_len, &nb, &n_splits, &split_len);
  const dim3 grid(static_cast<unsigned>(batch * n_kv_heads * n_splits)), block(kThreads);
  const float qscale = scale * kLog2e;
#define IQ_LAUNCH_F16(NB_)                                                                      \
  hipLaunchKernelGGL((decode_f16_kernel<NB_>), grid, block, 0, stream, q, k, v, seq_lens,       \
                     partials, out, capacity, static_cast<int>(max_seq_len),                   \
                     static_cast<int>(n_kv_heads), static_cast<int>(group),                    \
                     static_cast<int>(n_splits), static_cast<int>(split_len), qscale)
  switch (nb) {
    case 1: IQ_LAUNCH_F16(1); break;
    case 2: IQ_LAUNCH_F16(2); break;
    case 3: IQ_LAUNCH_F16(3); break;
    default: IQ_LAUNCH_F16(4); break;
  }
#undef IQ_LAUNCH_F16
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_splits == 1) return e;
  hipLaunchKernelGGL(merge_f16_kernel, dim3(static_cast<unsigned>(batch * n_kv_heads * group)),
                     dim3(kMergeThreads), 0, stream, partials, out, static_cast<int>(n_kv_heads),
                     static_cast<int>(group), static_cast<int>(n_splits));
  return hipGetLastError();
}

}  // namespace iq
