// Decode attention on the packed 3-bit cache for groups of 8 query heads per
// KV head (App. A; Table 2 A-D; Sec. 3.4), gfx950, one launch per call.
//
// Work decomposition: one 256-thread workgroup per (sequence b, KV head g,
// split of 64*NB positions); each of its 4 waves owns NB consecutive batches
// of 16 positions.  Every load of the wave (packed keys, packed values and
// both scale arrays for all its batches) is issued before any arithmetic, so
// the whole cache is in flight at once.
//
// The two contractions of a batch are dense 8-head x 128-dim x 16-position
// products and run on the matrix cores (v_mfma_f32_16x16x32_f16):
//
//  QK (Table 2 A): S[t][n] = sum_k Khat[t][k] Qt[k][n], rows t = 16 positions,
//    columns n = 16 = the group's 8 heads twice, k = 32 dims per instruction.
//    The fp32 rotated query is split into fp16 hi + lo parts and both are
//    multiplied into the same accumulator, so the scores carry ~22 bits.
//    A lane (t, gk) supplies 8 dims 32gk+8kb..+7 of position t, i.e. 4
//    consecutive 6-bit fields (2 codes each) of its 12-byte slice of the
//    record; each field indexes a 64-entry LDS table holding the pair of
//    fp16 codebook levels, which is directly the MFMA operand dword.
//  PV (Table 2 C): O[(h, s)][u] = sum_(t, s') P'[(h, s)][(t, s')] Vhat[(t, s')][u]
//    with rows (head h, slot s) and columns u = 16 dim pairs per instruction.
//    The operand dword of position t is the decoded field (v_{2F}, v_{2F+1});
//    row (h, s) carries the fp16 weight in half s of its dword and zero in
//    the other half, so row (h, 0) accumulates dim 2F and row (h, 1) dim
//    2F+1.  Lane group gk of the PV operands holds positions 4gk..4gk+3,
//    exactly the rows the QK accumulator left in that lane group, so the
//    weights never leave their lanes.
//
// Softmax (Table 2 B) is two-phase per wave: all QK products of the wave's
// positions first (scores kept in registers), one max per head, then the
// weights and the PV products; scores are in log2 units (the rotated query
// is pre-scaled by scale * log2 e) so exp2 is a single instruction.  The
// value scales s^V are divided by the wave's largest value scale before the
// fp16 conversion, keeping the weights in [0, 1].
//
// Merge: the 4 waves merge in LDS; workgroups of one (b, g) then merge
// through the workspace, the last workgroup to finish (an atomic ticket per
// (b, g), reset by that workgroup) merges all splits, divides by the sum and
// applies the single inverse rotation R^T = H_128 M^T (Table 2 D).
#include <hip/hip_runtime.h>
#include <math.h>

#include "iq_device.h"
#include "iq_internal.h"

namespace iq {
namespace {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_a4_t __attribute__((ext_vector_type(2), aligned(4)));

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kHeads = 8;                 // query heads per KV head
constexpr int kPart = 2 + kDim;           // m, l, o[128] per head
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kInvSqrtDim = 0.08838834764831845f;

__device__ __forceinline__ f32x4_t mfma(u32x4_t a, u32x4_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a),
                                                __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
}

// 6-bit field F (codes of dims 2F', 2F'+1) of a 96-bit slice w0:w1:w2 at bit 6F.
template <int F>
__device__ __forceinline__ uint32_t slice_field(uint32_t w0, uint32_t w1, uint32_t w2) {
  constexpr int bit = 6 * F, word = bit / 32, off = bit % 32;
  const uint32_t lo = word == 0 ? w0 : (word == 1 ? w1 : w2);
  if constexpr (off <= 26) {
    return __builtin_amdgcn_ubfe(lo, off, 6);
  } else {
    const uint32_t hi = word == 0 ? w1 : w2;
    return __builtin_amdgcn_alignbit(hi, lo, off) & 63u;
  }
}

// Workgroup barrier that orders LDS only.  __syncthreads() also fences
// global memory, which would make every wave wait for all of its outstanding
// cache loads at the first barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// Inverse rotation of 8 heads in LDS (buf[h][128], already divided by l):
// per block z = M^T o_blk, then the normalized WHT, written to dst.
__device__ void inverse_rotate_store(float* buf, const float* qparam, float* __restrict__ dst,
                                     int tid) {
  // 8 heads x 32 blocks = 256 (head, block) tasks, one per thread; qparam
  // holds the parameters of block tid % 32
  {
    const int h = tid >> 5, blk = tid & 31;
    float m[4][4];
    so4_matrix(qparam, m);
    float* o = buf + h * kDim + 4 * blk;
    const float o0 = o[0], o1 = o[1], o2 = o[2], o3 = o[3];
    float z[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) z[r] = m[0][r] * o0 + m[1][r] * o1 + m[2][r] * o2 + m[3][r] * o3;
    o[0] = z[0];
    o[1] = z[1];
    o[2] = z[2];
    o[3] = z[3];
  }
  lds_barrier();
  for (int st = 1; st < kDim; st <<= 1) {
    // 8 heads x 64 butterflies per stage, 2 per thread
#pragma unroll
    for (int rep = 0; rep < 2; ++rep) {
      const int e = tid + rep * kThreads;          // 0..511
      const int h = e >> 6, p = e & 63;
      const int i = ((p & ~(st - 1)) << 1) | (p & (st - 1));   // lower index of the pair
      float* v = buf + h * kDim;
      const float a = v[i], b = v[i + st];
      v[i] = a + b;
      v[i + st] = a - b;
    }
    lds_barrier();
  }
  for (int e = tid; e < kHeads * kDim; e += kThreads) dst[e] = buf[e] * kInvSqrtDim;
}

template <int NB>
__global__ __launch_bounds__(kThreads) void decode_g8_kernel(
    const float* __restrict__ q, const uint8_t* __restrict__ k_codes,
    const float* __restrict__ k_norms, const uint8_t* __restrict__ v_codes,
    const float* __restrict__ v_norms, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ quats, float* __restrict__ partials, float* __restrict__ out,
    int64_t capacity, int64_t max_seq_len, int n_kv_heads, int n_splits, int split_len,
    float qscale, Codebook cb) {
  __shared__ uint32_t lut[64];
  __shared__ float qbuf[kHeads * kDim];
  __shared__ float wave_o[kWaves][kHeads * kDim];
  __shared__ float wave_ml[kWaves][2][kHeads];
  __shared__ float qmax_s[kWaves];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;

  const int split = blockIdx.x % n_splits;
  const int bg = blockIdx.x / n_splits;
  const int g = bg % n_kv_heads;
  const int b = bg / n_kv_heads;
  const int n_q_heads = n_kv_heads * kHeads;

  int64_t seq = seq_lens[b];
  if (seq > max_seq_len) seq = max_seq_len;
  if (seq < 0) seq = 0;
  const int used = static_cast<int>((seq + split_len - 1) / split_len);
  float* out_bg = out + (static_cast<int64_t>(b) * n_q_heads + static_cast<int64_t>(g) * kHeads) * kDim;
  if (split >= used) {
    if (seq == 0 && split == 0)
      for (int e = tid; e < kHeads * kDim; e += kThreads) out_bg[e] = 0.f;
    return;
  }
  const int64_t start = static_cast<int64_t>(split) * split_len;
  const int64_t end = seq < start + split_len ? seq : start + split_len;
  const int64_t wbase = start + static_cast<int64_t>(wave) * NB * 16;   // first position of the wave
  const int64_t last = end - 1;                                           // last position of the split
  const int64_t last4 = last & ~static_cast<int64_t>(3);
  const int64_t row = (static_cast<int64_t>(b) * n_kv_heads + g) * capacity;

  // ---- issue every load of the wave -------------------------------------
  // the group's 8 query heads first (one float4 per thread), then the cache
  const f32x4_t qv = *reinterpret_cast<const f32x4_t*>(
      q + (static_cast<int64_t>(b) * n_q_heads + static_cast<int64_t>(g) * kHeads) * kDim +
      4 * tid);
  // this thread's SO(4) block parameters (block tid % 32 of KV head g)
  const float* quats_g = quats + static_cast<int64_t>(g) * kQuatFloats;
  float qparam[8];
  {
    const f32x4_t p0 = *reinterpret_cast<const f32x4_t*>(quats_g + 8 * (tid & 31));
    const f32x4_t p1 = *reinterpret_cast<const f32x4_t*>(quats_g + 8 * (tid & 31) + 4);
    qparam[0] = p0[0]; qparam[1] = p0[1]; qparam[2] = p0[2]; qparam[3] = p0[3];
    qparam[4] = p1[0]; qparam[5] = p1[1]; qparam[6] = p1[2]; qparam[7] = p1[3];
  }
  // keys: lane (t = col, gk = grp) takes dwords 3gk..3gk+2 of position t
  uint32_t kw[NB][3];
  // values: lane (u = col, grp) takes 8 bytes covering bytes 3u..3u+2 of
  // positions 4 grp + r, r = 0..3
  uint32_t vw[NB][4][2];
  f32x4_t ks[NB], vs[NB];
  const int vdw = (3 * col) / 4 < 10 ? (3 * col) / 4 : 10;
  const uint32_t vshift = static_cast<uint32_t>(8 * (3 * col - 4 * vdw));   // 0..40
  // keys and key scales of every batch first: the score phase can start on
  // the first batch while the values are still arriving
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int64_t base = wbase + 16 * i;
    int64_t t = base + col;
    t = t < last ? t : last;
    const uint32_t* p = reinterpret_cast<const uint32_t*>(k_codes + (row + t) * kRecordBytes) + 3 * grp;
    kw[i][0] = p[0];
    kw[i][1] = p[1];
    kw[i][2] = p[2];
    // one 16-byte load of scales; the 4-aligned group holding the last valid
    // position is the furthest one read (capacity % 4 == 0); positions past
    // the end are masked below
    int64_t t4 = base + 4 * grp;
    t4 = t4 < last4 ? t4 : last4;
    ks[i] = *reinterpret_cast<const f32x4_t*>(k_norms + row + t4);
  }
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int64_t base = wbase + 16 * i;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int64_t t = base + 4 * grp + r;
      t = t < last ? t : last;
      const u32x2_a4_t d =
          *reinterpret_cast<const u32x2_a4_t*>(v_codes + (row + t) * kRecordBytes + 4 * vdw);
      vw[i][r][0] = d[0];
      vw[i][r][1] = d[1];
    }
    int64_t t4 = base + 4 * grp;
    t4 = t4 < last4 ? t4 : last4;
    vs[i] = *reinterpret_cast<const f32x4_t*>(v_norms + row + t4);
  }

  // ---- while the loads fly: LUT and the rotated query --------------------
  if (tid < 64) {
    const uint32_t lo = __builtin_bit_cast(uint16_t, static_cast<_Float16>(cb.level[tid & 7]));
    const uint32_t hi = __builtin_bit_cast(uint16_t, static_cast<_Float16>(cb.level[tid >> 3]));
    lut[tid] = lo | (hi << 16);
  }
  qbuf[4 * tid] = qv[0];
  qbuf[4 * tid + 1] = qv[1];
  qbuf[4 * tid + 2] = qv[2];
  qbuf[4 * tid + 3] = qv[3];
  lds_barrier();
  // forward rotation q_tilde = diag(M) H q (App. A), scaled by qscale
  for (int st = 1; st < kDim; st <<= 1) {
#pragma unroll
    for (int rep = 0; rep < 2; ++rep) {
      const int e = tid + rep * kThreads;
      const int h = e >> 6, p = e & 63;
      const int i = ((p & ~(st - 1)) << 1) | (p & (st - 1));
      float* v = qbuf + h * kDim;
      const float a = v[i], bb = v[i + st];
      v[i] = a + bb;
      v[i + st] = a - bb;
    }
    lds_barrier();
  }
  {
    const int h = tid >> 5, blk = tid & 31;
    float m[4][4];
    so4_matrix(qparam, m);
    float* z = qbuf + h * kDim + 4 * blk;
    const float s = kInvSqrtDim * qscale;
    const float z0 = z[0] * s, z1 = z[1] * s, z2 = z[2] * s, z3 = z[3] * s;
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) y[r] = m[r][0] * z0 + m[r][1] * z1 + m[r][2] * z2 + m[r][3] * z3;
    z[0] = y[0];
    z[1] = y[1];
    z[2] = y[2];
    z[3] = y[3];
    float am = fmaxf(fmaxf(fabsf(y[0]), fabsf(y[1])), fmaxf(fabsf(y[2]), fabsf(y[3])));
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) am = fmaxf(am, __shfl_xor(am, o));
    if (lane == 0) qmax_s[wave] = am;
  }
  lds_barrier();
  // fp16 operands are kept in the normal range by exact power-of-two
  // scaling: the rotated queries so that the largest entry is below 2^14
  // (hi and lo parts both normal), undone on the scores.
  int qexp = 0;
  {
    const float am = fmaxf(fmaxf(qmax_s[0], qmax_s[1]), fmaxf(qmax_s[2], qmax_s[3]));
    if (am > 0.f) {
      int e = 0;
      frexpf(am, &e);                      // am < 2^e
      qexp = 14 - e;
      qexp = qexp > 100 ? 100 : (qexp < -100 ? -100 : qexp);
    }
  }
  const float qup = ldexpf(1.0f, qexp), qdown = ldexpf(1.0f, -qexp);
  // QK B operands: column col -> head col % 8; MFMA kb, lane group grp ->
  // dims 32 grp + 8 kb + 0..7; hi and lo fp16 parts.
  u32x4_t qhi[4], qlo[4];
  {
    const float* qh = qbuf + (col & 7) * kDim + 32 * grp;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float x0 = qh[8 * kb + 2 * j] * qup, x1 = qh[8 * kb + 2 * j + 1] * qup;
        const _Float16 h0 = static_cast<_Float16>(x0), h1 = static_cast<_Float16>(x1);
        const _Float16 l0 = static_cast<_Float16>(x0 - static_cast<float>(h0));
        const _Float16 l1 = static_cast<_Float16>(x1 - static_cast<float>(h1));
        qhi[kb][j] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h0)) |
                     (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h1)) << 16);
        qlo[kb][j] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l0)) |
                     (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l1)) << 16);
      }
    }
  }

  const int64_t nvalid = end - wbase;   // valid positions of this wave (may be <= 0)
  float m_run = -INFINITY, l_run = 0.f, vmax = 0.f;
  f32x4_t o_acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) o_acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (nvalid > 0) {
    // ---- phase 1: scores ---------------------------------------------------
    f32x4_t sc[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const uint32_t w0 = kw[i][0], w1 = kw[i][1], w2 = kw[i][2];
      u32x4_t a[4];
      a[0] = u32x4_t{lut[slice_field<0>(w0, w1, w2)], lut[slice_field<1>(w0, w1, w2)],
                     lut[slice_field<2>(w0, w1, w2)], lut[slice_field<3>(w0, w1, w2)]};
      a[1] = u32x4_t{lut[slice_field<4>(w0, w1, w2)], lut[slice_field<5>(w0, w1, w2)],
                     lut[slice_field<6>(w0, w1, w2)], lut[slice_field<7>(w0, w1, w2)]};
      a[2] = u32x4_t{lut[slice_field<8>(w0, w1, w2)], lut[slice_field<9>(w0, w1, w2)],
                     lut[slice_field<10>(w0, w1, w2)], lut[slice_field<11>(w0, w1, w2)]};
      a[3] = u32x4_t{lut[slice_field<12>(w0, w1, w2)], lut[slice_field<13>(w0, w1, w2)],
                     lut[slice_field<14>(w0, w1, w2)], lut[slice_field<15>(w0, w1, w2)]};
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        acc = mfma(a[kb], qhi[kb], acc);
        acc = mfma(a[kb], qlo[kb], acc);
      }
      // lane (col, grp) now holds positions 16 i + 4 grp + r of head col % 8
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t p = 16 * i + 4 * grp + r;
        float s = acc[r] * (ks[i][r] * qdown);
        if (p >= nvalid) s = -INFINITY;
        sc[i][r] = s;
        m_run = fmaxf(m_run, s);
        if (p < nvalid) vmax = fmaxf(vmax, vs[i][r]);
      }
    }
    m_run = wave_max(m_run);
    vmax = wave_max(vmax);
    // weights scaled by 2^15 / vmax: in [0, 2^15], fp16-normal down to
    // ~2e-9 of the largest weight; split into fp16 hi + lo parts
    const float vinv = vmax > 0.f ? 32768.0f / vmax : 0.f;

    // ---- phase 2: weights and values ---------------------------------------
    const uint32_t slot_shift = (col >= 8) ? 16u : 0u;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      u32x4_t pw_hi, pw_lo;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = __builtin_amdgcn_exp2f(sc[i][r] - m_run);
        l_run += e;
        const float sv = (16 * i + 4 * grp + r < nvalid) ? vs[i][r] : 0.f;
        const float pf = e * (sv * vinv);
        const _Float16 ph = static_cast<_Float16>(pf);
        const _Float16 pl = static_cast<_Float16>(pf - static_cast<float>(ph));
        pw_hi[r] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, ph)) << slot_shift;
        pw_lo[r] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, pl)) << slot_shift;
      }
      u32x4_t vb[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t lo = col == 15 ? vw[i][r][1] : vw[i][r][0];
        const uint32_t win = __builtin_amdgcn_alignbit(vw[i][r][1], lo, vshift & 31u);
        vb[0][r] = lut[win & 63u];
        vb[1][r] = lut[__builtin_amdgcn_ubfe(win, 6, 6)];
        vb[2][r] = lut[__builtin_amdgcn_ubfe(win, 12, 6)];
        vb[3][r] = lut[__builtin_amdgcn_ubfe(win, 18, 6)];
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        o_acc[nb] = mfma(pw_hi, vb[nb], o_acc[nb]);
        o_acc[nb] = mfma(pw_lo, vb[nb], o_acc[nb]);
      }
    }
    l_run = wave_sum(l_run);
  }

  // ---- merge the 4 waves in LDS ---------------------------------------------
  // lane (u = col, grp) holds rows 4 grp + r = (head (4 grp + r) % 8, slot
  // grp / 2) of MFMA nb, i.e. dim 2 (4 u + nb) + slot.
#pragma unroll
  for (int nb = 0; nb < 4; ++nb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = (4 * grp + r) & 7, s = grp >> 1;
      wave_o[wave][h * kDim + 8 * col + 2 * nb + s] = o_acc[nb][r] * (vmax * (1.0f / 32768.0f));
    }
  if (lane < kHeads) {
    wave_ml[wave][0][lane] = m_run;     // lanes 0..7 hold heads 0..7
    wave_ml[wave][1][lane] = l_run;
  }
  lds_barrier();

  // thread -> (head h = tid / 32, dims 4 (tid % 32) .. +3)
  const int mh = tid >> 5, md = (tid & 31) * 4;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wave_ml[w][0][mh]);
  float L = 0.f, O0 = 0.f, O1 = 0.f, O2 = 0.f, O3 = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const float mw = wave_ml[w][0][mh];
    const float c = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - M);
    L += c * wave_ml[w][1][mh];
    const float* ow = wave_o[w] + mh * kDim + md;
    O0 += c * ow[0];
    O1 += c * ow[1];
    O2 += c * ow[2];
    O3 += c * ow[3];
  }

  if (used == 1) {
    const float il = 1.0f / L;
    float* ob = qbuf + mh * kDim + md;
    ob[0] = O0 * il;
    ob[1] = O1 * il;
    ob[2] = O2 * il;
    ob[3] = O3 * il;
    lds_barrier();
    inverse_rotate_store(qbuf, qparam, out_bg, tid);
    return;
  }

  // ---- partial result of this split ------------------------------------------
  float* pp = partials + (static_cast<int64_t>(bg) * n_splits + split) * (kHeads * kPart) +
              mh * kPart;
  if ((tid & 31) == 0) {
    pp[0] = M;
    pp[1] = L;
  }
  *reinterpret_cast<f32x4_t*>(pp + 2 + md) = f32x4_t{O0, O1, O2, O3};
}

// Merge of the split partials of one (sequence b, query head h): one
// 256-thread workgroup; thread (sg, dq) takes splits sg, sg + 8, ... and dims
// 4 dq .. 4 dq + 3, with up to 16 splits' loads in flight per thread.  Then
// o = sum_s c_s O_s / sum_s c_s l_s with c_s = 2^(m_s - max m), and the single
// inverse rotation.
__global__ __launch_bounds__(kThreads) void merge_g8_kernel(
    const float* __restrict__ partials, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ quats, float* __restrict__ out, int64_t max_seq_len,
    int n_kv_heads, int n_splits, int split_len) {
  constexpr int kUnroll = 16;
  __shared__ float red_o[8][kDim];
  __shared__ float red_m[8], red_l[8];
  __shared__ float obuf[kDim];
  const int tid = threadIdx.x;
  const int n_q_heads = n_kv_heads * kHeads;
  const int h = blockIdx.x % n_q_heads;
  const int b = blockIdx.x / n_q_heads;
  const int g = h / kHeads, hh = h % kHeads;
  int64_t seq = seq_lens[b];
  if (seq > max_seq_len) seq = max_seq_len;
  if (seq < 0) seq = 0;
  const int used = static_cast<int>((seq + split_len - 1) / split_len);
  if (used <= 1) return;   // empty sequence or a single split: written by the split kernel
  const int sg = tid >> 5, dq = tid & 31;
  const float* base = partials + static_cast<int64_t>(b * n_kv_heads + g) * n_splits * (kHeads * kPart) +
                      hh * kPart;
  // block parameters for the inverse rotation (threads 0..31: block tid)
  float qparam[8];
  {
    const float* qg = quats + static_cast<int64_t>(g) * kQuatFloats + 8 * dq;
    const f32x4_t p0 = *reinterpret_cast<const f32x4_t*>(qg);
    const f32x4_t p1 = *reinterpret_cast<const f32x4_t*>(qg + 4);
    qparam[0] = p0[0]; qparam[1] = p0[1]; qparam[2] = p0[2]; qparam[3] = p0[3];
    qparam[4] = p1[0]; qparam[5] = p1[1]; qparam[6] = p1[2]; qparam[7] = p1[3];
  }
  float M = -INFINITY, L = 0.f;
  f32x4_t O = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int s0 = sg; s0 < used; s0 += 8 * kUnroll) {
    float mv[kUnroll], lv[kUnroll];
    f32x4_t ov[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int s = s0 + 8 * u;
      const int sc = s < used ? s : s0;
      const float* p = base + static_cast<int64_t>(sc) * (kHeads * kPart);
      mv[u] = s < used ? p[0] : -INFINITY;
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
      const float c = (mv[u] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mv[u] - Mn);
      L += c * lv[u];
      O += c * ov[u];
    }
    M = Mn;
  }
  // combine the 8 split groups
  if (dq == 0) red_m[sg] = M;
  lds_barrier();
  float Mt = red_m[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) Mt = fmaxf(Mt, red_m[j]);
  const float c = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mt);
  red_o[sg][4 * dq] = c * O[0];
  red_o[sg][4 * dq + 1] = c * O[1];
  red_o[sg][4 * dq + 2] = c * O[2];
  red_o[sg][4 * dq + 3] = c * O[3];
  if (dq == 0) red_l[sg] = c * L;
  lds_barrier();
  if (tid < kDim) {
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      o += red_o[j][tid];
      l += red_l[j];
    }
    obuf[tid] = o / l;
  }
  lds_barrier();
  // inverse rotation: z = M^T o per block, then the normalized WHT
  if (tid < 32) {
    float m[4][4];
    so4_matrix(qparam, m);
    float* ob = obuf + 4 * tid;
    const float o0 = ob[0], o1 = ob[1], o2 = ob[2], o3 = ob[3];
    float z[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) z[r] = m[0][r] * o0 + m[1][r] * o1 + m[2][r] * o2 + m[3][r] * o3;
    ob[0] = z[0];
    ob[1] = z[1];
    ob[2] = z[2];
    ob[3] = z[3];
  }
  lds_barrier();
  for (int st = 1; st < kDim; st <<= 1) {
    if (tid < 64) {
      const int i = ((tid & ~(st - 1)) << 1) | (tid & (st - 1));
      const float a = obuf[i], bb = obuf[i + st];
      obuf[i] = a + bb;
      obuf[i + st] = a - bb;
    }
    lds_barrier();
  }
  if (tid < kDim)
    out[(static_cast<int64_t>(b) * n_q_heads + h) * kDim + tid] = obuf[tid] * kInvSqrtDim;
}

}  // namespace

// Split plan of the group-8 path: splits per (sequence, KV head) and their
// length.  At least ceil(T / 512) splits (a wave handles at most 8 batches of
// 16 positions); while the grid is small (<= 4 rounds of 256 workgroups) the
// split count is raised so that the grid fills whole rounds of the 256 CUs.
void g8_plan(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len, int* nb,
             int64_t* n_splits, int64_t* split_len) {
  const int64_t t = max_seq_len > 0 ? max_seq_len : 1;
  const int64_t bg = batch * n_kv_heads > 0 ? batch * n_kv_heads : 1;
  int64_t s = (t + 511) / 512;
  const int64_t wgs = bg * s;
  if (wgs <= 4 * 256) {
    const int64_t rounds = (wgs + 255) / 256;
    const int64_t s_fill = (rounds * 256) / bg;
    if (s_fill > s) s = s_fill;
  }
  if (s > t) s = t;
  int64_t len = (t + s - 1) / s;
  len = (len + 15) / 16 * 16;
  s = (t + len - 1) / len;
  *split_len = len;
  *n_splits = s;
  *nb = static_cast<int>((len + kWaves * 16 - 1) / (kWaves * 16));
}

hipError_t launch_decode_g8(int nb, int64_t n_splits, int64_t split_len, const float* q,
                            const uint8_t* k_codes,
                            const float* k_norms, const uint8_t* v_codes, const float* v_norms,
                            const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                            const float* quats, int64_t batch, int64_t n_kv_heads, float scale,
                            float* out, float* partials, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(batch * n_kv_heads * n_splits)), block(kThreads);
  const float qscale = scale * kLog2e;
  const Codebook& cb = codebook();
#define IQ_LAUNCH_G8(NB_)                                                                        \
  hipLaunchKernelGGL(decode_g8_kernel<NB_>, grid, block, 0, stream, q, k_codes, k_norms,       \
                     v_codes, v_norms, seq_lens, quats, partials, out, capacity, max_seq_len,  \
                     static_cast<int>(n_kv_heads), static_cast<int>(n_splits),                \
                     static_cast<int>(split_len), qscale, cb)
  switch (nb) {
    case 1: IQ_LAUNCH_G8(1); break;
    case 2: IQ_LAUNCH_G8(2); break;
    case 3: IQ_LAUNCH_G8(3); break;
    case 4: IQ_LAUNCH_G8(4); break;
    case 5: IQ_LAUNCH_G8(5); break;
    case 6: IQ_LAUNCH_G8(6); break;
    case 7: IQ_LAUNCH_G8(7); break;
    default: IQ_LAUNCH_G8(8); break;
  }
#undef IQ_LAUNCH_G8
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // splits of every (sequence, query head) merged by a second launch
  if (n_splits > 1) {
    hipLaunchKernelGGL(merge_g8_kernel, dim3(static_cast<unsigned>(batch * n_kv_heads * kHeads)),
                       dim3(kThreads), 0, stream, partials, seq_lens, quats, out, max_seq_len,
                       static_cast<int>(n_kv_heads), static_cast<int>(n_splits),
                       static_cast<int>(split_len));
    e = hipGetLastError();
  }
  return e;
}

}  // namespace iq
