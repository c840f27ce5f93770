// Multi-token decode on the packed cache for groups of 8 query heads per KV
// head (App. A applied to each of 2-4 query tokens; Table 2 A-D), gfx950:
// the verification step of speculative decoding, the tokens causal among
// themselves.  Same split grid, loads, record decoding and merge as the
// single-token kernel (iq_decode_g8.hip); see the kernel comment.  Records
// of 2, 3 or 4 bits (Algorithm 1 with C_b), and a fused step that appends
// the kT new tokens itself.
#include <hip/hip_runtime.h>
#include <math.h>

#include "iq_g8_device.h"

namespace iq {
namespace {

// Multi-token decode (speculative verification): kT query tokens per
// sequence over the same cache.  Every batch of keys and values is decoded
// once and feeds kT sets of matrix instructions (the QK B operand of token t
// is read from LDS per batch).  The softmax is two-phase as in
// decode_g8_kernel: all scores of every token first (kept in registers), one
// max per token and head, then the weights and values.  Partials per (split,
// token, head); the merge kernel takes the token axis.
//
// Without kAppend the caller has already compressed the kT new tokens into
// the last kT of the seq_lens[b] positions, and token t attends the
// positions before seq_lens[b] - kT + 1 + t.
//
// kAppend, the fused step: one more workgroup per (b, g), split index
// n_splits, compresses the kT new keys and values (Alg. 1) and writes their
// records at positions seq_lens[b] .. seq_lens[b] + kT - 1, then publishes,
// per token t, the partial (m, l, O) over the new positions u <= t (causal
// among the new tokens; a new position at or past max_seq_len is not
// attended).  The attention workgroups serve the cached positions before
// seq_lens[b], which every token attends.  When the kT records do not all
// fit the capacity nothing is written, the capacity flag is raised, the new
// positions are not attended, and the partial's l entry carries -1, so that
// the merge leaves the length as it is; otherwise the merge advances it by
// kT.  No attention workgroup reads the records being written.
//
// kPaged: the cache is a page pool (PageTable), as in decode_g8_kernel
// (3-bit records, decode only).  kBits: the records' code width.
template <int NB, bool kWide, int kT, bool kPaged, int kBits, bool kAppend>
__global__ __launch_bounds__(kThreads) void decode_g8_multi_kernel(
    const float* __restrict__ q, uint8_t* __restrict__ k_codes, float* __restrict__ k_norms,
    uint8_t* __restrict__ v_codes, float* __restrict__ v_norms,
    const int32_t* __restrict__ seq_lens, const float* __restrict__ quats,
    float* __restrict__ partials, float* __restrict__ out, int64_t capacity, int max_seq_len,
    int n_kv_heads, int n_splits, int split_len, float qscale, CodebookB<kBits> cb,
    PageTable pages, const void* __restrict__ k_new, const void* __restrict__ v_new,
    int new_f16, int32_t* __restrict__ status) {
  static_assert(kT >= 2 && kT <= 4, "2 to 4 tokens");
  static_assert(!kPaged || (kBits == 3 && !kAppend), "paged pools: 3-bit decode only");
  constexpr int kRB = record_bytes<kBits>();
  constexpr int kLut = 1 << (2 * kBits);
  constexpr int kNew = kAppend ? 2 * kT : 1;
  struct Smem {
    uint32_t lut[kLut];   // fp16 pair table (address 0: a lookup address is field * 4)
    uint32_t qop[kT][2][kHeads][kQRowWords];
    int qexp[kT][kHeads];
    float wave_ml[kWaves][2][kHeads];
    uint32_t new_rec[kNew][4 * kBits];   // append: record of token w / 2's key (w even) or value
    float new_scale[kNew];
    union {
      WaveStageB<kBits> stage[kWaves];
      f32x4_t wave_o[kWaves][4][64];
    };
  };
  __shared__ __attribute__((aligned(16))) Smem sm;
  uint32_t* lut = sm.lut;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int split = blockIdx.x;
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int bg = b * n_kv_heads + g;
  const int n_q_heads = n_kv_heads * kHeads;
  const int n_parts = kAppend ? n_splits + 1 : n_splits;

  // queries of the kT tokens (thread (head qh, block qblk) for tid < 256)
  const int qh = (tid >> 5) & 7, qblk = tid & 31;
  f32x4_t qv[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t)
    qv[t] = *reinterpret_cast<const f32x4_t*>(
        q + ((static_cast<int64_t>(b) * kT + t) * n_q_heads + static_cast<int64_t>(g) * kHeads +
             qh) * kDim + 4 * qblk);
  const f32x4_t* qpar = reinterpret_cast<const f32x4_t*>(
      quats + static_cast<int64_t>(g) * kQuatFloats + 8 * qblk);
  const f32x4_t ql = qpar[0], qr = qpar[1];
  float* part_bg = partials + static_cast<int64_t>(bg) * n_parts * kT * (kHeads * kPart);
  const int64_t row = kPaged ? 0 : static_cast<int64_t>(bg) * capacity;

  if constexpr (kAppend) if (split == n_splits) {
    // ---- the append workgroup ------------------------------------------------
    const int seq0 = seq_lens[b];
    const bool fits = seq0 >= 0 && seq0 <= capacity - kT;
    if (!fits && status != nullptr && g == 0 && tid == 0)
      atomicOr(status, static_cast<int32_t>(IQ_ERR_CAPACITY));
    // waves 0 .. 2 kT - 1: wave w compresses token w / 2's key (w even) or
    // value (w odd); lane l holds dims 2l, 2l + 1 and the parameters of
    // SO(4) block l / 2
    if (wave < 2 * kT) {
      const int t = wave >> 1, which = wave & 1;
      const void* src = which ? v_new : k_new;
      const int64_t off = ((static_cast<int64_t>(b) * kT + t) * n_kv_heads + g) * kDim;
      float x0, x1;
      if (new_f16) {
        const uint32_t w = reinterpret_cast<const uint32_t*>(static_cast<const __half*>(src) +
                                                             off)[lane];
        x0 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w)));
        x1 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
      } else {
        const f32x2_t w =
            reinterpret_cast<const f32x2_t*>(static_cast<const float*>(src) + off)[lane];
        x0 = w[0];
        x1 = w[1];
      }
      const f32x4_t* qs = reinterpret_cast<const f32x4_t*>(
          quats + static_cast<int64_t>(g) * kQuatFloats + 8 * (lane >> 1));
      const f32x4_t p0 = qs[0], p1 = qs[1];
      const float qp[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
      const WaveCode wc = compress_vector_wave<kBits>(x0, x1, qp, cb, lane);
      if (lane < 4 * kBits) sm.new_rec[wave][lane] = wc.word;
      if (lane == 0) sm.new_scale[wave] = wc.scale;
      if (fits) {
        const int64_t rec = row + seq0 + t;
        uint8_t* codes = which ? v_codes : k_codes;
        float* norms = which ? v_norms : k_norms;
        if (lane < 4 * kBits) reinterpret_cast<uint32_t*>(codes + rec * kRB)[lane] = wc.word;
        if (lane == 0) norms[rec] = wc.scale;
      }
    }
    if (tid < kLut) {
      constexpr int kMask = (1 << kBits) - 1;
      const uint32_t lo =
          __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid & kMask)));
      const uint32_t hi =
          __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid >> kBits)));
      lut[tid] = lo | (hi << 16);
    }
    f32x4_t y[kT];
#pragma unroll
    for (int t = 0; t < kT; ++t)
      y[t] = tid < kRotThreads ? rotate_forward(qv[t], ql, qr, qblk, kInvSqrtDim * qscale)
                               : f32x4_t{0.f, 0.f, 0.f, 0.f};
    lds_barrier();   // new_rec, new_scale, lut
    if (tid >= kRotThreads) return;
    // scores of the new keys u <= t for head qh, in log2 units (y carries
    // the score scale): s^K_u (q_tilde_t . C[code_u]) over this thread's dims
    // 4 qblk .. +3, summed over the head's 32 lanes
    const int md = 4 * qblk;
    float sc[kT][kT];
    f32x4_t v4[kT];
#pragma unroll
    for (int u = 0; u < kT; ++u) {
      const f32x4_t k4 = decode_record_dims<kBits>(sm.new_rec[2 * u], lut, md);
      v4[u] = sm.new_scale[2 * u + 1] * decode_record_dims<kBits>(sm.new_rec[2 * u + 1], lut, md);
#pragma unroll
      for (int t = u; t < kT; ++t) {
        float dot = y[t][0] * k4[0] + y[t][1] * k4[1] + y[t][2] * k4[2] + y[t][3] * k4[3];
        dot += xor_lane<1>(dot);
        dot += xor_lane<2>(dot);
        dot += xor_lane<4>(dot);
        dot += xor_lane<8>(dot);
        dot += xor_lane<16>(dot);
        sc[t][u] = dot * sm.new_scale[2 * u];
      }
    }
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      float m = -INFINITY;
#pragma unroll
      for (int u = 0; u <= t; ++u)
        if (fits && seq0 + u < max_seq_len) m = fmaxf(m, sc[t][u]);
      float l = 0.f;
      f32x4_t o = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u <= t; ++u) {
        if (fits && seq0 + u < max_seq_len) {
          const float c = __builtin_amdgcn_exp2f(sc[t][u] - m);
          l += c;
          o += c * v4[u];
        }
      }
      float* pp = part_bg + (static_cast<int64_t>(n_splits) * kT + t) * (kHeads * kPart) +
                  qh * kPart;
      if (qblk == 0) {
        pp[0] = m;
        // > 0: the records were written (the merge then advances the length)
        pp[1] = !fits ? -1.0f : (m == -INFINITY ? 1.0f : l);
      }
      *reinterpret_cast<f32x4_t*>(pp + 2 + md) = o;
    }
    return;
  }

  const uint8_t* kc = k_codes + row * kRB;
  const uint8_t* vc = v_codes + row * kRB;

  // this wave's run of batches (as in decode_g8_kernel)
  const int start = split * split_len;
  const int nbat = split_len >> 4;
  const int nb_base = nbat / kWaves, nb_rem = nbat % kWaves;
  const int nb_w = nb_base + (wave < nb_rem ? 1 : 0);
  const int wbase = start + 16 * (wave * nb_base + (wave < nb_rem ? wave : nb_rem));
  int seq0 = 0;
  int lim = start + split_len < max_seq_len ? start + split_len : max_seq_len;
  auto last_batch = [&](int l) {
    int c = (l > 0 ? l - 1 : 0) & ~15;
    c = c < wbase + 16 * (nb_w - 1) ? c : wbase + 16 * (nb_w - 1);
    return c > 0 ? c : 0;
  };
  int clamp16 = last_batch(lim);
  if constexpr (kWide) {
    seq0 = seq_lens[b];
    const int seq_w = seq0 < 0 ? 0 : (seq0 > max_seq_len ? max_seq_len : seq0);
    if (start >= seq_w) {
      // nothing to attend for any token
      if (n_parts > 1) {
        if (tid < kT * kHeads)
          part_bg[(static_cast<int64_t>(split) * kT + tid / kHeads) * (kHeads * kPart) +
                  (tid % kHeads) * kPart] = -INFINITY;
      } else {
        for (int e = tid; e < kT * kHeads * kDim; e += kThreads) {
          const int t = e / (kHeads * kDim), r = e % (kHeads * kDim);
          out[((static_cast<int64_t>(b) * kT + t) * n_q_heads +
               static_cast<int64_t>(g) * kHeads) * kDim + r] = 0.f;
        }
      }
      return;
    }
    lim = lim < seq_w ? lim : seq_w;
    clamp16 = last_batch(lim);
  }
  const float* kn = k_norms + row;
  const float* vn = v_norms + row;
  // paged: each batch's record delta from its page-table entry, the NB
  // entries read together and an invalid one replaced by page 0
  int64_t dlt[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) dlt[i] = 0;
  if constexpr (kPaged) {
    const int32_t* trow = pages.tables + static_cast<int64_t>(b) * pages.max_pages;
    int32_t pg[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int t = wbase + 16 * i < clamp16 ? wbase + 16 * i : clamp16;
      pg[i] = trow[t >> pages.page_shift];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int t = wbase + 16 * i < clamp16 ? wbase + 16 * i : clamp16;
      const int64_t page =
          static_cast<uint32_t>(pg[i]) < static_cast<uint32_t>(pages.n_pages) ? pg[i] : 0;
      dlt[i] = ((page * n_kv_heads + g) << pages.page_shift) -
               static_cast<int64_t>((t >> pages.page_shift) << pages.page_shift);
    }
  }
  uint32_t kw[NB][kBits], vw[NB][kBits];
  f32x4_t ksl, vsl;
  load_keys<NB, kPaged, kBits>(kc, kn, vn, dlt, wbase, clamp16, lane, col, grp, kw, ksl, vsl);
  const uint32_t koff = static_cast<uint32_t>(col * kRB + 4 * kBits * grp);
  int tb[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) tb[i] = wbase + 16 * i < clamp16 ? wbase + 16 * i : clamp16;
  // every value batch goes out behind the keys
#pragma unroll
  for (int i = 0; i < NB; ++i)
    load_value_batch<kBits>(kPaged ? vc + dlt[i] * kRB : vc, tb[i], koff, vw[i]);
  // the word of the value window of lane u = col (see value_pairs)
  int vdw;
  uint32_t vsh;
  if constexpr (kBits == 3) {
    vdw = (3 * col) / 4;
    vsh = static_cast<uint32_t>(8 * (3 * col - 4 * vdw));   // 0, 8, 16 or 24
  } else if constexpr (kBits == 4) {
    vdw = col;
    vsh = 0;
  } else {
    vdw = col >> 1;
    vsh = static_cast<uint32_t>(16 * (col & 1));
  }

  if constexpr (!kWide) seq0 = seq_lens[b];
  const int seq = seq0 < 0 ? 0 : (seq0 > max_seq_len ? max_seq_len : seq0);
  // positions of this wave each token attends (may be <= 0): with kAppend
  // every token attends the whole cache (the new positions are the append
  // workgroup's)
  int nv[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    int st = kAppend ? seq : seq - (kT - 1 - t);
    st = st > 0 ? st : 0;
    const int end = st < start + split_len ? st : start + split_len;
    int n = end - wbase;
    nv[t] = n < 16 * nb_w ? n : 16 * nb_w;
  }
  const int nvalid = nv[kT - 1];

  // ---- while the loads fly: LUT and the rotated queries --------------------
  if (tid < kLut) {
    constexpr int kMask = (1 << kBits) - 1;
    const uint32_t lo =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid & kMask)));
    const uint32_t hi =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid >> kBits)));
    lut[tid] = lo | (hi << 16);
  }
  if (tid < kRotThreads) {
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      const f32x4_t y = rotate_forward(qv[t], ql, qr, qblk, kInvSqrtDim * qscale);
      int qexp = 0;
      const float am = group32_max(
          fmaxf(fmaxf(fabsf(y[0]), fabsf(y[1])), fmaxf(fabsf(y[2]), fabsf(y[3]))));
      if (am > 0.f) {
        int e = 0;
        frexpf(am, &e);
        qexp = 14 - e;
        qexp = qexp > 100 ? 100 : (qexp < -100 ? -100 : qexp);
      }
      const float qup = ldexpf(1.0f, qexp);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const float x0 = y[2 * j] * qup, x1 = y[2 * j + 1] * qup;
        const _Float16 h0 = static_cast<_Float16>(x0), h1 = static_cast<_Float16>(x1);
        const _Float16 l0 = static_cast<_Float16>(x0 - static_cast<float>(h0));
        const _Float16 l1 = static_cast<_Float16>(x1 - static_cast<float>(h1));
        sm.qop[t][0][qh][2 * qblk + j] =
            static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h0)) |
            (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h1)) << 16);
        sm.qop[t][1][qh][2 * qblk + j] =
            static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l0)) |
            (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l1)) << 16);
      }
      if (qblk == 0) sm.qexp[t][qh] = qexp;
    }
  }
  lds_barrier();   // lut, qop, qexp
  float qdown[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) qdown[t] = ldexpf(1.0f, -sm.qexp[t][col & 7]);
  // scales to the wave's stage; value scales past the last token's length
  // are 0 and the rest are brought to [0, 2^15] by the wave's largest
  WaveStageB<kBits>& st = sm.stage[wave];
  float vmax;
  {
    f32x4_t v = vsl;
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = (4 * lane + r < nvalid) ? v[r] : 0.f;
    vmax = wave64_max(fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
    const float vinv = vmax > 0.f ? 32768.0f * __builtin_amdgcn_rcpf(vmax) : 0.f;
    st.vs[lane] = v * vinv;
  }
  st.ks[lane] = ksl;
  wave_lds_fence();

  // phase 1 (Table 2 A): every batch's keys decoded once, the scores of all
  // kT tokens kept in registers; one max per token and head afterwards.
  // Lanes col and col ^ 8 hold the same four scores; the lane with col < 8
  // keeps positions r = 0, 1 of its row group and its partner r = 2, 3
  // (rs), so each weight is computed once (see phase 2).
  const bool upper = col >= 8;
  const int rs = upper ? 2 : 0;
  float m_run[kT], l_run[kT];
  f32x2_t sc[kT][NB];
#pragma unroll
  for (int t = 0; t < kT; ++t) m_run[t] = -INFINITY;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (16 * i >= nvalid) break;
    u32x4_t a[4];
    key_pairs<kBits>(lut, kw[i], a);
    const f32x4_t ks = st.ks[4 * i + grp];
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const u32x4_t qb =
            *reinterpret_cast<const u32x4_t*>(&sm.qop[t][col >> 3][col & 7][16 * grp + 4 * kb]);
        acc = mfma(a[kb], qb, acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] += xor_lane<8>(acc[r]);
      const f32x4_t x = acc * ks;
      f32x2_t xs = upper ? f32x2_t{x[2], x[3]} : f32x2_t{x[0], x[1]};
#pragma unroll
      for (int j = 0; j < 2; ++j) xs[j] = (16 * i + 4 * grp + rs + j < nv[t]) ? xs[j] : -INFINITY;
      sc[t][i] = xs;
      m_run[t] = fmaxf(fmaxf(m_run[t], xs[0]), xs[1]);
    }
  }
#pragma unroll
  for (int t = 0; t < kT; ++t) m_run[t] = wave_max(fmaxf(m_run[t], xor_lane<8>(m_run[t])));

  // phase 2 (Table 2 B, C): value records of all batches to the stage behind
  // one fence, then per batch the decoded values feed every token's weights
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (16 * i >= nvalid) break;
#pragma unroll
    for (int j = 0; j < kBits; ++j)
      st.rec[i][col * rec_stride<kBits>() + kBits * grp + j] = vw[i][j];
  }
  wave_lds_fence();
  f32x4_t o_acc[kT][4];
  float mq[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    l_run[t] = 0.f;
    // a token with nothing to attend in this wave keeps m = -inf: its
    // weights are exp2(-inf) = 0
    mq[t] = (m_run[t] == -INFINITY) ? 0.f : -m_run[t] * qdown[t];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) o_acc[t][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  // PV operand dwords from the packed (hi, lo) fp16 parts of this lane's
  // weights and its partner's (one DPP move), as in the single-token kernel:
  // v_perm_b32 puts the hi or lo part in half `upper` of the dword and zero
  // (a copy of a weight part's sign bit, 0) in the other half; the sources
  // (own, partner) for positions r < 2 and (partner, own) for r >= 2 share
  // one selector per part.
  const uint32_t sel_hi = upper ? 0x01000808u : 0x08080504u;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (16 * i >= nvalid) break;
    u32x4_t vb[4];
    value_pairs<kBits>(lut, st.rec[i], grp, vdw, vsh, vb);
    // this lane's two positions (0 past the last token's length)
    const f32x2_t wv =
        *reinterpret_cast<const f32x2_t*>(reinterpret_cast<const float*>(&st.vs[4 * i + grp]) + rs);
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      // p_hi: p with its low 13 mantissa bits cleared (exact in fp16),
      // p_lo = p - p_hi, packed hi in bits 0..15
      uint32_t pk[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[t][i][j], qdown[t], mq[t]));
        l_run[t] += e;
        const float pf = e * wv[j];
        const float ph = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, pf) & 0xFFFFE000u);
        pk[j] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(ph, pf - ph));
      }
      const uint32_t pp0 = static_cast<uint32_t>(
          __builtin_amdgcn_mov_dpp(static_cast<int>(pk[0]), 0x128, 0xF, 0xF, true));
      const uint32_t pp1 = static_cast<uint32_t>(
          __builtin_amdgcn_mov_dpp(static_cast<int>(pk[1]), 0x128, 0xF, 0xF, true));
      uint32_t sel_lo = sel_hi;
      asm volatile("" : "+v"(sel_lo));
      sel_lo |= 0x02020202u;
      const u32x4_t pw_hi = u32x4_t{__builtin_amdgcn_perm(pk[0], pp0, sel_hi),
                                    __builtin_amdgcn_perm(pk[1], pp1, sel_hi),
                                    __builtin_amdgcn_perm(pp0, pk[0], sel_hi),
                                    __builtin_amdgcn_perm(pp1, pk[1], sel_hi)};
      const u32x4_t pw_lo = u32x4_t{__builtin_amdgcn_perm(pk[0], pp0, sel_lo),
                                    __builtin_amdgcn_perm(pk[1], pp1, sel_lo),
                                    __builtin_amdgcn_perm(pp0, pk[0], sel_lo),
                                    __builtin_amdgcn_perm(pp1, pk[1], sel_lo)};
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        o_acc[t][nb] = mfma(pw_hi, vb[nb], o_acc[t][nb]);
        o_acc[t][nb] = mfma(pw_lo, vb[nb], o_acc[t][nb]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    l_run[t] = wave_sum(l_run[t] + xor_lane<8>(l_run[t]));
    m_run[t] *= qdown[t];   // log2 units
  }

  // ---- per token: merge the 8 waves in LDS, then the partial or the row ----
  const float oscale = vmax * (1.0f / 32768.0f);
  const int mh = qh, md = 4 * qblk;
  const int o_r = mh & 3, o_lane = (md >> 3) + 16 * ((mh >> 2) & 1), o_nb = (md & 7) >> 1;
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    lds_barrier();   // the stage (t = 0) or the previous token's wave_o is done
#pragma unroll
    for (int r = 0; r < 4; ++r)
      sm.wave_o[wave][r][lane] =
          f32x4_t{o_acc[t][0][r], o_acc[t][1][r], o_acc[t][2][r], o_acc[t][3][r]} * oscale;
    if (lane < kHeads) {
      sm.wave_ml[wave][0][lane] = m_run[t];
      sm.wave_ml[wave][1][lane] = l_run[t];
    }
    lds_barrier();
    if (tid < kRotThreads) {
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.wave_ml[w][0][mh]);
      float L = 0.f;
      f32x4_t O = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float mw = sm.wave_ml[w][0][mh];
        const float c = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - M);
        L += c * sm.wave_ml[w][1][mh];
        const f32x2_t s0 = *reinterpret_cast<const f32x2_t*>(
            reinterpret_cast<const float*>(&sm.wave_o[w][o_r][o_lane]) + o_nb);
        const f32x2_t s1 = *reinterpret_cast<const f32x2_t*>(
            reinterpret_cast<const float*>(&sm.wave_o[w][o_r][o_lane + 32]) + o_nb);
        O += c * f32x4_t{s0[0], s1[0], s0[1], s1[1]};
      }
      if (n_parts == 1) {
        const f32x4_t o = L > 0.f ? rotate_inverse(O * (1.0f / L), ql, qr, qblk)
                                  : f32x4_t{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<f32x4_t*>(
            out + ((static_cast<int64_t>(b) * kT + t) * n_q_heads +
                   static_cast<int64_t>(g) * kHeads + mh) * kDim + md) = o;
      } else {
        float* pp = part_bg + (static_cast<int64_t>(split) * kT + t) * (kHeads * kPart) +
                    mh * kPart;
        if (qblk == 0) {
          pp[0] = M;
          pp[1] = L;
        }
        *reinterpret_cast<f32x4_t*>(pp + 2 + md) = O;
      }
    }
  }
}

}  // namespace

hipError_t launch_decode_g8_multi(int nb, int64_t n_splits, int64_t split_len, int n_tok,
                                  const float* q, uint8_t* k_codes, float* k_norms,
                                  uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                                  int64_t capacity, int64_t max_seq_len, const float* quats,
                                  int64_t batch, int64_t n_kv_heads, float scale, float* out,
                                  float* partials, const PageTable* pages, int bits,
                                  const StepAppend* append, hipStream_t stream,
                                  const iq_codebook_t* cb) {
  if (n_tok < 2 || n_tok > 4) return hipErrorInvalidValue;
  if (bits != 2 && bits != 3 && bits != 4) return hipErrorInvalidValue;
  if (pages && (bits != 3 || append)) return hipErrorInvalidValue;
  const PageTable pt = pages ? *pages : PageTable{nullptr, 0, 4, 1};
  const int64_t n_parts = append ? n_splits + 1 : n_splits;
  const dim3 grid(static_cast<unsigned>(n_parts), static_cast<unsigned>(n_kv_heads),
                  static_cast<unsigned>(batch)),
      block(kThreads);
  constexpr int64_t kCus = 256;
  const bool wide = n_parts * n_kv_heads * batch > kCus;
  const size_t lds_pad = wide ? 0 : kOneWorkgroupPadBytes;
  const float qscale = scale * kLog2e;
  const void* k_new = append ? append->k_new : nullptr;
  const void* v_new = append ? append->v_new : nullptr;
  const int new_f16 = append ? append->f16 : 0;
  int32_t* status = append ? append->status : nullptr;
#define IQ_LAUNCH_MTK(NB_, WIDE_, T_, P_, B_, A_)                                                \
  hipLaunchKernelGGL((decode_g8_multi_kernel<NB_, WIDE_, T_, P_, B_, A_>), grid, block, lds_pad,  \
                     stream, q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, partials,    \
                     out, capacity, static_cast<int>(max_seq_len), static_cast<int>(n_kv_heads),  \
                     static_cast<int>(n_splits), static_cast<int>(split_len), qscale,             \
                     codebook_for<B_>(cb), pt, k_new, v_new, new_f16, status)
#define IQ_LAUNCH_MTA(NB_, WIDE_, T_, B_)            \
  if (append) {                                      \
    IQ_LAUNCH_MTK(NB_, WIDE_, T_, false, B_, true);  \
  } else {                                           \
    IQ_LAUNCH_MTK(NB_, WIDE_, T_, false, B_, false); \
  }
#define IQ_LAUNCH_MT(NB_, WIDE_, T_)                  \
  if (pages) {                                        \
    IQ_LAUNCH_MTK(NB_, WIDE_, T_, true, 3, false);    \
  } else if (bits == 2) {                             \
    IQ_LAUNCH_MTA(NB_, WIDE_, T_, 2)                  \
  } else if (bits == 4) {                             \
    IQ_LAUNCH_MTA(NB_, WIDE_, T_, 4)                  \
  } else {                                            \
    IQ_LAUNCH_MTA(NB_, WIDE_, T_, 3)                  \
  }
#define IQ_LAUNCH_MT_W(NB_, T_)       \
  if (wide) {                         \
    IQ_LAUNCH_MT(NB_, true, T_)       \
  } else {                            \
    IQ_LAUNCH_MT(NB_, false, T_)      \
  }
#define IQ_LAUNCH_MT_NB(T_)                   \
  switch (nb) {                               \
    case 1: IQ_LAUNCH_MT_W(1, T_) break;       \
    case 2: IQ_LAUNCH_MT_W(2, T_) break;       \
    case 3: IQ_LAUNCH_MT_W(3, T_) break;       \
    case 4: IQ_LAUNCH_MT_W(4, T_) break;       \
    default: IQ_LAUNCH_MT_W(5, T_) break;      \
  }
  if (n_tok == 2) {
    IQ_LAUNCH_MT_NB(2)
  } else if (n_tok == 3) {
    IQ_LAUNCH_MT_NB(3)
  } else {
    IQ_LAUNCH_MT_NB(4)
  }
#undef IQ_LAUNCH_MT_NB
#undef IQ_LAUNCH_MT_W
#undef IQ_LAUNCH_MT
#undef IQ_LAUNCH_MTA
#undef IQ_LAUNCH_MTK
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_parts == 1) return e;
  // the partials of every (sequence, token, query head) merged by a second
  // launch, which in the fused step also advances the lengths by n_tok
  const dim3 mgrid(static_cast<unsigned>(n_kv_heads * kHeads),
                   static_cast<unsigned>(batch * n_tok));
#define IQ_LAUNCH_MT_MERGE(A_, T_)                                                             \
  hipLaunchKernelGGL((merge_g8_kernel<A_, T_>), mgrid, dim3(kMergeThreads), 0, stream,         \
                     partials, quats, out, static_cast<int>(n_kv_heads),                        \
                     static_cast<int>(n_parts), seq_lens, capacity, kHeads)
#define IQ_LAUNCH_MT_MERGE_T(A_)                            \
  if (n_tok == 2) {                                         \
    IQ_LAUNCH_MT_MERGE(A_, 2);                              \
  } else if (n_tok == 3) {                                  \
    IQ_LAUNCH_MT_MERGE(A_, 3);                              \
  } else {                                                  \
    IQ_LAUNCH_MT_MERGE(A_, 4);                              \
  }
  if (append) {
    IQ_LAUNCH_MT_MERGE_T(true)
  } else {
    IQ_LAUNCH_MT_MERGE_T(false)
  }
#undef IQ_LAUNCH_MT_MERGE_T
#undef IQ_LAUNCH_MT_MERGE
  return hipGetLastError();
}

}  // namespace iq
