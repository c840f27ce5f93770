// Decode attention on the packed 3-bit cache for groups of 8 query heads per
// KV head (App. A; Table 2 A-D; Sec. 3.4), gfx950.  The same kernel runs on
// 2- and 4-bit records (Algorithm 1 at b = 2, 4); the notes below describe
// the 3-bit case, the others differ only in how a lane's slice of a record
// splits into code pairs.
//
// Work decomposition: one 512-thread workgroup (8 waves, two per SIMD) per
// (split of 16 * nbat positions, KV head g, sequence b), the grid's three
// dimensions; the split's nbat batches of 16 positions are dealt to the 8
// waves in contiguous runs of nbat / 8 or nbat / 8 + 1 batches.  With one
// workgroup per CU the SIMDs carry equal work.  A wave's loads (query,
// rotation parameters, both scale arrays and the keys of all its batches,
// then each batch's values as its scores start) are issued in the order the
// data is used, so each wait covers only the data it needs and the waves
// compute while the rest of the cache is still arriving.  In grids of one
// round the loads do not wait for the sequence length (see the kernel).
// The fused step adds one workgroup per (b, g) for the new token.
//
// The two contractions of a batch are dense 8-head x 128-dim x 16-position
// products and run on the matrix cores (v_mfma_f32_16x16x32_f16):
//
//  QK (Table 2 A): S[t][n] = sum_k Khat[t][k] Qt[k][n], rows t = 16 positions,
//    columns n = 16, k = 32 dims per instruction.  The fp32 rotated query is
//    split into fp16 hi + lo parts: columns 0..7 hold the 8 heads' hi parts,
//    columns 8..15 their lo parts, and lanes n and n ^ 8 add their products,
//    so the scores carry ~22 bits.
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
//    weights never leave their lanes.  Each weight is split into fp16 hi +
//    lo parts, one product each: with the weights rounded to fp16 once the
//    outputs of long contexts drift past 2e-3 of the fp64 result.
//
// Softmax (Table 2 B) is two-phase per wave: all QK products of the wave's
// positions first (scores kept in registers), one max per head, then the
// weights and the PV products; scores are in log2 units (the rotated query
// is pre-scaled by scale * log2 e) so exp2 is a single instruction.  The
// value scales s^V are divided by the wave's largest value scale before the
// fp16 conversion, keeping the weights in [0, 2^15].
//
// Merge: the 8 waves merge in LDS; with several splits per (b, g) each
// workgroup writes its partial (m, l, O) per head and a second kernel merges
// them, divides by the sum and applies the single inverse rotation
// R^T = H_128 M^T (Table 2 D); with one split the workgroup does it itself.
#include <hip/hip_runtime.h>
#include <math.h>

#include "iq_g8_device.h"

namespace iq {
namespace {

// Scores, softmax and value accumulation of one wave over the batches that
// hold its nvalid (> 0) positions; only the last of them can be partial.
// kFull: exactly NBX full batches, straight-line code (the scheduler can
// overlap batches); otherwise up to NBX batches with per-batch checks.
// Scores are kept in the per-head scaled domain (x = acc * s^K, the query
// operand carried 2^qexp); qdown = 2^-qexp turns them into log2 units inside
// the exponent.  On return m_run is in log2 units.
// Scale group g of batch i (positions 16 i + 4 g ..) is st.ks[4 i + g].  The
// value scales st.vs[4 i + g]: kWide, staged already multiplied by 2^15 /
// vmax (vmax = the wave's largest attended value scale, computed by the
// caller) and 0 past nvalid; otherwise staged as loaded, and vmax (in: 0) is
// computed here.
// lut: the pair table.  Each batch's value records go through st.rec[i]
// (lane (t, gk) writes its 12 bytes of record t, lane (u, grp) reads the
// 8-byte window holding bytes 3u..3u+2 of records 4 grp + r); the wave's own
// LDS operations complete in order.
//
// kRope (the content / RoPE sub-block split, Sec. 5): every position also
// has a 64-dim positional key kept in fp16, neither rotated nor quantized;
// its scores come from two more matrix instructions per batch on the
// positional keys as loaded (rp: lane (t, gk) holds dims 32 m + 8 gk .. + 7
// of position t in rk[i][m], batch 0 loaded by the caller, batch i + 1 as
// batch i starts) against the positional query operands qbr.
template <int NB, int NBX, bool kFull, bool kWide, bool kPaged, int kBits, bool kRope = false>
__device__ __forceinline__ void attend_wave(const uint32_t (&kw)[NB][kBits],
                                            uint32_t (&vw)[NB][kBits], const uint8_t* vc,
                                            uint32_t koff, const int (&tb)[NB],
                                            const int64_t (&dlt)[NB], WaveStageB<kBits>& st,
                                            const u32x4_t (&qb)[4],
                                            const uint32_t* lut, int col, int grp, int nvalid,
                                            int vdw, uint32_t vsh, float qdown, float& m_run,
                                            float& l_run, float& vmax, f32x4_t (&o_acc)[4],
                                            const uint16_t* rp = nullptr,
                                            const u32x4_t* rk0 = nullptr,
                                            const u32x4_t* qbr = nullptr) {
  // ---- phase 1: scores (Table 2 A) -----------------------------------------
  // the value load of batch i goes out as batch i's scores start, so that
  // phase 1 begins without waiting to issue every value load first.
  // Lanes col and col ^ 8 hold the same four scores (positions 4 grp + r);
  // from here on the lane with col < 8 keeps positions r = 0, 1 and its
  // partner r = 2, 3 (rs = 0 or 2), so each weight is computed once.
  const bool upper = col >= 8;
  const int rs = upper ? 2 : 0;
  f32x2_t sc[NBX];
  u32x4_t rk[NBX][2];
  if constexpr (kRope) {
    rk[0][0] = rk0[0];
    rk[0][1] = rk0[1];
  }
#pragma unroll
  for (int i = 0; i < NBX; ++i) {
    if (!kFull && 16 * i >= nvalid) break;
    __builtin_amdgcn_sched_barrier(kNoVmemAcross);
    load_value_batch<kBits>(kPaged ? vc + dlt[i] * record_bytes<kBits>() : vc, tb[i], koff,
                            vw[i]);
    if constexpr (kRope) {
      if (i + 1 < NBX) {
        const u32x4_t* src =
            reinterpret_cast<const u32x4_t*>(rp + static_cast<int64_t>(tb[i + 1] + col) * 64);
        rk[i + 1][0] = src[grp];
        rk[i + 1][1] = src[4 + grp];
      }
    }
    __builtin_amdgcn_sched_barrier(kNoVmemAcross);
    u32x4_t a[4];
    key_pairs<kBits>(lut, kw[i], a);
    f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) acc = mfma(a[kb], qb[kb], acc);
    // lane (col, grp) holds positions 16 i + 4 grp + r of head col % 8
    f32x4_t x;
    if constexpr (kRope) {
      f32x4_t accr = f32x4_t{0.f, 0.f, 0.f, 0.f};
      accr = mfma(rk[i][0], qbr[0], accr);
      accr = mfma(rk[i][1], qbr[1], accr);
      // content score (times the key scale) plus positional score, then the
      // hi and lo columns of the head joined as below
      x = acc * st.ks[4 * i + grp] + accr;
#pragma unroll
      for (int r = 0; r < 4; ++r) x[r] += xor_lane<8>(x[r]);
    } else {
      // column col holds the hi (col < 8) or lo (col >= 8) product of head
      // col % 8: both lanes of the pair get the sum
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] += xor_lane<8>(acc[r]);
      x = acc * st.ks[4 * i + grp];
    }
    f32x2_t xs = upper ? f32x2_t{x[2], x[3]} : f32x2_t{x[0], x[1]};
    if (!kFull && 16 * i + 16 > nvalid) {
#pragma unroll
      for (int j = 0; j < 2; ++j) xs[j] = (16 * i + 4 * grp + rs + j < nvalid) ? xs[j] : -INFINITY;
    }
    sc[i] = xs;
    m_run = fmaxf(fmaxf(m_run, xs[0]), xs[1]);
  }
  m_run = wave_max(fmaxf(m_run, xor_lane<8>(m_run)));
  // weight scales s^V * 2^15 / vmax.  Wide grids: staged that way in the
  // prologue and read per batch, so the kernel stays within 128 VGPRs.
  // Otherwise: the batches' value scales are read into registers here,
  // before the fence below (which would hold the reads back), with vmax
  // taken over them (off the prologue's critical path).
  f32x2_t wvv[NBX];
  if constexpr (!kWide) {
#pragma unroll
    for (int i = 0; i < NBX; ++i) {
      if (!kFull && 16 * i >= nvalid) break;
      f32x2_t v = *reinterpret_cast<const f32x2_t*>(
          reinterpret_cast<const float*>(&st.vs[4 * i + grp]) + rs);
      if (!kFull && 16 * i + 16 > nvalid) {
#pragma unroll
        for (int j = 0; j < 2; ++j) v[j] = (16 * i + 4 * grp + rs + j < nvalid) ? v[j] : 0.f;
      }
      wvv[i] = v;
      vmax = fmaxf(fmaxf(vmax, v[0]), v[1]);
    }
    vmax = wave_max(fmaxf(vmax, xor_lane<8>(vmax)));
    const float vinv = vmax > 0.f ? 32768.0f * __builtin_amdgcn_rcpf(vmax) : 0.f;
#pragma unroll
    for (int i = 0; i < NBX; ++i) wvv[i] *= vinv;
  }
  // v_perm_b32 selectors of the PV operand dwords.  Operand dword r of the
  // lane holds the hi (lo) part of position r's weight in half `upper`, zero
  // in the other half.  Position j (j = 0, 1) comes from the lower lane of
  // the pair, position 2 + j from the upper one; perm(x, y, sel) reads the
  // packed pair x as bytes 4..7 and y as bytes 0..3, so with (own, partner)
  // for positions j and (partner, own) for positions 2 + j one selector
  // serves both.  The zero bytes use selector values 8 and 10 (a copy of
  // the sign bit of a weight part, 0: the weights are not negative), so
  // the lo selector is the hi one with bit 1 of every byte set.
  const uint32_t sel_hi = upper ? 0x01000808u : 0x08080504u;
  const float mq = -m_run * qdown;

  // ---- phase 2: weights (Table 2 B) and values (Table 2 C) -----------------
  // every batch's value records go to their own staging rows first, so the
  // reads of all batches may be scheduled freely after one fence
#pragma unroll
  for (int i = 0; i < NBX; ++i) {
    if (!kFull && 16 * i >= nvalid) break;
#pragma unroll
    for (int j = 0; j < kBits; ++j)
      st.rec[i][col * rec_stride<kBits>() + kBits * grp + j] = vw[i][j];
  }
  wave_lds_fence();
#pragma unroll
  for (int i = 0; i < NBX; ++i) {
    if (!kFull && 16 * i >= nvalid) break;
    const uint32_t* rec = st.rec[i];
    // the weight scales of this lane's two positions (0 past nvalid)
    const f32x2_t wv =
        kWide ? *reinterpret_cast<const f32x2_t*>(
                    reinterpret_cast<const float*>(&st.vs[4 * i + grp]) + rs)
              : wvv[i];
    // weight p split into p_hi (p with its low 13 mantissa bits cleared:
    // exact in fp16 over the weights' range) and p_lo = p - p_hi (exact in
    // fp32, then fp16), packed as one dword (hi in bits 0..15)
    uint32_t pk[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[i][j], qdown, mq));
      l_run += e;
      const float pf = e * wv[j];
      const float ph = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, pf) & 0xFFFFE000u);
      pk[j] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(ph, pf - ph));
    }
    // the partner lane's pairs (row_ror:8 inside each row of 16 lanes)
    const uint32_t pp0 = static_cast<uint32_t>(
        __builtin_amdgcn_mov_dpp(static_cast<int>(pk[0]), 0x128, 0xF, 0xF, true));
    const uint32_t pp1 = static_cast<uint32_t>(
        __builtin_amdgcn_mov_dpp(static_cast<int>(pk[1]), 0x128, 0xF, 0xF, true));
    const u32x4_t pw_hi = u32x4_t{__builtin_amdgcn_perm(pk[0], pp0, sel_hi),
                                  __builtin_amdgcn_perm(pk[1], pp1, sel_hi),
                                  __builtin_amdgcn_perm(pp0, pk[0], sel_hi),
                                  __builtin_amdgcn_perm(pp1, pk[1], sel_hi)};
    // (formed per batch: one instruction rather than a register held
    // across the loop)
    uint32_t sel_lo = sel_hi;
    asm volatile("" : "+v"(sel_lo));
    sel_lo |= 0x02020202u;
    const u32x4_t pw_lo = u32x4_t{__builtin_amdgcn_perm(pk[0], pp0, sel_lo),
                                  __builtin_amdgcn_perm(pk[1], pp1, sel_lo),
                                  __builtin_amdgcn_perm(pp0, pk[0], sel_lo),
                                  __builtin_amdgcn_perm(pp1, pk[1], sel_lo)};
    u32x4_t vb[4];
    value_pairs<kBits>(lut, rec, grp, vdw, vsh, vb);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      o_acc[nb] = mfma(pw_hi, vb[nb], o_acc[nb]);
      o_acc[nb] = mfma(pw_lo, vb[nb], o_acc[nb]);
    }
  }
  l_run = wave_sum(l_run + xor_lane<8>(l_run));
  m_run *= qdown;
}

// The waves' staging areas while attending and their outputs afterwards
// (wave_o[w][r][lane] = the lane's accumulator entries r of the four PV
// products, as written by the matrix cores).  kSepO: separate, so each wave
// stores its outputs as soon as it is done (one-round grids, which have LDS
// to spare); otherwise they share the space (grids of several rounds, two
// workgroups per CU).
template <int kBits, bool kSepO>
struct G8Stage;
template <int kBits>
struct G8Stage<kBits, false> {
  union {
    WaveStageB<kBits> stage[kWaves];
    f32x4_t wave_o[kWaves][4][64];
  };
};
template <int kBits>
struct G8Stage<kBits, true> {
  WaveStageB<kBits> stage[kWaves];
  f32x4_t wave_o[kWaves][4][64];
};

// LDS of the decode kernel, the pair table first (address 0: a lookup
// address is just field * 4).
template <int kBits, bool kRope, bool kSepO>
struct G8Smem {
  uint32_t lut[1 << (2 * kBits)];   // fp16 pair table: entry f = (C[f % 2^b], C[f / 2^b])
  uint32_t qop[2][kHeads][kQRowWords];
  // positional query operands (kRope): fp16 hi / lo pair rows of 32 words
  uint32_t qop_r[kRope ? 2 : 1][kHeads][kRope ? kRopeRowWords : 1];
  int qexp[kHeads];
  float wave_ml[kWaves][2][kHeads];
  uint32_t new_rec[2][4 * kBits];   // append: the new key / value record
  float new_scale[2];
  // persistent workgroups: each wave's copy of the current chunk of 64
  // sequences' inclusive item offsets and clamped lengths
  int chunk_incl[kWaves][64];
  int chunk_len[kWaves][64];
  G8Stage<kBits, kSepO> st;
};

// Writes the fp16 pair table of the codebook (threads 0 .. 2^(2b) - 1).
template <class Smem, int kBits>
__device__ __forceinline__ void build_pair_table(Smem& sm, const CodebookB<kBits>& cb, int tid) {
  constexpr int kLut = 1 << (2 * kBits);
  if (tid < kLut) {
    constexpr int kMask = (1 << kBits) - 1;
    const uint32_t lo =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid & kMask)));
    const uint32_t hi =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid >> kBits)));
    sm.lut[tid] = lo | (hi << 16);
  }
}

// The kernel's arguments, as passed (see decode_g8_kernel).
template <int kBits>
struct G8Args {
  const float* q;
  uint8_t* k_codes;
  float* k_norms;
  uint8_t* v_codes;
  float* v_norms;
  const int32_t* seq_lens;
  const float* quats;
  float* partials;
  float* out;
  int64_t capacity;
  int max_seq_len, n_kv_heads, n_splits, split_len;
  float qscale;
  CodebookB<kBits> cb;
  const void* k_new;
  const void* v_new;
  int new_f16;
  int32_t* status;
  PageTable pages;
  int group, batch;
  int32_t* lens0;   // fused steps on grids of several rounds: each sequence's length
};

// The fused step's new token for (sequence b, KV head g, head group vg):
// compresses the new key and value (Alg. 1), writes their records at
// position seq_lens[b] and publishes the new token's score and value as the
// partial of split index n_splits (m = -inf when the token is not attended:
// at capacity, or at or past max_seq_len).  No attention work reads the
// records being written, and seq_lens is advanced by the merge kernel after
// every workgroup has read it.  lens0 (grids of several rounds): the
// sequence's length as read here, for the merge.
template <bool kPaged, int kBits, bool kRope, class Smem>
__device__ __forceinline__ void append_token(Smem& sm, const G8Args<kBits>& a,
                                             int gsize, int g, int vg, int b, int bgv,
                                             bool build_lut) {
  constexpr int kRB = record_bytes<kBits>();
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));   // recomputed per item (see attend_split)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int n_q_heads = a.n_kv_heads * gsize;
  const int hq0 = g * gsize + kHeads * vg;
  const int nh = gsize - kHeads * vg < kHeads ? gsize - kHeads * vg : kHeads;
  const int n_parts = a.n_splits + 1;
  const int qh = (tid >> 5) & 7, qblk = tid & 31;
  const f32x4_t qload = *reinterpret_cast<const f32x4_t*>(
      a.q + (static_cast<int64_t>(b) * n_q_heads + hq0 + (qh < nh ? qh : nh - 1)) * kDim +
      4 * qblk);
  const f32x4_t qv = qh < nh ? qload : f32x4_t{0.f, 0.f, 0.f, 0.f};
  const f32x4_t* qpar = reinterpret_cast<const f32x4_t*>(
      a.quats + static_cast<int64_t>(g) * kQuatFloats + 8 * qblk);
  const f32x4_t ql = qpar[0], qr = qpar[1];
  float* part_bg = a.partials + static_cast<int64_t>(bgv) * n_parts * (kHeads * kPart);
  const int64_t row = kPaged ? 0 : static_cast<int64_t>(b * a.n_kv_heads + g) * a.capacity;

  const int seq0 = a.seq_lens[b];
  // record index of the new token (its page's slot, or the row position);
  // -1 when there is no room: the sequence is at capacity, or (paged) the
  // slot's page is not mapped.  Then nothing is written, the token is not
  // attended, the capacity flag is raised, and the new-token partial's l
  // entry carries -1 so that the merge leaves the length as it is.
  const int64_t rec = !(seq0 >= 0 && seq0 < a.capacity)
                          ? -1
                          : (kPaged ? paged_record(a.pages, a.n_kv_heads, b, g, seq0) : row + seq0);
  const bool written = rec >= 0;
  const bool attend_new = written && seq0 < a.max_seq_len;
  if (!written && a.status != nullptr && g == 0 && vg == 0 && tid == 0)
    atomicOr(a.status, static_cast<int32_t>(IQ_ERR_CAPACITY));
  // the length the merge counts the live splits of (grids of several rounds)
  if (a.lens0 != nullptr && g == 0 && vg == 0 && tid == 0) a.lens0[b] = seq0;
  // waves 4 and 5 compress the new key and value: lane l holds dims 2l,
  // 2l + 1 and the parameters of SO(4) block l / 2
  if (wave == 4 || wave == 5) {
    const void* src = wave == 4 ? a.k_new : a.v_new;
    const int64_t off = (static_cast<int64_t>(b) * a.n_kv_heads + g) * kDim;
    float x0, x1;
    if (a.new_f16) {
      const uint32_t w =
          reinterpret_cast<const uint32_t*>(static_cast<const __half*>(src) + off)[lane];
      x0 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w)));
      x1 = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
    } else {
      const f32x2_t w =
          reinterpret_cast<const f32x2_t*>(static_cast<const float*>(src) + off)[lane];
      x0 = w[0];
      x1 = w[1];
    }
    const f32x4_t* qs = reinterpret_cast<const f32x4_t*>(
        a.quats + static_cast<int64_t>(g) * kQuatFloats + 8 * (lane >> 1));
    const f32x4_t p0 = qs[0], p1 = qs[1];
    const float qp[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
    const WaveCode wc = compress_vector_wave<kBits>(x0, x1, qp, a.cb, lane);
    const int which = wave - 4;
    if (lane < 4 * kBits) sm.new_rec[which][lane] = wc.word;
    if (lane == 0) sm.new_scale[which] = wc.scale;
    if (written && vg == 0) {   // one head group of the KV head writes
      uint8_t* codes = which == 0 ? a.k_codes : a.v_codes;
      float* norms = which == 0 ? a.k_norms : a.v_norms;
      if (lane < 4 * kBits) reinterpret_cast<uint32_t*>(codes + rec * kRB)[lane] = wc.word;
      if (lane == 0) norms[rec] = wc.scale;
    }
  }
  if (build_lut) build_pair_table(sm, a.cb, tid);
  f32x4_t y = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if (tid < kRotThreads) y = rotate_forward(qv, ql, qr, qblk, kInvSqrtDim * a.qscale);
  lds_barrier();   // new_rec, new_scale, lut
  if (tid >= kRotThreads) return;
  // score of the new key for head qh: s^K (q_tilde . C[code]) over this
  // thread's dims 4 qblk .. +3, summed over the head's 32 lanes (y already
  // carries the score scale, in log2 units)
  const int md = 4 * qblk;
  const f32x4_t k4 = decode_record_dims<kBits>(sm.new_rec[0], sm.lut, md);
  const f32x4_t v4 = decode_record_dims<kBits>(sm.new_rec[1], sm.lut, md);
  float dot = y[0] * k4[0] + y[1] * k4[1] + y[2] * k4[2] + y[3] * k4[3];
  dot += xor_lane<1>(dot);
  dot += xor_lane<2>(dot);
  dot += xor_lane<4>(dot);
  dot += xor_lane<8>(dot);
  dot += xor_lane<16>(dot);
  float* pp = part_bg + static_cast<int64_t>(a.n_splits) * (kHeads * kPart) + qh * kPart;
  if (qblk == 0) {
    pp[0] = attend_new ? dot * sm.new_scale[0] : -INFINITY;
    pp[1] = written ? 1.0f : -1.0f;
  }
  *reinterpret_cast<f32x4_t*>(pp + 2 + md) = sm.new_scale[1] * v4;
}

// One attention work item: split `split` of the row (KV head g, head group
// vg) of sequence b, partial row bgv.  It attends the positions before
// min(seq_lens[b], max_seq_len).  One-round grids: the work split does not
// depend on the length, so every cache load is addressed from the split range
// alone (clamped to max_seq_len, hence inside the capacity) and issued before
// the length is read; positions at or past the length are masked.  kWide:
// the clamped length is known (seq_w) and the loads cover exactly the
// positions attended.  With several splits the item writes its partial
// (m, l, O) per head; with one it writes the output row itself.
// build_lut: the item writes the pair table (the workgroup's first item).
template <int NB, bool kAppend, bool kWide, bool kPaged, int kBits, bool kRope, class Smem>
__device__ __forceinline__ void attend_split(Smem& sm, const G8Args<kBits>& a,
                                             int gsize, int split, int g, int vg, int b,
                                             int bgv, int seq_w, bool build_lut) {
  constexpr int kRB = record_bytes<kBits>();
  const uint16_t* __restrict__ k_rope = static_cast<const uint16_t*>(a.k_new);
  const float* __restrict__ q_rope = static_cast<const float*>(a.v_new);
  const int rope_shared = a.new_f16;
  uint32_t* lut = sm.lut;
  uint32_t(*qop)[kHeads][kQRowWords] = sm.qop;
  int* qexp_s = sm.qexp;
  float(*wave_ml)[2][kHeads] = sm.wave_ml;
  WaveStageB<kBits>* stage = sm.st.stage;
  f32x4_t(*wave_o)[4][64] = sm.st.wave_o;

  // the thread index, opaque to the compiler: in a persistent workgroup's
  // loop over items, values derived from it are then recomputed per item
  // rather than held in registers across the loop
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  // the wave index as a scalar: every per-wave branch is then a scalar
  // branch, and per-wave positions are scalars
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int n_q_heads = a.n_kv_heads * gsize;
  const int hq0 = g * gsize + kHeads * vg;
  const int nh = gsize - kHeads * vg < kHeads ? gsize - kHeads * vg : kHeads;
  const int n_parts = kAppend ? a.n_splits + 1 : a.n_splits;
  const int split_len = a.split_len, max_seq_len = a.max_seq_len;
  float* out_bg = a.out + (static_cast<int64_t>(b) * n_q_heads + hq0) * kDim;
  const int start = split * split_len;
  if constexpr (kWide) {
    if (start >= seq_w) {
      // nothing to attend (an empty sequence, with a single split): a zero
      // output row
      if (n_parts == 1)
        for (int e = tid; e < nh * kDim; e += kThreads) out_bg[e] = 0.f;
      return;
    }
  }

  // The query and rotation loads go out first (thread (head qh, SO(4) block
  // qblk) for tid < 256; the other waves load the same values).
  const int qh = (tid >> 5) & 7, qblk = tid & 31;
  const f32x4_t qload = *reinterpret_cast<const f32x4_t*>(
      a.q + (static_cast<int64_t>(b) * n_q_heads + hq0 + (qh < nh ? qh : nh - 1)) * kDim +
      4 * qblk);
  const f32x4_t qv = qh < nh ? qload : f32x4_t{0.f, 0.f, 0.f, 0.f};
  // positional query part (kRope): thread (qh, qblk < 16) holds its dims
  // 4 qblk .. 4 qblk + 3
  f32x4_t qrv = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if constexpr (kRope) {
    const f32x4_t t = *reinterpret_cast<const f32x4_t*>(
        q_rope + (static_cast<int64_t>(b) * n_q_heads + hq0 + (qh < nh ? qh : nh - 1)) *
                     kRopeDim +
        4 * (qblk & 15));
    qrv = (qh < nh && qblk < 16) ? t : f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const f32x4_t* qpar = reinterpret_cast<const f32x4_t*>(
      a.quats + static_cast<int64_t>(g) * kQuatFloats + 8 * qblk);
  const f32x4_t ql = qpar[0], qr = qpar[1];
  float* part_bg = a.partials + static_cast<int64_t>(bgv) * n_parts * (kHeads * kPart);
  // contiguous: the (b, g) row; paged: the pools (positions are placed by
  // the per-batch deltas)
  const int64_t row = kPaged ? 0 : static_cast<int64_t>(b * a.n_kv_heads + g) * a.capacity;
  const uint8_t* kc = a.k_codes + row * kRB;
  const uint8_t* vc = a.v_codes + row * kRB;

  // this wave's run of batches: nbat / 8 each, one more for the first
  // nbat % 8 waves
  const int nbat = split_len >> 4;
  const int nb_base = nbat / kWaves, nb_rem = nbat % kWaves;
  const int nb_w = nb_base + (wave < nb_rem ? 1 : 0);
  const int wbase = start + 16 * (wave * nb_base + (wave < nb_rem ? wave : nb_rem));
  int lim = start + split_len < max_seq_len ? start + split_len : max_seq_len;
  if constexpr (kWide) lim = lim < seq_w ? lim : seq_w;
  // start of the wave's last batch before lim (the clamp of the loads):
  // lim <= max_seq_len <= capacity, a multiple of 16, so every loaded batch
  // lies in the row (in a mapped or the fallback page when paged)
  int clamp16 = (lim > 0 ? lim - 1 : 0) & ~15;
  clamp16 = clamp16 < wbase + 16 * (nb_w - 1) ? clamp16 : wbase + 16 * (nb_w - 1);
  clamp16 = clamp16 > 0 ? clamp16 : 0;
  // paged: each batch's record delta (its page's record base minus the
  // page's first logical position; page 0 for an invalid page index).  All
  // NB table entries are read before any is used, and an invalid entry is
  // replaced by a select, so the reads go out together (one round trip).
  int64_t dlt[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) dlt[i] = 0;
  if constexpr (kPaged) {
    const PageTable& pages = a.pages;
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
      dlt[i] = ((page * a.n_kv_heads + g) << pages.page_shift) -
               static_cast<int64_t>((t >> pages.page_shift) << pages.page_shift);
    }
  }
  const float* kn = a.k_norms + row;
  const float* vn = a.v_norms + row;

  // ---- the cache loads (keys and scales now, values as the scores proceed)
  uint32_t kw[NB][kBits], vw[NB][kBits];
  f32x4_t ksl, vsl;
  load_keys<NB, kPaged, kBits>(kc, kn, vn, dlt, wbase, clamp16, lane, col, grp, kw, ksl, vsl);
  // kRope: the positional keys of the wave's first batch (the others are
  // loaded one batch ahead while attending); lane (t, gk) takes dims
  // 8 gk .. + 7 and 32 + 8 gk .. + 7 of position t
  const uint16_t* rp = nullptr;
  u32x4_t rk0[2];
  if constexpr (kRope) {
    rp = k_rope + (static_cast<int64_t>(b) * (rope_shared ? 1 : a.n_kv_heads) +
                   (rope_shared ? 0 : g)) *
                      a.capacity * kRopeDim;
    const int tb0 = wbase < clamp16 ? wbase : clamp16;
    const u32x4_t* src =
        reinterpret_cast<const u32x4_t*>(rp + static_cast<int64_t>(tb0 + col) * kRopeDim);
    rk0[0] = src[grp];
    rk0[1] = src[4 + grp];
  }
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

  // one-round grids: the length, read once the loads are in flight
  int seq;
  if constexpr (kWide) {
    seq = seq_w;
  } else {
    const int seq0 = a.seq_lens[b];
    seq = seq0 < 0 ? 0 : (seq0 > max_seq_len ? max_seq_len : seq0);
  }
  const int end = seq < start + split_len ? seq : start + split_len;
  int nvalid = end - wbase;   // this wave's positions (may be <= 0)
  nvalid = nvalid < 16 * nb_w ? nvalid : 16 * nb_w;

  // ---- while the loads fly: LUT and the rotated query --------------------
  if (build_lut) build_pair_table(sm, a.cb, tid);
  // the 32 blocks of a head are 32 consecutive lanes of one wave, so the
  // rotation needs no barrier
  if (tid < kRotThreads) {
    const f32x4_t y = rotate_forward(qv, ql, qr, qblk, kInvSqrtDim * a.qscale);
    // fp16 operands are kept in the normal range by an exact power-of-two
    // scale per head: the largest rotated entry is brought below 2^14 (hi
    // and lo parts both normal) and the scale is undone on the scores
    int qexp = 0;
    // kRope: the positional part, scaled like the scores but not rotated,
    // shares the head's power-of-two operand scale
    const f32x4_t yr = qrv * a.qscale;
    float amx = fmaxf(fmaxf(fabsf(y[0]), fabsf(y[1])), fmaxf(fabsf(y[2]), fabsf(y[3])));
    if constexpr (kRope)
      amx = fmaxf(amx, fmaxf(fmaxf(fabsf(yr[0]), fabsf(yr[1])), fmaxf(fabsf(yr[2]), fabsf(yr[3]))));
    const float am = group32_max(amx);
    if (am > 0.f) {
      int e = 0;
      frexpf(am, &e);   // am < 2^e
      qexp = 14 - e;
      qexp = qexp > 100 ? 100 : (qexp < -100 ? -100 : qexp);
    }
    // fp16 hi and lo pairs of this thread's 4 dims, stored once per workgroup
    const float qup = ldexpf(1.0f, qexp);
    uint32_t hw[2], lw[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const float x0 = y[2 * j] * qup, x1 = y[2 * j + 1] * qup;
      const _Float16 h0 = static_cast<_Float16>(x0), h1 = static_cast<_Float16>(x1);
      const _Float16 l0 = static_cast<_Float16>(x0 - static_cast<float>(h0));
      const _Float16 l1 = static_cast<_Float16>(x1 - static_cast<float>(h1));
      hw[j] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h0)) |
              (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h1)) << 16);
      lw[j] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l0)) |
              (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l1)) << 16);
    }
    qop[0][qh][2 * qblk] = hw[0];
    qop[0][qh][2 * qblk + 1] = hw[1];
    qop[1][qh][2 * qblk] = lw[0];
    qop[1][qh][2 * qblk + 1] = lw[1];
    if constexpr (kRope) {
      if (qblk < 16) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const float x0 = yr[2 * j] * qup, x1 = yr[2 * j + 1] * qup;
          const _Float16 h0 = static_cast<_Float16>(x0), h1 = static_cast<_Float16>(x1);
          const _Float16 l0 = static_cast<_Float16>(x0 - static_cast<float>(h0));
          const _Float16 l1 = static_cast<_Float16>(x1 - static_cast<float>(h1));
          sm.qop_r[0][qh][2 * qblk + j] =
              static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h0)) |
              (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, h1)) << 16);
          sm.qop_r[1][qh][2 * qblk + j] =
              static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l0)) |
              (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, l1)) << 16);
        }
      }
    }
    if (qblk == 0) qexp_s[qh] = qexp;
  }
  lds_barrier();   // lut, qop, qexp_s
  const uint32_t koff = static_cast<uint32_t>(col * kRB + 4 * kBits * grp);
  int tb[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) tb[i] = wbase + 16 * i < clamp16 ? wbase + 16 * i : clamp16;
  // QK B operands: column col -> head col % 8, hi part for col < 8, lo part
  // for col >= 8; MFMA kb, lane group grp -> dims 32 grp + 8 kb + 0..7 (fp16
  // pair words 16 grp + 4 kb .. +3)
  u32x4_t qb[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    qb[kb] = *reinterpret_cast<const u32x4_t*>(&qop[col >> 3][col & 7][16 * grp + 4 * kb]);
  // positional operands: MFMA m, lane group grp -> dims 32 m + 8 grp .. + 7
  // (pair words 16 m + 4 grp .. + 3)
  u32x4_t qbr[2];
  if constexpr (kRope) {
#pragma unroll
    for (int m = 0; m < 2; ++m)
      qbr[m] = *reinterpret_cast<const u32x4_t*>(&sm.qop_r[col >> 3][col & 7][16 * m + 4 * grp]);
  }
  const float qdown = ldexpf(1.0f, -qexp_s[col & 7]);
  // this wave's scales to its LDS stage (read back per batch).  Lane j
  // holds positions 4j .. 4j+3 of the wave; the value scales of positions at
  // or past nvalid count as 0.  The largest of the rest, vmax, sets the
  // weight scale 2^15 / vmax: weights in [0, 2^15], fp16-normal down to ~2e-9
  // of the largest weight (they are split into fp16 hi + lo parts).  Wide
  // grids apply it here; otherwise attend_wave does, after the scores.
  float vmax = 0.f;
  if constexpr (kWide) {
    f32x4_t v = vsl;
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = (4 * lane + r < nvalid) ? v[r] : 0.f;
    vmax = wave64_max(fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
    const float vinv = vmax > 0.f ? 32768.0f * __builtin_amdgcn_rcpf(vmax) : 0.f;
    stage[wave].vs[lane] = v * vinv;
  } else {
    stage[wave].vs[lane] = vsl;   // scaled in attend_wave
  }
  stage[wave].ks[lane] = ksl;
  wave_lds_fence();

  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o_acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) o_acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if (nvalid == 16 * NB)
    attend_wave<NB, NB, true, kWide, kPaged, kBits, kRope>(
        kw, vw, vc, koff, tb, dlt, stage[wave], qb, lut, col, grp, nvalid, vdw, vsh, qdown,
        m_run, l_run, vmax, o_acc, rp, rk0, qbr);
  else if (NB > 1 && nvalid == 16 * (NB - 1))
    attend_wave<NB, (NB > 1 ? NB - 1 : 1), true, kWide, kPaged, kBits, kRope>(
        kw, vw, vc, koff, tb, dlt, stage[wave], qb, lut, col, grp, nvalid, vdw, vsh, qdown,
        m_run, l_run, vmax, o_acc, rp, rk0, qbr);
  else if (nvalid > 0)
    attend_wave<NB, NB, false, kWide, kPaged, kBits, kRope>(
        kw, vw, vc, koff, tb, dlt, stage[wave], qb, lut, col, grp, nvalid, vdw, vsh, qdown,
        m_run, l_run, vmax, o_acc, rp, rk0, qbr);

  // ---- merge the 8 waves in LDS ---------------------------------------------
  // (a shared output area: once every wave is done with its staging area)
  if constexpr (kWide) lds_barrier();
  // lane (u = col, grp) holds rows 4 grp + r = (head (4 grp + r) % 8, slot
  // grp / 2) of MFMA nb, i.e. dim 8 u + 2 nb + slot; stored as one 16-byte
  // vector per (r, lane) over nb (consecutive lanes: no bank conflicts)
  const float oscale = vmax * (1.0f / 32768.0f);
#pragma unroll
  for (int r = 0; r < 4; ++r)
    wave_o[wave][r][lane] = f32x4_t{o_acc[0][r], o_acc[1][r], o_acc[2][r], o_acc[3][r]} * oscale;
  if (lane < kHeads) {
    wave_ml[wave][0][lane] = m_run;     // lanes 0..7 hold heads 0..7
    wave_ml[wave][1][lane] = l_run;
  }
  lds_barrier();   // wave_o, wave_ml
  if (tid >= kRotThreads) return;

  // thread -> (head h = tid / 32, dims 4 (tid % 32) .. +3), the same
  // (head, block) as in the query rotation.  An item with nothing to attend
  // (split at or past the length) ends with M = -inf, L = 0, O = 0.
  const int mh = qh, md = 4 * qblk;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) M = fmaxf(M, wave_ml[w][0][mh]);
  // dims md + j, j = 0..3: column u = md / 8, MFMA nb = (md % 8) / 2 + j / 2,
  // slot j % 2, row r = mh % 4 of lane u + 16 grp with grp = (mh / 4) % 2 +
  // 2 slot; entries (nb, nb + 1) of a lane are one aligned 8-byte pair
  const int o_r = mh & 3, o_lane = (md >> 3) + 16 * ((mh >> 2) & 1), o_nb = (md & 7) >> 1;
  float L = 0.f;
  f32x4_t O = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const float mw = wave_ml[w][0][mh];
    const float c = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - M);
    L += c * wave_ml[w][1][mh];
    const f32x2_t s0 = *reinterpret_cast<const f32x2_t*>(   // slot 0
        reinterpret_cast<const float*>(&wave_o[w][o_r][o_lane]) + o_nb);
    const f32x2_t s1 = *reinterpret_cast<const f32x2_t*>(   // slot 1
        reinterpret_cast<const float*>(&wave_o[w][o_r][o_lane + 32]) + o_nb);
    O += c * f32x4_t{s0[0], s1[0], s0[1], s1[1]};
  }

  if (n_parts == 1) {
    // thread (mh, md / 4) holds block md / 4 of head mh: rotate back in
    // place (an empty sequence gives a zero row)
    const f32x4_t o = L > 0.f ? rotate_inverse(O * (1.0f / L), ql, qr, qblk)
                              : f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (mh < nh) *reinterpret_cast<f32x4_t*>(out_bg + mh * kDim + md) = o;
    return;
  }
  // ---- partial result of this split ------------------------------------------
  float* pp = part_bg + static_cast<int64_t>(split) * (kHeads * kPart) + mh * kPart;
  if (qblk == 0) {
    pp[0] = M;
    pp[1] = L;
  }
  *reinterpret_cast<f32x4_t*>(pp + 2 + md) = O;
}

// The decode kernel.  Rows of a sequence: (KV head g, head group vg) with vg
// < ceil(group / 8); row (g, vg) serves query heads g * group + 8 vg + 0 ..
// nh - 1 (nh = 8, fewer in the last head group when group is not a multiple
// of 8), whose other query rows of the products are zero and unused.
//
// One-round grids (kWide false; at most one workgroup per CU): grid (split,
// row, sequence b), one work item per workgroup, bound by latency (the
// loads go out before the length is read).  The fused step (kAppend) adds
// split index n_splits per (b, row) for the new token.
//
// Grids of several rounds (kWide): gridDim.x persistent workgroups.  The
// work items are the fused step's new tokens (batch * rows of them, kAppend)
// and then the live splits, enumerated sequence by sequence (a sequence of
// clamped length L has ceil(L / split_len) live splits, each with its rows;
// exactly one when there is a single split, so that an empty sequence still
// gets its zero row); workgroup w takes items w, w + gridDim.x, ...  The
// lengths are read 64 at a time (one per lane) and turned into item offsets
// by a prefix sum across the lanes; every wave computes the same mapping.
// Splits past a length take no workgroup, and the merge kernel reads only
// the splits before each length.
//
// kPaged: the cache is a page pool (PageTable); capacity is then the logical
// capacity max_pages * page_size, and every batch of 16 positions and the
// new token's slot are located through the page table.
//
// kBits: the records' code width, 3 (the paper's cache) or 2 / 4 (Algorithm
// 1 with C_2 / C_4: records of 32 / 64 bytes).  Paged pools hold 3-bit
// records only.
//
// kRope: the content / RoPE sub-block split (Sec. 5, "MLA/RoPE hard
// blocker"): each key also has a 64-dim positional part in fp16
// (k_rope [b][rope row][capacity][64], rope row g, or 0 when rope_shared),
// never rotated or quantized, and each query head a positional part
// (q_rope [b][head][64] fp32); the score adds their dot product.  Decode
// only (no append), contiguous 3-bit caches; the three arguments of the
// append (k_new, v_new, new_f16) carry k_rope, q_rope and rope_shared.
//
// kAnyGroup: `group` query heads per KV head (1 .. 16) in head groups of 8;
// otherwise exactly 8 (the argument is not read).
template <int NB, bool kAppend, bool kWide, bool kPaged, int kBits, bool kRope = false,
          bool kAnyGroup = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kWide && !kRope ? 4 : 2)))
void decode_g8_kernel(
    const float* __restrict__ q, uint8_t* __restrict__ k_codes, float* __restrict__ k_norms,
    uint8_t* __restrict__ v_codes, float* __restrict__ v_norms,
    const int32_t* __restrict__ seq_lens, const float* __restrict__ quats,
    float* __restrict__ partials, float* __restrict__ out, int64_t capacity, int max_seq_len,
    int n_kv_heads, int n_splits, int split_len, float qscale, CodebookB<kBits> cb,
    const void* __restrict__ k_new, const void* __restrict__ v_new, int new_f16,
    int32_t* __restrict__ status, PageTable pages, int group, int batch,
    int32_t* __restrict__ lens0) {
  static_assert(kBits == 3 || !kPaged, "paged pools hold 3-bit records");
  static_assert(!kRope || (!kAppend && !kPaged && kBits == 3 && kAnyGroup),
                "the positional split runs on contiguous 3-bit caches, decode only");
  // the arguments gathered for the device functions (the pointers keep the
  // kernel parameters' no-alias property: the lengths, for one, are then
  // read through the scalar cache)
  const G8Args<kBits> a{q,        k_codes,  k_norms, v_codes,    v_norms,     seq_lens,
                        quats,    partials, out,     capacity,   max_seq_len, n_kv_heads,
                        n_splits, split_len, qscale, cb,         k_new,       v_new,
                        new_f16,  status,   pages,   group,      batch,       lens0};
  __shared__ __attribute__((aligned(16))) G8Smem<kBits, kRope, !kWide> sm;
  const int gsize = kAnyGroup ? a.group : kHeads;
  const int vshift = kAnyGroup && gsize > kHeads ? 1 : 0;
  const int n_rows = a.n_kv_heads << vshift;

  if constexpr (!kWide) {
    const int split = blockIdx.x, yrow = blockIdx.y, b = blockIdx.z;
    const int g = yrow >> vshift, vg = yrow & vshift;
    const int bgv = b * n_rows + yrow;
    if constexpr (kAppend) {
      if (split == a.n_splits) {
        append_token<kPaged, kBits, kRope>(sm, a, gsize, g, vg, b, bgv, true);
        return;
      }
    }
    attend_split<NB, kAppend, false, kPaged, kBits, kRope>(sm, a, gsize, split, g, vg, b, bgv,
                                                          0, true);
  } else {
    const int lane = threadIdx.x & 63;
    const int n_parts = kAppend ? a.n_splits + 1 : a.n_splits;
    const int n_app = kAppend ? a.batch * n_rows : 0;
    const int stride = static_cast<int>(gridDim.x);
    int j = static_cast<int>(blockIdx.x);   // this workgroup's next item
    bool first = true;
    // the pair table, once (ordered before its first use by the first
    // item's barriers)
    build_pair_table(sm, a.cb, threadIdx.x);
    if constexpr (kAppend) {
      for (; j < n_app; j += stride) {
        if (!first) lds_barrier();   // the previous item is done with the LDS
        const int b = j / n_rows, yrow = j - b * n_rows;
        append_token<kPaged, kBits, kRope>(sm, a, gsize, yrow >> vshift, yrow & vshift, b, j,
                                           false);
        first = false;
      }
    }
    int base = n_app;   // items before the current chunk of sequences
    for (int c0 = 0; c0 < a.batch; c0 += 64) {
      // the chunk's clamped lengths (lane l: sequence c0 + l) and the
      // inclusive prefix sum of their items
      int len = 0;
      if (c0 + lane < a.batch) {
        const int s = a.seq_lens[c0 + lane];
        len = s < 0 ? 0 : (s > a.max_seq_len ? a.max_seq_len : s);
      }
      // (the divisor opaque here: its reciprocal is then not held in a
      // register across the loop)
      int sl = a.split_len;
      asm volatile("" : "+s"(sl));
      const int live = c0 + lane < a.batch ? (n_parts == 1 ? 1 : (len + sl - 1) / sl) : 0;
      int incl = live * n_rows;
      {
        // the lane index opaque here, so that the permute addresses are not
        // computed once and held in registers for the whole kernel
        int ln = lane;
        asm volatile("" : "+v"(ln));
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int t = __builtin_amdgcn_ds_bpermute(((ln - d) & 63) << 2, incl);
          incl += ln >= d ? t : 0;
        }
      }
      const int total = __builtin_amdgcn_readlane(incl, 63);
      // kept in the wave's LDS copy rather than in registers across the items
      const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
      sm.chunk_incl[wv][lane] = incl;
      sm.chunk_len[wv][lane] = len;
      for (; j < base + total; j += stride) {
        const int r = j - base;
        // the item's sequence: the lanes whose inclusive prefix is <= r
        // (a prefix of the lanes: the sums do not decrease) come before it.
        // The wave's own LDS writes are complete before its later reads.
        const int inc = sm.chunk_incl[wv][threadIdx.x & 63];
        const int bi = __builtin_popcountll(__ballot(inc <= r));
        const int excl = bi > 0 ? __builtin_amdgcn_readlane(inc, bi - 1) : 0;
        const int seq_w = sm.chunk_len[wv][bi];
        const int rr = r - excl;
        const int split = rr / n_rows, yrow = rr - split * n_rows;
        const int b = c0 + bi;
        if (!first) lds_barrier();   // the previous item is done with the LDS
        attend_split<NB, kAppend, true, kPaged, kBits, kRope>(
            sm, a, gsize, split, yrow >> vshift, yrow & vshift, b, b * n_rows + yrow, seq_w,
            false);
        first = false;
      }
      base += total;
    }
  }
}
}  // namespace

// Split plan of the group-8 path: splits per (sequence, KV head) and their
// length (a multiple of 16).  A workgroup covers at most 8 waves x 5 batches
// x 16 = 640 positions (at 640 every wave has 5 batches and every SIMD the
// same load; a cap of 560 left three SIMDs with one batch more than the
// fourth for the same per-item time); while the grid is small (<= 4 rounds of one workgroup per CU) the
// split count is raised so that the grid, with the fused step's append
// workgroup per (sequence, KV head), fills whole rounds, but a split keeps at
// least one batch per wave.  n_rows: the (KV head, head group) rows of the
// grid per sequence (n_kv_heads * ceil(group / 8)).
void g8_plan(int64_t batch, int64_t n_rows, int64_t max_seq_len, int* nb, int64_t* n_splits,
             int64_t* split_len) {
  constexpr int64_t kCus = 256;
  constexpr int64_t kMaxLen = 640;
  const int64_t t = max_seq_len > 0 ? max_seq_len : 1;
  const int64_t bg = batch * n_rows > 0 ? batch * n_rows : 1;
  int64_t s = (t + kMaxLen - 1) / kMaxLen;
  const int64_t wgs = bg * (s + 1);
  if (wgs <= 4 * kCus) {
    const int64_t rounds = (wgs + kCus - 1) / kCus;
    int64_t s_fill = (rounds * kCus) / bg - 1;
    const int64_t s_min_len = (t + 16 * kWaves - 1) / (16 * kWaves);   // >= 1 batch per wave
    if (s_fill > s_min_len) s_fill = s_min_len;
    if (s_fill > s) s = s_fill;
  }
  int64_t len = (t + s - 1) / s;
  len = (len + 15) / 16 * 16;
  s = (t + len - 1) / len;
  *split_len = len;
  *n_splits = s;
  const int64_t nbat = len / 16;
  *nb = static_cast<int>((nbat + kWaves - 1) / kWaves);
}

hipError_t launch_decode_g8(int nb, int64_t n_splits, int64_t split_len, const float* q,
                            uint8_t* k_codes, float* k_norms, uint8_t* v_codes, float* v_norms,
                            int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                            const float* quats, int64_t batch, int64_t n_kv_heads,
                            int64_t group, float scale, float* out, float* partials,
                            const StepAppend* append, const PageTable* pages, int bits,
                            hipStream_t stream, const iq_codebook_t* cb,
                            const RopeKeys* rope) {
  if (bits != 3 && pages) return hipErrorInvalidValue;
  if (rope && (append || pages || bits != 3)) return hipErrorInvalidValue;
  if (group < 1 || group > 2 * kHeads) return hipErrorInvalidValue;
  // partials per (sequence, KV head, head group): the splits, and the fused
  // step's new token
  const int64_t n_rows = n_kv_heads * ((group + kHeads - 1) / kHeads);
  const int64_t n_parts = append ? n_splits + 1 : n_splits;
  // Up to 5 batches per wave the kernel needs at most 128 VGPRs and ~55 KB of
  // LDS, so two workgroups fit on a CU.  A grid of at most one round gets one
  // workgroup per work item, and its LDS request is padded so that no CU
  // takes two while another idles.  Larger grids run two persistent
  // workgroups per CU over the work items (fewer when there are fewer
  // items): one workgroup's prologue and merge then run beside the other's
  // attention, and splits past a length take no workgroup.
  constexpr int64_t kCus = 256;
  const bool wide = n_parts * n_rows * batch > kCus;
  const size_t lds_pad = wide ? 0 : kOneWorkgroupPadBytes;
  const int64_t n_items = n_parts * n_rows * batch;
  if (n_items > (int64_t{1} << 30)) return hipErrorInvalidValue;   // 32-bit item indices
  // (the positional split's wide instances hold one workgroup per CU)
  const int64_t workers = (rope ? 1 : 2) * kCus;
  const dim3 grid = wide ? dim3(static_cast<unsigned>(n_items < workers ? n_items : workers))
                         : dim3(static_cast<unsigned>(n_parts), static_cast<unsigned>(n_rows),
                                static_cast<unsigned>(batch));
  const dim3 block(kThreads);
  const float qscale = scale * kLog2e;
  const void* k_new = append ? append->k_new : nullptr;
  const void* v_new = append ? append->v_new : nullptr;
  const int new_f16 = append ? append->f16 : 0;
  int32_t* status = append ? append->status : nullptr;
  const PageTable pt = pages ? *pages : PageTable{nullptr, 0, 4, 1};
  // the positional split passes its arguments in the append's three
  const void* k_side = rope ? static_cast<const void*>(rope->k_rope) : k_new;
  const void* v_side = rope ? static_cast<const void*>(rope->q_rope) : v_new;
  const int flag = rope ? rope->shared : new_f16;
  const bool any_group = group != kHeads;
  // fused steps on grids of several rounds: each sequence's length at the
  // step's start, after the partials (the merge's count of live splits)
  int32_t* const lens0 =
      wide && append && n_parts > 1
          ? reinterpret_cast<int32_t*>(reinterpret_cast<char*>(partials) +
                                       g8_partial_region_bytes(batch, n_rows, n_splits))
          : nullptr;
#define IQ_LAUNCH_G8_K(NB_, APP_, WIDE_, PAGED_, BITS_, ROPE_, ANY_)                           \
  hipLaunchKernelGGL((decode_g8_kernel<NB_, APP_, WIDE_, PAGED_, BITS_, ROPE_, ANY_>), grid,     \
                     block, lds_pad, stream, q, k_codes, k_norms, v_codes, v_norms, seq_lens,   \
                     quats, partials, out, capacity, static_cast<int>(max_seq_len),             \
                     static_cast<int>(n_kv_heads), static_cast<int>(n_splits),                  \
                     static_cast<int>(split_len), qscale, codebook_for<BITS_>(cb), k_side,      \
                     v_side, flag, status, pt, static_cast<int>(group), static_cast<int>(batch), \
                     lens0)
#define IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, PAGED_, BITS_)         \
  if (any_group) {                                                \
    IQ_LAUNCH_G8_K(NB_, APP_, WIDE_, PAGED_, BITS_, false, true);  \
  } else {                                                        \
    IQ_LAUNCH_G8_K(NB_, APP_, WIDE_, PAGED_, BITS_, false, false); \
  }
#define IQ_LAUNCH_G8_W(NB_, APP_, WIDE_)                \
  if (pages) {                                          \
    IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, true, 3);        \
  } else if (bits == 2) {                               \
    IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, false, 2);       \
  } else if (bits == 4) {                               \
    IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, false, 4);       \
  } else {                                              \
    IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, false, 3);       \
  }
#define IQ_LAUNCH_G8(NB_, APP_)          \
  if (wide) {                            \
    IQ_LAUNCH_G8_W(NB_, APP_, true)      \
  } else {                               \
    IQ_LAUNCH_G8_W(NB_, APP_, false)     \
  }
#define IQ_LAUNCH_G8_NB(APP_)            \
  switch (nb) {                          \
    case 1: IQ_LAUNCH_G8(1, APP_); break; \
    case 2: IQ_LAUNCH_G8(2, APP_); break; \
    case 3: IQ_LAUNCH_G8(3, APP_); break; \
    case 4: IQ_LAUNCH_G8(4, APP_); break; \
    default: IQ_LAUNCH_G8(5, APP_); break; \
  }
#define IQ_LAUNCH_G8_ROPE(NB_)                              \
  if (wide) {                                               \
    IQ_LAUNCH_G8_K(NB_, false, true, false, 3, true, true);  \
  } else {                                                  \
    IQ_LAUNCH_G8_K(NB_, false, false, false, 3, true, true); \
  }
  if (rope) {
    switch (nb) {
      case 1: IQ_LAUNCH_G8_ROPE(1); break;
      case 2: IQ_LAUNCH_G8_ROPE(2); break;
      case 3: IQ_LAUNCH_G8_ROPE(3); break;
      case 4: IQ_LAUNCH_G8_ROPE(4); break;
      default: IQ_LAUNCH_G8_ROPE(5); break;
    }
  } else if (append) {
    IQ_LAUNCH_G8_NB(true)
  } else {
    IQ_LAUNCH_G8_NB(false)
  }
#undef IQ_LAUNCH_G8_ROPE
#undef IQ_LAUNCH_G8_NB
#undef IQ_LAUNCH_G8
#undef IQ_LAUNCH_G8_W
#undef IQ_LAUNCH_G8_WPB
#undef IQ_LAUNCH_G8_K
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the partials of every (sequence, query head) merged by a second launch,
  // which in the fused step also advances the lengths
  if (n_parts > 1) {
    const dim3 mgrid(static_cast<unsigned>(n_kv_heads * group), static_cast<unsigned>(batch));
    // grids of several rounds leave the splits past each length unwritten:
    // their merge reads the live ones only.  Rows of more than 64 partials
    // (one sequence's long context over few KV heads) are read in passes of
    // 128 or 256 partials by variants that hold them all in registers (fewer
    // waves per SIMD: for merge grids of at most 256 workgroups)
    const bool wide_pass = n_parts > 64 && n_kv_heads * group * batch <= kCus;
#define IQ_LAUNCH_MERGE_U(APP_, ANY_, LIVE_, U_)                                               \
  hipLaunchKernelGGL((merge_g8_kernel<APP_, 1, ANY_, LIVE_, U_>), mgrid, dim3(kMergeThreads), 0, \
                     stream, partials, quats, out, static_cast<int>(n_kv_heads),                \
                     static_cast<int>(n_parts), seq_lens, capacity, static_cast<int>(group),    \
                     static_cast<int>(split_len), static_cast<int>(max_seq_len), lens0)
#define IQ_LAUNCH_MERGE_L(APP_, ANY_, LIVE_)        \
  if (wide_pass && n_parts > 128) {                 \
    IQ_LAUNCH_MERGE_U(APP_, ANY_, LIVE_, 32);       \
  } else if (wide_pass) {                           \
    IQ_LAUNCH_MERGE_U(APP_, ANY_, LIVE_, 16);       \
  } else {                                          \
    IQ_LAUNCH_MERGE_U(APP_, ANY_, LIVE_, 8);        \
  }
#define IQ_LAUNCH_MERGE(APP_, ANY_)        \
  if (wide) {                              \
    IQ_LAUNCH_MERGE_L(APP_, ANY_, true)    \
  } else {                                 \
    IQ_LAUNCH_MERGE_L(APP_, ANY_, false)   \
  }
    if (append && any_group) {
      IQ_LAUNCH_MERGE(true, true)
    } else if (append) {
      IQ_LAUNCH_MERGE(true, false)
    } else if (any_group) {
      IQ_LAUNCH_MERGE(false, true)
    } else {
      IQ_LAUNCH_MERGE(false, false)
    }
#undef IQ_LAUNCH_MERGE
#undef IQ_LAUNCH_MERGE_L
#undef IQ_LAUNCH_MERGE_U
    e = hipGetLastError();
  }
  return e;
}

}  // namespace iq
