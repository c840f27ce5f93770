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
//    weights never leave their lanes.
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

#include "iq_device.h"
#include "iq_internal.h"

namespace iq {
namespace {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_a4_t __attribute__((ext_vector_type(2), aligned(4)));

constexpr int kWaves = 8;                 // waves of a decode workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kRotThreads = 256;          // (head, SO(4) block) tasks: waves 0..3
constexpr int kMaxBatches = 5;            // 16-position batches per wave (register budget)
constexpr int kMergeThreads = 256;
// dynamic LDS that, added to the kernel's own, leaves room for one
// workgroup per CU (160 KB of LDS per CU)
constexpr size_t kOneWorkgroupPadBytes = 48 * 1024;
constexpr int kRecStride = kRecordWords + 1;   // staged record stride (words): spreads banks
constexpr int kQRowWords = kDim / 2 + 4;  // fp16-pair row of one head, padded (68 words)
constexpr int kHeads = 8;                 // query heads per KV head
constexpr int kPart = 2 + kDim;           // m, l, o[128] per head
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kInvSqrtDim = 0.08838834764831845f;

__device__ __forceinline__ f32x4_t mfma(u32x4_t a, u32x4_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a),
                                                __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
}

// Pair-table byte offsets (4 * field) of 6-bit fields that lie inside one
// byte of a word, one instruction each through the byte selects of SDWA:
// top6x4<K>(w) = 4 * bits 8K+2 .. 8K+7 (a field at bit 8K + 2),
// low6x4<K>(w) = 4 * bits 8K .. 8K+5 (a field at bit 8K; the shifted byte is
// truncated to 8 bits, dropping the byte's top two bits).
template <int K>
__device__ __forceinline__ uint32_t top6x4(uint32_t w) {
  static_assert(K >= 0 && K < 4, "byte index");
  uint32_t r;
  if constexpr (K == 0)
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 "
        "src1_sel:DWORD" : "=v"(r) : "v"(w), "s"(0xFCu));
  else if constexpr (K == 1)
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 "
        "src1_sel:DWORD" : "=v"(r) : "v"(w), "s"(0xFCu));
  else if constexpr (K == 2)
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 "
        "src1_sel:DWORD" : "=v"(r) : "v"(w), "s"(0xFCu));
  else
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 "
        "src1_sel:DWORD" : "=v"(r) : "v"(w), "s"(0xFCu));
  return r;
}
template <int K>
__device__ __forceinline__ uint32_t low6x4(uint32_t w) {
  static_assert(K >= 0 && K < 4, "byte index");
  uint32_t r;
  if constexpr (K == 0)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_0" : "=v"(r) : "v"(w));
  else if constexpr (K == 1)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_1" : "=v"(r) : "v"(w));
  else if constexpr (K == 2)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_2" : "=v"(r) : "v"(w));
  else
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:BYTE_0 dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_3" : "=v"(r) : "v"(w));
  return r;
}
// 4 * byte K of w (a 4-bit code pair, 256-entry table), one SDWA shift.
template <int K>
__device__ __forceinline__ uint32_t byte4x4(uint32_t w) {
  static_assert(K >= 0 && K < 4, "byte index");
  uint32_t r;
  if constexpr (K == 0)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_0" : "=v"(r) : "v"(w));
  else if constexpr (K == 1)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_1" : "=v"(r) : "v"(w));
  else if constexpr (K == 2)
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_2" : "=v"(r) : "v"(w));
  else
    asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
        "src1_sel:BYTE_3" : "=v"(r) : "v"(w));
  return r;
}
// 4 * a nibble (a 2-bit code pair, 16-entry table): byte K of u masked with
// 0x3C, one SDWA AND.  With u = w << 2 that is the low nibble of byte K of
// w, with u = w >> 2 its high nibble.
template <int K>
__device__ __forceinline__ uint32_t nib4x4(uint32_t u) {
  static_assert(K >= 0 && K < 4, "byte index");
  uint32_t r;
  if constexpr (K == 0)
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 "
        "src1_sel:DWORD" : "=v"(r) : "v"(u), "s"(0x3Cu));
  else if constexpr (K == 1)
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 "
        "src1_sel:DWORD" : "=v"(r) : "v"(u), "s"(0x3Cu));
  else if constexpr (K == 2)
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 "
        "src1_sel:DWORD" : "=v"(r) : "v"(u), "s"(0x3Cu));
  else
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 "
        "src1_sel:DWORD" : "=v"(r) : "v"(u), "s"(0x3Cu));
  return r;
}
// Pair-table entry at byte offset a4 (the table sits at LDS address 0).
__device__ __forceinline__ uint32_t lut_at(const uint32_t* lut, uint32_t a4) {
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + a4);
}

// Workgroup barrier that orders LDS only.  __syncthreads() also fences
// global memory, which would make every wave wait for all of its outstanding
// cache loads at the first barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Orders this wave's LDS accesses across lanes: a value one lane wrote is
// read by another lane of the same wave after this point.  The wave's LDS
// operations execute in order, so no hardware wait is needed; this keeps the
// compiler from moving the accesses across it.
__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
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

// One Walsh-Hadamard stage across lanes: the pair (i, i ^ kM) becomes
// (x_i + x_(i^kM), x_i - x_(i^kM)); blk = this lane's index in its 32-group.
template <int kM>
__device__ __forceinline__ void lane_butterfly(f32x4_t& x, int blk) {
  const float sg = (blk & kM) ? -1.0f : 1.0f;
#pragma unroll
  for (int r = 0; r < 4; ++r) x[r] = __builtin_fmaf(sg, x[r], xor_lane<kM>(x[r]));
}

// Unnormalized H_32 over the block index held by 32 consecutive lanes (each
// lane holds its block's 4 entries).  With the in-block H_4 this is H_128:
// the transform factors over index bits (bits 0..1 inside the block, bits
// 2..6 = block index).
__device__ __forceinline__ void lane_wht32(f32x4_t& x, int blk) {
  lane_butterfly<1>(x, blk);
  lane_butterfly<2>(x, blk);
  lane_butterfly<4>(x, blk);
  lane_butterfly<8>(x, blk);
  lane_butterfly<16>(x, blk);
}

// Largest value over all 64 lanes, returned wave-uniform: quad and row
// rotations (DPP) give every 16-lane row its maximum, the row broadcasts
// (row_bcast:15 into rows 1 and 3, row_bcast:31 into rows 2 and 3) carry
// the lower rows into row 3, and its last lane is read out.
__device__ __forceinline__ float wave64_max(float x) {
  x = fmaxf(x, xor_lane<1>(x));
  x = fmaxf(x, xor_lane<2>(x));
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x),
                                                                  0x124, 0xF, 0xF, true)));
  x = fmaxf(x, xor_lane<8>(x));
  int xi = __builtin_bit_cast(int, x);
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(xi, xi, 0x142, 0xA, 0xF,
                                                                     false)));
  xi = __builtin_bit_cast(int, x);
  x = fmaxf(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(xi, xi, 0x143, 0xC, 0xF,
                                                                     false)));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

// Largest value over the lane's group of 32 lanes.
__device__ __forceinline__ float group32_max(float v) {
  v = fmaxf(v, xor_lane<1>(v));
  v = fmaxf(v, xor_lane<2>(v));
  v = fmaxf(v, xor_lane<4>(v));
  v = fmaxf(v, xor_lane<8>(v));
  v = fmaxf(v, xor_lane<16>(v));
  return v;
}

// Hamilton product a b of quaternions (w, x, y, z).
__device__ __forceinline__ f32x4_t quat_mul(f32x4_t a, f32x4_t b) {
  return f32x4_t{a[0] * b[0] - a[1] * b[1] - a[2] * b[2] - a[3] * b[3],
                 a[0] * b[1] + a[1] * b[0] + a[2] * b[3] - a[3] * b[2],
                 a[0] * b[2] - a[1] * b[3] + a[2] * b[0] + a[3] * b[1],
                 a[0] * b[3] + a[1] * b[2] - a[2] * b[1] + a[3] * b[0]};
}
__device__ __forceinline__ f32x4_t quat_conj(f32x4_t a) {
  return f32x4_t{a[0], -a[1], -a[2], -a[3]};
}

// Forward rotation (App. A) of one head held by 32 lanes, 4 dims per lane:
// the block map v -> q_L v conj(q_R) (Sec. 3.3) applied to (H_4 (H_32 x))_blk,
// times `scale` (1/sqrt(128) and any score scale).  ql, qr: this lane's block
// parameters.
__device__ __forceinline__ f32x4_t rotate_forward(f32x4_t x, f32x4_t ql, f32x4_t qr, int blk,
                                                  float scale) {
  lane_wht32(x, blk);
  float a = x[0], b = x[1], c = x[2], d = x[3];
  wht4(a, b, c, d);
  return quat_mul(quat_mul(ql, f32x4_t{a, b, c, d}), quat_conj(qr)) * scale;
}

// Inverse rotation R^T = H_128 diag(M^T) / sqrt(128) (Table 2 D) of one head
// held by 32 lanes, 4 dims per lane.  M^T z = conj(q_L) z q_R: the matrices
// of left and right multiplication by a quaternion transpose to those of its
// conjugate.
__device__ __forceinline__ f32x4_t rotate_inverse(f32x4_t o, f32x4_t ql, f32x4_t qr, int blk) {
  f32x4_t x = quat_mul(quat_mul(quat_conj(ql), o), qr);
  float a = x[0], b = x[1], c = x[2], d = x[3];
  wht4(a, b, c, d);
  x = f32x4_t{a, b, c, d};
  lane_wht32(x, blk);
  return x * kInvSqrtDim;
}

// Codebook values of dims d..d+3 (d % 4 == 0) of a packed record held in
// LDS (12 words): codes at bits 3d .. 3d+11, two 6-bit fields looked up in
// the fp16 pair table.
__device__ __forceinline__ f32x4_t decode_record_dims(const uint32_t* rec, const uint32_t* lut,
                                                      int d) {
  const int bit = 3 * d, w = bit >> 5, off = bit & 31;
  const uint32_t lo = rec[w];
  const uint32_t hi = w + 1 < kRecordWords ? rec[w + 1] : 0u;
  const uint32_t bits = __builtin_amdgcn_alignbit(hi, lo, off);
  const uint32_t p0 = lut[bits & 63u], p1 = lut[(bits >> 6) & 63u];
  return f32x4_t{static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(p0))),
                 static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(p0 >> 16))),
                 static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(p1))),
                 static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(p1 >> 16)))};
}

// Staged record stride (words) for b-bit records of 4b words: 13 for the
// 3-bit records; 10 and 20 put the four lane groups of the value reads
// (record 4 gk + r, word u or u / 2) on disjoint banks.
template <int kBits>
constexpr int rec_stride() {
  return kBits == 3 ? kRecStride : (kBits == 2 ? 10 : 20);
}

// Per-wave LDS staging: the two scale arrays of the wave (a 16-byte group
// per lane, 64 groups) and the value records of all its batches.
template <int kBits>
struct WaveStageB {
  f32x4_t ks[64];
  f32x4_t vs[64];
  uint32_t rec[kMaxBatches][16 * rec_stride<kBits>()];
};
using WaveStage = WaveStageB<3>;

// Cache loads of one wave, in the order the data is used: both scale arrays
// (one 16-byte load per lane: lane j takes positions 4j .. 4j+3 of the
// wave), then per batch of 16 positions the keys (load_keys), and later the
// values (load_value_batch, one batch at a time as the scores proceed).  Keys and values are loaded the same way: lane
// (t = col, gk = grp) takes dwords 3gk .. 3gk+2 of position t, one coalesced
// 768-byte load per batch.
// Batch starts are multiples of 16 and the capacity is a multiple of 16, so a
// batch holding any position before the end of the split lies inside the
// row.  Batch starts are clamped to `clamp16`, the wave's last batch holding
// positions (a batch past it re-reads the same lines and is skipped).  Per
// batch the start is a scalar and the lane offsets are constants: one
// straight-line sequence for every wave, so the compiler keeps exact counts
// of the loads in flight.
// kPaged: batch i of the wave lies at record index dlt[i] + (its position)
// of the pools (dlt[i] = the batch page's record base minus the page's first
// logical position); contiguous caches use the row pointers as they are.
template <int NB, bool kPaged, int kBits>
__device__ __forceinline__ void load_keys(const uint8_t* kc, const float* kn, const float* vn,
                                          const int64_t (&dlt)[NB], int wbase, int clamp16,
                                          int lane, int col, int grp, uint32_t (&kw)[NB][kBits],
                                          f32x4_t& ksl, f32x4_t& vsl) {
  constexpr int kRB = record_bytes<kBits>();
  const uint32_t koff = static_cast<uint32_t>(col * kRB + 4 * kBits * grp);
  // scales: lane j -> batch j / 4 (clamped like the batches), group j % 4
  {
    const int jb = lane >> 2 < NB ? lane >> 2 : NB - 1;
    const int tj = (wbase + 16 * jb < clamp16 ? wbase + 16 * jb : clamp16) + 4 * (lane & 3);
    int64_t d = 0;
    if constexpr (kPaged) {
      d = dlt[0];
#pragma unroll
      for (int i = 1; i < NB; ++i) d = jb == i ? dlt[i] : d;
    }
    ksl = *reinterpret_cast<const f32x4_t*>(kn + d + tj);
    vsl = *reinterpret_cast<const f32x4_t*>(vn + d + tj);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int tb = wbase + 16 * i < clamp16 ? wbase + 16 * i : clamp16;
    const uint8_t* kb = kPaged ? kc + dlt[i] * kRB : kc;
    const uint32_t* p =
        reinterpret_cast<const uint32_t*>(kb + static_cast<uint32_t>(tb * kRB) + koff);
#pragma unroll
    for (int j = 0; j < kBits; ++j) kw[i][j] = p[j];
  }
  __builtin_amdgcn_sched_barrier(0);
}

// Scheduling-barrier mask: every instruction type may move across except
// vector-memory ones (keeps the value loads in their place and order).
constexpr int kNoVmemAcross = 0x1 | 0x2 | 0x4 | 0x8 | 0x80 | 0x100 | 0x200 | 0x400;

// Value slice of one batch: lane (t = col, gk = grp) takes dwords b gk ..
// b gk + b - 1 of position tb + t (one coalesced 16 x 8b-byte load; 768
// bytes at b = 3).
template <int kBits>
__device__ __forceinline__ void load_value_batch(const uint8_t* vc, int tb, uint32_t koff,
                                                 uint32_t (&v)[kBits]) {
  const uint32_t* p = reinterpret_cast<const uint32_t*>(
      vc + static_cast<uint32_t>(tb * record_bytes<kBits>()) + koff);
#pragma unroll
  for (int j = 0; j < kBits; ++j) v[j] = p[j];
}

// QK operand dwords of one lane: pairs F = 4 kb + e (e = 0..3) of its slice
// w (the lane's 32 dims), each a byte offset into the pair table.
template <int kBits>
__device__ __forceinline__ void key_pairs(const uint32_t* lut, const uint32_t (&w)[kBits],
                                          u32x4_t (&a)[4]) {
  if constexpr (kBits == 3) {
    // fields F = 0..15 at bit 6F of the 96-bit slice w0:w1:w2: those at
    // bits 0 or 2 mod 8 are byte selects of w0..w2, the others byte selects
    // of the slice shifted right by 4 (u0..u2)
    const uint32_t w0 = w[0], w1 = w[1], w2 = w[2];
    const uint32_t u0 = __builtin_amdgcn_alignbit(w1, w0, 4);
    const uint32_t u1 = __builtin_amdgcn_alignbit(w2, w1, 4);
    const uint32_t u2 = w2 >> 4;
    a[0] = u32x4_t{lut_at(lut, low6x4<0>(w0)), lut_at(lut, top6x4<0>(u0)),
                   lut_at(lut, low6x4<1>(u0)), lut_at(lut, top6x4<2>(w0))};
    a[1] = u32x4_t{lut_at(lut, low6x4<3>(w0)), lut_at(lut, top6x4<3>(u0)),
                   lut_at(lut, low6x4<0>(u1)), lut_at(lut, top6x4<1>(w1))};
    a[2] = u32x4_t{lut_at(lut, low6x4<2>(w1)), lut_at(lut, top6x4<2>(u1)),
                   lut_at(lut, low6x4<3>(u1)), lut_at(lut, top6x4<0>(w2))};
    a[3] = u32x4_t{lut_at(lut, low6x4<1>(w2)), lut_at(lut, top6x4<1>(u2)),
                   lut_at(lut, low6x4<2>(u2)), lut_at(lut, top6x4<3>(w2))};
  } else if constexpr (kBits == 4) {
    // pair F = byte F of the 16-byte slice: byte e of word kb
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      a[kb] = u32x4_t{lut_at(lut, byte4x4<0>(w[kb])), lut_at(lut, byte4x4<1>(w[kb])),
                      lut_at(lut, byte4x4<2>(w[kb])), lut_at(lut, byte4x4<3>(w[kb]))};
  } else {
    static_assert(kBits == 2, "2, 3 or 4 bits");
    // pair F = nibble F of the 8-byte slice: nibbles 0..3 of bytes 2 (kb % 2)
    // and 2 (kb % 2) + 1 of word kb / 2
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t lo = w[h] << 2, hi = w[h] >> 2;
      a[2 * h] = u32x4_t{lut_at(lut, nib4x4<0>(lo)), lut_at(lut, nib4x4<0>(hi)),
                         lut_at(lut, nib4x4<1>(lo)), lut_at(lut, nib4x4<1>(hi))};
      a[2 * h + 1] = u32x4_t{lut_at(lut, nib4x4<2>(lo)), lut_at(lut, nib4x4<2>(hi)),
                             lut_at(lut, nib4x4<3>(lo)), lut_at(lut, nib4x4<3>(hi))};
    }
  }
}

// PV operand dwords of lane u = col for the position rows 4 gk + r of a
// staged batch: pairs F = 4u + nb (nb = 0..3), i.e. dims 8u .. 8u + 7.
// 3 bits: bytes 3u .. 3u + 2 of the record, found in the 8-byte window at
// word vdw shifted right by vsh; 4 bits: word u (vdw = u); 2 bits: the half
// of word u / 2 (vdw) at bit vsh = 16 (u % 2).
template <int kBits>
__device__ __forceinline__ void value_pairs(const uint32_t* lut, const uint32_t* rec, int grp,
                                            int vdw, uint32_t vsh, u32x4_t (&vb)[4]) {
  constexpr int kStride = rec_stride<kBits>();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t* wp = rec + (4 * grp + r) * kStride + vdw;
    if constexpr (kBits == 3) {
      // bytes 3u .. 3u+2 of the 8-byte window (a 64-bit shift: lane 15's
      // bytes start 5 bytes in)
      const uint64_t w64 = (static_cast<uint64_t>(wp[1]) << 32) | wp[0];
      // fields at bits 0, 6, 12, 18 of the window: bits 0 and 18 are byte
      // selects of it, bits 6 and 12 of the window shifted right by 4
      const uint32_t win = static_cast<uint32_t>(w64 >> vsh);
      const uint32_t wu = static_cast<uint32_t>(w64 >> (vsh + 4));
      vb[0][r] = lut_at(lut, low6x4<0>(win));
      vb[1][r] = lut_at(lut, top6x4<0>(wu));
      vb[2][r] = lut_at(lut, low6x4<1>(wu));
      vb[3][r] = lut_at(lut, top6x4<2>(win));
    } else if constexpr (kBits == 4) {
      const uint32_t x = wp[0];
      vb[0][r] = lut_at(lut, byte4x4<0>(x));
      vb[1][r] = lut_at(lut, byte4x4<1>(x));
      vb[2][r] = lut_at(lut, byte4x4<2>(x));
      vb[3][r] = lut_at(lut, byte4x4<3>(x));
    } else {
      const uint32_t x = wp[0] >> vsh;
      const uint32_t lo = x << 2, hi = x >> 2;
      vb[0][r] = lut_at(lut, nib4x4<0>(lo));
      vb[1][r] = lut_at(lut, nib4x4<0>(hi));
      vb[2][r] = lut_at(lut, nib4x4<1>(lo));
      vb[3][r] = lut_at(lut, nib4x4<1>(hi));
    }
  }
}

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
template <int NB, int NBX, bool kFull, bool kWide, bool kPaged, int kBits>
__device__ __forceinline__ void attend_wave(const uint32_t (&kw)[NB][kBits],
                                            uint32_t (&vw)[NB][kBits], const uint8_t* vc,
                                            uint32_t koff, const int (&tb)[NB],
                                            const int64_t (&dlt)[NB], WaveStageB<kBits>& st,
                                            const u32x4_t (&qb)[4],
                                            const uint32_t* lut, int col, int grp, int nvalid,
                                            int vdw, uint32_t vsh, float qdown, float& m_run,
                                            float& l_run, float& vmax, f32x4_t (&o_acc)[4]) {
  // ---- phase 1: scores (Table 2 A) -----------------------------------------
  // the value load of batch i goes out as batch i's scores start, so that
  // phase 1 begins without waiting to issue every value load first
  f32x4_t sc[NBX];
#pragma unroll
  for (int i = 0; i < NBX; ++i) {
    if (!kFull && 16 * i >= nvalid) break;
    __builtin_amdgcn_sched_barrier(kNoVmemAcross);
    load_value_batch<kBits>(kPaged ? vc + dlt[i] * record_bytes<kBits>() : vc, tb[i], koff,
                            vw[i]);
    __builtin_amdgcn_sched_barrier(kNoVmemAcross);
    u32x4_t a[4];
    key_pairs<kBits>(lut, kw[i], a);
    f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) acc = mfma(a[kb], qb[kb], acc);
    // column col holds the hi (col < 8) or lo (col >= 8) product of head
    // col % 8: both lanes of the pair get the sum
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] += xor_lane<8>(acc[r]);
    // lane (col, grp) holds positions 16 i + 4 grp + r of head col % 8
    f32x4_t x = acc * st.ks[4 * i + grp];
    if (!kFull && 16 * i + 16 > nvalid) {
#pragma unroll
      for (int r = 0; r < 4; ++r) x[r] = (16 * i + 4 * grp + r < nvalid) ? x[r] : -INFINITY;
    }
    sc[i] = x;
    m_run = fmaxf(fmaxf(m_run, x[0]), x[1]);
    m_run = fmaxf(fmaxf(m_run, x[2]), x[3]);
  }
  m_run = wave_max(m_run);
  // weight scales s^V * 2^15 / vmax.  Wide grids: staged that way in the
  // prologue and read per batch, so the kernel stays within 128 VGPRs.
  // Otherwise: the batches' value scales are read into registers here,
  // before the fence below (which would hold the reads back), with vmax
  // taken over them (off the prologue's critical path).
  f32x4_t wvv[NBX];
  if constexpr (!kWide) {
#pragma unroll
    for (int i = 0; i < NBX; ++i) {
      if (!kFull && 16 * i >= nvalid) break;
      f32x4_t v = st.vs[4 * i + grp];
      if (!kFull && 16 * i + 16 > nvalid) {
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = (16 * i + 4 * grp + r < nvalid) ? v[r] : 0.f;
      }
      wvv[i] = v;
      vmax = fmaxf(fmaxf(vmax, v[0]), v[1]);
      vmax = fmaxf(fmaxf(vmax, v[2]), v[3]);
    }
    vmax = wave_max(vmax);
    const float vinv = vmax > 0.f ? 32768.0f * __builtin_amdgcn_rcpf(vmax) : 0.f;
#pragma unroll
    for (int i = 0; i < NBX; ++i) wvv[i] *= vinv;
  }
  const uint32_t slot_shift = (col >= 8) ? 16u : 0u;
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
    const f32x4_t wv = kWide ? st.vs[4 * i + grp] : wvv[i];   // 0 past nvalid
    u32x4_t pw_hi, pw_lo;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[i][r], qdown, mq));
      l_run += e;
      const float pf = e * wv[r];
      const _Float16 ph = static_cast<_Float16>(pf);
      const _Float16 pl = static_cast<_Float16>(pf - static_cast<float>(ph));
      pw_hi[r] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, ph)) << slot_shift;
      pw_lo[r] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, pl)) << slot_shift;
    }
    u32x4_t vb[4];
    value_pairs<kBits>(lut, rec, grp, vdw, vsh, vb);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      o_acc[nb] = mfma(pw_hi, vb[nb], o_acc[nb]);
      o_acc[nb] = mfma(pw_lo, vb[nb], o_acc[nb]);
    }
  }
  l_run = wave_sum(l_run);
  m_run *= qdown;
}

// Grid (split, KV head g, sequence b).  The attention workgroups attend the
// positions before min(seq_lens[b], max_seq_len); their work split does not
// depend on the length, so every cache load is addressed from the split
// range alone (clamped to max_seq_len, hence inside the capacity) and issued
// before the length is read; positions at or past the length are masked.
// With several splits each workgroup writes its partial (m, l, O) per head;
// with one it writes the output row itself.
//
// kAppend, the fused decode step: one more workgroup per (b, g), split index
// n_splits, compresses the new key and value (Alg. 1), writes their records
// at position seq_lens[b] and publishes the new token's score and value as
// the partial of that extra split (m = -inf when the token is not attended:
// at capacity, or at or past max_seq_len).  No attention workgroup reads the
// records being written, and seq_lens is advanced by the merge kernel after
// every workgroup has read it.
//
// kPaged: the cache is a page pool (PageTable); capacity is then the logical
// capacity max_pages * page_size, and every batch of 16 positions and the
// new token's slot are located through the page table.
//
// kBits: the records' code width, 3 (the paper's cache) or 2 / 4 (Algorithm
// 1 with C_2 / C_4: records of 32 / 64 bytes).  The fused step and paged
// pools run on 3-bit records only.
template <int NB, bool kAppend, bool kWide, bool kPaged, int kBits>
__global__ __launch_bounds__(kThreads) void decode_g8_kernel(
    const float* __restrict__ q, uint8_t* __restrict__ k_codes, float* __restrict__ k_norms,
    uint8_t* __restrict__ v_codes, float* __restrict__ v_norms,
    const int32_t* __restrict__ seq_lens, const float* __restrict__ quats,
    float* __restrict__ partials, float* __restrict__ out, int64_t capacity, int max_seq_len,
    int n_kv_heads, int n_splits, int split_len, float qscale, CodebookB<kBits> cb,
    const void* __restrict__ k_new, const void* __restrict__ v_new, int new_f16,
    int32_t* __restrict__ status, PageTable pages) {
  static_assert(kBits == 3 || (!kAppend && !kPaged), "fused step and pages: 3-bit records");
  constexpr int kRB = record_bytes<kBits>();
  constexpr int kLut = 1 << (2 * kBits);   // pairs of codes
  // All LDS of the kernel in one object, the pair table first (address 0:
  // a lookup address is just field * 4).
  struct Smem {
    uint32_t lut[kLut];   // fp16 pair table: entry f = (C[f % 2^b], C[f / 2^b])
    uint32_t qop[2][kHeads][kQRowWords];
    int qexp[kHeads];
    float wave_ml[kWaves][2][kHeads];
    uint32_t new_rec[2][kRecordWords];   // append workgroup: the new key / value record
    float new_scale[2];
    // the waves' staging areas while attending, their outputs afterwards
    // (wave_o[w][r][lane] = the lane's accumulator entries r of the four
    // PV products, as written by the matrix cores)
    union {
      WaveStageB<kBits> stage[kWaves];
      f32x4_t wave_o[kWaves][4][64];
    };
  };
  __shared__ __attribute__((aligned(16))) Smem sm;
  uint32_t* lut = sm.lut;
  uint32_t(*qop)[kHeads][kQRowWords] = sm.qop;
  int* qexp_s = sm.qexp;
  float(*wave_ml)[2][kHeads] = sm.wave_ml;
  WaveStageB<kBits>* stage = sm.stage;
  f32x4_t(*wave_o)[4][64] = sm.wave_o;

  const int tid = threadIdx.x;
  // the wave index as a scalar: every per-wave branch is then a scalar
  // branch, and per-wave positions are scalars
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;

  const int split = blockIdx.x;
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int bg = b * n_kv_heads + g;
  const int n_q_heads = n_kv_heads * kHeads;
  const int n_parts = kAppend ? n_splits + 1 : n_splits;

  // The query and rotation loads go out first (thread (head qh, SO(4) block
  // qblk) for tid < 256; the other waves load the same values).
  const int qh = (tid >> 5) & 7, qblk = tid & 31;
  const f32x4_t qv = *reinterpret_cast<const f32x4_t*>(
      q + (static_cast<int64_t>(b) * n_q_heads + static_cast<int64_t>(g) * kHeads + qh) * kDim +
      4 * qblk);
  const f32x4_t* qpar = reinterpret_cast<const f32x4_t*>(
      quats + static_cast<int64_t>(g) * kQuatFloats + 8 * qblk);
  const f32x4_t ql = qpar[0], qr = qpar[1];
  float* out_bg =
      out + (static_cast<int64_t>(b) * n_q_heads + static_cast<int64_t>(g) * kHeads) * kDim;
  float* part_bg = partials + static_cast<int64_t>(bg) * n_parts * (kHeads * kPart);
  // contiguous: the (b, g) row; paged: the pools (positions are placed by
  // the per-batch deltas)
  const int64_t row = kPaged ? 0 : static_cast<int64_t>(bg) * capacity;
  uint8_t* kc = k_codes + row * kRB;
  uint8_t* vc = v_codes + row * kRB;

  if constexpr (kAppend) if (split == n_splits) {
    // ---- the append workgroup ------------------------------------------------
    const int seq0 = seq_lens[b];
    const bool appended = seq0 >= 0 && seq0 < capacity;
    const bool attend_new = appended && seq0 < max_seq_len;
    if (!appended && status != nullptr && g == 0 && tid == 0)
      atomicOr(status, static_cast<int32_t>(IQ_ERR_CAPACITY));
    // waves 4 and 5 compress the new key and value: lane l holds dims 2l,
    // 2l + 1 and the parameters of SO(4) block l / 2
    if (wave == 4 || wave == 5) {
      const void* src = wave == 4 ? k_new : v_new;
      const int64_t off = (static_cast<int64_t>(b) * n_kv_heads + g) * kDim;
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
      const WaveCode wc = compress_vector_wave(x0, x1, qp, cb, lane);
      const int which = wave - 4;
      if (lane < kRecordWords) sm.new_rec[which][lane] = wc.word;
      if (lane == 0) sm.new_scale[which] = wc.scale;
      // record index of the new token (its page's slot, or the row position)
      const int64_t rec =
          !appended ? -1 : (kPaged ? paged_record(pages, n_kv_heads, b, g, seq0) : row + seq0);
      if (rec >= 0) {
        uint8_t* codes = which == 0 ? k_codes : v_codes;
        float* norms = which == 0 ? k_norms : v_norms;
        if (lane < kRecordWords)
          reinterpret_cast<uint32_t*>(codes + rec * kRecordBytes)[lane] = wc.word;
        if (lane == 0) norms[rec] = wc.scale;
      }
    }
    if (tid < 64) {
      const uint32_t lo =
          __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid & 7)));
      const uint32_t hi =
          __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid >> 3)));
      lut[tid] = lo | (hi << 16);
    }
    f32x4_t y = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (tid < kRotThreads) y = rotate_forward(qv, ql, qr, qblk, kInvSqrtDim * qscale);
    lds_barrier();   // new_rec, new_scale, lut
    if (tid >= kRotThreads) return;
    // score of the new key for head qh: s^K (q_tilde . C[code]) over this
    // thread's dims 4 qblk .. +3, summed over the head's 32 lanes (y already
    // carries the score scale, in log2 units)
    const int md = 4 * qblk;
    const f32x4_t k4 = decode_record_dims(sm.new_rec[0], lut, md);
    const f32x4_t v4 = decode_record_dims(sm.new_rec[1], lut, md);
    float dot = y[0] * k4[0] + y[1] * k4[1] + y[2] * k4[2] + y[3] * k4[3];
    dot += xor_lane<1>(dot);
    dot += xor_lane<2>(dot);
    dot += xor_lane<4>(dot);
    dot += xor_lane<8>(dot);
    dot += xor_lane<16>(dot);
    float* pp = part_bg + static_cast<int64_t>(n_splits) * (kHeads * kPart) + qh * kPart;
    if (qblk == 0) {
      pp[0] = attend_new ? dot * sm.new_scale[0] : -INFINITY;
      pp[1] = 1.0f;
    }
    *reinterpret_cast<f32x4_t*>(pp + 2 + md) = sm.new_scale[1] * v4;
    return;
  }

  // ---- attention workgroups -------------------------------------------------
  // this wave's run of batches: nbat / 8 each, one more for the first
  // nbat % 8 waves
  const int start = split * split_len;
  const int nbat = split_len >> 4;
  const int nb_base = nbat / kWaves, nb_rem = nbat % kWaves;
  const int nb_w = nb_base + (wave < nb_rem ? 1 : 0);
  const int wbase = start + 16 * (wave * nb_base + (wave < nb_rem ? wave : nb_rem));
  // Grids of one round (at most one workgroup per CU) are bound by latency:
  // their loads are addressed from the split range clamped to max_seq_len
  // and go out before the length is read.  Grids of several rounds read the
  // length first and skip splits past it, whose loads would take bandwidth
  // from the other workgroups.
  int seq0 = 0;
  int lim = start + split_len < max_seq_len ? start + split_len : max_seq_len;
  // start of the wave's last batch before lim (the clamp of the loads):
  // lim <= max_seq_len <= capacity, a multiple of 16, so every loaded batch
  // lies in the row (in a mapped or the fallback page when paged)
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
      // nothing to attend: an empty partial (m = -inf) for the merge, or a
      // zero output row for an empty sequence
      if (n_parts > 1) {
        if (tid < kHeads)
          part_bg[static_cast<int64_t>(split) * (kHeads * kPart) + tid * kPart] = -INFINITY;
      } else {
        for (int e = tid; e < kHeads * kDim; e += kThreads) out_bg[e] = 0.f;
      }
      return;
    }
    lim = lim < seq_w ? lim : seq_w;
    clamp16 = last_batch(lim);
  }
  // paged: each batch's record delta (its page's record base minus the
  // page's first logical position; page 0 for an invalid page index).  All
  // NB table entries are read before any is used, and an invalid entry is
  // replaced by a select, so the reads go out together (one round trip).
  // In grids of several rounds they follow the length read: issued beside
  // it, they would hold every empty split until they return.
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
  const float* kn = k_norms + row;
  const float* vn = v_norms + row;

  // ---- the cache loads (keys and scales now, values as the scores proceed)
  uint32_t kw[NB][kBits], vw[NB][kBits];
  f32x4_t ksl, vsl;
  load_keys<NB, kPaged, kBits>(kc, kn, vn, dlt, wbase, clamp16, lane, col, grp, kw, ksl, vsl);
  // the word of the value window of lane u = col (see value_pairs)
  int vdw;
  uint32_t vsh;
  if constexpr (kBits == 3) {
    vdw = (3 * col) / 4 < 10 ? (3 * col) / 4 : 10;
    vsh = static_cast<uint32_t>(8 * (3 * col - 4 * vdw));   // 0..40
  } else if constexpr (kBits == 4) {
    vdw = col;
    vsh = 0;
  } else {
    vdw = col >> 1;
    vsh = static_cast<uint32_t>(16 * (col & 1));
  }

  // one-round grids: the length, read once the loads are in flight
  if constexpr (!kWide) seq0 = seq_lens[b];
  const int seq = seq0 < 0 ? 0 : (seq0 > max_seq_len ? max_seq_len : seq0);
  const int end = seq < start + split_len ? seq : start + split_len;
  int nvalid = end - wbase;   // this wave's positions (may be <= 0)
  nvalid = nvalid < 16 * nb_w ? nvalid : 16 * nb_w;

  // ---- while the loads fly: LUT and the rotated query --------------------
  if (tid < kLut) {
    constexpr int kMask = (1 << kBits) - 1;
    const uint32_t lo =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid & kMask)));
    const uint32_t hi =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid >> kBits)));
    lut[tid] = lo | (hi << 16);
  }
  // the 32 blocks of a head are 32 consecutive lanes of one wave, so the
  // rotation needs no barrier
  if (tid < kRotThreads) {
    const f32x4_t y = rotate_forward(qv, ql, qr, qblk, kInvSqrtDim * qscale);
    // fp16 operands are kept in the normal range by an exact power-of-two
    // scale per head: the largest rotated entry is brought below 2^14 (hi
    // and lo parts both normal) and the scale is undone on the scores
    int qexp = 0;
    const float am = group32_max(
        fmaxf(fmaxf(fabsf(y[0]), fabsf(y[1])), fmaxf(fabsf(y[2]), fabsf(y[3]))));
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
    attend_wave<NB, NB, true, kWide, kPaged, kBits>(kw, vw, vc, koff, tb, dlt, stage[wave], qb,
                                                    lut, col, grp, nvalid, vdw, vsh, qdown,
                                                    m_run, l_run, vmax, o_acc);
  else if (NB > 1 && nvalid == 16 * (NB - 1))
    attend_wave<NB, (NB > 1 ? NB - 1 : 1), true, kWide, kPaged, kBits>(
        kw, vw, vc, koff, tb, dlt, stage[wave], qb, lut, col, grp, nvalid, vdw, vsh, qdown,
        m_run, l_run, vmax, o_acc);
  else if (nvalid > 0)
    attend_wave<NB, NB, false, kWide, kPaged, kBits>(kw, vw, vc, koff, tb, dlt, stage[wave], qb,
                                                     lut, col, grp, nvalid, vdw, vsh, qdown,
                                                     m_run, l_run, vmax, o_acc);

  // ---- merge the 8 waves in LDS ---------------------------------------------
  lds_barrier();   // every wave is done with its staging area
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
  // (head, block) as in the query rotation.  A workgroup with nothing to
  // attend (split at or past the length) ends with M = -inf, L = 0, O = 0.
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
    *reinterpret_cast<f32x4_t*>(out_bg + mh * kDim + md) = o;
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

// Multi-token decode (speculative verification): kT query tokens per
// sequence over the same cache, token t attending positions before
// seq - kT + 1 + t (causal among the new tokens, which the caller has
// already compressed into the last kT positions).  Same grid, split plan,
// loads and record decoding as decode_g8_kernel on 3-bit records: every
// batch of keys and values is decoded once and feeds kT sets of matrix
// instructions (the QK B operand of token t is read from LDS per batch).  The
// softmax is two-phase as in decode_g8_kernel: all scores of every token
// first (kept in registers), one max per token and head, then the weights
// and values.  Partials per (split, token, head); the merge kernel takes the
// token axis.
template <int NB, bool kWide, int kT>
__global__ __launch_bounds__(kThreads) void decode_g8_multi_kernel(
    const float* __restrict__ q, const uint8_t* __restrict__ k_codes,
    const float* __restrict__ k_norms, const uint8_t* __restrict__ v_codes,
    const float* __restrict__ v_norms, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ quats, float* __restrict__ partials, float* __restrict__ out,
    int64_t capacity, int max_seq_len, int n_kv_heads, int n_splits, int split_len, float qscale,
    Codebook cb) {
  static_assert(kT >= 2 && kT <= 4, "2 to 4 tokens");
  struct Smem {
    uint32_t lut[64];
    uint32_t qop[kT][2][kHeads][kQRowWords];
    int qexp[kT][kHeads];
    float wave_ml[kWaves][2][kHeads];
    union {
      WaveStage stage[kWaves];
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
  float* part_bg = partials + static_cast<int64_t>(bg) * n_splits * kT * (kHeads * kPart);
  const int64_t row = static_cast<int64_t>(bg) * capacity;
  const uint8_t* kc = k_codes + row * kRecordBytes;
  const uint8_t* vc = v_codes + row * kRecordBytes;

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
      if (n_splits > 1) {
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
  int64_t dlt[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) dlt[i] = 0;
  uint32_t kw[NB][3], vw[NB][3];
  f32x4_t ksl, vsl;
  load_keys<NB, false, 3>(kc, kn, vn, dlt, wbase, clamp16, lane, col, grp, kw, ksl, vsl);
  const uint32_t koff = static_cast<uint32_t>(col * kRecordBytes + 12 * grp);
  int tb[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) tb[i] = wbase + 16 * i < clamp16 ? wbase + 16 * i : clamp16;
  // every value batch goes out behind the keys
#pragma unroll
  for (int i = 0; i < NB; ++i) load_value_batch<3>(vc, tb[i], koff, vw[i]);
  const int vdw = (3 * col) / 4 < 10 ? (3 * col) / 4 : 10;
  const uint32_t vsh = static_cast<uint32_t>(8 * (3 * col - 4 * vdw));

  if constexpr (!kWide) seq0 = seq_lens[b];
  const int seq = seq0 < 0 ? 0 : (seq0 > max_seq_len ? max_seq_len : seq0);
  // positions of this wave each token attends (may be <= 0)
  int nv[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    int st = seq - (kT - 1 - t);
    st = st > 0 ? st : 0;
    const int end = st < start + split_len ? st : start + split_len;
    int n = end - wbase;
    nv[t] = n < 16 * nb_w ? n : 16 * nb_w;
  }
  const int nvalid = nv[kT - 1];

  // ---- while the loads fly: LUT and the rotated queries --------------------
  if (tid < 64) {
    const uint32_t lo =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid & 7)));
    const uint32_t hi =
        __builtin_bit_cast(uint16_t, static_cast<_Float16>(codebook_level(cb, tid >> 3)));
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
  WaveStage& st = sm.stage[wave];
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
  // kT tokens kept in registers; one max per token and head afterwards
  float m_run[kT], l_run[kT];
  f32x4_t sc[kT][NB];
#pragma unroll
  for (int t = 0; t < kT; ++t) m_run[t] = -INFINITY;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (16 * i >= nvalid) break;
    u32x4_t a[4];
    key_pairs<3>(lut, kw[i], a);
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
      f32x4_t x = acc * ks;
#pragma unroll
      for (int r = 0; r < 4; ++r) x[r] = (16 * i + 4 * grp + r < nv[t]) ? x[r] : -INFINITY;
      sc[t][i] = x;
      m_run[t] = fmaxf(fmaxf(m_run[t], fmaxf(x[0], x[1])), fmaxf(x[2], x[3]));
    }
  }
#pragma unroll
  for (int t = 0; t < kT; ++t) m_run[t] = wave_max(m_run[t]);

  // phase 2 (Table 2 B, C): value records of all batches to the stage behind
  // one fence, then per batch the decoded values feed every token's weights
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (16 * i >= nvalid) break;
#pragma unroll
    for (int j = 0; j < 3; ++j) st.rec[i][col * kRecStride + 3 * grp + j] = vw[i][j];
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
  const uint32_t slot_shift = (col >= 8) ? 16u : 0u;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (16 * i >= nvalid) break;
    u32x4_t vb[4];
    value_pairs<3>(lut, st.rec[i], grp, vdw, vsh, vb);
    const f32x4_t wv = st.vs[4 * i + grp];   // 0 past the last token's length
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      u32x4_t pw_hi, pw_lo;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[t][i][r], qdown[t], mq[t]));
        l_run[t] += e;
        const float pf = e * wv[r];
        const _Float16 ph = static_cast<_Float16>(pf);
        const _Float16 pl = static_cast<_Float16>(pf - static_cast<float>(ph));
        pw_hi[r] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, ph)) << slot_shift;
        pw_lo[r] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, pl)) << slot_shift;
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        o_acc[t][nb] = mfma(pw_hi, vb[nb], o_acc[t][nb]);
        o_acc[t][nb] = mfma(pw_lo, vb[nb], o_acc[t][nb]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    l_run[t] = wave_sum(l_run[t]);
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
      if (n_splits == 1) {
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

// Merge of the split partials of one (sequence b, query head h): grid
// (query head, sequence), one 256-thread workgroup each; thread (sg, dq)
// takes partials sg, sg + 8, ... and dims 4 dq .. 4 dq + 3, with up to 8
// partials' loads in flight per thread.  Then o = sum_s c_s O_s / sum_s c_s
// l_s with c_s = 2^(m_s - max m), and the single inverse rotation.  Splits
// with nothing to attend carry m = -inf (their other entries are never read),
// so the merge needs no sequence length.  kAppend: the last of the n_parts
// partials is the new token's, and workgroup (b, head 0) then advances
// seq_lens[b] past the token the decode kernel appended.
//
// kTok > 1 (multi-token decode): the partials of each split hold kTok
// tokens' rows; grid (query head, sequence x token), output row (b, t).
template <bool kAppend, int kTok = 1>
__global__ __launch_bounds__(kMergeThreads) void merge_g8_kernel(
    const float* __restrict__ partials, const float* __restrict__ quats, float* __restrict__ out,
    int n_kv_heads, int n_parts, int32_t* __restrict__ seq_lens, int64_t capacity) {
  static_assert(kTok == 1 || !kAppend, "the fused step decodes one token");
  constexpr int kUnroll = 8;   // 8 x 8 = 64 splits per pass, all loads in flight
  __shared__ __attribute__((aligned(16))) float red_o[8][kDim];
  __shared__ float red_m[8], red_l[8];
  const int tid = threadIdx.x;
  const int n_q_heads = n_kv_heads * kHeads;
  const int h = blockIdx.x;
  const int bt = blockIdx.y;   // sequence (x token)
  const int b = kTok == 1 ? bt : bt / kTok;
  const int tok = kTok == 1 ? 0 : bt % kTok;
  const int g = h / kHeads, hh = h % kHeads;
  int seq0 = 0;
  if (kAppend && h == 0 && tid == 0) seq0 = seq_lens[b];
  const int sg = tid >> 5, dq = tid & 31;
  constexpr int kSplitStride = kTok * kHeads * kPart;
  const float* base = partials +
                      (static_cast<int64_t>(b * n_kv_heads + g) * n_parts * kTok + tok) *
                          (kHeads * kPart) +
                      hh * kPart;
  // block parameters for the inverse rotation (threads 0..31: block tid)
  const f32x4_t* qg =
      reinterpret_cast<const f32x4_t*>(quats + static_cast<int64_t>(g) * kQuatFloats + 8 * dq);
  const f32x4_t ql = qg[0], qr = qg[1];
  float M = -INFINITY, L = 0.f;
  f32x4_t O = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int s0 = sg; s0 < n_parts; s0 += 8 * kUnroll) {
    float mv[kUnroll], lv[kUnroll];
    f32x2_t mlv[kUnroll];
    f32x4_t ov[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int s = s0 + 8 * u;
      const int sc = s < n_parts ? s : s0;
      const float* p = base + static_cast<int64_t>(sc) * kSplitStride;
      mlv[u] = *reinterpret_cast<const f32x2_t*>(p);   // (m, l)
      ov[u] = *reinterpret_cast<const f32x4_t*>(p + 2 + 4 * dq);
    }
    // every load of the pass is issued before the first use
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      mv[u] = s0 + 8 * u < n_parts ? mlv[u][0] : -INFINITY;
      lv[u] = mlv[u][1];
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) Mn = fmaxf(Mn, mv[u]);
    const float cM = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    L *= cM;
    O *= cM;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      // an empty split's l and O were never written: select, do not scale
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
  // lanes 0..31 of wave 0: block tid of the head, divided by the sum, then
  // the inverse rotation in registers
  if (tid < 32) {
    f32x4_t o = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      o += *reinterpret_cast<const f32x4_t*>(&red_o[j][4 * tid]);
      l += red_l[j];
    }
    // an empty sequence (every split empty) gives a zero row
    const f32x4_t r = l > 0.f ? rotate_inverse(o * (1.0f / l), ql, qr, tid)
                              : f32x4_t{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4_t*>(out + (static_cast<int64_t>(bt) * n_q_heads + h) * kDim +
                                4 * tid) = r;
  }
  if (kAppend && h == 0 && tid == 0 && seq0 >= 0 && seq0 < capacity) seq_lens[b] = seq0 + 1;
}

}  // namespace

// Split plan of the group-8 path: splits per (sequence, KV head) and their
// length (a multiple of 16).  A workgroup covers at most 8 waves x 5 batches
// x 16 = 640 positions, capped at 560 so that long contexts keep more
// splits; while the grid is small (<= 4 rounds of one workgroup per CU) the
// split count is raised so that the grid, with the fused step's append
// workgroup per (sequence, KV head), fills whole rounds, but a split keeps at
// least one batch per wave.
void g8_plan(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len, int* nb,
             int64_t* n_splits, int64_t* split_len) {
  constexpr int64_t kCus = 256;
  constexpr int64_t kMaxLen = 560;
  const int64_t t = max_seq_len > 0 ? max_seq_len : 1;
  const int64_t bg = batch * n_kv_heads > 0 ? batch * n_kv_heads : 1;
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
                            const float* quats, int64_t batch, int64_t n_kv_heads, float scale,
                            float* out, float* partials, const StepAppend* append,
                            const PageTable* pages, int bits, hipStream_t stream) {
  if (bits != 3 && (append || pages)) return hipErrorInvalidValue;
  // partials per (sequence, KV head): the splits, and the fused step's new
  // token
  const int64_t n_parts = append ? n_splits + 1 : n_splits;
  const dim3 grid(static_cast<unsigned>(n_parts), static_cast<unsigned>(n_kv_heads),
                  static_cast<unsigned>(batch)),
      block(kThreads);
  // Up to 5 batches per wave the kernel needs at most 128 VGPRs and ~55 KB of
  // LDS, so two workgroups fit on a CU: a grid of several rounds then runs
  // one workgroup's prologue and merge beside another's attention.  A grid
  // of at most one round would instead pile two workgroups on some CUs and
  // leave others idle; padding its LDS request keeps one workgroup per CU.
  constexpr int64_t kCus = 256;
  const bool wide = n_parts * n_kv_heads * batch > kCus;
  const size_t lds_pad = wide ? 0 : kOneWorkgroupPadBytes;
  const float qscale = scale * kLog2e;
  const void* k_new = append ? append->k_new : nullptr;
  const void* v_new = append ? append->v_new : nullptr;
  const int new_f16 = append ? append->f16 : 0;
  int32_t* status = append ? append->status : nullptr;
  const PageTable pt = pages ? *pages : PageTable{nullptr, 0, 4, 1};
#define IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, PAGED_, BITS_)                                     \
  hipLaunchKernelGGL((decode_g8_kernel<NB_, APP_, WIDE_, PAGED_, BITS_>), grid, block, lds_pad, \
                     stream, q, k_codes, k_norms, v_codes, v_norms, seq_lens, quats, partials,  \
                     out, capacity, static_cast<int>(max_seq_len),                              \
                     static_cast<int>(n_kv_heads), static_cast<int>(n_splits),                  \
                     static_cast<int>(split_len), qscale, codebook_b<BITS_>(), k_new, v_new,    \
                     new_f16, status, pt)
#define IQ_LAUNCH_G8_W(NB_, APP_, WIDE_)                \
  if (pages) {                                          \
    IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, true, 3);        \
  } else if (APP_ || bits == 3) {                       \
    IQ_LAUNCH_G8_WPB(NB_, APP_, WIDE_, false, 3);       \
  } else if (bits == 2) {                               \
    IQ_LAUNCH_G8_WPB(NB_, false, WIDE_, false, 2);      \
  } else {                                              \
    IQ_LAUNCH_G8_WPB(NB_, false, WIDE_, false, 4);      \
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
  if (append) {
    IQ_LAUNCH_G8_NB(true)
  } else {
    IQ_LAUNCH_G8_NB(false)
  }
#undef IQ_LAUNCH_G8_NB
#undef IQ_LAUNCH_G8
#undef IQ_LAUNCH_G8_W
#undef IQ_LAUNCH_G8_WPB
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the partials of every (sequence, query head) merged by a second launch,
  // which in the fused step also advances the lengths
  if (n_parts > 1) {
    const dim3 mgrid(static_cast<unsigned>(n_kv_heads * kHeads), static_cast<unsigned>(batch));
    if (append)
      hipLaunchKernelGGL(merge_g8_kernel<true>, mgrid, dim3(kMergeThreads), 0, stream, partials,
                         quats, out, static_cast<int>(n_kv_heads), static_cast<int>(n_parts),
                         seq_lens, capacity);
    else
      hipLaunchKernelGGL(merge_g8_kernel<false>, mgrid, dim3(kMergeThreads), 0, stream, partials,
                         quats, out, static_cast<int>(n_kv_heads), static_cast<int>(n_parts),
                         seq_lens, capacity);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_decode_g8_multi(int nb, int64_t n_splits, int64_t split_len, int n_tok,
                                  const float* q, const uint8_t* k_codes, const float* k_norms,
                                  const uint8_t* v_codes, const float* v_norms,
                                  const int32_t* seq_lens, int64_t capacity,
                                  int64_t max_seq_len, const float* quats, int64_t batch,
                                  int64_t n_kv_heads, float scale, float* out, float* partials,
                                  hipStream_t stream) {
  if (n_tok < 2 || n_tok > 4) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(n_splits), static_cast<unsigned>(n_kv_heads),
                  static_cast<unsigned>(batch)),
      block(kThreads);
  constexpr int64_t kCus = 256;
  const bool wide = n_splits * n_kv_heads * batch > kCus;
  const size_t lds_pad = wide ? 0 : kOneWorkgroupPadBytes;
  const float qscale = scale * kLog2e;
  const Codebook& cb = codebook();
#define IQ_LAUNCH_MT(NB_, WIDE_, T_)                                                            \
  hipLaunchKernelGGL((decode_g8_multi_kernel<NB_, WIDE_, T_>), grid, block, lds_pad, stream, q, \
                     k_codes, k_norms, v_codes, v_norms, seq_lens, quats, partials, out,        \
                     capacity, static_cast<int>(max_seq_len), static_cast<int>(n_kv_heads),     \
                     static_cast<int>(n_splits), static_cast<int>(split_len), qscale, cb)
#define IQ_LAUNCH_MT_W(NB_, T_)       \
  if (wide) {                         \
    IQ_LAUNCH_MT(NB_, true, T_);      \
  } else {                            \
    IQ_LAUNCH_MT(NB_, false, T_);     \
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
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_splits == 1) return e;
  const dim3 mgrid(static_cast<unsigned>(n_kv_heads * kHeads),
                   static_cast<unsigned>(batch * n_tok));
#define IQ_LAUNCH_MT_MERGE(T_)                                                                 \
  hipLaunchKernelGGL((merge_g8_kernel<false, T_>), mgrid, dim3(kMergeThreads), 0, stream,       \
                     partials, quats, out, static_cast<int>(n_kv_heads),                        \
                     static_cast<int>(n_splits), nullptr, capacity)
  if (n_tok == 2) IQ_LAUNCH_MT_MERGE(2);
  else if (n_tok == 3) IQ_LAUNCH_MT_MERGE(3);
  else IQ_LAUNCH_MT_MERGE(4);
#undef IQ_LAUNCH_MT_MERGE
  return hipGetLastError();
}

}  // namespace iq
