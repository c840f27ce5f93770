// Device helpers of the group-8 decode kernels (iq_decode_g8.hip, the
// single-token kernel and the fused step; iq_decode_multi.hip, multi-token
// decode), and the split merge kernel both launch: constants, the matrix
// instruction, SDWA field selects, LDS barriers, cross-lane reductions, the
// forward and inverse rotation in registers, the per-wave staging layout,
// the cache loads and the decoding of record slices into operand dwords.
// Internal to the library.
#pragma once

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
constexpr int kRopeDim = 64;              // positional key / query part (RoPE sub-block)
constexpr int kRopeRowWords = kRopeDim / 2 + 4;   // its fp16-pair row, padded (36 words)
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
// LDS (4b words): codes at bits b d .. b d + 4b - 1, two 2b-bit fields looked
// up in the fp16 pair table.
template <int kBits = 3>
__device__ __forceinline__ f32x4_t decode_record_dims(const uint32_t* rec, const uint32_t* lut,
                                                      int d) {
  constexpr uint32_t kMask = (1u << (2 * kBits)) - 1;
  const int bit = kBits * d, w = bit >> 5, off = bit & 31;
  const uint32_t lo = rec[w];
  const uint32_t hi = w + 1 < 4 * kBits ? rec[w + 1] : 0u;
  const uint32_t bits = __builtin_amdgcn_alignbit(hi, lo, off);
  const uint32_t p0 = lut[bits & kMask], p1 = lut[(bits >> (2 * kBits)) & kMask];
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
// dlt[j] for a per-lane j < NB, as a chain of selects on compile-time
// indices (an index that is a loop variable before unrolling can leave the
// array in scratch memory when registers are tight).
template <int I, int NB>
__device__ __forceinline__ int64_t pick_batch(const int64_t (&dlt)[NB], int j) {
  if constexpr (I == NB - 1)
    return dlt[I];
  else
    return j == I ? dlt[I] : pick_batch<I + 1, NB>(dlt, j);
}

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
    if constexpr (kPaged) d = pick_batch<0, NB>(dlt, jb);
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
// 3 bits: bytes 3u .. 3u + 2 of the record, at bit vsh (0, 8, 16 or 24) of
// words vdw, vdw + 1 (vdw = 3u / 4; for u = 15 the second word is the
// staged row's padding word, whose bits are never used); 4 bits: word u
// (vdw = u); 2 bits: the half of word u / 2 (vdw) at bit vsh = 16 (u % 2).
template <int kBits>
__device__ __forceinline__ void value_pairs(const uint32_t* lut, const uint32_t* rec, int grp,
                                            int vdw, uint32_t vsh, u32x4_t (&vb)[4]) {
  constexpr int kStride = rec_stride<kBits>();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t* wp = rec + (4 * grp + r) * kStride + vdw;
    if constexpr (kBits == 3) {
      // the 32-bit window starting at byte 3u (one funnel shift of the word
      // pair); fields at bits 0, 6, 12, 18 of it: bits 0 and 18 are byte
      // selects of it, bits 6 and 12 of the window shifted right by 4
      const uint32_t lo = wp[0], hi = wp[1];
      const uint32_t win = __builtin_amdgcn_alignbit(hi, lo, vsh);
      const uint32_t wu = __builtin_amdgcn_alignbit(hi, lo, vsh + 4);
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

// Merge of the split partials of one (sequence b, query head h): grid
// (query head, sequence), one 256-thread workgroup each; thread (sg, dq)
// takes partials sg, sg + 8, ... and dims 4 dq .. 4 dq + 3, with up to
// kUnroll partials' loads in flight per thread.  Then o = sum_s c_s O_s / sum_s c_s
// l_s with c_s = 2^(m_s - max m), and the single inverse rotation.  Splits
// with nothing to attend carry m = -inf (their other entries are never read),
// so the merge needs no sequence length.  kAppend: the last of the n_parts
// partials is the new token's, and workgroup (b, head 0) then advances
// seq_lens[b] past the token the decode kernel appended, unless that
// partial's l entry is negative (no room: nothing was written).
//
// kTok > 1 (multi-token decode): the partials of each split hold kTok
// tokens' rows; grid (query head, sequence x token), output row (b, t).
// With kAppend (the fused multi-token step) the last partial holds the new
// tokens' rows, and workgroup (b, token 0, head 0) advances seq_lens[b] by
// kTok.
// kAnyGroup: group query heads per KV head (1 .. 16); the partial rows are
// per (sequence, KV head, head group of 8), the layout of the decode
// kernels' grid.  Otherwise 8 (group is not read).
//
// kLive (grids of several rounds, whose decode workgroups skip the splits
// past a sequence's length): only the splits holding positions before
// min(seq_lens[b], max_seq_len) are read (ceil of that over split_len), and
// the new-token partial; the others were never written.  With kAppend the
// length is lens0[b], the one the decode kernel saw (seq_lens[b] may already
// be advanced by this launch's workgroup of head 0).
template <bool kAppend, int kTok = 1, bool kAnyGroup = false, bool kLive = false,
          int kUnroll = 8>
__global__ __launch_bounds__(kMergeThreads) void merge_g8_kernel(
    const float* __restrict__ partials, const float* __restrict__ quats, float* __restrict__ out,
    int n_kv_heads, int n_parts, int32_t* __restrict__ seq_lens, int64_t capacity, int group,
    int split_len = 0, int max_seq_len = 0, const int32_t* __restrict__ lens0 = nullptr) {
  static_assert(kTok == 1 || !kLive, "multi-token partials are read in full");
  // 8 x kUnroll splits per pass, all of a pass's loads in flight (rows of
  // more than 64 partials take passes of 256)
  __shared__ __attribute__((aligned(16))) float red_o[8][kDim];
  __shared__ float red_m[8], red_l[8];
  const int tid = threadIdx.x;
  const int gsize = kAnyGroup ? group : kHeads;
  const int n_q_heads = n_kv_heads * gsize;
  const int n_vg = (gsize + kHeads - 1) / kHeads;
  const int h = blockIdx.x;
  const int bt = blockIdx.y;   // sequence (x token)
  const int b = kTok == 1 ? bt : bt / kTok;
  const int tok = kTok == 1 ? 0 : bt % kTok;
  const int g = h / gsize, hr = h - g * gsize;
  const int hh = hr % kHeads;
  const int bgv = (b * n_kv_heads + g) * n_vg + hr / kHeads;   // the partial row
  int seq0 = 0;
  float written = 0.f;
  if (kAppend && h == 0 && tok == 0 && tid == 0) {
    seq0 = seq_lens[b];
    // the new-token partial (token 0) of KV head 0 (every KV head shares
    // the outcome)
    written = partials[(static_cast<int64_t>(b) * n_kv_heads * n_vg * n_parts + n_parts - 1) *
                           kTok * (kHeads * kPart) + 1];
  }
  const int sg = tid >> 5, dq = tid & 31;
  constexpr int kSplitStride = kTok * kHeads * kPart;
  const float* base = partials +
                      (static_cast<int64_t>(bgv) * n_parts * kTok + tok) * (kHeads * kPart) +
                      hh * kPart;
  // block parameters for the inverse rotation (threads 0..31: block tid)
  const f32x4_t* qg =
      reinterpret_cast<const f32x4_t*>(quats + static_cast<int64_t>(g) * kQuatFloats + 8 * dq);
  const f32x4_t ql = qg[0], qr = qg[1];
  float M = -INFINITY, L = 0.f;
  f32x4_t O = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // partials read: n_iter of them; with kLive the live splits, then (fused
  // step) the new token's at index n_parts - 1
  int n_iter = n_parts;
  if constexpr (kLive) {
    // the fused step: the length as the decode kernel read it (workgroup
    // (b, head 0) of this launch advances seq_lens[b])
    int seq = kAppend ? lens0[b] : seq_lens[b];
    seq = seq < 0 ? 0 : (seq > max_seq_len ? max_seq_len : seq);
    n_iter = (seq + split_len - 1) / split_len + (kAppend ? 1 : 0);
  }
  auto part_index = [&](int s) {
    return (kLive && kAppend && s == n_iter - 1) ? n_parts - 1 : s;
  };
  for (int s0 = sg; s0 < n_iter; s0 += 8 * kUnroll) {
    float mv[kUnroll], lv[kUnroll];
    f32x2_t mlv[kUnroll];
    f32x4_t ov[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int s = s0 + 8 * u;
      const int sc = part_index(s < n_iter ? s : s0);
      const float* p = base + static_cast<int64_t>(sc) * kSplitStride;
      mlv[u] = *reinterpret_cast<const f32x2_t*>(p);   // (m, l)
      ov[u] = *reinterpret_cast<const f32x4_t*>(p + 2 + 4 * dq);
    }
    // every load of the pass is issued before the first use
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      mv[u] = s0 + 8 * u < n_iter ? mlv[u][0] : -INFINITY;
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
  // combine the 8 split groups: each stores its (M, L, O) as it is, and
  // lanes 0..31 of wave 0 (block tid of the head) rescale them to the common
  // maximum while summing, divide by the sum and apply the inverse rotation
  // in registers
  *reinterpret_cast<f32x4_t*>(&red_o[sg][4 * dq]) = O;
  if (dq == 0) {
    red_m[sg] = M;
    red_l[sg] = L;
  }
  lds_barrier();
  if (tid < 32) {
    float Mt = red_m[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) Mt = fmaxf(Mt, red_m[j]);
    f32x4_t o = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float mj = red_m[j];
      const float c = (mj == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mj - Mt);
      o += c * *reinterpret_cast<const f32x4_t*>(&red_o[j][4 * tid]);
      l += c * red_l[j];
    }
    // an empty sequence (every split empty) gives a zero row
    const f32x4_t r = l > 0.f ? rotate_inverse(o * (1.0f / l), ql, qr, tid)
                              : f32x4_t{0.f, 0.f, 0.f, 0.f};
    *reinterpret_cast<f32x4_t*>(out + (static_cast<int64_t>(bt) * n_q_heads + h) * kDim +
                                4 * tid) = r;
  }
  if (kAppend && h == 0 && tok == 0 && tid == 0 && seq0 >= 0 && seq0 <= capacity - kTok &&
      written > 0.f)
    seq_lens[b] = seq0 + kTok;
}

}  // namespace
}  // namespace iq
