// Device-side building blocks of the IsoQuant rotation and quantizer
// (Sec. 3.2 Steps 2-4, Sec. 3.3, App. B), shared by the kernels of libisoquant.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "iq_internal.h"

namespace iq {

// 4 x 4 matrix (row-major) of the block map v -> q_L v conj(q_R), with the
// block's components (v0, v1, v2, v3) read as the quaternion v0 + v1 i + v2 j
// + v3 k.  Built as L(q_L) R(conj q_R): L(p) is left multiplication by p,
// R(p) right multiplication by p, both written out from the Hamilton
// product.  qv = (q_L.w, q_L.x, q_L.y, q_L.z, q_R.w, q_R.x, q_R.y, q_R.z).
__device__ __forceinline__ void so4_matrix(const float* qv, float (&m)[4][4]) {
  const float p0 = qv[0], p1 = qv[1], p2 = qv[2], p3 = qv[3];
  const float r0 = qv[4], r1 = -qv[5], r2 = -qv[6], r3 = -qv[7];  // conj(q_R)
  const float l[4][4] = {{p0, -p1, -p2, -p3},
                         {p1, p0, -p3, p2},
                         {p2, p3, p0, -p1},
                         {p3, -p2, p1, p0}};
  const float r[4][4] = {{r0, -r1, -r2, -r3},
                         {r1, r0, r3, -r2},
                         {r2, -r3, r0, r1},
                         {r3, r2, -r1, r0}};
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      m[i][j] = l[i][0] * r[0][j] + l[i][1] * r[1][j] + l[i][2] * r[2][j] + l[i][3] * r[3][j];
}

// Unnormalized 4-point Walsh-Hadamard butterfly on bits 0 and 1 of a block.
__device__ __forceinline__ void wht4(float& a, float& b, float& c, float& d) {
  const float s0 = a + b, d0 = a - b, s1 = c + d, d1 = c - d;
  a = s0 + s1;
  b = d0 + d1;
  c = s0 - s1;
  d = d0 - d1;
}

// M' = M H_4 (H_4 unnormalized Sylvester, symmetric): each row of M goes
// through the 4-point butterfly.  Since the Walsh-Hadamard transform factors
// over index bits, H_128 = (H_32 on bits 2..6)(H_4 on bits 0..1) and the two
// factors commute, so R x = diag(M_i H_4) (H_32 (x) I_4) x / sqrt(128).
__device__ __forceinline__ void so4_matrix_h4(const float* qv, float (&m)[4][4]) {
  so4_matrix(qv, m);
#pragma unroll
  for (int i = 0; i < 4; ++i) wht4(m[i][0], m[i][1], m[i][2], m[i][3]);
}

// Level i (0 .. 2^b - 1) of a codebook held in kernel arguments.  A select chain
// over compile-time indices: indexing the argument struct with a lane value
// would turn into a memory load, whose wait would also wait for every load
// issued before it.
template <int kBits>
__device__ __forceinline__ float codebook_level(const CodebookB<kBits>& cb, int i) {
  // readfirstlane pins each level to a register value, so that the selects
  // are not folded back into an address computation
  constexpr int n = 1 << kBits;
  float lv[n];
#pragma unroll
  for (int j = 0; j < n; ++j)
    lv[j] = __builtin_bit_cast(
        float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, cb.level[j])));
  float v = lv[0];
#pragma unroll
  for (int j = 1; j < n; ++j) v = (i == j) ? lv[j] : v;
  return v;
}

// Code of y for ascending thresholds t: #{j : t[j] <= y}, by a three-level
// binary search (ties go to the upper level; NaN gives 0).
__device__ __forceinline__ uint32_t quantize3(float y, const float (&t)[7]) {
  const bool b2 = y >= t[3];
  const float tb = b2 ? t[5] : t[1];
  const bool b1 = y >= tb;
  const float tc = b2 ? (b1 ? t[6] : t[4]) : (b1 ? t[2] : t[0]);
  const bool b0 = y >= tc;
  return (b2 ? 4u : 0u) | (b1 ? 2u : 0u) | (b0 ? 1u : 0u);
}

// OR a 3-bit code into a 12-word record image at code index i (LSB-first bit
// string, code i at bits 3i .. 3i+2).  i is a compile-time constant after
// unrolling, so the word array stays in registers.
__device__ __forceinline__ void put_code(uint32_t (&w)[kRecordWords], int i, uint32_t code) {
  const int bit = 3 * i;
  const int word = bit >> 5, off = bit & 31;
  w[word] |= code << off;
  if (off > 29) w[word + 1] |= code >> (32 - off);
}

// Value of lane (lane ^ kM) within the lane's group of 32 lanes (kM < 32):
// quad permutations through DPP for 1 and 2, the swizzle unit otherwise.
template <int kM>
__device__ __forceinline__ float xor_lane(float v) {
  const int x = __builtin_bit_cast(int, v);
  // every lane reads a lane inside its own row, so bound_ctrl never applies;
  // setting it lets the compiler fold the move into the instruction using it
  if constexpr (kM == 1) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, true));
  } else if constexpr (kM == 2) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, true));
  } else if constexpr (kM == 8) {
    // rotation by 8 inside each row of 16 lanes (row_ror:8) is xor 8
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, true));
  } else {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(x, (kM << 10) | 0x1F));
  }
}

// Value of lane (lane ^ m) for any m < 64 (xor 32 through the permute unit).
template <int kM>
__device__ __forceinline__ float xor_lane64(float v) {
  if constexpr (kM < 32) {
    return xor_lane<kM>(v);
  } else {
    return __shfl_xor(v, kM);
  }
}

// ---- one vector per wave -------------------------------------------------
// Used where only a few vectors are compressed at once (the per-step append):
// the 128 dims are spread over the 64 lanes (lane l holds dims 2l, 2l+1), so
// the serial chain is short.

template <int kM>
__device__ __forceinline__ double xor_lane64_f64(double v) {
  const float2 p = __builtin_bit_cast(float2, v);
  return __builtin_bit_cast(double, float2{xor_lane64<kM>(p.x), xor_lane64<kM>(p.y)});
}

// One butterfly stage of the cross-lane Walsh-Hadamard transform (partner
// lane l ^ kM), on the lane's two partial sums.
template <int kM>
__device__ __forceinline__ void wave_butterfly(float& a, float& c, int lane) {
  const float pa = xor_lane64<kM>(a), pc = xor_lane64<kM>(c);
  const bool upper = (lane & kM) != 0;
  a = upper ? pa - a : a + pa;
  c = upper ? pc - c : c + pc;
}

// dims 2 lane, 2 lane + 1 of a 128-dim vector of fp32 or fp16
__device__ __forceinline__ void load_pair(const float* src, int lane, float& a, float& b) {
  const float2 f = reinterpret_cast<const float2*>(src)[lane];
  a = f.x;
  b = f.y;
}
__device__ __forceinline__ void load_pair(const __half* src, int lane, float& a, float& b) {
  const uint32_t w = reinterpret_cast<const uint32_t*>(src)[lane];
  a = __half2float(__ushort_as_half(static_cast<unsigned short>(w & 0xFFFFu)));
  b = __half2float(__ushort_as_half(static_cast<unsigned short>(w >> 16)));
}

struct WaveCode {
  uint32_t word;   // record word `lane` (meaningful in lanes 0 .. 4b - 1)
  float scale;     // s = ||x||_2
};

// Algorithm 1 for one vector held by one wave (lane l: x0 = x[2l],
// x1 = x[2l+1]); qp holds (q_L, q_R) of SO(4) block l / 2 of the vector's
// head.  Every lane of the wave must take part.
//   Step 1: fp64 sum of squares, wave reduction.
//   Step 2: H_128 as 7 butterfly stages (stage 1 in-lane, stages 2..7 with
//           the partner lane l ^ (st/2)), then the SO(4) block of the lane
//           pair (2 blk, 2 blk + 1).
//   Step 3: codes against the thresholds scaled by s sqrt(128).
//   Step 4: lane w < 4b gathers the 2b-bit fields (the lanes' code pairs)
//           overlapping record word w (at most 7 at b = 3, where fields
//           straddle words; 8 or 4 whole fields at b = 2 or 4).
template <int kBits>
__device__ __forceinline__ WaveCode compress_vector_wave(float x0, float x1, const float* qp,
                                                        const CodebookB<kBits>& cb, int lane) {
  constexpr int kThr = (1 << kBits) - 1;
  double ss = static_cast<double>(x0) * static_cast<double>(x0) +
              static_cast<double>(x1) * static_cast<double>(x1);
  ss += xor_lane64_f64<1>(ss);
  ss += xor_lane64_f64<2>(ss);
  ss += xor_lane64_f64<4>(ss);
  ss += xor_lane64_f64<8>(ss);
  ss += xor_lane64_f64<16>(ss);
  ss += xor_lane64_f64<32>(ss);
  const double s = sqrt(ss);
  float a = x0 + x1, c = x0 - x1;   // stage 1 (dims 2l, 2l+1)
  wave_butterfly<1>(a, c, lane);
  wave_butterfly<2>(a, c, lane);
  wave_butterfly<4>(a, c, lane);
  wave_butterfly<8>(a, c, lane);
  wave_butterfly<16>(a, c, lane);
  wave_butterfly<32>(a, c, lane);
  // block blk = lane / 2 covers dims 4 blk .. 4 blk + 3 = (a, c) of lanes
  // 2 blk and 2 blk + 1
  const float oa = xor_lane<1>(a), oc = xor_lane<1>(c);
  const bool odd = lane & 1;
  const float z0 = odd ? oa : a, z1 = odd ? oc : c, z2 = odd ? a : oa, z3 = odd ? c : oc;
  float m[4][4];
  so4_matrix(qp, m);
  const int r0 = odd ? 2 : 0;
  const float y0 = m[r0][0] * z0 + m[r0][1] * z1 + m[r0][2] * z2 + m[r0][3] * z3;
  const float y1 = m[r0 + 1][0] * z0 + m[r0 + 1][1] * z1 + m[r0 + 1][2] * z2 + m[r0 + 1][3] * z3;
  float thr[kThr];
  if (ss > 0.0) {
    const double sc = s * 11.313708498984760390;   // s sqrt(128)
#pragma unroll
    for (int j = 0; j < kThr; ++j)
      thr[j] = static_cast<float>(static_cast<double>(cb.thr[j]) * sc);
  } else {
#pragma unroll
    for (int j = 0; j < kThr; ++j) thr[j] = cb.thr[j];
  }
  uint32_t fld;
  if constexpr (kBits == 3) {
    fld = quantize3(y0, thr) | (quantize3(y1, thr) << 3);
  } else {
    // #{j : t_j <= y} as a plain count (ties upward, NaN gives 0)
    uint32_t c0 = 0u, c1 = 0u;
#pragma unroll
    for (int j = 0; j < kThr; ++j) {
      c0 += y0 >= thr[j] ? 1u : 0u;
      c1 += y1 >= thr[j] ? 1u : 0u;
    }
    fld = c0 | (c1 << kBits);
  }
  constexpr int kFw = 2 * kBits;              // field width (a lane's pair)
  constexpr int kFields = 32 / kFw + 2;        // fields overlapping a word
  const int w = lane < 4 * kBits ? lane : 0;
  const int f_lo = (32 * w) / kFw;
  uint32_t word = 0u;
#pragma unroll
  for (int k = 0; k < kFields; ++k) {
    const int f = f_lo + k;
    const uint32_t v = static_cast<uint32_t>(__shfl(static_cast<int>(fld), f & 63));
    const int sh = kFw * f - 32 * w;
    if (f < 64 && sh < 32) word |= sh >= 0 ? (v << sh) : (v >> (-sh));
  }
  return WaveCode{word, static_cast<float>(s)};
}

}  // namespace iq
