// Device-side building blocks of the IsoQuant rotation and quantizer
// (Sec. 3.2 Steps 2-4, Sec. 3.3, App. B), shared by the kernels of libisoquant.
#pragma once

#include <hip/hip_runtime.h>
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

}  // namespace iq
