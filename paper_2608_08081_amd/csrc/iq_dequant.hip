// Materialization of the packed cache: the "Dequant R^-1 -> FP16 tensors"
// stage of the reconstruct-then-compute pipeline (Sec. 1, Fig. 1 top), the
// baseline that compressed-space attention avoids.  gfx950.
//
// Per token: x_hat = s R^T C[code] with R = diag(M_i) H_128 / sqrt(128)
// (Eq. 2), so R^T = H_128 diag(M_i^T) / sqrt(128); H_128 factors over the
// index bits into H_4 (bits 0..1, inside an SO(4) block) and H_32 (bits 2..6,
// the block index), and the block-local part is the 4 x 4 matrix
// B_i = H_4 M_i^T:
//   z_i = B_i (C[code_4i], .., C[code_4i+3])     per block,
//   x_hat = s / sqrt(128) * (H_32 (x) I_4) z.
//
// Work decomposition: 8 lanes per token, 8 tokens per wave and pass.  Lane l
// takes chunk c = (l & 3) | ((l >> 1) & 4) of the token (dims 16c..16c+15 =
// blocks 4c..4c+3) for token slot ((l >> 2) & 1) | ((l >> 3) & 6).  Of the
// block index bits, bits 0..1 live inside the lane and bits 2..4 are chunk
// bits 0..2, i.e. lane bits 0, 1 and 3: H_32 is two in-lane butterfly stages
// and three cross-lane stages with partners l ^ 1, l ^ 2 and l ^ 8, all
// three DPP lane permutations.  Each lane keeps its 4 blocks' B_i in
// registers for the workgroup's whole token range, reads the 48 code bits of
// its chunk as two words, looks the codes up in a 64-entry LDS table of
// level pairs and writes its 16 outputs as 32 (fp16) or 64 (fp32)
// contiguous bytes, so the 8 lanes of a token write its row in one piece.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "iq_device.h"
#include "iq_internal.h"

namespace iq {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

constexpr int kDqWaves = 4;
constexpr int kDqThreads = 64 * kDqWaves;
constexpr int kDqPasses = 8;                              // passes of 8 tokens per wave
constexpr int kDqTokens = 8 * kDqWaves * kDqPasses;       // tokens per workgroup (256)
constexpr float kInvSqrtDim = 0.08838834764831845f;

// 4-point unnormalized Walsh-Hadamard butterfly
__device__ __forceinline__ void wht4v(float& a, float& b, float& c, float& d) {
  const float s0 = a + b, d0 = a - b, s1 = c + d, d1 = c - d;
  a = s0 + s1;
  b = d0 + d1;
  c = s0 - s1;
  d = d0 - d1;
}

// One cross-lane Walsh-Hadamard stage on the lane pair (l, l ^ kM) holding
// the same component of two blocks: the pair becomes (x_lo + x_up,
// x_lo - x_up).  Computed as a + sgn * partner with sgn = -1 in the upper
// lane, which leaves the upper lane's result negated; the negation is
// carried as a per-lane sign (the stages' partner lanes always carry the
// same sign as the lane itself, since each stage flips the sign of upper
// lanes only by a bit the later partners share) and removed with the final
// scaling.  One fused multiply-add per value and stage.
template <int kM>
__device__ __forceinline__ float xstage(float a, float sgn) {
  return __builtin_fmaf(xor_lane<kM>(a), sgn, a);
}

template <typename TOut>
__device__ __forceinline__ void store_chunk(TOut* dst, const float (&x)[16]);

template <>
__device__ __forceinline__ void store_chunk<__half>(__half* dst, const float (&x)[16]) {
  uint32_t w[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const __half2 h = __floats2half2_rn(x[2 * i], x[2 * i + 1]);
    w[i] = __builtin_bit_cast(uint32_t, h);
  }
  uint4* p = reinterpret_cast<uint4*>(dst);
  p[0] = uint4{w[0], w[1], w[2], w[3]};
  p[1] = uint4{w[4], w[5], w[6], w[7]};
}

template <>
__device__ __forceinline__ void store_chunk<float>(float* dst, const float (&x)[16]) {
  f32x4_t* p = reinterpret_cast<f32x4_t*>(dst);
#pragma unroll
  for (int i = 0; i < 4; ++i) p[i] = f32x4_t{x[4 * i], x[4 * i + 1], x[4 * i + 2], x[4 * i + 3]};
}

// Workgroup: (K|V side, sequence b, KV head g, 256-token chunk).  Tokens
// t0 .. t0 + 255 of the output come from cache positions src_offset + t;
// tokens at or past n_tokens, or whose cache position is at or past
// seq_lens[b] (when given), are not written.
template <typename TOut>
__global__ __launch_bounds__(kDqThreads) void dequant_kernel(
    const uint8_t* __restrict__ codes0, const float* __restrict__ norms0, TOut* __restrict__ out0,
    const uint8_t* __restrict__ codes1, const float* __restrict__ norms1, TOut* __restrict__ out1,
    const float* __restrict__ quats, const int32_t* __restrict__ seq_lens, int n_heads,
    int64_t n_bh, int64_t n_tokens, int64_t chunks, int64_t capacity, int64_t src_offset,
    Codebook cb) {
  __shared__ f32x2_t pair_tab[64];   // field f -> (C[f & 7], C[f >> 3])
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int64_t chunk = blockIdx.x % chunks;
  const int64_t rest = blockIdx.x / chunks;
  const int64_t bh = rest % n_bh;
  const int which = static_cast<int>(rest / n_bh);
  const int64_t b = bh / n_heads;
  const int g = static_cast<int>(bh % n_heads);
  const uint8_t* codes = which ? codes1 : codes0;
  const float* norms = which ? norms1 : norms0;
  TOut* out = which ? out1 : out0;

  // tokens of this workgroup that exist: [t0, t_end)
  int64_t t_end = n_tokens;
  if (seq_lens) {
    const int64_t lim = static_cast<int64_t>(seq_lens[b]) - src_offset;
    if (lim < t_end) t_end = lim;
  }
  const int64_t t0 = chunk * kDqTokens;
  if (t0 >= t_end) return;   // uniform over the workgroup

  if (tid < 64) pair_tab[tid] = f32x2_t{codebook_level(cb, tid & 7), codebook_level(cb, tid >> 3)};

  const int c = (lane & 3) | ((lane >> 1) & 4);
  const int slot = ((lane >> 2) & 1) | ((lane >> 3) & 6);
  const int w0 = (3 * c) >> 1;           // first record word of the chunk's 48 bits
  const int sh = (c & 1) ? 16 : 0;       // bit offset of the chunk in that word

  // every load of the workgroup's token range first: code words and scales
  const int64_t row0 = bh * capacity + src_offset;
  uint32_t wlo[kDqPasses], whi[kDqPasses];
  float sv[kDqPasses];
#pragma unroll
  for (int p = 0; p < kDqPasses; ++p) {
    int64_t t = t0 + (p * kDqWaves + wave) * 8 + slot;
    t = t < t_end ? t : t0;   // in range; such a token is not stored
    const uint32_t* rec = reinterpret_cast<const uint32_t*>(codes + (row0 + t) * kRecordBytes);
    wlo[p] = rec[w0];
    whi[p] = rec[w0 + 1];
    sv[p] = norms[row0 + t];
  }

  // B_i = H_4 M_i^T of blocks 4c .. 4c+3 (column k of B_i = H_4 (row k of M_i))
  float bm[4][4][4];   // [block][row r][column k]
  const float* qh = quats + static_cast<int64_t>(g) * kQuatFloats;
#pragma unroll
  for (int bb = 0; bb < 4; ++bb) {
    float m[4][4];
    so4_matrix(qh + (4 * c + bb) * 8, m);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float r0 = m[k][0], r1 = m[k][1], r2 = m[k][2], r3 = m[k][3];
      wht4v(r0, r1, r2, r3);
      bm[bb][0][k] = r0;
      bm[bb][1][k] = r1;
      bm[bb][2][k] = r2;
      bm[bb][3][k] = r3;
    }
  }
  __syncthreads();   // pair table

  const float sg1 = (lane & 1) ? -1.f : 1.f, sg2 = (lane & 2) ? -1.f : 1.f;
  const float sg8 = (lane & 8) ? -1.f : 1.f;
  const float out_sign = sg1 * sg2 * sg8;   // sign the three stages leave on this lane
#pragma unroll
  for (int p = 0; p < kDqPasses; ++p) {
    const int64_t t = t0 + (p * kDqWaves + wave) * 8 + slot;
    // the chunk's 48 code bits: lo = bits 0..31, hi = bits 32..47 (low half)
    const uint32_t lo = __builtin_amdgcn_alignbit(whi[p], wlo[p], sh);
    const uint32_t hi = whi[p] >> sh;
    uint32_t f[8];
#pragma unroll
    for (int k = 0; k < 5; ++k) f[k] = (lo >> (6 * k)) & 63u;
    f[5] = __builtin_amdgcn_alignbit(hi, lo, 30) & 63u;
    f[6] = (hi >> 4) & 63u;
    f[7] = (hi >> 10) & 63u;
    float y[16];   // levels of dims 16c .. 16c+15
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const f32x2_t lv = pair_tab[f[k]];
      y[2 * k] = lv[0];
      y[2 * k + 1] = lv[1];
    }
    // block-local part: z_i = B_i y_i
    float z[4][4];   // [block bb][component r]
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        z[bb][r] = bm[bb][r][0] * y[4 * bb] + bm[bb][r][1] * y[4 * bb + 1] +
                   bm[bb][r][2] * y[4 * bb + 2] + bm[bb][r][3] * y[4 * bb + 3];
    // H_32: block-index bits 0..1 inside the lane, bits 2..4 across lanes
#pragma unroll
    for (int r = 0; r < 4; ++r) wht4v(z[0][r], z[1][r], z[2][r], z[3][r]);
    const float scale = sv[p] * (kInvSqrtDim * out_sign);
    float x[16];
#pragma unroll
    for (int bb = 0; bb < 4; ++bb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = z[bb][r];
        v = xstage<1>(v, sg1);
        v = xstage<2>(v, sg2);
        v = xstage<8>(v, sg8);
        x[4 * bb + r] = v * scale;
      }
    if (t < t_end) store_chunk<TOut>(out + ((bh * n_tokens) + t) * kDim + 16 * c, x);
  }
}

}  // namespace

hipError_t launch_dequant(const uint8_t* k_codes, const float* k_norms, const uint8_t* v_codes,
                          const float* v_norms, const float* quats, const int32_t* seq_lens,
                          int64_t batch, int64_t n_heads, int64_t n_tokens, int64_t capacity,
                          int64_t src_offset, int out_f16, void* k_out, void* v_out,
                          hipStream_t stream, const iq_codebook_t* codebook_arg) {
  // side 0 is whichever of K and V is present first, side 1 the other
  const bool has_k = k_codes != nullptr, has_v = v_codes != nullptr;
  const uint8_t* c0 = has_k ? k_codes : v_codes;
  const float* n0 = has_k ? k_norms : v_norms;
  void* o0 = has_k ? k_out : v_out;
  const uint8_t* c1 = (has_k && has_v) ? v_codes : nullptr;
  const float* n1 = (has_k && has_v) ? v_norms : nullptr;
  void* o1 = (has_k && has_v) ? v_out : nullptr;
  const int nwhich = (has_k && has_v) ? 2 : 1;
  const int64_t n_bh = batch * n_heads;
  const int64_t chunks = (n_tokens + kDqTokens - 1) / kDqTokens;
  const int64_t blocks = chunks * n_bh * nwhich;
  if (blocks == 0) return hipSuccess;
  const Codebook cb = codebook_for<3>(codebook_arg);
  const dim3 grid(static_cast<unsigned>(blocks)), block(kDqThreads);
  if (out_f16) {
    hipLaunchKernelGGL(dequant_kernel<__half>, grid, block, 0, stream, c0, n0,
                       static_cast<__half*>(o0), c1, n1, static_cast<__half*>(o1), quats,
                       seq_lens, static_cast<int>(n_heads), n_bh, n_tokens, chunks, capacity,
                       src_offset, cb);
  } else {
    hipLaunchKernelGGL(dequant_kernel<float>, grid, block, 0, stream, c0, n0,
                       static_cast<float*>(o0), c1, n1, static_cast<float*>(o1), quats, seq_lens,
                       static_cast<int>(n_heads), n_bh, n_tokens, chunks, capacity, src_offset,
                       cb);
  }
  return hipGetLastError();
}

}  // namespace iq
