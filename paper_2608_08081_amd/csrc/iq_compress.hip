// IsoQuant compression kernels (Algorithm 1; Sec. 3.2 Steps 1-4) for gfx950.
//
// Bulk compression: two adjacent lanes compress one 128-dim vector in
// registers, lane 2j + h holding dims 64 h .. 64 h + 63 of vector j.  A
// workgroup (4 waves) takes 128 consecutive tokens of one (K|V, sequence, KV
// head); it first builds the head's 32 block matrices M_i H_4 in LDS (2 KB),
// which the lanes then read as 16-byte rows (two addresses per read, one per
// half: LDS broadcasts).  Half a vector per lane keeps about 100 registers
// per lane, so five waves share a SIMD and the vector-ALU work of one wave
// runs while the others wait on memory.
//
// Per vector:
//   s^2  = sum x_i^2 in fp64 (products of fp16/fp32 inputs are exact in fp64),
//          each half summed in its lane, the two sums added (Step 1);
//          stored scale = fp32(sqrt(s^2));
//   y    = diag(M_i H_4) (H_32 (x) I_4) x   unnormalized, fp32  (Step 2).
//          H_32 acts on index bits 2..6; bit 6 is the lane of the pair, so
//          its butterfly is one fused multiply-add per value with the
//          partner's value (a cross-lane read): the lower lane gets a + b,
//          the upper lane b - a = -(a - b).  The upper lane's values then
//          carry a factor -1 through the remaining (linear) butterflies on
//          bits 2..5, which it undoes by using -M_i for its blocks 16..31;
//   code = #{j : y >= t_j * s * sqrt(128)}  (Step 3; comparing the
//          unnormalized y against scaled thresholds is the same test as
//          comparing R x / s against t_j, and saves 128 multiplies).  The
//          codebook is symmetric (t_{6-j} = -t_j, t_3 = 0), so the code is
//          4 + m for y >= 0 and 3 - m = (4 + m) ^ 7 for y < 0, where
//          m = #{k = 1..3 : |y| >= T_k} comes from a two-step search; the
//          two rules differ only when |y| equals a threshold exactly;
//   pack = 3-bit codes into 12 words; codes 0..63 fill words 0..5 (lower
//          lane) and codes 64..127 words 6..11 (upper lane), each lane
//          storing its 24 bytes (Step 4).
// The same kernel compresses to b = 2 or b = 4 bit codes (Algorithm 1 with
// C_2 or C_4: 2^(b-1) - 1 positive thresholds, records of 4b words, 2b per
// lane).
// A vector whose s^2 is not finite (NaN or infinite input) gets the record of
// all-NaN coordinates, code 0 everywhere, as #{j : t_j <= NaN} = 0.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "iq_device.h"
#include "iq_internal.h"

namespace iq {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kCompressThreads = 256;
constexpr int kCompressTokens = kCompressThreads / 2;   // two lanes per vector
constexpr int kHalfDim = kDim / 2;

// One half (64 dims) of a vector of fp16 or fp32 input.
__device__ __forceinline__ void load_half(const __half* src, float (&x)[kHalfDim]) {
  const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
  for (int i = 0; i < kHalfDim / 8; ++i) {
    const uint4 u = p[i];
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[8 * i + 2 * j] = __half2float(__ushort_as_half(static_cast<unsigned short>(w[j] & 0xFFFFu)));
      x[8 * i + 2 * j + 1] = __half2float(__ushort_as_half(static_cast<unsigned short>(w[j] >> 16)));
    }
  }
}

__device__ __forceinline__ void load_half(const float* src, float (&x)[kHalfDim]) {
  const float4* p = reinterpret_cast<const float4*>(src);
#pragma unroll
  for (int i = 0; i < kHalfDim / 4; ++i) {
    const float4 f = p[i];
    x[4 * i] = f.x;
    x[4 * i + 1] = f.y;
    x[4 * i + 2] = f.z;
    x[4 * i + 3] = f.w;
  }
}

// Code of y against the scaled positive thresholds T1 < T2 < T3 of a
// symmetric codebook (see the file comment), already shifted to bit `off`
// of its record word: ((4 + m) ^ (y < 0 ? 7 : 0)) << off, built from three
// selects of shifted constants.
__device__ __forceinline__ uint32_t quantize_sym(float y, float t1, float t2, float t3, int off) {
  const float a = fabsf(y);
  const bool b1 = a >= t2;
  const bool b0 = a >= (b1 ? t3 : t1);
  const uint32_t hi = b1 ? (6u << off) : (4u << off);
  const uint32_t lo = b0 ? (1u << off) : 0u;
  const uint32_t flip = y >= 0.f ? 0u : (7u << off);
  return (hi | lo) ^ flip;
}

// The same rule for b = 2 and b = 4 (h = 2^(b-1) levels per sign, positive
// thresholds t[0] < ... < t[h-2]): code (h + m) ^ (y < 0 ? 2h - 1 : 0) with
// m = #{k : |y| >= t[k]}.  Codes of 2 and 4 bits never
// straddle a 32-bit word.
template <int kBits>
__device__ __forceinline__ uint32_t quantize_sym_b(float y, const float (&t)[(1 << (kBits - 1)) - 1],
                                                   int off) {
  constexpr uint32_t h = 1u << (kBits - 1);
  const float a = fabsf(y);
  uint32_t m;
  if constexpr (kBits == 2) {
    m = a >= t[0] ? 1u : 0u;
  } else {
    static_assert(kBits == 4, "2 or 4 bits");
    // a plain count: a select tree over 7 thresholds, interleaved across
    // coordinates, more than doubles the register footprint
    m = 0u;
#pragma unroll
    for (int k = 0; k < 7; ++k) m += a >= t[k] ? 1u : 0u;
  }
  const uint32_t flip = y >= 0.f ? 0u : (2 * h - 1);
  return ((h + m) ^ flip) << off;
}

// OR the code of coordinate i of a half (bits 3i .. 3i+2 of the half
// record) into w.
__device__ __forceinline__ void put_code_sym(uint32_t (&w)[kRecordWords / 2], int i, float y,
                                             float t1, float t2, float t3) {
  const int bit = 3 * i;
  const int word = bit >> 5, off = bit & 31;
  if (off <= 29) {
    w[word] |= quantize_sym(y, t1, t2, t3, off);
  } else {
    const uint32_t c = quantize_sym(y, t1, t2, t3, 0);
    w[word] |= c << off;
    w[word + 1] |= c >> (32 - off);
  }
}

// x[i] += x_partner[i] * sg for i = i0 .. i0 + 7, the partner lane being
// lane ^ 1: one multiply-add per value whose first operand is read from the
// partner lane (DPP quad permutation [1, 0, 3, 2]).  Written out because the
// compiler keeps the lane move as a separate instruction.  The leading
// s_nop 1 gives the two wait states a DPP read needs after the VALU write of
// its source register; the eight instructions read only registers written
// before the block.
__device__ __forceinline__ void cross_butterfly8(float (&x)[kDim / 2], int i0, float sg) {
  asm volatile(
      "s_nop 1\n\t"
      "v_fmac_f32_dpp %0, %0, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %1, %1, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %2, %2, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %3, %3, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %4, %4, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %5, %5, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %6, %6, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %7, %7, %8 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf"
      : "+v"(x[i0]), "+v"(x[i0 + 1]), "+v"(x[i0 + 2]), "+v"(x[i0 + 3]), "+v"(x[i0 + 4]),
        "+v"(x[i0 + 5]), "+v"(x[i0 + 6]), "+v"(x[i0 + 7])
      : "v"(sg));
}

// Compress one half of a vector (Algorithm 1) and write its half of the
// record (and, lower lane, the scale).  half: 0 for dims 0..63, 1 for dims
// 64..127; the partner lane (lane ^ 1) holds the other half and must run
// the same code.  mtab: rows of the head's block matrices M_i H_4 (row r of
// block i at mtab[4 i + r]), negated for blocks 16..31.
template <typename T, int kBits>
__device__ __forceinline__ void compress_half(const T* __restrict__ src, const f32x4_t* mtab,
                                              uint8_t* __restrict__ dst_code,
                                              float* __restrict__ dst_norm,
                                              const CodebookB<kBits>& cb, int half) {
  constexpr int kWords = 2 * kBits;   // this lane's half of the record
  constexpr int kHalf = 1 << (kBits - 1);
  float x[kHalfDim];
  load_half(src + kHalfDim * half, x);

  // Step 1: fp64 sum of squares of this half (four independent chains),
  // plus the partner's
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
#pragma unroll
  for (int i = 0; i < kHalfDim; i += 4) {
    a0 = fma(static_cast<double>(x[i]), static_cast<double>(x[i]), a0);
    a1 = fma(static_cast<double>(x[i + 1]), static_cast<double>(x[i + 1]), a1);
    a2 = fma(static_cast<double>(x[i + 2]), static_cast<double>(x[i + 2]), a2);
    a3 = fma(static_cast<double>(x[i + 3]), static_cast<double>(x[i + 3]), a3);
  }
  double ss = (a0 + a1) + (a2 + a3);
  // the two halves' sums (the same sum in both lanes: addition commutes)
  ss += xor_lane64_f64<1>(ss);
  const double s = sqrt(ss);
  const bool finite = ss < static_cast<double>(INFINITY);

  // Positive thresholds in the unnormalized domain: t_j * s * sqrt(128).  A
  // zero vector keeps the plain thresholds, so its all-zero y maps to the
  // first non-negative level.
  const double sc = ss > 0.0 ? s * 11.313708498984760390 : 1.0;   // sqrt(128)
  float tp[kHalf - 1];
#pragma unroll
  for (int j = 0; j < kHalf - 1; ++j) {
    tp[j] = static_cast<float>(static_cast<double>(cb.thr[kHalf + j]) * sc);
    // opaque from here on: otherwise the threshold selects of the search
    // are pushed above the fp64 scaling, which then runs once per coordinate
    asm volatile("" : "+v"(tp[j]));
  }

  // Step 2a: the butterfly on index bit 6 (across the lane pair: the lower
  // lane a + b, the upper lane b - a), then bits 2..5 in the lane.
  const float sg = half ? -1.0f : 1.0f;
#pragma unroll
  for (int i = 0; i < kHalfDim; i += 8) cross_butterfly8(x, i, sg);
#pragma unroll
  for (int st = 4; st < kHalfDim; st <<= 1) {
#pragma unroll
    for (int i = 0; i < kHalfDim; ++i) {
      if (!(i & st)) {
        const float a = x[i], b = x[i + st];
        x[i] = a + b;
        x[i + st] = a - b;
      }
    }
  }

  // Step 2b + 3 + 4: per block, y = (M_i H_4) z, quantize, pack.
  const f32x4_t* mt = mtab + 64 * half;   // blocks 16 half .. 16 half + 15
  uint32_t w[kWords];
#pragma unroll
  for (int i = 0; i < kWords; ++i) w[i] = 0u;
#pragma unroll
  for (int blk = 0; blk < kNumBlocks / 2; ++blk) {
    const float z0 = x[4 * blk], z1 = x[4 * blk + 1], z2 = x[4 * blk + 2], z3 = x[4 * blk + 3];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const f32x4_t m = mt[4 * blk + r];
      const float y = m[0] * z0 + m[1] * z1 + m[2] * z2 + m[3] * z3;
      const int i = 4 * blk + r;
      if constexpr (kBits == 3) {
        put_code_sym(w, i, y, tp[0], tp[1], tp[2]);
      } else {
        const int bit = kBits * i;
        w[bit >> 5] |= quantize_sym_b<kBits>(y, tp, bit & 31);
      }
    }
  }
  if (!finite) {
#pragma unroll
    for (int i = 0; i < kWords; ++i) w[i] = 0u;
  }

  uint32_t* out = reinterpret_cast<uint32_t*>(dst_code) + kWords * half;
  if constexpr (kWords % 4 == 0) {
#pragma unroll
    for (int j = 0; j < kWords / 4; ++j)
      reinterpret_cast<uint4*>(out)[j] = make_uint4(w[4 * j], w[4 * j + 1], w[4 * j + 2],
                                                    w[4 * j + 3]);
  } else {
    // 24 bytes at byte 0 or 24 of the record: 8-byte aligned
#pragma unroll
    for (int j = 0; j < kWords / 2; ++j)
      reinterpret_cast<uint2*>(out)[j] = make_uint2(w[2 * j], w[2 * j + 1]);
  }
  if (half == 0) *dst_norm = static_cast<float>(s);
}

// Bulk compression.  1-D grid of 256-thread workgroups:
//   blockIdx.x = (which * (B*H) + bh) * chunks + chunk,  thread 2 j + h =
//   half h of token j of the chunk (128 tokens).
// kPaged: the destination is a page pool; a token whose page index is
// invalid is not written.
template <typename T, bool kPaged, int kBits>
__global__ __launch_bounds__(kCompressThreads) void compress_kernel(
    const T* __restrict__ src0, const T* __restrict__ src1, const float* __restrict__ quats,
    uint8_t* __restrict__ codes0, float* __restrict__ norms0, uint8_t* __restrict__ codes1,
    float* __restrict__ norms1, int n_heads, int64_t n_bh, int64_t n_tokens, int64_t chunks,
    int64_t capacity, int64_t dst_offset, CodebookB<kBits> cb, PageTable pages) {
  __shared__ f32x4_t mtab[kNumBlocks * 4];
  const int64_t blk = blockIdx.x;
  const int64_t chunk = blk % chunks;
  const int64_t rest = blk / chunks;
  const int64_t bh = rest % n_bh;
  const int which = static_cast<int>(rest / n_bh);
  const int h = static_cast<int>(bh % n_heads);
  const int tid = threadIdx.x;
  // rows of M_i H_4: thread tid < 128 builds row tid % 4 of block tid / 4,
  // negated for blocks 16..31 (whose lane holds its values negated)
  if (tid < kNumBlocks * 4) {
    float m[4][4];
    so4_matrix_h4(quats + static_cast<int64_t>(h) * kQuatFloats + 8 * (tid >> 2), m);
    const int r = tid & 3;
    f32x4_t row = f32x4_t{m[0][0], m[0][1], m[0][2], m[0][3]};
#pragma unroll
    for (int i = 1; i < 4; ++i)
      if (r == i) row = f32x4_t{m[i][0], m[i][1], m[i][2], m[i][3]};
    mtab[tid] = (tid >> 2) >= kNumBlocks / 2 ? -row : row;
  }
  __syncthreads();
  const int64_t t = chunk * kCompressTokens + (tid >> 1);
  if (t >= n_tokens) return;
  const T* src = which ? src1 : src0;
  uint8_t* codes = which ? codes1 : codes0;
  float* norms = which ? norms1 : norms0;
  int64_t pos = bh * capacity + dst_offset + t;
  if constexpr (kPaged) {
    pos = paged_record(pages, n_heads, static_cast<int>(bh / n_heads), h, dst_offset + t);
    if (pos < 0) return;
  }
  compress_half<T, kBits>(src + (bh * n_tokens + t) * kDim, mtab,
                          codes + pos * record_bytes<kBits>(), norms + pos, cb, tid & 1);
}

// Per-step append: one workgroup per sequence, one wave per vector (keys and
// values of every KV head), each vector compressed by compress_vector_wave,
// which keeps the serial chain short (a lane-per-vector kernel would run a
// ~2.7K-instruction chain for a handful of vectors).  seq_lens[b] is read
// once, before any write, and bumped by thread 0 after its own vectors.
constexpr int kAppendMaxWaves = 16;

template <typename T>
__global__ __launch_bounds__(64 * kAppendMaxWaves) void append_kernel(
    const T* __restrict__ src0, const T* __restrict__ src1, const float* __restrict__ quats,
    uint8_t* __restrict__ codes0, float* __restrict__ norms0, uint8_t* __restrict__ codes1,
    float* __restrict__ norms1, int n_heads, int n_vectors, int64_t capacity,
    int32_t* __restrict__ seq_lens, int32_t* __restrict__ status, Codebook cb) {
  __shared__ int32_t pos_s;
  const int b = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n_waves = blockDim.x >> 6;
  if (threadIdx.x == 0) pos_s = seq_lens[b];
  __syncthreads();
  const int64_t pos = pos_s;
  if (pos < 0 || pos >= capacity) {
    if (threadIdx.x == 0 && status != nullptr)
      atomicOr(status, static_cast<int32_t>(IQ_ERR_CAPACITY));
    return;
  }
  for (int idx = wave; idx < n_vectors; idx += n_waves) {
    const int which = idx / n_heads;
    const int h = idx % n_heads;
    const int64_t bh = static_cast<int64_t>(b) * n_heads + h;
    float x0, x1;
    load_pair((which ? src1 : src0) + bh * kDim, lane, x0, x1);
    float qp[8];
    {
      const float4* qs = reinterpret_cast<const float4*>(
          quats + static_cast<int64_t>(h) * kQuatFloats + 8 * (lane >> 1));
      const float4 p0 = qs[0], p1 = qs[1];
      qp[0] = p0.x; qp[1] = p0.y; qp[2] = p0.z; qp[3] = p0.w;
      qp[4] = p1.x; qp[5] = p1.y; qp[6] = p1.z; qp[7] = p1.w;
    }
    const WaveCode wc = compress_vector_wave(x0, x1, qp, cb, lane);
    if (lane < kRecordWords) {
      uint8_t* codes = which ? codes1 : codes0;
      reinterpret_cast<uint32_t*>(codes + (bh * capacity + pos) * kRecordBytes)[lane] = wc.word;
      if (lane == 0) (which ? norms1 : norms0)[bh * capacity + pos] = wc.scale;
    }
  }
  if (threadIdx.x == 0) seq_lens[b] = static_cast<int32_t>(pos + 1);
}

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, int64_t n_words) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n_words;
       i += stride)
    p[i] = 0u;
}

}  // namespace

namespace {

hipError_t launch_compress_any(const void* k, const void* v, int dtype, int64_t batch,
                               int64_t n_heads, int64_t n_tokens, const float* quats,
                               uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                               float* v_norms, int64_t capacity, int64_t dst_offset,
                               const PageTable* pages, int bits, hipStream_t stream,
                               const iq_codebook_t* cb) {
  // slot 0 is whichever side is present first, slot 1 the other (if any)
  const void* s0 = k ? k : v;
  uint8_t* c0 = k ? k_codes : v_codes;
  float* n0 = k ? k_norms : v_norms;
  const void* s1 = (k && v) ? v : nullptr;
  uint8_t* c1 = (k && v) ? v_codes : nullptr;
  float* n1 = (k && v) ? v_norms : nullptr;
  const int nwhich = s1 ? 2 : 1;
  const int64_t n_bh = batch * n_heads;
  const int64_t chunks = (n_tokens + kCompressTokens - 1) / kCompressTokens;
  const int64_t blocks = chunks * n_bh * nwhich;
  if (blocks == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(blocks)), block(kCompressThreads);
  const PageTable pt = pages ? *pages : PageTable{nullptr, 0, 4, 1};
  // paged pools hold the paper's 3-bit records only
  if (pages && bits != 3) return hipErrorInvalidValue;
#define IQ_LAUNCH_COMPRESS(T_, P_, B_)                                                         \
  hipLaunchKernelGGL((compress_kernel<T_, P_, B_>), grid, block, 0, stream,                     \
                     static_cast<const T_*>(s0), static_cast<const T_*>(s1), quats, c0, n0, c1, \
                     n1, static_cast<int>(n_heads), n_bh, n_tokens, chunks, capacity,           \
                     dst_offset, codebook_for<B_>(cb), pt)
#define IQ_LAUNCH_COMPRESS_T(T_)                   \
  if (pages) IQ_LAUNCH_COMPRESS(T_, true, 3);      \
  else if (bits == 2) IQ_LAUNCH_COMPRESS(T_, false, 2); \
  else if (bits == 4) IQ_LAUNCH_COMPRESS(T_, false, 4); \
  else IQ_LAUNCH_COMPRESS(T_, false, 3);
  if (dtype == IQ_DTYPE_F16) {
    IQ_LAUNCH_COMPRESS_T(__half)
  } else {
    IQ_LAUNCH_COMPRESS_T(float)
  }
#undef IQ_LAUNCH_COMPRESS_T
#undef IQ_LAUNCH_COMPRESS
  return hipGetLastError();
}

}  // namespace

hipError_t launch_compress(const void* k, const void* v, int dtype, int64_t batch,
                           int64_t n_heads, int64_t n_tokens, const float* quats,
                           uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                           float* v_norms, int64_t capacity, int64_t dst_offset, int bits,
                           hipStream_t stream, const iq_codebook_t* cb) {
  return launch_compress_any(k, v, dtype, batch, n_heads, n_tokens, quats, k_codes, k_norms,
                             v_codes, v_norms, capacity, dst_offset, nullptr, bits, stream, cb);
}

hipError_t launch_compress_paged(const void* k, const void* v, int dtype, int64_t batch,
                                 int64_t n_heads, int64_t n_tokens, const float* quats,
                                 uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                                 float* v_norms, const PageTable& pages, int64_t dst_offset,
                                 hipStream_t stream) {
  return launch_compress_any(k, v, dtype, batch, n_heads, n_tokens, quats, k_codes, k_norms,
                             v_codes, v_norms, (pages.max_pages << pages.page_shift), dst_offset,
                             &pages, 3, stream, nullptr);
}

hipError_t launch_append(const void* k, const void* v, int dtype, int64_t batch,
                         int64_t n_heads, const float* quats, uint8_t* k_codes,
                         float* k_norms, uint8_t* v_codes, float* v_norms,
                         int64_t capacity, int32_t* seq_lens, int32_t* status,
                         hipStream_t stream, const iq_codebook_t* codebook_arg) {
  if (batch == 0) return hipSuccess;
  const void* s0 = k ? k : v;
  uint8_t* c0 = k ? k_codes : v_codes;
  float* n0 = k ? k_norms : v_norms;
  const void* s1 = (k && v) ? v : nullptr;
  uint8_t* c1 = (k && v) ? v_codes : nullptr;
  float* n1 = (k && v) ? v_norms : nullptr;
  const int n_vectors = static_cast<int>(n_heads * (s1 ? 2 : 1));
  const int waves = n_vectors < kAppendMaxWaves ? n_vectors : kAppendMaxWaves;
  const dim3 block(static_cast<unsigned>(64 * waves));
  const Codebook cb = codebook_for<3>(codebook_arg);
  if (dtype == IQ_DTYPE_F16) {
    hipLaunchKernelGGL(append_kernel<__half>, dim3(static_cast<unsigned>(batch)), block, 0,
                       stream, static_cast<const __half*>(s0), static_cast<const __half*>(s1),
                       quats, c0, n0, c1, n1, static_cast<int>(n_heads), n_vectors, capacity,
                       seq_lens, status, cb);
  } else {
    hipLaunchKernelGGL(append_kernel<float>, dim3(static_cast<unsigned>(batch)), block, 0,
                       stream, static_cast<const float*>(s0), static_cast<const float*>(s1), quats,
                       c0, n0, c1, n1, static_cast<int>(n_heads), n_vectors, capacity, seq_lens,
                       status, cb);
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream) {
  const int64_t words = static_cast<int64_t>(bytes / 4);
  if (words == 0) return hipSuccess;
  int64_t blocks = (words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                     static_cast<uint32_t*>(ptr), words);
  return hipGetLastError();
}

}  // namespace iq
