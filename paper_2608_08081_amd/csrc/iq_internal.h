// Internal declarations of libisoquant shared by the host API and the
// kernel translation units.  Not installed; the public ABI is isoquant.h.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "isoquant.h"

namespace iq {

constexpr int kDim = 128;           // head_dim (Sec. 3.2, d = 128)
constexpr int kRecordBytes = 48;    // 128 codes x 3 bits
constexpr int kRecordWords = 12;
constexpr int kNumBlocks = 32;      // SO(4) blocks per head (d / 4)
constexpr int kQuatFloats = 256;    // stored parameters per head (App. B)
constexpr int kMaxGroup = 16;       // query heads per KV head supported

// Codebook C_b of b-bit codes, passed to kernels by value.  level[]
// ascending (fp16-exact values), thr[j] = midpoint of level[j] and
// level[j+1].  The cache format of the paper is b = 3 (Codebook); b = 2 and
// b = 4 run through the same steps with 2^b levels.
template <int kBits>
struct CodebookB {
  float level[1 << kBits];
  float thr[(1 << kBits) - 1];
};
using Codebook = CodebookB<3>;

// Bytes of one packed record of 128 b-bit codes.
template <int kBits>
constexpr int record_bytes() {
  return kDim * kBits / 8;
}

// Computed on first use (host), immutable afterwards.  codebook_b<b>() for
// b = 2, 3, 4; codebook() is codebook_b<3>().
template <int kBits>
const CodebookB<kBits>& codebook_b();
const Codebook& codebook();

// The codebook a launch uses: the caller's (an iq_codebook_t of kBits bits,
// already validated), or the library's C_b when cb is null.
template <int kBits>
CodebookB<kBits> codebook_for(const iq_codebook_t* cb) {
  if (cb == nullptr) return codebook_b<kBits>();
  CodebookB<kBits> r;
  for (int i = 0; i < (1 << kBits); ++i) r.level[i] = cb->levels[i];
  for (int i = 0; i < (1 << kBits) - 1; ++i) r.thr[i] = cb->thresholds[i];
  return r;
}

// A paged cache: records of logical position t of (sequence b, KV head g)
// live in page tables[b * max_pages + t / page_size], slot t % page_size, of
// pools laid out [n_pages][n_kv_heads][page_size][48] (codes) and
// [n_pages][n_kv_heads][page_size] (scales).  page_size is a power of two
// (page_shift its log2), at least 16, so a batch of 16 positions never
// straddles a page.  A page index outside [0, n_pages) is a caller error:
// reads then use page 0 and writes are skipped, so no access leaves the
// pools.
struct PageTable {
  const int32_t* tables;   // [batch][max_pages]
  int64_t max_pages;
  int32_t page_shift;
  int32_t n_pages;
};

// Record index (into the pools viewed as [n_pages * n_kv_heads * page_size]
// records) of logical position t, or -1 if its page index is invalid.
__device__ __forceinline__ int64_t paged_record(const PageTable& pt, int n_kv_heads, int b,
                                                int g, int64_t t) {
  const int32_t page = pt.tables[static_cast<int64_t>(b) * pt.max_pages + (t >> pt.page_shift)];
  if (static_cast<uint32_t>(page) >= static_cast<uint32_t>(pt.n_pages)) return -1;
  const int64_t slot = t & ((int64_t(1) << pt.page_shift) - 1);
  return ((static_cast<int64_t>(page) * n_kv_heads + g) << pt.page_shift) + slot;
}

// Split-K plan for one decode call.  Deterministic function of the shapes so
// that iq_decode_workspace_bytes and iq_decode_attention agree.
struct DecodePlan {
  int kernel;               // reserved
  int64_t split_len;        // generic path: positions per split
  int64_t n_splits;         // generic path: splits per (sequence, KV head)
  size_t partial_bytes;     // generic path: B * H_q * n_splits * 130 floats
  // matrix-core path (any group <= 16, in head groups of 8 query heads)
  int g8_batches;           // 16-position batches per wave (0 = n/a)
  int64_t g8_splits;        // splits per (sequence, KV head, head group)
  int64_t g8_split_len;     // positions per split
  size_t ticket_bytes;      // reserved (0)
  size_t g8_partial_bytes;  // g8_partial_region_bytes + one int32 per sequence
  size_t total_bytes;       // max over both paths
};
bool plan_decode(int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                 int64_t max_seq_len, DecodePlan* plan);

// Workspace of the matrix-core path after the reserved bytes: the partials
// of every (sequence, row, split or new token) in this many bytes (rows =
// KV heads x head groups), then one int32 per sequence: in fused steps on
// grids of several rounds, the length each sequence had when the step
// began, recorded by its append workgroup for the merge (whose workgroup of
// head 0 advances seq_lens while the others still need the old length).
inline size_t g8_partial_region_bytes(int64_t batch, int64_t rows, int64_t n_splits) {
  const size_t b = static_cast<size_t>(batch) * rows * (n_splits + 1) * 8 * (2 + kDim) * 4;
  return (b + 255) / 256 * 256;
}

// Kernel launchers (return the launch's hipError_t).
// bits: 3 (the cache format), or 2 / 4 (records of 16 * bits bytes).
hipError_t launch_compress(const void* k, const void* v, int dtype, int64_t batch,
                           int64_t n_heads, int64_t n_tokens, const float* quats,
                           uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                           float* v_norms, int64_t capacity, int64_t dst_offset, int bits,
                           hipStream_t stream, const iq_codebook_t* cb = nullptr);

// Bulk compression into a paged cache: tokens [0, n_tokens) of every
// sequence to logical positions dst_offset ..
hipError_t launch_compress_paged(const void* k, const void* v, int dtype, int64_t batch,
                                 int64_t n_heads, int64_t n_tokens, const float* quats,
                                 uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                                 float* v_norms, const PageTable& pages, int64_t dst_offset,
                                 hipStream_t stream);

hipError_t launch_append(const void* k, const void* v, int dtype, int64_t batch,
                         int64_t n_heads, const float* quats, uint8_t* k_codes,
                         float* k_norms, uint8_t* v_codes, float* v_norms,
                         int64_t capacity, int32_t* seq_lens, int32_t* status,
                         hipStream_t stream, const iq_codebook_t* cb = nullptr);

// The new token of a fused decode step (keys and values of every KV head).
struct StepAppend {
  const void* k_new;
  const void* v_new;
  int f16;            // 1: fp16 inputs, 0: fp32
  int32_t* status;    // optional IQ_ERR_CAPACITY flag
};

// Decode attention; with `append`, the fused step: append the new token at
// seq_lens[b], attend over seq_lens[b] + 1 positions, advance seq_lens.
hipError_t launch_decode(const DecodePlan& plan, const float* q, uint8_t* k_codes,
                         float* k_norms, uint8_t* v_codes, float* v_norms,
                         int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                         const float* quats, int64_t batch, int64_t n_q_heads,
                         int64_t n_kv_heads, float scale, float* out, void* workspace,
                         const StepAppend* append, hipStream_t stream,
                         const iq_codebook_t* cb = nullptr);

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);

// n_rows: (KV head, head group of 8 query heads) rows per sequence.
void g8_plan(int64_t batch, int64_t n_rows, int64_t max_seq_len, int* nb, int64_t* n_splits,
             int64_t* split_len);
// pages: null for a contiguous cache ([B][H_kv][capacity] records), else
// the page table (capacity is then max_pages * page_size).  bits: the
// records' code width (2, 3 or 4; paged pools need 3).
// The positional parts of a decode with the content / RoPE sub-block split:
// k_rope fp16 [batch][shared ? 1 : n_kv_heads][capacity][64], q_rope fp32
// [batch][n_q_heads][64].
struct RopeKeys {
  const uint16_t* k_rope;
  const float* q_rope;
  int shared;
};

// group: query heads per KV head (1 .. 16), served in head groups of 8.
// rope: the positional parts (decode of contiguous 3-bit caches only).
hipError_t launch_decode_g8(int nb, int64_t n_splits, int64_t split_len, const float* q,
                            uint8_t* k_codes, float* k_norms, uint8_t* v_codes, float* v_norms,
                            int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                            const float* quats, int64_t batch, int64_t n_kv_heads,
                            int64_t group, float scale, float* out, float* partials,
                            const StepAppend* append, const PageTable* pages, int bits,
                            hipStream_t stream, const iq_codebook_t* cb = nullptr,
                            const RopeKeys* rope = nullptr);

// Multi-token decode on records of `bits` bits (group 8): n_tok (2..4)
// query tokens per sequence, q / out [batch][n_tok][8 n_kv_heads][128]; the
// plan is g8_plan's, partials [batch][n_kv_heads][n_parts][n_tok][8][130]
// floats with n_parts = n_splits (+ 1 with `append`); pages: null for a
// contiguous cache, else the page table (3-bit records, no append).  With
// `append` (k_new / v_new [batch][n_tok][n_kv_heads][128]), the fused
// step: the n_tok tokens are appended at seq_lens[b], attended causally and
// seq_lens advanced by n_tok.
hipError_t launch_decode_g8_multi(int nb, int64_t n_splits, int64_t split_len, int n_tok,
                                  const float* q, uint8_t* k_codes, float* k_norms,
                                  uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                                  int64_t capacity, int64_t max_seq_len, const float* quats,
                                  int64_t batch, int64_t n_kv_heads, float scale, float* out,
                                  float* partials, const PageTable* pages, int bits,
                                  const StepAppend* append, hipStream_t stream,
                                  const iq_codebook_t* cb = nullptr);

// Reconstruct-then-compute baseline (Fig. 1 top): materialize the packed
// cache as fp16 or fp32 vectors, and decode attention on an fp16 cache.
hipError_t launch_dequant(const uint8_t* k_codes, const float* k_norms, const uint8_t* v_codes,
                          const float* v_norms, const float* quats, const int32_t* seq_lens,
                          int64_t batch, int64_t n_heads, int64_t n_tokens, int64_t capacity,
                          int64_t src_offset, int out_f16, void* k_out, void* v_out,
                          hipStream_t stream, const iq_codebook_t* cb = nullptr);

void f16_plan(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len, int* nb,
              int64_t* n_splits, int64_t* split_len);
size_t f16_workspace_bytes(int64_t batch, int64_t n_kv_heads, int64_t max_seq_len);
hipError_t launch_decode_f16(const float* q, const __half* k, const __half* v,
                             const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                             int64_t batch, int64_t n_kv_heads, int64_t group, float scale,
                             float* out, float* partials, hipStream_t stream);

}  // namespace iq
