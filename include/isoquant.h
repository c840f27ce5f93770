/*
 * isoquant.h - C ABI of libisoquant: IsoQuant 3-bit KV-cache compression and
 * decode attention computed directly on the packed cache, for AMD Instinct
 * MI355X (gfx950).
 *
 * Method: arXiv 2608.08081, "RotaryQuant: Fitting 120B MoE Models on Consumer
 * Hardware via Fused Compressed-Space Attention".  Citations below name the
 * paper's sections, equations, algorithms and tables.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - head_dim must be 128, and the code width is 3 bits (the configuration of
 *   Sec. 3.2 Step 4) except in the *_bits entry points (2, 3 or 4 bits; see
 *   "Other code widths"); anything else returns IQ_ERR_UNSUPPORTED.
 * - Sections below: the contiguous cache (rotation, compression, append,
 *   decode, fused step), the paged cache, the reconstruct-then-compute
 *   baseline, other code widths, multi-token decode.
 * - Device pointers are plain HIP device allocations owned by the caller.
 *   The library never allocates, frees or retains device memory and keeps no
 *   mutable global state (the codebook is an immutable constant computed once
 *   per process on first use), so calls are thread-safe.  The one exception
 *   is iq_decode_step_noalloc, whose scratch is a static device array of the
 *   library (one per GPU, shared by every call of that entry point).
 * - Every device entry point is asynchronous on `stream` (0 = the null
 *   stream) and never synchronizes.  Arguments are validated on the host
 *   before any HIP call; on a validation error nothing is launched.
 * - A failed kernel launch returns IQ_ERR_HIP.  Device-side faults surface,
 *   as usual in HIP, at the caller's next synchronizing call.
 *
 * Cache layout (one layer)
 * ------------------------
 * codes  : uint8 [batch][n_kv_heads][capacity][48]   one record per token
 * norms  : fp32  [batch][n_kv_heads][capacity]        per-token scale s
 * Keys and values use separate, identically laid out arrays.  Record format
 * (the paper fixes only "48 bytes per 128-dim vector", Sec. 3.2 Step 4): code
 * i of the vector occupies bits 3i..3i+2 of the record read as a
 * little-endian bit string (bit n = bit n%8 of byte n/8), LSB first.  Codes
 * number the codebook levels in ascending order.
 * Rotation parameters: fp32 [n_kv_heads][32][2][4]: per SO(4) block the pair
 * (q_L, q_R), each quaternion as (w, x, y, z), 256 floats per head (App. B);
 * device copies passed to the kernels must be 16-byte aligned.
 */
#ifndef ISOQUANT_H_
#define ISOQUANT_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define IQ_HEAD_DIM 128
#define IQ_BITS 3
#define IQ_LEVELS 8
#define IQ_RECORD_BYTES 48
#define IQ_PARAMS_PER_HEAD 256

typedef enum iq_status {
  IQ_OK = 0,
  IQ_ERR_INVALID_ARGUMENT = 1,   /* null/misaligned pointer, bad size, range */
  IQ_ERR_UNSUPPORTED = 2,        /* head_dim != 128, unknown dtype, group > 16 */
  IQ_ERR_WORKSPACE_TOO_SMALL = 3,
  IQ_ERR_HIP = 4,                /* a HIP runtime call or launch failed */
  IQ_ERR_CAPACITY = 5            /* written to status_dev by iq_append_token */
} iq_status;

/* Element types of K/V inputs and outputs.  Entry points take them as an
 * int32_t `dtype` argument (any other value returns IQ_ERR_UNSUPPORTED). */
typedef enum iq_dtype {
  IQ_DTYPE_F32 = 0,
  IQ_DTYPE_F16 = 1
} iq_dtype;

/* Human-readable name of a status code (static string, never NULL; unknown
 * codes give "unknown status"). */
const char* iq_status_string(int32_t s);

/* ABI version of this header (major * 100 + minor). */
int iq_version(void);

/*
 * iq_codebook - the 3-bit Lloyd-Max codebook C_b (Sec. 3.2 Step 3).
 * Levels minimize expected squared error for one coordinate of a unit vector
 * spread uniformly over the sphere S^127 (density proportional to
 * (1 - t^2)^62.5), each rounded to the nearest fp16 value; thresholds are
 * the midpoints of adjacent stored levels.  Host memory out:
 * levels[8] ascending, thresholds[7] ascending.  Either pointer may be NULL.
 */
iq_status iq_codebook(float* levels, float* thresholds);

/*
 * iq_make_rotation - seeded SO(4) parameters for n_kv_heads heads (Sec. 3.3
 * "SO(4) parameterization", App. B).  Host memory out:
 * quats_host[n_kv_heads][32][2][4].  Each unit quaternion is drawn from one
 * SplitMix64 stream seeded with `seed`, in the order head, block, q_L then
 * q_R: four draws (top 53 bits * 2^-53, mapped to [-1, 1)) rejected unless
 * the squared norm lies in (1e-6, 1], divided by the norm in fp64, rounded to
 * fp32.  Pure host function (no HIP call).
 */
iq_status iq_make_rotation(uint64_t seed, int64_t n_kv_heads, int64_t head_dim,
                           float* quats_host);

/* Designs of the rotation ablation (Sec. 4.6, "Rotation Design Ablation")
 * that keep the structure R = R_blocks H_128, so every kernel runs them
 * unchanged. */
typedef enum iq_rotation_variant {
  IQ_ROTATION_SO4 = 0,        /* v3, the method: paired (q_L, q_R) SO(4) blocks after H */
  IQ_ROTATION_SO3 = 1,        /* H, then single-quaternion blocks v -> q v conj(q) (SO(3)) */
  IQ_ROTATION_WHT_ONLY = 2    /* H alone: identity quaternions */
} iq_rotation_variant;

/*
 * iq_make_rotation_variant - parameters of one rotation design, same layout
 * as iq_make_rotation (host quats_host[n_kv_heads][32][2][4]).
 * IQ_ROTATION_SO4 equals iq_make_rotation; IQ_ROTATION_SO3 takes the same
 * draws and sets q_R = q_L in every block, so each block acts as SO(3) and
 * fixes its real axis (App. B); IQ_ROTATION_WHT_ONLY writes (1, 0, 0, 0)
 * everywhere.  The ablation's v1 and v2 (blocks without H) are not of this
 * form and exist only in the CPU oracle.  IQ_ERR_UNSUPPORTED for another
 * variant or head_dim != 128.  Pure host function (no HIP call).
 */
iq_status iq_make_rotation_variant(uint64_t seed, int64_t n_kv_heads, int64_t head_dim,
                                   int32_t variant, float* quats_host);

/*
 * iq_fit_rotation - fitted SO(4) block parameters (Sec. 3.2: the blocks
 * fine-tune the rotation after H_128, 6 degrees of freedom each, 192
 * "learnable" parameters per head; the paper gives no procedure).  Reading:
 * per KV head and block, the rotation of the block's four post-WHT
 * coordinates that minimizes their mean squared quantization error (the
 * objective Step 3 states for the quantizer) on the calibration vectors,
 * found by `sweeps` Jacobi sweeps over the six coordinate planes from the
 * identity (a grid of 24 angles, then golden-section refinement; a plane
 * rotation is kept only if it lowers the error), so the fitted error never
 * exceeds that of H_128 alone on the calibration set.  Host memory:
 * calib[n_kv_heads][n_vectors][128] fp32 in (zero and non-finite vectors
 * are skipped), quats_host[n_kv_heads][32][2][4] out, the layout of
 * iq_make_rotation.  1 <= n_vectors <= 2^24, sweeps >= 0 (0 gives identity
 * quaternions).  Pure host function (no HIP call); runs the 32 blocks of a
 * head on up to 8 host threads.
 */
iq_status iq_fit_rotation(const float* calib, int64_t n_vectors, int64_t n_kv_heads,
                          int64_t head_dim, int32_t sweeps, float* quats_host);

/*
 * iq_so4_to_quaternions - the pair (q_L, q_R) with m v = q_L v conj(q_R)
 * for a rotation m of R^4 (App. B: SO(4) is covered by S^3 x S^3), block
 * component 0 the real part.  m: host fp64 4 x 4, row-major; q_pair: host
 * fp32 out (q_L.w, q_L.x, q_L.y, q_L.z, q_R.w, ..., q_R.z), unit, defined
 * up to the common sign (q_L, q_R) -> (-q_L, -q_R).  IQ_ERR_INVALID_ARGUMENT
 * if m is not orthogonal to 1e-6 or has determinant -1.  Pure host function.
 */
iq_status iq_so4_to_quaternions(const double* m, float* q_pair);

/*
 * iq_compress_kv - Algorithm 1 (Sec. 3.2 Steps 1-4) over a block of tokens:
 * for every vector x: s = ||x||_2 (accumulated in fp64, stored as fp32),
 * x_tilde = R_SO(4)(H_128 x / s) (Eq. 2), each coordinate replaced by the
 * index of its nearest codebook level, codes bit-packed into a 48-byte
 * record.  This is the deferred bulk compression at the prefill-to-decode
 * boundary (Sec. 3.4 "Deferred prefill", App. C).
 *
 * k, v        : device, [batch][n_kv_heads][n_tokens][128] of `dtype`,
 *               16-byte aligned.  Either side may be NULL together with its
 *               outputs (compress keys only / values only); not both.
 * quats       : device fp32 [n_kv_heads][32][2][4] (one rotation per KV head,
 *               shared by keys, values and the query heads of the group).
 * k_codes/v_codes : device uint8 [batch][n_kv_heads][capacity][48], 16-byte
 *               aligned.  k_norms/v_norms: device fp32 [batch][n_kv_heads][capacity].
 * Token t of the input is written at cache position dst_offset + t.
 * Requires 0 <= dst_offset and dst_offset + n_tokens <= capacity.
 * n_tokens == 0 or batch == 0 is a valid no-op.
 */
iq_status iq_compress_kv(const void* k, const void* v, int32_t dtype,
                         int64_t batch, int64_t n_kv_heads, int64_t n_tokens,
                         int64_t head_dim, const float* quats,
                         uint8_t* k_codes, float* k_norms,
                         uint8_t* v_codes, float* v_norms,
                         int64_t capacity, int64_t dst_offset, hipStream_t stream);

/*
 * iq_append_token - per-step compression of one new token per sequence
 * (Alg. 1 applied to the decode step's new key and value; the paper's
 * packed-cache write of App. D, done in place).
 *
 * k_new, v_new : device [batch][n_kv_heads][128] of `dtype` (either may be
 *                NULL with its cache arrays, not both).
 * seq_lens     : device int32 [batch], read and updated in place: the token of
 *                sequence b is written at position seq_lens[b], then
 *                seq_lens[b] is incremented.
 * status_dev   : optional device int32; if sequence b is already at capacity
 *                its token is dropped, seq_lens[b] is left unchanged and
 *                IQ_ERR_CAPACITY is OR-ed into *status_dev.  Never cleared by
 *                the library.
 */
iq_status iq_append_token(const void* k_new, const void* v_new, int32_t dtype,
                          int64_t batch, int64_t n_kv_heads, int64_t head_dim,
                          const float* quats,
                          uint8_t* k_codes, float* k_norms,
                          uint8_t* v_codes, float* v_norms,
                          int64_t capacity, int32_t* seq_lens, int32_t* status_dev,
                          hipStream_t stream);

/*
 * iq_decode_workspace_bytes - size of the device workspace iq_decode_attention
 * and iq_decode_step need for these shapes (the split-K partial results and,
 * for the fused step, each sequence's length at the step's start, which the
 * merge of the partials reads while the step advances seq_lens).  Returns 0
 * for invalid shapes.
 */
size_t iq_decode_workspace_bytes(int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                 int64_t max_seq_len, int64_t head_dim);

/*
 * iq_decode_workspace_init - zero-fill a workspace (a fill kernel on `stream`,
 * safe under graph capture).  Optional: iq_decode_attention and iq_decode_step
 * write every workspace byte they read within the same call, so the workspace
 * needs no initialization.
 */
iq_status iq_decode_workspace_init(void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * iq_decode_attention - single-token decode attention computed on the packed
 * cache without materializing keys or values (App. A; Table 2; Fig. 1
 * bottom): per query head h of KV head g = h / (n_q_heads / n_kv_heads),
 *   q_tilde = R_g q_h;  score_j = s^K_j (q_tilde . C[codeK_j]) * scale;
 *   alpha = softmax(score);  o = R_g^T sum_j alpha_j s^V_j C[codeV_j].
 * The sum over positions is split across workgroups (flash-decoding) and the
 * partial results are merged before the single inverse rotation.
 *
 * q         : device fp32 [batch][n_q_heads][128], original (unrotated) space.
 * caches    : as written by iq_compress_kv / iq_append_token.
 * seq_lens  : device int32 [batch]; positions 0 .. seq_lens[b]-1 are attended.
 *             Values above max_seq_len are treated as max_seq_len; a length of
 *             0 yields a zero output row.
 * max_seq_len : host-side upper bound of seq_lens[] (sizes the launch, so no
 *             device-to-host synchronization is needed); <= capacity.
 * softmax_scale : <= 0 selects 1/sqrt(128).
 * out       : device fp32 [batch][n_q_heads][128], original space.
 * workspace : device, >= iq_decode_workspace_bytes(...) bytes, 256-byte
 *             aligned, contents ignored on entry.  Calls that share a
 *             workspace must not overlap in time.
 * n_q_heads / n_kv_heads must be an integer <= 16.  Caches whose capacity
 * is a multiple of 16 (>= 16, capacity * 48 < 2^31) with 16-byte aligned
 * scale arrays run on the matrix cores (query heads in groups of 8 per KV
 * head; batch and n_kv_heads * ceil(group / 8) <= 65535), other caches on a
 * vector-unit path with the same results to rounding.
 */
iq_status iq_decode_attention(const float* q,
                              const uint8_t* k_codes, const float* k_norms,
                              const uint8_t* v_codes, const float* v_norms,
                              const int32_t* seq_lens, int64_t capacity,
                              int64_t max_seq_len, const float* quats,
                              int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                              int64_t head_dim, float softmax_scale, float* out,
                              void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/*
 * iq_decode_step - one fused decode step: iq_append_token of (k_new, v_new)
 * followed by iq_decode_attention of q over the advanced lengths (Alg. 1 on
 * the step's new key and value, then App. A / Table 2 on the packed cache;
 * the per-step cache write of App. D), issued as one launch sequence.  The
 * new record is written at position seq_lens[b] by an extra workgroup per
 * (sequence, KV head) of the attention launch, which also contributes the
 * new token to the attention from its fresh record.
 *
 * Results are those of the two separate calls:
 *   - if 0 <= seq_lens[b] < capacity, the token is written at seq_lens[b],
 *     positions 0 .. seq_lens[b] are attended and seq_lens[b] is incremented;
 *   - otherwise the token is dropped, IQ_ERR_CAPACITY is OR-ed into
 *     *status_dev (if not NULL), seq_lens[b] is unchanged and positions
 *     0 .. seq_lens[b]-1 are attended.
 * Attended lengths above max_seq_len are treated as max_seq_len (the token is
 * still written); max_seq_len bounds the lengths after the append and must
 * be >= 1.
 *
 * k_new, v_new : device [batch][n_kv_heads][128] of `dtype`, 16-byte aligned,
 *                both required.
 * Every other argument is as for iq_decode_attention (same workspace size,
 * iq_decode_workspace_bytes) and iq_append_token; seq_lens is read and
 * updated in place.
 */
iq_status iq_decode_step(const float* q, const void* k_new, const void* v_new, int32_t dtype,
                         uint8_t* k_codes, float* k_norms, uint8_t* v_codes, float* v_norms,
                         int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                         const float* quats, int64_t batch, int64_t n_q_heads,
                         int64_t n_kv_heads, int64_t head_dim, float softmax_scale, float* out,
                         void* workspace, size_t workspace_bytes, int32_t* status_dev,
                         hipStream_t stream);

/*
 * iq_decode_step_noalloc - iq_decode_step without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  The split
 * partials go to a static device array of IQ_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends; nothing is
 * allocated or freed by the call.  The array's device address is looked up
 * (hipGetSymbolAddress) on the first call made with each device current,
 * before the arguments are checked.
 *
 * Arguments, results and errors as for iq_decode_step; shapes whose
 * workspace (iq_decode_workspace_bytes) exceeds IQ_NOALLOC_SCRATCH_BYTES
 * return IQ_ERR_WORKSPACE_TOO_SMALL (the 64 MiB hold, e.g., batch 64 with 16
 * query and 2 KV heads at 33K positions, 34.6 MB).  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other streams, other host threads) race
 * and must be serialized by the caller.  The array needs no clearing (every
 * byte a call reads was written earlier in the same call).
 */
#define IQ_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

iq_status iq_decode_step_noalloc(const float* q, const void* k_new, const void* v_new,
                                 int32_t dtype, uint8_t* k_codes, float* k_norms,
                                 uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                                 int64_t capacity, int64_t max_seq_len, const float* quats,
                                 int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                 int64_t head_dim, float softmax_scale, float* out,
                                 int32_t* status_dev, hipStream_t stream);

/*
 * Paged cache (serving with page pools)
 * -------------------------------------
 * The same records (48-byte codes + fp32 scale per vector, Sec. 3.2 Step 4)
 * in a pool of pages shared by all sequences, located through per-sequence
 * page tables instead of one contiguous row per (sequence, KV head):
 *   k_codes / v_codes : device uint8 [n_pages][n_kv_heads][page_size][48],
 *                       16-byte aligned;
 *   k_norms / v_norms : device fp32 [n_pages][n_kv_heads][page_size],
 *                       16-byte aligned (iq_compress_kv_paged: 4);
 *   block_tables      : device int32 [batch][max_pages]: logical position t of
 *                       sequence b lives in page block_tables[b][t / page_size],
 *                       slot t % page_size;
 *   page_size         : positions per page, a power of two, 16 .. 2^20;
 *   capacity          : max_pages * page_size (logical positions per
 *                       sequence), with capacity * 48 < 2^31.
 * A page index outside [0, n_pages) is a caller error: reads then use page 0
 * and writes are skipped, so no access leaves the pools; a fused step whose
 * new position lies on such a page treats it as having no room (nothing
 * written or attended for that token, seq_lens[b] unchanged, IQ_ERR_CAPACITY
 * OR-ed into *status_dev).  The decode entry
 * points run on the matrix cores only: n_q_heads / n_kv_heads an integer
 * <= 16 (IQ_ERR_UNSUPPORTED above), batch and n_kv_heads * ceil(group / 8)
 * <= 65535 (multi-token decode: n_q_heads == 8 * n_kv_heads).  Results
 * equal those of the contiguous entry points on a cache holding the same
 * records; the workspace is sized by iq_decode_workspace_bytes.
 */

/* iq_compress_kv_paged - iq_compress_kv into a paged cache: tokens
 * [0, n_tokens) of every sequence to logical positions dst_offset ..
 * dst_offset + n_tokens - 1 (<= capacity). */
iq_status iq_compress_kv_paged(const void* k, const void* v, int32_t dtype, int64_t batch,
                               int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                               const float* quats, uint8_t* k_codes, float* k_norms,
                               uint8_t* v_codes, float* v_norms, int64_t page_size,
                               int64_t n_pages, const int32_t* block_tables, int64_t max_pages,
                               int64_t dst_offset, hipStream_t stream);

/* iq_decode_attention_paged - iq_decode_attention on a paged cache
 * (max_seq_len <= capacity). */
iq_status iq_decode_attention_paged(const float* q, const uint8_t* k_codes,
                                    const float* k_norms, const uint8_t* v_codes,
                                    const float* v_norms, int64_t page_size, int64_t n_pages,
                                    const int32_t* block_tables, int64_t max_pages,
                                    const int32_t* seq_lens, int64_t max_seq_len,
                                    const float* quats, int64_t batch, int64_t n_q_heads,
                                    int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                                    float* out, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/* iq_decode_step_paged - iq_decode_step on a paged cache: the new token goes
 * to logical position seq_lens[b] (the caller has mapped its page), if
 * below capacity. */
iq_status iq_decode_step_paged(const float* q, const void* k_new, const void* v_new,
                               int32_t dtype, uint8_t* k_codes, float* k_norms,
                               uint8_t* v_codes, float* v_norms, int64_t page_size,
                               int64_t n_pages, const int32_t* block_tables, int64_t max_pages,
                               int32_t* seq_lens, int64_t max_seq_len, const float* quats,
                               int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                               int64_t head_dim, float softmax_scale, float* out,
                               void* workspace, size_t workspace_bytes, int32_t* status_dev,
                               hipStream_t stream);

/*
 * Reconstruct-then-compute baseline (Sec. 1, Fig. 1 top)
 * ------------------------------------------------------
 * The pipeline the compressed-space path replaces: dequantize the packed
 * cache and apply R^-1 to every token, materializing fp16 tensors, then run
 * ordinary attention on them.  These entry points exist so that the two
 * pipelines can be compared on the same shapes; iq_decode_attention_f16 is
 * also plain decode attention on an uncompressed fp16 cache.
 */

/*
 * iq_dequantize_kv - materialize cache records as original-space vectors
 * (the "Dequant R^-1" stage of Fig. 1 top): x_hat = s R_g^T C[code] for
 * every token, with R_g = diag(M_i) H_128 / sqrt(128) the rotation of Eq. 2
 * and C the codebook of iq_codebook.  Computed in fp32 and rounded once to
 * the output type.
 *
 * k_codes/k_norms, v_codes/v_norms : device, a cache as written by
 *               iq_compress_kv ([batch][n_kv_heads][capacity][48] uint8 and
 *               [batch][n_kv_heads][capacity] fp32).  Either side may be NULL
 *               together with its output; not both.
 * quats       : device fp32 [n_kv_heads][32][2][4], 16-byte aligned.
 * seq_lens    : optional device int32 [batch]; when given, output token t of
 *               sequence b is written only if src_offset + t < seq_lens[b].
 * k_out/v_out : device [batch][n_kv_heads][n_tokens][128] of `out_dtype`
 *               (IQ_DTYPE_F16 or IQ_DTYPE_F32), 16-byte aligned; token t
 *               comes from cache position src_offset + t.  Tokens not written
 *               keep their contents.
 * Requires 0 <= src_offset and src_offset + n_tokens <= capacity.
 * n_tokens == 0 or batch == 0 is a valid no-op.
 */
iq_status iq_dequantize_kv(const uint8_t* k_codes, const float* k_norms,
                           const uint8_t* v_codes, const float* v_norms,
                           const float* quats, const int32_t* seq_lens,
                           int64_t batch, int64_t n_kv_heads, int64_t n_tokens,
                           int64_t head_dim, int64_t capacity, int64_t src_offset,
                           int32_t out_dtype, void* k_out, void* v_out,
                           hipStream_t stream);

/*
 * iq_decode_f16_workspace_bytes - device workspace iq_decode_attention_f16
 * needs for these shapes (split partial results).  0 for invalid shapes.
 */
size_t iq_decode_f16_workspace_bytes(int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                     int64_t max_seq_len, int64_t head_dim);

/*
 * iq_decode_attention_f16 - single-token decode attention on an fp16 cache
 * (the "GEMM Q K^T, softmax, . V" stages of Fig. 1 top): per query head h of
 * KV head g = h / (n_q_heads / n_kv_heads),
 *   o = sum_j softmax_j(scale * q_h . k_j) v_j,   j < seq_lens[b],
 * split over workgroups (flash-decoding) and merged; fp32 accumulation.
 *
 * q        : device fp32 [batch][n_q_heads][128], 16-byte aligned;
 *            |q_i| * scale must stay below 4e4 (the query is carried as fp16
 *            hi + lo parts).
 * k, v     : device fp16 [batch][n_kv_heads][capacity][128], 16-byte aligned
 *            (e.g. the output of iq_dequantize_kv with n_tokens = capacity).
 * seq_lens, capacity, max_seq_len, softmax_scale, out : as for
 *            iq_decode_attention.
 * workspace : device, >= iq_decode_f16_workspace_bytes(...) bytes, 256-byte
 *            aligned, contents ignored; calls sharing it must not overlap.
 * n_q_heads / n_kv_heads must be an integer <= 8 (IQ_ERR_UNSUPPORTED above).
 */
iq_status iq_decode_attention_f16(const float* q, const void* k, const void* v,
                                  const int32_t* seq_lens, int64_t capacity,
                                  int64_t max_seq_len, int64_t batch, int64_t n_q_heads,
                                  int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                                  float* out, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/*
 * Other code widths (Algorithm 1 at b = 2 and b = 4)
 * ---------------------------------------------------
 * Algorithm 1 quantizes to b bits per coordinate with the Lloyd-Max codebook
 * C_b of the same sphere marginal and packs the codes into d*b/8 bytes
 * (Sec. 3.2 Steps 3-4); the paper's cache uses b = 3.  These entry points
 * take b explicitly: records are 16*b bytes (32 at b = 2, 48 at b = 3, 64 at
 * b = 4), code i at bits b*i .. b*i+b-1 of the little-endian bit string,
 * scales and every other layout and argument as for the 3-bit entry points.
 * b = 3 gives exactly the results of iq_codebook / iq_compress_kv /
 * iq_decode_attention / iq_decode_step.  Any other b returns
 * IQ_ERR_UNSUPPORTED.
 */

/* C_b: levels[2^b] and thresholds[2^b - 1] (host memory, either may be
 * NULL), built as for iq_codebook. */
iq_status iq_codebook_bits(int bits, float* levels, float* thresholds);

/* iq_compress_kv writing b-bit records: k_codes / v_codes are
 * [batch][n_kv_heads][capacity][16*bits] uint8, 16-byte aligned. */
iq_status iq_compress_kv_bits(const void* k, const void* v, int32_t dtype,
                              int64_t batch, int64_t n_kv_heads, int64_t n_tokens,
                              int64_t head_dim, const float* quats,
                              uint8_t* k_codes, float* k_norms,
                              uint8_t* v_codes, float* v_norms,
                              int64_t capacity, int64_t dst_offset, int bits,
                              hipStream_t stream);

/* iq_decode_attention on b-bit records (workspace as sized by
 * iq_decode_workspace_bytes).  b = 2 and b = 4 run on the matrix-core path
 * only: capacity a multiple of 16 (>= 16) with capacity * 16 * bits < 2^31,
 * 16-byte aligned scale arrays, batch and n_kv_heads * ceil(group / 8) <=
 * 65535 (group = n_q_heads / n_kv_heads <= 16); otherwise
 * IQ_ERR_UNSUPPORTED. */
iq_status iq_decode_attention_bits(const float* q,
                                   const uint8_t* k_codes, const float* k_norms,
                                   const uint8_t* v_codes, const float* v_norms,
                                   const int32_t* seq_lens, int64_t capacity,
                                   int64_t max_seq_len, const float* quats,
                                   int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                   int64_t head_dim, float softmax_scale, float* out,
                                   void* workspace, size_t workspace_bytes, int bits,
                                   hipStream_t stream);

/* iq_decode_step on b-bit records: the new key and value are compressed at
 * b bits into position seq_lens[b] (Algorithm 1 with C_b), then attended
 * with the cache; requirements as for iq_decode_attention_bits, status and
 * length advance as for iq_decode_step. */
iq_status iq_decode_step_bits(const float* q, const void* k_new, const void* v_new,
                              int32_t dtype, uint8_t* k_codes, float* k_norms,
                              uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                              int64_t capacity, int64_t max_seq_len, const float* quats,
                              int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                              int64_t head_dim, float softmax_scale, float* out, void* workspace,
                              size_t workspace_bytes, int32_t* status_dev, int bits,
                              hipStream_t stream);

/*
 * Multi-token decode (the verification step of speculative decoding)
 * ------------------------------------------------------------------
 * n_tokens query tokens per sequence attend one packed cache that
 * already holds them at its last n_tokens positions: token t of sequence b
 * attends positions 0 .. L_b - n_tokens + t, with L_b = min(seq_lens[b],
 * max_seq_len) (causal among the new tokens; a token with no position gives
 * a zero row).  Each token is App. A decode attention with that length; the
 * cache is read once for all tokens.
 *   q, out    : device fp32 [batch][n_tokens][n_q_heads][128], 16-byte
 *               aligned (original space).
 *   n_tokens  : 1 .. 4 (1 is iq_decode_attention);
 *   iq_decode_attention_multi reads 3-bit records (the paper's cache);
 *   workspace : >= iq_decode_multi_workspace_bytes(...) bytes, 256-byte
 *               aligned, contents ignored on entry.
 * Other arguments as for iq_decode_attention.  n_tokens >= 2 runs on the
 * matrix-core path only (n_q_heads == 8 * n_kv_heads, capacity a multiple
 * of 16 and >= 16, 16-byte aligned scale arrays, batch and n_kv_heads <=
 * 65535, batch * n_tokens <= 65535); otherwise IQ_ERR_UNSUPPORTED, and
 * iq_decode_multi_workspace_bytes returns 0 for such shapes.
 */
size_t iq_decode_multi_workspace_bytes(int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                                       int64_t n_kv_heads, int64_t max_seq_len,
                                       int64_t head_dim);

iq_status iq_decode_attention_multi(const float* q,
                                    const uint8_t* k_codes, const float* k_norms,
                                    const uint8_t* v_codes, const float* v_norms,
                                    const int32_t* seq_lens, int64_t capacity,
                                    int64_t max_seq_len, const float* quats,
                                    int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                                    int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                                    float* out, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/* iq_decode_attention_multi on a paged cache (pools, page_size, n_pages,
 * block_tables, max_pages as for iq_decode_attention_paged; capacity is
 * max_pages * page_size); workspace as sized by
 * iq_decode_multi_workspace_bytes.  Results equal those of
 * iq_decode_attention_multi on a contiguous cache holding the same records. */
iq_status iq_decode_attention_multi_paged(const float* q,
                                          const uint8_t* k_codes, const float* k_norms,
                                          const uint8_t* v_codes, const float* v_norms,
                                          int64_t page_size, int64_t n_pages,
                                          const int32_t* block_tables, int64_t max_pages,
                                          const int32_t* seq_lens, int64_t max_seq_len,
                                          const float* quats, int64_t batch, int64_t n_tokens,
                                          int64_t n_q_heads, int64_t n_kv_heads,
                                          int64_t head_dim, float softmax_scale, float* out,
                                          void* workspace, size_t workspace_bytes,
                                          hipStream_t stream);

/* iq_decode_attention_multi on records of `bits` bits (2, 3 or 4; Algorithm
 * 1 with C_b, records of 4 * bits words written by iq_compress_kv_bits).
 * n_tokens == 1 is iq_decode_attention_bits. */
iq_status iq_decode_attention_multi_bits(const float* q,
                                         const uint8_t* k_codes, const float* k_norms,
                                         const uint8_t* v_codes, const float* v_norms,
                                         const int32_t* seq_lens, int64_t capacity,
                                         int64_t max_seq_len, const float* quats,
                                         int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                                         int64_t n_kv_heads, int64_t head_dim,
                                         float softmax_scale, float* out, void* workspace,
                                         size_t workspace_bytes, int bits,
                                         hipStream_t stream);

/* The fused multi-token step (speculative verification with its append):
 * the n_tokens new keys and values of each sequence (k_new, v_new: device
 * [batch][n_tokens][n_kv_heads][128] of `dtype`, 16-byte aligned) are
 * compressed to `bits`-bit records (Algorithm 1 with C_b) and written at
 * positions seq_lens[b] .. seq_lens[b] + n_tokens - 1; token t attends the
 * cached positions before seq_lens[b] and the new positions 0 .. t (causal
 * among the new tokens; a position at or past max_seq_len is not attended);
 * seq_lens[b] is then advanced by n_tokens.  The result equals that of
 * iq_compress_kv_bits of the new tokens at dst_offset seq_lens[b] followed
 * by iq_decode_attention_multi_bits with the advanced lengths.  When the
 * n_tokens records do not all fit (seq_lens[b] + n_tokens > capacity) none
 * is written, the length is left as it was, the tokens attend the cached
 * positions only, and IQ_ERR_CAPACITY is ORed into *status_dev (optional,
 * device int32).  n_tokens == 1 is iq_decode_step_bits.  Other arguments
 * and restrictions as for iq_decode_attention_multi_bits; the workspace as
 * sized by iq_decode_multi_workspace_bytes. */
iq_status iq_decode_step_multi(const float* q, const void* k_new, const void* v_new,
                               int32_t dtype, uint8_t* k_codes, float* k_norms,
                               uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                               int64_t capacity, int64_t max_seq_len, const float* quats,
                               int64_t batch, int64_t n_tokens, int64_t n_q_heads,
                               int64_t n_kv_heads, int64_t head_dim, float softmax_scale,
                               float* out, void* workspace, size_t workspace_bytes,
                               int32_t* status_dev, int bits, hipStream_t stream);

/*
 * Content / RoPE sub-block split (Sec. 5, "MLA/RoPE hard blocker"; Sec. 6)
 * -------------------------------------------------------------------------
 * Latent-attention models (e.g. DeepSeek-V2) split each key into a content
 * part and a positional part that carries the rotary phase; the positional
 * part must be neither rotated nor quantized.  Here the content part of
 * every key (128 dims) is compressed as any other key (iq_compress_kv), the
 * positional part (64 dims) is stored by the caller as fp16 as it is, and
 * values are content only.  For query head h of KV head g:
 *   score_j = scale * ( s^K_j (R_g q_h) . C[codeK_j] + q_rope_h . k_rope_j )
 *   o       = R_g^T sum_j softmax_j(score) s^V_j C[codeV_j].
 *
 * q, caches, seq_lens, capacity, max_seq_len, quats, out, workspace : as for
 *            iq_decode_attention (same workspace size).
 * q_rope   : device fp32 [batch][n_q_heads][64], 16-byte aligned.
 * k_rope   : device fp16 [batch][n_rope_heads][capacity][64], 16-byte
 *            aligned; n_rope_heads 1 (one positional key per token shared by
 *            every head, the latent-attention layout) or n_kv_heads.
 * rope_dim : 64 (IQ_ERR_UNSUPPORTED otherwise).
 * softmax_scale : <= 0 selects 1/sqrt(128 + 64).
 * |q_rope_i| * scale must stay below 4e4 (carried as fp16 hi + lo parts).
 * Runs on the matrix-core path only (capacity a multiple of 16 and >= 16,
 * 16-byte aligned scale arrays, group <= 16; IQ_ERR_UNSUPPORTED otherwise).
 */
iq_status iq_decode_attention_rope(const float* q, const float* q_rope, const uint8_t* k_codes,
                                   const float* k_norms, const void* k_rope,
                                   int64_t n_rope_heads, const uint8_t* v_codes,
                                   const float* v_norms, const int32_t* seq_lens,
                                   int64_t capacity, int64_t max_seq_len, const float* quats,
                                   int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                                   int64_t head_dim, int64_t rope_dim, float softmax_scale,
                                   float* out, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Fitted codebooks (Sec. 3.2 Step 3 on calibration data)
 * ------------------------------------------------------
 * Step 3 quantizes with the Lloyd-Max levels of the marginal of one rotated
 * coordinate; the library's C_b reads that marginal analytically (the sphere
 * marginal, iq_codebook).  The paper also counts codebook entries among the
 * method's fitted parameters ("Why structured rotation works").  These entry
 * points fit the levels to measured data and run compression, decode and
 * the fused step with such a codebook.  A codebook is passed by host pointer
 * (read during the call, not retained):
 *   bits       : 2, 3 or 4;
 *   levels     : the first 2^bits entries, strictly ascending, each exactly
 *                representable in fp16, |level| < 1 (levels of the
 *                normalized, rotated coordinate), and symmetric:
 *                levels[i] == -levels[2^bits - 1 - i];
 *   thresholds : the first 2^bits - 1 entries, exactly the fp32 midpoints
 *                of adjacent levels.
 * Anything else returns IQ_ERR_INVALID_ARGUMENT (IQ_ERR_UNSUPPORTED for
 * bits).  A cache written with one codebook must be decoded with the same
 * codebook; the record layout is that of the *_bits entry points.
 */
typedef struct iq_codebook_t {
  int32_t bits;
  float levels[16];
  float thresholds[15];
} iq_codebook_t;

/*
 * iq_fit_codebook - Lloyd-Max levels of the empirical distribution of the
 * rotated, normalized calibration coordinates y = R x / ||x|| (Eq. 2, R from
 * quats_host, the parameters the cache will be written with): the sample of
 * every coordinate of every non-zero finite calibration vector of every
 * head, together with its negation (the marginal is symmetric, and the
 * compression quantizer relies on it); Lloyd's iteration (thresholds =
 * midpoints, level = mean of its cell, cell j = {t_(j-1) <= y < t_j}, an
 * empty cell keeps its level) from C_b until no cell changes; levels then
 * rounded to the nearest fp16 value and made exactly symmetric, thresholds
 * their midpoints.  Host memory: calib[n_kv_heads][n_vectors][128] fp32,
 * quats_host[n_kv_heads][32][2][4], *out written on success.
 * 1 <= n_vectors, n_vectors * n_kv_heads <= 2^24.  IQ_ERR_INVALID_ARGUMENT
 * also when no calibration vector is usable.  Pure host function.
 */
iq_status iq_fit_codebook(const float* calib, int64_t n_vectors, int64_t n_kv_heads,
                          int64_t head_dim, const float* quats_host, int32_t bits,
                          iq_codebook_t* out);

/* iq_compress_kv with codebook *cb: records of cb->bits bits (layout of
 * iq_compress_kv_bits). */
iq_status iq_compress_kv_cb(const void* k, const void* v, int32_t dtype, int64_t batch,
                            int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                            const float* quats, const iq_codebook_t* cb, uint8_t* k_codes,
                            float* k_norms, uint8_t* v_codes, float* v_norms, int64_t capacity,
                            int64_t dst_offset, hipStream_t stream);

/* iq_decode_attention on records written with codebook *cb (paths and
 * restrictions of iq_decode_attention_bits at cb->bits). */
iq_status iq_decode_attention_cb(const float* q, const uint8_t* k_codes, const float* k_norms,
                                 const uint8_t* v_codes, const float* v_norms,
                                 const int32_t* seq_lens, int64_t capacity, int64_t max_seq_len,
                                 const float* quats, const iq_codebook_t* cb, int64_t batch,
                                 int64_t n_q_heads, int64_t n_kv_heads, int64_t head_dim,
                                 float softmax_scale, float* out, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* iq_decode_step with codebook *cb for the new records and the attention
 * (restrictions of iq_decode_step_bits at cb->bits). */
iq_status iq_decode_step_cb(const float* q, const void* k_new, const void* v_new,
                            int32_t dtype, uint8_t* k_codes, float* k_norms, uint8_t* v_codes,
                            float* v_norms, int32_t* seq_lens, int64_t capacity,
                            int64_t max_seq_len, const float* quats, const iq_codebook_t* cb,
                            int64_t batch, int64_t n_q_heads, int64_t n_kv_heads,
                            int64_t head_dim, float softmax_scale, float* out, void* workspace,
                            size_t workspace_bytes, int32_t* status_dev, hipStream_t stream);

/* iq_dequantize_kv of records written with codebook *cb (3-bit codebooks
 * only; IQ_ERR_UNSUPPORTED otherwise). */
iq_status iq_dequantize_kv_cb(const uint8_t* k_codes, const float* k_norms,
                              const uint8_t* v_codes, const float* v_norms, const float* quats,
                              const iq_codebook_t* cb, const int32_t* seq_lens, int64_t batch,
                              int64_t n_kv_heads, int64_t n_tokens, int64_t head_dim,
                              int64_t capacity, int64_t src_offset, int32_t out_dtype,
                              void* k_out, void* v_out, hipStream_t stream);

/*
 * Measurement support (not part of the method)
 * ---------------------------------------------
 * The decode step is bound by HBM bandwidth (its algorithmic bytes are the
 * records and scales it streams, Sec. 3.4 and Table 2).  iq_stream_read is
 * the reference point for what one launch can reach: it reads `bytes` of
 * `src` with 16-byte loads, loads_per_thread per thread, all issued before
 * any is used, consecutive threads on consecutive 16-byte words; workgroups
 * of block_threads threads (64, 128, 256, 512 or 1024), loads_per_thread
 * 1, 2, 4, 8 or 16.
 *
 * src        : device, 16-byte aligned, `bytes` a multiple of 16 (0 = no-op).
 * sink       : device uint32 [sink_words], sink_words >=
 *              iq_stream_read_sink_words(bytes, block_threads,
 *              loads_per_thread) (the number of workgroups); word w is
 *              written only if the XOR of every word workgroup w read equals
 *              `sentinel`, so a run normally writes nothing.
 * Returns IQ_ERR_INVALID_ARGUMENT for any other shape or a null or
 * misaligned pointer, IQ_ERR_HIP if the launch fails.
 */
size_t iq_stream_read_sink_words(size_t bytes, int32_t block_threads, int32_t loads_per_thread);

iq_status iq_stream_read(const void* src, size_t bytes, uint32_t* sink, size_t sink_words,
                         int32_t block_threads, int32_t loads_per_thread, uint32_t sentinel,
                         hipStream_t stream);

#ifdef __cplusplus
}  /* extern "C" */
#endif

#endif  /* ISOQUANT_H_ */
