// The fused decode step (iq_decode_step) without a caller workspace, for
// callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops, harnesses that forbid allocation).  Its split
// partials live in a file-scope device array of IQ_NOALLOC_SCRATCH_BYTES,
// one copy per GPU, held until the process ends.
//
// In host code the array's name is only a stand-in for the symbol: its
// device address is looked up once per device (hipGetSymbolAddress, with
// that device current) and that address is what the kernels receive.
// Nothing in the array has to start at zero: every byte a decode call reads
// was written earlier in the same call.  Calls that overlap on one GPU share
// the array and race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "isoquant.h"

namespace {

static __device__ __align__(256) unsigned char scratch[IQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch`, per device

// Device address of this device's scratch array (looked up on the first
// call made with the device current).
iq_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return IQ_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return IQ_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return IQ_OK;
}

}  // namespace

extern "C" iq_status iq_decode_step_noalloc(const float* q, const void* k_new, const void* v_new,
                                            int32_t dtype, uint8_t* k_codes, float* k_norms,
                                            uint8_t* v_codes, float* v_norms, int32_t* seq_lens,
                                            int64_t capacity, int64_t max_seq_len,
                                            const float* quats, int64_t batch,
                                            int64_t n_q_heads, int64_t n_kv_heads,
                                            int64_t head_dim, float softmax_scale, float* out,
                                            int32_t* status_dev, hipStream_t stream) {
  if (head_dim != IQ_HEAD_DIM) return IQ_ERR_UNSUPPORTED;
  // the workspace these shapes need must fit the static array
  const size_t need =
      iq_decode_workspace_bytes(batch, n_q_heads, n_kv_heads, max_seq_len, head_dim);
  if (need == 0) return IQ_ERR_INVALID_ARGUMENT;
  if (need > IQ_NOALLOC_SCRATCH_BYTES) return IQ_ERR_WORKSPACE_TOO_SMALL;
  void* ws = nullptr;
  const iq_status st = scratch_address(&ws);
  if (st != IQ_OK) return st;
  // every other check, and the launches, as in iq_decode_step
  return iq_decode_step(q, k_new, v_new, dtype, k_codes, k_norms, v_codes, v_norms, seq_lens,
                        capacity, max_seq_len, quats, batch, n_q_heads, n_kv_heads, head_dim,
                        softmax_scale, out, ws, IQ_NOALLOC_SCRATCH_BYTES, status_dev, stream);
}
