// Measurement support, not part of the method: a plain streaming read of a
// device buffer, the reference point for the bandwidth a single launch of
// the decode step can reach on this machine.  The decode step's roofline
// is HBM (its algorithmic bytes are the packed records and scales it
// streams, Sec. 3.4 and Table 2), so its achieved bandwidth is reported
// against both the nominal HBM peak and what this kernel reaches on a
// buffer of the same size, read cold.
//
// Each thread issues kLoads 16-byte loads before it uses any of them
// (consecutive threads read consecutive 16-byte words, so every wave load
// is one coalesced 1 KiB access), folds them into one word, and writes only
// if the fold equals a sentinel the host passes at run time: the loads
// cannot be removed, and a real run writes nothing.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "isoquant.h"

namespace iq {
namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int kLoads>
__global__ void stream_read_kernel(const u32x4_t* __restrict__ src, uint64_t n16,
                                   uint32_t* __restrict__ sink, uint32_t sentinel) {
  const uint64_t base = static_cast<uint64_t>(blockIdx.x) * blockDim.x * kLoads + threadIdx.x;
  u32x4_t v[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const uint64_t i = base + static_cast<uint64_t>(j) * blockDim.x;
    v[j] = i < n16 ? src[i] : u32x4_t{0u, 0u, 0u, 0u};
  }
  uint32_t f = 0;
#pragma unroll
  for (int j = 0; j < kLoads; ++j) f ^= v[j][0] ^ v[j][1] ^ v[j][2] ^ v[j][3];
  if (f == sentinel) sink[blockIdx.x] = f;
}

}  // namespace
}  // namespace iq

extern "C" {

size_t iq_stream_read_sink_words(size_t bytes, int32_t block_threads, int32_t loads_per_thread) {
  if (block_threads <= 0 || loads_per_thread <= 0) return 0;
  const size_t per = static_cast<size_t>(block_threads) * loads_per_thread * 16;
  return bytes == 0 ? 0 : (bytes + per - 1) / per;
}

iq_status iq_stream_read(const void* src, size_t bytes, uint32_t* sink, size_t sink_words,
                         int32_t block_threads, int32_t loads_per_thread, uint32_t sentinel,
                         hipStream_t stream) {
  if (block_threads != 64 && block_threads != 128 && block_threads != 256 &&
      block_threads != 512 && block_threads != 1024)
    return IQ_ERR_INVALID_ARGUMENT;
  if (loads_per_thread != 1 && loads_per_thread != 2 && loads_per_thread != 4 &&
      loads_per_thread != 8 && loads_per_thread != 16)
    return IQ_ERR_INVALID_ARGUMENT;
  if (bytes % 16) return IQ_ERR_INVALID_ARGUMENT;
  if (bytes == 0) return IQ_OK;
  if (!src || !sink || reinterpret_cast<uintptr_t>(src) % 16 ||
      reinterpret_cast<uintptr_t>(sink) % 4)
    return IQ_ERR_INVALID_ARGUMENT;
  const size_t grid = iq_stream_read_sink_words(bytes, block_threads, loads_per_thread);
  if (grid > 0x7fffffff || sink_words < grid) return IQ_ERR_INVALID_ARGUMENT;
  const auto* s = static_cast<const iq::u32x4_t*>(src);
  const uint64_t n16 = bytes / 16;
  const dim3 g(static_cast<unsigned>(grid)), b(static_cast<unsigned>(block_threads));
  switch (loads_per_thread) {
    case 1: hipLaunchKernelGGL(iq::stream_read_kernel<1>, g, b, 0, stream, s, n16, sink, sentinel); break;
    case 2: hipLaunchKernelGGL(iq::stream_read_kernel<2>, g, b, 0, stream, s, n16, sink, sentinel); break;
    case 4: hipLaunchKernelGGL(iq::stream_read_kernel<4>, g, b, 0, stream, s, n16, sink, sentinel); break;
    case 8: hipLaunchKernelGGL(iq::stream_read_kernel<8>, g, b, 0, stream, s, n16, sink, sentinel); break;
    default: hipLaunchKernelGGL(iq::stream_read_kernel<16>, g, b, 0, stream, s, n16, sink, sentinel); break;
  }
  return hipGetLastError() == hipSuccess ? IQ_OK : IQ_ERR_HIP;
}

}  // extern "C"
