// Plain streaming kernel for the benchmark's practical ceiling (see tg_probe.h).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "tg_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;

// Workgroup g reads read16 / n_chunks 16-byte words starting at its share of src and
// writes chunk16 words at g * chunk16 of dst; the read words are folded into the
// written values so the loads cannot be dropped.
__global__ __launch_bounds__(kThreads) void stream_kernel(const u32x4 *src, int64_t read16,
                                                          u32x4 *dst, int64_t write16,
                                                          int64_t chunk16, int64_t n_chunks) {
  const int64_t g = blockIdx.x;
  const int64_t r0 = read16 * g / n_chunks, r1 = read16 * (g + 1) / n_chunks;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int64_t i = r0 + threadIdx.x; i < r1; i += kThreads) acc ^= src[i];
  const int64_t w0 = g * chunk16, w1 = w0 + chunk16 < write16 ? w0 + chunk16 : write16;
  for (int64_t i = w0 + threadIdx.x; i < w1; i += kThreads)
    __builtin_nontemporal_store(acc + static_cast<uint32_t>(i), dst + i);
}

}  // namespace

extern "C" int tg_probe_stream(const void *src, int64_t read_bytes, void *dst,
                               int64_t write_bytes, int32_t chunk, void *stream) {
  if (!src || !dst || read_bytes < 0 || write_bytes <= 0 || read_bytes % 16 ||
      write_bytes % 16 || chunk < 4096 || chunk % 4096 ||
      reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
    return -1;
  const int64_t n_chunks = (write_bytes + chunk - 1) / chunk;
  if (n_chunks > 0x7FFFFFFF) return -1;
  hipLaunchKernelGGL(stream_kernel, dim3(static_cast<uint32_t>(n_chunks)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4 *>(src),
                     read_bytes / 16, static_cast<u32x4 *>(dst), write_bytes / 16, chunk / 16,
                     n_chunks);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
