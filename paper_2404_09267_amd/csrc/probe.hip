// Plain streaming kernel for the benchmark's practical ceiling (see tg_probe.h).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "tg_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;

// Workgroup g reads read16 / n_chunks 16-byte words starting at its share of src and
// writes chunk16 words: run16 words at g * run16 of each of the `planes` planes of
// plane16 words. The read words are folded into the written values so the loads cannot
// be dropped.
__global__ __launch_bounds__(kThreads) void stream_kernel(const u32x4 *src, int64_t read16,
                                                          u32x4 *dst, int64_t plane16,
                                                          int64_t run16, int32_t planes,
                                                          int64_t n_chunks) {
  const int64_t g = blockIdx.x;
  const int64_t r0 = read16 * g / n_chunks, r1 = read16 * (g + 1) / n_chunks;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int64_t i = r0 + threadIdx.x; i < r1; i += kThreads) acc ^= src[i];
  const int64_t w0 = g * run16, w1 = w0 + run16 < plane16 ? w0 + run16 : plane16;
  for (int p = 0; p < planes; ++p)
    for (int64_t i = w0 + threadIdx.x; i < w1; i += kThreads)
      __builtin_nontemporal_store(acc + static_cast<uint32_t>(i),
                                  dst + static_cast<int64_t>(p) * plane16 + i);
}

}  // namespace

extern "C" int tg_probe_stream_planes(const void *src, int64_t read_bytes, void *dst,
                                      int64_t write_bytes, int32_t chunk, int32_t planes,
                                      void *stream) {
  if (!src || !dst || read_bytes < 0 || write_bytes <= 0 || read_bytes % 16 || planes < 1 ||
      planes > 4 || write_bytes % (16 * planes) || chunk < 4096 || chunk % 4096 ||
      reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
    return -1;
  const int64_t plane16 = write_bytes / 16 / planes;
  const int64_t run16 = (chunk / 16 + planes - 1) / planes;
  const int64_t n_chunks = (plane16 + run16 - 1) / run16;
  if (n_chunks > 0x7FFFFFFF) return -1;
  hipLaunchKernelGGL(stream_kernel, dim3(static_cast<uint32_t>(n_chunks)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4 *>(src),
                     read_bytes / 16, static_cast<u32x4 *>(dst), plane16, run16, planes,
                     n_chunks);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int tg_probe_stream(const void *src, int64_t read_bytes, void *dst,
                               int64_t write_bytes, int32_t chunk, void *stream) {
  return tg_probe_stream_planes(src, read_bytes, dst, write_bytes, chunk, 1, stream);
}
