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

// Workgroup g replays one stitch unit's memory traffic with no work of its own: it reads
// the 16-byte words covering the byte ranges [off[k], off[k] + len[k]) of src for k in
// [begin[g], begin[g + 1]) -- every thread a strided share of their concatenation,
// kReplayChunks ranges at a time -- and then writes the unit's run of run16 words in each
// of the three planes of its canvas (canvas g / runs, run g % runs; planes of plane16
// words, canvases of three planes). The read words are folded into the written values.
constexpr int kReplayThreads = 128;
constexpr int kReplayChunks = 128;

__global__ __launch_bounds__(kReplayThreads) void replay_kernel(
    const u32x4 *src, const int64_t *off, const int32_t *len, const int32_t *begin, u32x4 *dst,
    int64_t plane16, int64_t run16, int32_t runs) {
  __shared__ int64_t s_first[kReplayChunks];   // first word of each range
  __shared__ int32_t s_start[kReplayChunks];   // its first position in the concatenation
  __shared__ int32_t s_wave[kReplayThreads / 64];
  const int g = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int k0 = begin[g], k1 = begin[g + 1];
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int kb = k0; kb < k1; kb += kReplayChunks) {
    const int nk = min(kReplayChunks, k1 - kb);
    int cnt = 0;
    int64_t a = 0;
    if (t < nk) {
      a = off[kb + t] >> 4;
      cnt = static_cast<int>(((off[kb + t] + len[kb + t] + 15) >> 4) - a);
    }
    int incl = cnt;
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if (lane >= o) incl += u;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    const int base = wave > 0 ? s_wave[0] : 0;
    const int total = s_wave[0] + s_wave[1];
    if (t < nk) {
      s_first[t] = a;
      s_start[t] = base + incl - cnt;
    }
    __syncthreads();
    // four words per thread and step, all four loads issued before any is used
    for (int w0 = t; w0 < total; w0 += 4 * kReplayThreads) {
      u32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int w = w0 + u * kReplayThreads;
        v[u] = u32x4{0u, 0u, 0u, 0u};
        if (w < total) {
          int c = 0;  // the last range starting at or before w
          for (int step = kReplayChunks / 2; step > 0; step >>= 1)
            if (c + step < nk && s_start[c + step] <= w) c += step;
          v[u] = src[s_first[c] + (w - s_start[c])];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) acc ^= v[u];
    }
    __syncthreads();
  }
  const int64_t cl = g / runs, r = g - cl * runs;
  const int64_t w0 = r * run16, w1 = w0 + run16 < plane16 ? w0 + run16 : plane16;
  for (int p = 0; p < 3; ++p)
    for (int64_t i = w0 + t; i < w1; i += kReplayThreads)
      __builtin_nontemporal_store(acc + static_cast<uint32_t>(i), dst + (cl * 3 + p) * plane16 + i);
}

}  // namespace

extern "C" int tg_probe_replay(const void *src, int64_t src_bytes, const int64_t *off,
                               const int32_t *len, const int32_t *begin, int32_t n_units,
                               int32_t units_per_canvas, void *dst, int64_t plane_bytes,
                               int64_t run_bytes, void *stream) {
  if (!src || !off || !len || !begin || !dst || n_units < 1 || units_per_canvas < 1 ||
      n_units % units_per_canvas || plane_bytes < 16 || plane_bytes % 16 || run_bytes < 16 ||
      run_bytes % 16 || src_bytes < 0 ||
      reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16)
    return -1;
  (void)src_bytes;  // the caller checks every range against it on the host
  hipLaunchKernelGGL(replay_kernel, dim3(static_cast<uint32_t>(n_units)), dim3(kReplayThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4 *>(src), off, len,
                     begin, static_cast<u32x4 *>(dst), plane_bytes / 16, run_bytes / 16,
                     units_per_canvas);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

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
