// tg_plan_upload: a step's plan from pinned host memory to the device in one kernel.
//
// The plan is made on the host (tg_plan_pack) and read by every stitch workgroup from
// device memory, so a serving loop moves it across PCIe once per step. A runtime copy
// from pinned memory costs a set-up of its own between kernels on the stream (about
// 10 us measured, against 3-4 us of copying for a 40 KB plan); this kernel instead reads
// the pinned buffer directly over PCIe and follows the previous kernel at once. It moves
// bytes only: no step of the method is computed here.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "tg.h"

namespace {

constexpr int kThreads = 256;
constexpr int kMaxBlocks = 1024;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Grid-stride copy: 16-byte words when both ends are 16-byte aligned, then the tail (or
// everything, when they are not) byte by byte.
__global__ __launch_bounds__(kThreads) void upload_kernel(const uint8_t *src, uint8_t *dst,
                                                          uint64_t bytes, int wide) {
  const uint64_t stride = uint64_t(gridDim.x) * kThreads;
  const uint64_t t = uint64_t(blockIdx.x) * kThreads + threadIdx.x;
  uint64_t done = 0;
  if (wide) {
    const uint64_t n16 = bytes / 16;
    const u32x4 *s = reinterpret_cast<const u32x4 *>(src);
    u32x4 *d = reinterpret_cast<u32x4 *>(dst);
    for (uint64_t i = t; i < n16; i += stride) d[i] = s[i];
    done = n16 * 16;
  }
  for (uint64_t i = done + t; i < bytes; i += stride) dst[i] = src[i];
}

}  // namespace

extern "C" int tg_plan_upload(const void *src, void *dst, size_t bytes, void *stream) {
  if (bytes == 0) return TG_OK;
  if (!src || !dst) return TG_E_INVAL;
  // the device's address of the pinned buffer; fails for memory that is not pinned
  void *dsrc = nullptr;
  if (hipHostGetDevicePointer(&dsrc, const_cast<void *>(src), 0) != hipSuccess || !dsrc) {
    (void)hipGetLastError();  // clear the failed lookup's error
    return TG_E_INVAL;
  }
  const int wide = (reinterpret_cast<uintptr_t>(dsrc) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(dst) % 16 == 0);
  const uint64_t words = wide ? (bytes + 15) / 16 : bytes;
  uint64_t blocks = (words + kThreads - 1) / kThreads;
  if (blocks > kMaxBlocks) blocks = kMaxBlocks;
  hipLaunchKernelGGL(upload_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint8_t *>(dsrc),
                     static_cast<uint8_t *>(dst), static_cast<uint64_t>(bytes), wide);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
