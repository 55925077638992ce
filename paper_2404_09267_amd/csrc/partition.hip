// tg_partition: adaptive frame partitioning of RoIs into zone patches.
//
// Small objects far from a high-resolution camera are easily missed by background
// modelling alone, so Tangram groups a frame's RoIs by zone and sends one patch per zone:
// the frame is divided into X x Y zones of equal size, every RoI joins the zone it
// overlaps most, and each zone with RoIs becomes the minimum rectangle enclosing them
// (Sec. III-A, Adaptive Frame Partitioning; Alg. 1). Zone i of X spans columns
// [floor(i W / X), floor((i + 1) W / X)) (rows alike), zones are numbered row-major and
// an overlap tie goes to the lower number; patches are listed frame by frame, zones in
// row-major order.
//
// Two launches on the caller's stream:
//  1. clear: zeroes the ticket and look-back words of launch 2.
//  2. zones: one 256-thread workgroup per frame, frames taken in ticket order. Each
//     thread scores its RoIs against the zones they touch and folds them into the winning
//     zone's enclosing rectangle with LDS atomic min/max; the workgroup then counts its
//     non-empty zones (ballot + mbcnt), finds its output offset with a single-pass
//     decoupled look-back over earlier frames, and writes its patches there.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

#include "lookback.h"
#include "tg.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxZones = 1024;                     // zones per frame, e.g. 32 x 32

struct PartitionParams {
  const tg_roi *boxes;
  const int32_t *frame_begin;
  int32_t n_boxes, n_frames, frame_w, frame_h, zones_x, zones_y;
  tg_roi *patches;
  int32_t *zone_of_box;
  int32_t *n_patches;
  uint32_t *ticket;
  uint64_t *state;  // one word per frame
};

// First pixel of zone k of n along an axis of `size` pixels.
__device__ __forceinline__ int zone_start(int k, int n, int size) {
  return static_cast<int>((static_cast<int64_t>(k) * size) / n);
}
// The zone holding pixel p: the largest k with zone_start(k) <= p.
__device__ __forceinline__ int zone_of(int p, int n, int size) {
  return static_cast<int>(((static_cast<int64_t>(p) + 1) * n - 1) / size);
}

__global__ void clear_kernel(uint64_t *words, int32_t n_words) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_words) words[i] = 0;
}

__global__ __launch_bounds__(kThreads) void zone_kernel(const PartitionParams P) {
  __shared__ int acc[kMaxZones][4];  // x0, y0, x1, y1 of each zone's enclosing rectangle
  __shared__ int s_frame, s_prefix;
  __shared__ int s_wave[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int X = P.zones_x, Y = P.zones_y, Z = X * Y, W = P.frame_w, H = P.frame_h;
  if (tid == 0)
    s_frame = static_cast<int>(__hip_atomic_fetch_add(P.ticket, 1u, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT));
  for (int r = tid; r < Z; r += kThreads) {
    acc[r][0] = INT_MAX;
    acc[r][1] = INT_MAX;
    acc[r][2] = INT_MIN;
    acc[r][3] = INT_MIN;
  }
  __syncthreads();
  const int f = s_frame;
  const int lo = min(max(P.frame_begin[f], 0), P.n_boxes);
  const int hi = min(max(P.frame_begin[f + 1], lo), P.n_boxes);
  for (int b = lo + tid; b < hi; b += kThreads) {
    const tg_roi r = P.boxes[b];
    int best = -1;
    if (r.frame == f && r.w > 0 && r.h > 0 && r.x >= 0 && r.y >= 0 && r.x <= W - r.w &&
        r.y <= H - r.h) {
      const int x1 = r.x + r.w, y1 = r.y + r.h;
      const int i0 = zone_of(r.x, X, W), i1 = zone_of(x1 - 1, X, W);
      const int j0 = zone_of(r.y, Y, H), j1 = zone_of(y1 - 1, Y, H);
      int64_t best_area = -1;
      for (int j = j0; j <= j1; ++j) {
        const int64_t hh = min(y1, zone_start(j + 1, Y, H)) - max(r.y, zone_start(j, Y, H));
        for (int i = i0; i <= i1; ++i) {
          const int64_t ww = min(x1, zone_start(i + 1, X, W)) - max(r.x, zone_start(i, X, W));
          if (ww * hh > best_area) {  // strict: the first (lowest) zone keeps a tie
            best_area = ww * hh;
            best = j * X + i;
          }
        }
      }
      atomicMin(&acc[best][0], r.x);
      atomicMin(&acc[best][1], r.y);
      atomicMax(&acc[best][2], x1);
      atomicMax(&acc[best][3], y1);
    }
    if (P.zone_of_box) P.zone_of_box[b] = best;
  }
  __syncthreads();

  // Non-empty zones of this frame, counted in zone order.
  int total = 0;
  for (int base = 0; base < Z; base += kThreads) {
    const int r = base + tid;
    const uint64_t used = __ballot(r < Z && acc[r][0] != INT_MAX);
    if (lane == 0) s_wave[wave] = __popcll(used);
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) total += s_wave[w];
    __syncthreads();
  }
  if (wave == 0) {
    bool failed;
    const int prefix = tg_detail::lookback_prefix(P.state, f, total, &failed);
    if (lane == 0) {
      s_prefix = prefix;
      if (f == P.n_frames - 1) *P.n_patches = failed ? TG_E_INTERNAL : prefix + total;
    }
  }
  __syncthreads();

  int pos = s_prefix;
  for (int base = 0; base < Z; base += kThreads) {
    const int r = base + tid;
    const bool u = r < Z && acc[r][0] != INT_MAX;
    const uint64_t used = __ballot(u);
    if (lane == 0) s_wave[wave] = __popcll(used);
    __syncthreads();
    int before = 0, round = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < wave) before += s_wave[w];
      round += s_wave[w];
    }
    if (u) {
      const int k = pos + before +
                    static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                        static_cast<uint32_t>(used >> 32),
                        __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(used), 0u)));
      P.patches[k] = tg_roi{f, acc[r][0], acc[r][1], acc[r][2] - acc[r][0],
                            acc[r][3] - acc[r][1]};
    }
    pos += round;
    __syncthreads();
  }
}

__global__ void zero_count_kernel(int32_t *n) { *n = 0; }

}  // namespace

extern "C" size_t tg_partition_workspace_bytes(int32_t n_frames) {
  if (n_frames <= 0) return 0;
  return sizeof(uint64_t) * (1 + static_cast<size_t>(n_frames));
}

extern "C" int tg_partition(const tg_partition_args *a, void *stream) {
  if (!a || a->n_boxes < 0 || a->n_frames < 0 || !a->n_patches) return TG_E_INVAL;
  if (a->frame_w < 1 || a->frame_h < 1 || a->zones_x < 1 || a->zones_y < 1 ||
      a->zones_x > a->frame_w || a->zones_y > a->frame_h ||
      int64_t(a->zones_x) * a->zones_y > kMaxZones)
    return TG_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (a->n_frames == 0) {
    hipLaunchKernelGGL(zero_count_kernel, dim3(1), dim3(1), 0, s, a->n_patches);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  if (!a->frame_begin || !a->patches || (a->n_boxes > 0 && !a->boxes)) return TG_E_INVAL;
  const size_t need = tg_partition_workspace_bytes(a->n_frames);
  if (!a->workspace || a->workspace_bytes < need ||
      reinterpret_cast<uintptr_t>(a->workspace) % 8 != 0)
    return TG_E_WORKSPACE;

  PartitionParams P;
  P.boxes = a->boxes;
  P.frame_begin = a->frame_begin;
  P.n_boxes = a->n_boxes;
  P.n_frames = a->n_frames;
  P.frame_w = a->frame_w;
  P.frame_h = a->frame_h;
  P.zones_x = a->zones_x;
  P.zones_y = a->zones_y;
  P.patches = a->patches;
  P.zone_of_box = a->zone_of_box;
  P.n_patches = a->n_patches;
  P.ticket = static_cast<uint32_t *>(a->workspace);
  P.state = static_cast<uint64_t *>(a->workspace) + 1;

  const int32_t words = 1 + a->n_frames;
  hipLaunchKernelGGL(clear_kernel, dim3((words + kThreads - 1) / kThreads), dim3(kThreads), 0,
                     s, static_cast<uint64_t *>(a->workspace), words);
  if (hipGetLastError() != hipSuccess) return TG_E_HIP;
  hipLaunchKernelGGL(zone_kernel, dim3(static_cast<uint32_t>(a->n_frames)), dim3(kThreads), 0,
                     s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
