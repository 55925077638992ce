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
// Three launches on the caller's stream, with no atomics outside LDS:
//  1. count: one 256-thread workgroup per frame scores the frame's RoIs against the zones
//     they touch, folds each into the winning zone's enclosing rectangle with LDS atomic
//     min/max, and stores the frame's number of non-empty zones.
//  2. scan: one workgroup turns the counts into each frame's first output position and
//     writes the total.
//  3. write: the per-frame pass of launch 1 again, then the frame's non-empty zones are
//     written from its first position in zone order (ranks from ballots and mbcnt).
// Launch 3 recomputes the rectangles instead of keeping them: a frame's RoIs are a few
// hundred bytes, while keeping its rectangles would take workspace by the zone count.
// (A single launch that orders frames by an atomic ticket and finds each frame's position
// with a look-back over the earlier frames pays for the ticket instead: one device-scope
// atomic on one address per frame, which the hardware serialises.)
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

#include "tg.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxZones = 1024;  // zones per frame, e.g. 32 x 32
constexpr int kScanThreads = 1024;

struct PartitionParams {
  const tg_roi *boxes;
  const int32_t *frame_begin;
  int32_t n_boxes, n_frames, frame_w, frame_h, zones_x, zones_y;
  tg_roi *patches;
  int32_t *zone_of_box;
  int32_t *n_patches;
  int32_t *first;  // [n_frames]: count of non-empty zones, then the frame's first position
};

// First pixel of zone k of n along an axis of `size` pixels.
__device__ __forceinline__ int zone_start(int k, int n, int size) {
  return static_cast<int>((static_cast<int64_t>(k) * size) / n);
}
// The zone holding pixel p: the largest k with zone_start(k) <= p.
__device__ __forceinline__ int zone_of(int p, int n, int size) {
  return static_cast<int>(((static_cast<int64_t>(p) + 1) * n - 1) / size);
}

// Inclusive prefix sum over the 64 lanes of a wave (DPP row shifts, then row broadcasts).
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Frame f's zone rectangles in acc (x0, y0, x1, y1; an empty zone keeps x0 = INT_MAX),
// and with `record` each RoI's zone in zone_of_box. Called by the whole workgroup; ends
// with a barrier.
__device__ void fold_frame(const PartitionParams &P, int f, int (*acc)[4], bool record) {
  const int tid = threadIdx.x;
  const int X = P.zones_x, Y = P.zones_y, Z = X * Y, W = P.frame_w, H = P.frame_h;
  for (int r = tid; r < Z; r += kThreads) {
    acc[r][0] = INT_MAX;
    acc[r][1] = INT_MAX;
    acc[r][2] = INT_MIN;
    acc[r][3] = INT_MIN;
  }
  __syncthreads();
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
    if (record) P.zone_of_box[b] = best;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kThreads) void count_kernel(const PartitionParams P) {
  __shared__ int acc[kMaxZones][4];
  __shared__ int s_wave[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int f = blockIdx.x, Z = P.zones_x * P.zones_y;
  fold_frame(P, f, acc, false);
  int used = 0;
  for (int r = tid; r < Z; r += kThreads) used += acc[r][0] != INT_MAX;
  for (int o = 32; o > 0; o >>= 1) used += __shfl_xor(used, o);
  if (lane == 0) s_wave[wave] = used;
  __syncthreads();
  if (tid == 0) {
    int total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) total += s_wave[w];
    P.first[f] = total;
  }
}

// Exclusive prefix sum of the counts, in place, and the total: thread t takes a
// contiguous chunk of frames.
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const PartitionParams P) {
  __shared__ int s_wave[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int F = P.n_frames;
  const int chunk = (F + kScanThreads - 1) / kScanThreads;
  const int a = static_cast<int>(min(int64_t(tid) * chunk, int64_t(F)));
  const int b = static_cast<int>(min(int64_t(a) + chunk, int64_t(F)));
  int sum = 0;
  for (int i = a; i < b; ++i) sum += P.first[i];
  const int incl = wave_inclusive_sum(sum);
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int run = incl - sum;
  for (int w = 0; w < wave; ++w) run += s_wave[w];
  for (int i = a; i < b; ++i) {
    const int c = P.first[i];
    P.first[i] = run;
    run += c;
  }
  if (tid == kScanThreads - 1) *P.n_patches = run;
}

__global__ __launch_bounds__(kThreads) void write_kernel(const PartitionParams P) {
  __shared__ int acc[kMaxZones][4];
  __shared__ int s_wave[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int f = blockIdx.x, Z = P.zones_x * P.zones_y;
  fold_frame(P, f, acc, P.zone_of_box != nullptr);
  int pos = P.first[f];
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
  P.first = static_cast<int32_t *>(a->workspace);

  const dim3 frames(static_cast<uint32_t>(a->n_frames));
  hipLaunchKernelGGL(count_kernel, frames, dim3(kThreads), 0, s, P);
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kScanThreads), 0, s, P);
  hipLaunchKernelGGL(write_kernel, frames, dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
