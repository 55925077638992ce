// tg_unstitch: map detector boxes from canvas pixels back to frame pixels.
//
// The paper scores detections per source frame (Sec. V-D) after inferring stitched
// canvases (Sec. III-C) but does not say how a detection finds its patch. This
// library's rule: a box belongs to the patch holding its centre (half-open on the
// right and bottom edges); it is optionally clipped to that patch and shifted by the
// patch's frame offset minus its canvas offset.
//
// Launches on the caller's stream:
//  0. pack (calls whose boxes test many patches in all): one 24-byte patch record per
//     plan position -- the placed rectangle of RoI order[k] in binary32, its canvas and
//     its id -- so that the assign reads a canvas's patches as consecutive records
//     instead of gathering placements and RoIs by id. Those gathers (two cache lines per
//     patch and box) bound the assign by the L2's request rate when many boxes meet
//     canvases of many patches.
//  1. assign: LPB lanes per box test the box canvas's patches LPB at a time; a wave
//     ballot picks the (unique) patch containing the centre and roi_of_box[b] is
//     written. With the overlap rule each lane scores its patch's overlap area and the
//     lanes of the box take the largest (ties: lower RoI id) with xor shuffles. The first
//     launch also clears the look-back state of the emit launch.
//  2. emit: four consecutive boxes per thread, 1024 per workgroup. Kept boxes are
//     ranked inside the workgroup with a wave prefix sum of per-thread counts, the
//     workgroup's offset comes from a single-pass decoupled look-back over earlier
//     workgroups (workgroup order is taken from an atomic ticket, so every workgroup a
//     block waits on has already started), and kept boxes are written in increasing
//     box index -- a stable compaction whose output does not depend on scheduling.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>

#include "lookback.h"
#include "tg.h"

// Built with -ffp-contract=off: every binary32 operation here is rounded on its own (no
// multiply-add fusion), so decisions taken in floating point match any plain IEEE
// implementation of the same steps.

namespace {

constexpr int kThreads = 256;
constexpr int kBoxesPerThread = 4;                  // emit: consecutive boxes per thread
constexpr int kEmitBoxes = kThreads * kBoxesPerThread;
// Calls whose boxes test at least this many patches in all read the plan through patch
// records (one pack launch more); smaller ones gather it directly.
constexpr int64_t kRecordsMinTests = int64_t(1) << 21;

struct UnstitchParams {
  const tg_box *boxes;
  const int32_t *box_canvas;
  int32_t n_boxes;
  const tg_roi *rois;
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin;
  int32_t n_rois, n_canvases, clip, rule;
  int32_t *roi_of_box;
  tg_det *dets;
  int32_t *n_out;
  uint32_t *ticket;
  uint64_t *state;  // one word per emit workgroup
  int32_t n_state_words;  // ticket word + state words, in uint64 units
  float4 *rect;  // patch records (null: the assign gathers the plan directly) ...
  int2 *meta;    // ... and their (canvas, RoI id)
};

// Patch records, one per plan position k: the placed rectangle of RoI order[k] as
// binary32 (dx, dy, dx + w, dy + h) and (its canvas, its id); an id out of range gets
// canvas -1, which no box names. Also clears the look-back state of the emit launch.
__global__ __launch_bounds__(kThreads) void pack_kernel(const UnstitchParams P) {
  const int64_t k = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (k < P.n_state_words) reinterpret_cast<uint64_t *>(P.ticket)[k] = 0;
  if (k >= P.n_rois) return;
  const int id = P.order[k];
  float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  int canvas = -1;
  if (id >= 0 && id < P.n_rois) {
    const tg_place pl = P.place[id];
    const tg_roi ro = P.rois[id];
    r = make_float4(float(pl.x), float(pl.y), float(pl.x + ro.w), float(pl.y + ro.h));
    canvas = pl.canvas;
  }
  P.rect[k] = r;
  P.meta[k] = make_int2(canvas, id);
}

// The patch at plan position k as the assign tests it: its placed rectangle, its canvas
// (-1 when order[k] is not a RoI id) and order[k] -- from the records or from the plan.
template <bool kRecords>
__device__ __forceinline__ void patch_at(const UnstitchParams &P, int k, float4 &r, int &canvas,
                                         int &id) {
  if (kRecords) {
    r = P.rect[k];
    const int2 m = P.meta[k];
    canvas = m.x;
    id = m.y;
    return;
  }
  id = P.order[k];
  r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  canvas = -1;
  if (id >= 0 && id < P.n_rois) {
    const tg_place pl = P.place[id];
    const tg_roi ro = P.rois[id];
    r = make_float4(float(pl.x), float(pl.y), float(pl.x + ro.w), float(pl.y + ro.h));
    canvas = pl.canvas;
  }
}

template <int LPB, bool kRecords>
__global__ __launch_bounds__(kThreads) void assign_kernel(const UnstitchParams P) {
  const int gtid = blockIdx.x * kThreads + threadIdx.x;
  if (!kRecords && gtid < P.n_state_words) reinterpret_cast<uint64_t *>(P.ticket)[gtid] = 0;

  constexpr int kBoxesPerBlock = kThreads / LPB;
  const int lane = threadIdx.x & 63;
  const int sub = threadIdx.x / LPB;
  const int sl = threadIdx.x % LPB;
  const int seg_shift = lane - sl;  // first lane of this box's segment within the wave
  const uint64_t seg_mask = LPB == 64 ? ~uint64_t(0) : ((uint64_t(1) << LPB) - 1);
  const int b = blockIdx.x * kBoxesPerBlock + sub;
  if (b >= P.n_boxes) return;  // whole segments leave together

  const int c = P.box_canvas[b];
  const tg_box box = P.boxes[b];
  const float cx = (box.x1 + box.x2) * 0.5f;
  const float cy = (box.y1 + box.y2) * 0.5f;
  int k_lo = 0, k_hi = 0;
  if (c >= 0 && c < P.n_canvases) {
    k_lo = min(max(P.canvas_begin[c], 0), P.n_rois);
    k_hi = min(max(P.canvas_begin[c + 1], k_lo), P.n_rois);
  }
  if (P.rule == 1) {
    // Largest overlap area (> 0), ties to the lower RoI id: each lane scores one patch per
    // round, the segment takes the best of its lanes (xor shuffles stay in the segment),
    // and the best of the rounds is kept.
    if (box.x1 != box.x1 || box.y1 != box.y1 || box.x2 != box.x2 || box.y2 != box.y2)
      k_hi = k_lo;  // a NaN coordinate matches nothing
    float best = 0.0f;
    int best_id = -1;
    for (int base = k_lo; base < k_hi; base += LPB) {
      const int k = base + sl;
      float a = 0.0f;
      int id = -1;
      if (k < k_hi) {
        float4 r;
        int pc;
        patch_at<kRecords>(P, k, r, pc, id);
        if (pc == c) {
          const float ow = fmaxf(0.0f, __fsub_rn(fminf(box.x2, r.z), fmaxf(box.x1, r.x)));
          const float oh = fmaxf(0.0f, __fsub_rn(fminf(box.y2, r.w), fmaxf(box.y1, r.y)));
          a = __fmul_rn(ow, oh);
        }
      }
#pragma unroll
      for (int o = 1; o < LPB; o <<= 1) {
        const float a2 = __shfl_xor(a, o);
        const int i2 = __shfl_xor(id, o);
        if (a2 > a || (a2 == a && a2 > 0.0f && i2 < id)) {
          a = a2;
          id = i2;
        }
      }
      if (a > best || (a == best && a > 0.0f && id < best_id)) {
        best = a;
        best_id = id;
      }
    }
    if (sl == 0) P.roi_of_box[b] = best > 0.0f ? best_id : -1;
    return;
  }
  for (int base = k_lo; base < k_hi; base += LPB) {
    const int k = base + sl;
    bool hit = false;
    int id = -1;
    if (k < k_hi) {
      float4 r;
      int pc;
      patch_at<kRecords>(P, k, r, pc, id);
      hit = pc == c && r.x <= cx && cx < r.z && r.y <= cy && cy < r.w;
    }
    const uint64_t m = (__ballot(hit) >> seg_shift) & seg_mask;
    if (m) {
      if (sl == __builtin_ctzll(m)) P.roi_of_box[b] = id;  // lowest k wins
      return;
    }
  }
  if (sl == 0) P.roi_of_box[b] = -1;
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

// Writes the detection of kept box b (patch roi) at position pos.
__device__ __forceinline__ void write_det(const UnstitchParams &P, int b, int roi, int pos) {
  const tg_roi r = P.rois[roi];
  const tg_place pl = P.place[roi];
  const tg_box box = P.boxes[b];
  float v[4] = {box.x1, box.y1, box.x2, box.y2};
  if (P.clip) {
    const float lo[2] = {float(pl.x), float(pl.y)};
    const float hi[2] = {float(pl.x + r.w), float(pl.y + r.h)};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (v[q] < lo[q & 1]) v[q] = lo[q & 1];
      if (v[q] > hi[q & 1]) v[q] = hi[q & 1];
    }
  }
  const float ox = float(r.x - pl.x), oy = float(r.y - pl.y);
  tg_det d;
  d.box = b;
  d.roi = roi;
  d.frame = r.frame;
  d.x1 = v[0] + ox;
  d.y1 = v[1] + oy;
  d.x2 = v[2] + ox;
  d.y2 = v[3] + oy;
  P.dets[pos] = d;
}

__global__ __launch_bounds__(kThreads) void emit_kernel(const UnstitchParams P) {
  __shared__ int s_blk, s_prefix;
  __shared__ int s_wave[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0)
    s_blk = static_cast<int>(__hip_atomic_fetch_add(P.ticket, 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT));
  __syncthreads();
  const int blk = s_blk;
  const int b0 = blk * kEmitBoxes + kBoxesPerThread * tid;  // this thread's first box
  int roi[kBoxesPerThread];
#pragma unroll
  for (int j = 0; j < kBoxesPerThread; ++j)
    roi[j] = b0 + j < P.n_boxes ? P.roi_of_box[b0 + j] : -1;
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < kBoxesPerThread; ++j) cnt += roi[j] >= 0;
  const int incl = wave_inclusive_sum(cnt);
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
  for (int w = 0; w < kThreads / 64; ++w) {
    if (w < wave) before += s_wave[w];
    total += s_wave[w];
  }
  if (wave == 0) {
    bool failed;
    const int prefix = tg_detail::lookback_prefix(P.state, blk, total, &failed);
    if (lane == 0) {
      s_prefix = prefix;
      if (blk == static_cast<int>(gridDim.x) - 1) *P.n_out = failed ? TG_E_INTERNAL : prefix + total;
    }
  }
  __syncthreads();
  int pos = s_prefix + before + incl - cnt;
#pragma unroll
  for (int j = 0; j < kBoxesPerThread; ++j)
    if (roi[j] >= 0) write_det(P, b0 + j, roi[j], pos++);
}

__global__ void zero_count_kernel(int32_t *n_out) { *n_out = 0; }

int emit_blocks(int32_t n) { return (n + kEmitBoxes - 1) / kEmitBoxes; }

// Bytes of the ticket and look-back words for n boxes, rounded up to 16 so that the
// patch records after them are aligned.
size_t lookback_bytes(int32_t n) {
  return (sizeof(uint64_t) * (1 + static_cast<size_t>(emit_blocks(n))) + 15) & ~size_t(15);
}

// Bytes of the patch records of a plan of n_rois RoIs: a float4 and an int2 each.
size_t record_bytes(int32_t n_rois) {
  return n_rois > 0 ? 24 * static_cast<size_t>(n_rois) : 0;
}

// Workspace of the allocation-free entry point: the ticket and look-back words for up
// to TG_UNSTITCH_NOALLOC_MAX_BOXES boxes, then patch records for plans of up to
// TG_UNSTITCH_NOALLOC_MAX_ROIS RoIs (3.3 MB in all). Each GPU the library runs on holds
// its own copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device.
constexpr size_t kScratchLookback =
    (8 * (1 + size_t(TG_UNSTITCH_NOALLOC_MAX_BOXES + kEmitBoxes - 1) / kEmitBoxes) + 15) & ~size_t(15);
constexpr size_t kScratchBytes = kScratchLookback + 24 * size_t(TG_UNSTITCH_NOALLOC_MAX_ROIS);
__device__ __align__(256) uint64_t scratch[kScratchBytes / 8];

// Device address of `scratch` on the current device, looked up once per device id (null
// when the lookup fails).
void *scratch_address() {
  static std::atomic<void *> cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  void *p = cached[dev].load(std::memory_order_acquire);
  if (p) return p;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
  cached[dev].store(p, std::memory_order_release);
  return p;
}

// Argument checks shared by both entry points (the workspace aside).
int check_args(const tg_unstitch_args *a) {
  if (!a || a->n_boxes < 0 || a->n_rois < 0 || a->n_canvases < 0) return TG_E_INVAL;
  if (a->rule != 0 && a->rule != 1) return TG_E_INVAL;
  if (!a->n_out) return TG_E_INVAL;
  if (a->n_boxes == 0) return TG_OK;
  if (!a->boxes || !a->box_canvas || !a->roi_of_box || !a->dets) return TG_E_INVAL;
  if (a->n_canvases > 0 && !a->canvas_begin) return TG_E_INVAL;
  if (a->n_rois > 0 && (!a->rois || !a->place || !a->order)) return TG_E_INVAL;
  return TG_OK;
}

template <bool kRecords>
void launch_assign(int lpb, int32_t n_boxes, hipStream_t s, const UnstitchParams &P) {
  const int64_t per_block = kThreads / lpb;
  const dim3 grid(static_cast<uint32_t>((int64_t(n_boxes) + per_block - 1) / per_block));
  if (lpb == 16)
    hipLaunchKernelGGL((assign_kernel<16, kRecords>), grid, dim3(kThreads), 0, s, P);
  else if (lpb == 32)
    hipLaunchKernelGGL((assign_kernel<32, kRecords>), grid, dim3(kThreads), 0, s, P);
  else
    hipLaunchKernelGGL((assign_kernel<64, kRecords>), grid, dim3(kThreads), 0, s, P);
}

// Enqueues the launches with `words` (device, 8-byte aligned, lookback_bytes(n_boxes)
// bytes) as the ticket and look-back words -- cleared by the first launch -- and
// `records` (16-byte aligned, record_bytes(n_rois) bytes, or null) for the patch records.
int launch(const tg_unstitch_args *a, void *words, void *records, hipStream_t s) {
  if (a->n_boxes == 0) {
    hipLaunchKernelGGL(zero_count_kernel, dim3(1), dim3(1), 0, s, a->n_out);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  UnstitchParams P;
  P.boxes = a->boxes;
  P.box_canvas = a->box_canvas;
  P.n_boxes = a->n_boxes;
  P.rois = a->rois;
  P.place = a->place;
  P.order = a->order;
  P.canvas_begin = a->canvas_begin;
  P.n_rois = a->n_rois;
  P.n_canvases = a->n_canvases;
  P.clip = a->clip;
  P.rule = a->rule;
  P.roi_of_box = a->roi_of_box;
  P.dets = a->dets;
  P.n_out = a->n_out;
  P.ticket = static_cast<uint32_t *>(words);
  P.state = static_cast<uint64_t *>(words) + 1;
  P.n_state_words = 1 + emit_blocks(a->n_boxes);
  const int64_t per_canvas = a->n_canvases > 0 ? (int64_t(a->n_rois) + a->n_canvases - 1) /
                                                     a->n_canvases
                                               : 1;
  // Patch records when the boxes test many patches in all (about n_boxes * per_canvas).
  const bool use_records = records && a->n_rois > 0 &&
                           int64_t(a->n_boxes) * per_canvas >= kRecordsMinTests;
  // Lanes per box. Gathering the plan directly, a round is two dependent gathers: 64
  // lanes, so one round usually settles a box, unless canvases hold at most 16 patches
  // (cam20_4k, 32 patches per canvas: 11.6 us with 64 lanes, 12.0 with 32, 14.9 with 16).
  // Reading records, a round costs little (consecutive records), so canvases of up to 32
  // patches take 16 lanes and two rounds at most (window_64x30, 29 patches per canvas:
  // 38.8 us instead of 44.2 with 32).
  const int lpb = use_records ? (per_canvas <= 32 ? 16 : 64) : (per_canvas <= 16 ? 16 : 64);
  P.rect = use_records ? static_cast<float4 *>(records) : nullptr;
  P.meta = use_records ? reinterpret_cast<int2 *>(P.rect + a->n_rois) : nullptr;
  if (use_records) {
    const int64_t pack_threads = std::max<int64_t>(a->n_rois, P.n_state_words);
    hipLaunchKernelGGL(pack_kernel, dim3(static_cast<uint32_t>((pack_threads + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, P);
    launch_assign<true>(lpb, a->n_boxes, s, P);
  } else {
    launch_assign<false>(lpb, a->n_boxes, s, P);
  }
  if (hipGetLastError() != hipSuccess) return TG_E_HIP;
  hipLaunchKernelGGL(emit_kernel, dim3(static_cast<uint32_t>(emit_blocks(a->n_boxes))),
                     dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}

}  // namespace

extern "C" size_t tg_unstitch_workspace_bytes(int32_t n_boxes, int32_t n_rois) {
  if (n_boxes <= 0) return 0;
  return lookback_bytes(n_boxes) + record_bytes(n_rois);
}

extern "C" int tg_unstitch(const tg_unstitch_args *a, void *stream) {
  const int rc = check_args(a);
  if (rc != TG_OK) return rc;
  if (a->n_boxes == 0) return launch(a, nullptr, nullptr, static_cast<hipStream_t>(stream));
  const size_t need = tg_unstitch_workspace_bytes(a->n_boxes, a->n_rois);
  if (!a->workspace || a->workspace_bytes < need ||
      reinterpret_cast<uintptr_t>(a->workspace) % 16 != 0)
    return TG_E_WORKSPACE;
  char *ws = static_cast<char *>(a->workspace);
  return launch(a, ws, ws + lookback_bytes(a->n_boxes), static_cast<hipStream_t>(stream));
}

extern "C" int tg_unstitch_noalloc(const tg_unstitch_args *a, void *stream) {
  const int rc = check_args(a);
  if (rc != TG_OK) return rc;
  if (a->n_boxes > TG_UNSTITCH_NOALLOC_MAX_BOXES) return TG_E_WORKSPACE;
  if (a->n_boxes == 0) return launch(a, nullptr, nullptr, static_cast<hipStream_t>(stream));
  char *ws = static_cast<char *>(scratch_address());
  if (!ws) return TG_E_HIP;
  // plans larger than the records area are gathered directly (same results)
  void *records = a->n_rois <= TG_UNSTITCH_NOALLOC_MAX_ROIS ? ws + kScratchLookback : nullptr;
  return launch(a, ws, records, static_cast<hipStream_t>(stream));
}
