// tg_merge: per-frame suppression of duplicate detections after tg_unstitch.
//
// When a frame is cut into zone patches (Sec. III-A, Alg. 1), neighbouring patches can
// overlap, so one object can come back from two patches once detections are mapped to
// their frame (Sec. V-D scores per frame). The paper does not spell out the merge; this
// library's reading: a frame's detections are ranked by score (higher first, equal scores
// by box index, a NaN score last), and walking that ranking a detection is kept unless one
// kept before it in the same frame (with cross_only: from another patch) overlaps it by
// IoU > threshold, decided as inter > threshold * union in binary32 with every operation
// rounded on its own. Kept detections are written in input order.
//
// Six launches on the caller's stream, all on device data (the detection count comes from
// tg_unstitch's n_out on the device):
//  1. clear the per-frame counters and look-back words;
//  2. count detections per frame (LDS histograms, one global atomic per frame and
//     workgroup);
//  3. exclusive scan of the counts (one workgroup);
//  4. scatter detection indices into frame groups (ranks inside a workgroup from LDS, one
//     range per frame and workgroup from a global cursor; the order inside a group does
//     not matter, the ranking below is a total order);
//  5. one 1024-thread workgroup per frame: bitonic sort of 64-bit keys (score, box) in LDS,
//     then the greedy pass 64 candidates at a time (all threads test the chunk against the
//     detections kept so far and fill the chunk's 64 x 64 suppression bits; one wave walks
//     the chunk); up to 2048 detections per frame, more are left unmerged (all kept) and
//     counted in n_overflow;
//  6. stable compaction of the kept detections (decoupled look-back, 1024 per workgroup).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "lookback.h"
#include "tg.h"

// Built with -ffp-contract=off: every binary32 operation here is rounded on its own (no
// multiply-add fusion), so decisions taken in floating point match any plain IEEE
// implementation of the same steps.

namespace {

constexpr int kThreads = 256;
constexpr int kMaxPerFrame = 2048;
constexpr int kPerThread = 4;  // compaction: consecutive detections per thread
constexpr int kCompactBlock = kThreads * kPerThread;
constexpr int kScanThreads = 1024;

struct MergeParams {
  const tg_det *dets;
  const int32_t *n_dets;
  int32_t n_max;
  const float *scores;
  int32_t n_scores, n_frames;
  float thr;
  int32_t cross_only;
  int32_t *keep;
  tg_det *out;
  int32_t *n_kept;
  int32_t *n_overflow;
  int32_t *counts;       // [n_frames]
  int32_t *cursor;       // [n_frames]
  int32_t *frame_begin;  // [n_frames + 1]
  int32_t *grouped;      // [n_max]
  uint32_t *ticket;
  uint64_t *state;       // [compaction workgroups]
};

__device__ __forceinline__ int count_of(const MergeParams &P) {
  return min(max(*P.n_dets, 0), P.n_max);
}

__global__ void clear_kernel(MergeParams P, int32_t n_words32, int32_t n_words64) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_words32) {
    P.counts[i] = 0;  // counts and cursor are contiguous
  }
  if (i < n_words64) reinterpret_cast<uint64_t *>(P.ticket)[i] = 0;  // ticket + states
  if (i == 0) *P.n_overflow = 0;
}

// Detections per frame. Up to kHistMax frames a workgroup first counts in LDS and then
// adds each non-empty bin to the global count once (many detections share few frames, so
// direct global atomics would queue on the same words).
constexpr int kHistMax = 4096;

__global__ __launch_bounds__(kThreads) void count_kernel(const MergeParams P) {
  __shared__ int hist[kHistMax];
  const int tid = threadIdx.x;
  const bool local = P.n_frames <= kHistMax;
  if (local)
    for (int f = tid; f < P.n_frames; f += kThreads) hist[f] = 0;
  __syncthreads();
  const int i = blockIdx.x * kThreads + tid;
  if (i < count_of(P)) {
    const int f = P.dets[i].frame;
    if (f >= 0 && f < P.n_frames)
      atomicAdd(local ? &hist[f] : &P.counts[f], 1);
    else
      P.keep[i] = 0;  // no frame to merge in: dropped
  }
  if (!local) return;
  __syncthreads();
  for (int f = tid; f < P.n_frames; f += kThreads)
    if (hist[f]) atomicAdd(&P.counts[f], hist[f]);
}

__global__ __launch_bounds__(kScanThreads) void scan_kernel(const MergeParams P) {
  __shared__ int s_wave[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int carry = 0;
  for (int base = 0; base < P.n_frames; base += kScanThreads) {
    const int f = base + tid;
    const int v = f < P.n_frames ? P.counts[f] : 0;
    int incl = v;
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o);
      if (lane >= o) incl += t;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) {
      if (w < wave) before += s_wave[w];
      total += s_wave[w];
    }
    if (f < P.n_frames) P.frame_begin[f] = carry + before + incl - v;
    carry += total;
    __syncthreads();
  }
  if (tid == 0) P.frame_begin[P.n_frames] = carry;
}

// Detection indices into frame groups. Up to kHistMax frames a workgroup ranks its
// detections per frame in LDS and reserves one range per non-empty frame.
__global__ __launch_bounds__(kThreads) void scatter_kernel(const MergeParams P) {
  __shared__ int hist[kHistMax];
  const int tid = threadIdx.x;
  const bool local = P.n_frames <= kHistMax;
  if (local)
    for (int f = tid; f < P.n_frames; f += kThreads) hist[f] = 0;
  __syncthreads();
  const int i = blockIdx.x * kThreads + tid;
  int f = -1, rank = 0;
  if (i < count_of(P)) {
    f = P.dets[i].frame;
    if (f < 0 || f >= P.n_frames)
      f = -1;
    else if (local)
      rank = atomicAdd(&hist[f], 1);
    else
      P.grouped[P.frame_begin[f] + atomicAdd(&P.cursor[f], 1)] = i;
  }
  if (!local) return;
  __syncthreads();
  for (int g = tid; g < P.n_frames; g += kThreads)  // this workgroup's range of frame g
    if (hist[g]) hist[g] = P.frame_begin[g] + atomicAdd(&P.cursor[g], hist[g]);
  __syncthreads();
  if (f >= 0) P.grouped[hist[f] + rank] = i;
}

// Ranking key, ascending = higher score first, then lower box index. NaN ranks as -inf;
// -0 and +0 are the same score.
__device__ __forceinline__ uint64_t rank_key(float s, int32_t box) {
  if (s != s) s = -__builtin_inff();
  if (s == 0.0f) s = 0.0f;
  uint32_t b = __float_as_uint(s);
  b ^= (b & 0x80000000u) ? 0xFFFFFFFFu : 0x80000000u;  // ascending order of floats
  return (static_cast<uint64_t>(~b) << 32) | static_cast<uint32_t>(box);
}

// Whether box a suppresses box b (x1, y1, x2, y2 in .x .y .z .w).
__device__ __forceinline__ bool suppresses(float4 a, float4 b, float thr) {
  const float w = fmaxf(0.0f, __fsub_rn(fminf(a.z, b.z), fmaxf(a.x, b.x)));
  const float h = fmaxf(0.0f, __fsub_rn(fminf(a.w, b.w), fmaxf(a.y, b.y)));
  const float inter = __fmul_rn(w, h);
  const float area_a = __fmul_rn(fmaxf(0.0f, __fsub_rn(a.z, a.x)), fmaxf(0.0f, __fsub_rn(a.w, a.y)));
  const float area_b = __fmul_rn(fmaxf(0.0f, __fsub_rn(b.z, b.x)), fmaxf(0.0f, __fsub_rn(b.w, b.y)));
  const float uni = __fsub_rn(__fadd_rn(area_a, area_b), inter);
  return inter > __fmul_rn(thr, uni);
}

// LDS of one frame: ranking keys and detection ids for the sort, then the ranked boxes,
// patches and flags, the list of detections kept so far and one chunk's bit matrix.
constexpr int kChunk = 64;  // candidates decided per round
constexpr int kFrameThreads = 1024;  // one workgroup per frame
static_assert(kChunk * kChunk % kFrameThreads == 0 && 32 % (kChunk * kChunk / kFrameThreads) == 0,
              "a thread's columns lie in one 32-bit word");
constexpr size_t kOffKey = 0;                                          // u64 [2048]
constexpr size_t kOffDet = kOffKey + sizeof(uint64_t) * kMaxPerFrame;  // i32 [2048]
constexpr size_t kOffBox = kOffDet + sizeof(int32_t) * kMaxPerFrame;   // float4 [2048]
constexpr size_t kOffRoi = kOffBox + sizeof(float4) * kMaxPerFrame;    // i32 [2048]
constexpr size_t kOffKeptBox = kOffRoi + sizeof(int32_t) * kMaxPerFrame;  // float4 [2048]
constexpr size_t kOffKeptRoi = kOffKeptBox + sizeof(float4) * kMaxPerFrame;  // i32 [2048]
constexpr size_t kOffBits = kOffKeptRoi + sizeof(int32_t) * kMaxPerFrame;   // u32 [64][2]
constexpr size_t kOffAlive = kOffBits + sizeof(uint32_t) * 2 * kChunk; // u8 [2048]
constexpr size_t kLdsBytes = kOffAlive + kMaxPerFrame;

__global__ __launch_bounds__(kFrameThreads) void frame_kernel(const MergeParams P) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsBytes];
  __shared__ int s_kept;
  uint64_t *key = reinterpret_cast<uint64_t *>(lds + kOffKey);
  int32_t *det = reinterpret_cast<int32_t *>(lds + kOffDet);
  float4 *box = reinterpret_cast<float4 *>(lds + kOffBox);
  int32_t *roi = reinterpret_cast<int32_t *>(lds + kOffRoi);
  float4 *kept_box = reinterpret_cast<float4 *>(lds + kOffKeptBox);
  int32_t *kept_roi = reinterpret_cast<int32_t *>(lds + kOffKeptRoi);
  uint32_t *bits = reinterpret_cast<uint32_t *>(lds + kOffBits);  // row a: bits[2a], bits[2a+1]
  uint8_t *alive = lds + kOffAlive;
  const int tid = threadIdx.x, lane = tid & 63;
  const int f = blockIdx.x;
  const int lo = P.frame_begin[f];
  const int n = P.frame_begin[f + 1] - lo;
  if (n <= 0) return;
  if (n > kMaxPerFrame) {  // left unmerged
    for (int k = tid; k < n; k += kFrameThreads) P.keep[P.grouped[lo + k]] = 1;
    if (tid == 0) atomicAdd(P.n_overflow, 1);
    return;
  }
  int pw = 1;
  while (pw < n) pw <<= 1;
  for (int k = tid; k < pw; k += kFrameThreads) {
    if (k < n) {
      const int i = P.grouped[lo + k];
      const int32_t b = P.dets[i].box;
      const float s = (b >= 0 && b < P.n_scores) ? P.scores[b] : __builtin_nanf("");
      key[k] = rank_key(s, b);
      det[k] = i;
    } else {
      key[k] = ~uint64_t(0);  // padding sorts last
      det[k] = -1;
    }
  }
  if (tid == 0) s_kept = 0;
  __syncthreads();
  // Bitonic sort of pw keys, ascending.
  for (int size = 2; size <= pw; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = tid; t < pw / 2; t += kFrameThreads) {
        const int i = 2 * t - (t & (stride - 1));
        const int j = i + stride;
        const bool up = (i & size) == 0;
        const uint64_t ki = key[i], kj = key[j];
        if ((ki > kj) == up) {
          key[i] = kj;
          key[j] = ki;
          const int32_t d = det[i];
          det[i] = det[j];
          det[j] = d;
        }
      }
      __syncthreads();
    }
  }
  for (int k = tid; k < n; k += kFrameThreads) {
    const tg_det d = P.dets[det[k]];
    box[k] = make_float4(d.x1, d.y1, d.x2, d.y2);
    roi[k] = d.roi;
    alive[k] = 1;
  }
  __syncthreads();
  // Greedy over the ranking, kChunk candidates per round: (1) candidates overlapped by a
  // detection kept in an earlier round die -- lane l of every wave holds candidate l, the
  // waves share out the kept list; (2) the chunk's own suppression bits; (3) one wave walks
  // the chunk in rank order with row a of the bits in lane a. Equal to walking candidate
  // by candidate.
  const int wave = tid >> 6;
  for (int c0 = 0; c0 < n; c0 += kChunk) {
    const int m = min(kChunk, n - c0);
    const int K = s_kept;
    if (lane < m) {
      const float4 bj = box[c0 + lane];
      const int rj = roi[c0 + lane];
      bool dead = false;
#pragma unroll 4
      for (int e = wave; e < K; e += kFrameThreads / 64)
        dead |= (!P.cross_only || kept_roi[e] != rj) && suppresses(kept_box[e], bj, P.thr);
      if (dead) alive[c0 + lane] = 0;  // every writer stores 0
    }
    if (tid < 2 * kChunk) bits[tid] = 0;
    __syncthreads();
    {
      constexpr int kCols = kChunk * kChunk / kFrameThreads;  // columns per thread
      const int a = tid / (kChunk / kCols), q = tid % (kChunk / kCols);  // row a, columns
      uint32_t part = 0;                                                 // [kCols q, +kCols)
      if (a < m) {
        const float4 ba = box[c0 + a];
        const int ra = roi[c0 + a];
        for (int b = max(kCols * q, a + 1); b < min(kCols * q + kCols, m); ++b)
          if ((!P.cross_only || roi[c0 + b] != ra) && suppresses(ba, box[c0 + b], P.thr))
            part |= 1u << (b & 31);
        if (part) atomicOr(&bits[2 * a + ((kCols * q) >> 5)], part);
      }
    }
    __syncthreads();
    if (tid < 64) {
      const uint32_t row_lo = lane < m ? bits[2 * lane] : 0;
      const uint32_t row_hi = lane < m ? bits[2 * lane + 1] : 0;
      uint64_t removed = __ballot(lane < m && !alive[c0 + lane]) | (m < 64 ? ~uint64_t(0) << m : 0);
      for (int a = 0; a < m; ++a) {
        if ((removed >> a) & 1) continue;
        // readlane returns int: widen through uint32_t so bit 31 does not sign-extend
        const uint32_t lo32 = static_cast<uint32_t>(__builtin_amdgcn_readlane(row_lo, a));
        const uint32_t hi32 = static_cast<uint32_t>(__builtin_amdgcn_readlane(row_hi, a));
        removed |= (static_cast<uint64_t>(hi32) << 32) | lo32;
      }
      const bool keep_me = lane < m && !((removed >> lane) & 1);
      const uint64_t kb = __ballot(keep_me);
      if (keep_me) {
        const int slot = K + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                 static_cast<uint32_t>(kb >> 32),
                                 __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(kb), 0u)));
        kept_box[slot] = box[c0 + lane];
        kept_roi[slot] = roi[c0 + lane];
      }
      if (lane < m) alive[c0 + lane] = keep_me ? 1 : 0;
      if (lane == 0) s_kept = K + __popcll(kb);
    }
    __syncthreads();
  }
  for (int k = tid; k < n; k += kFrameThreads) P.keep[det[k]] = alive[k];
}

__global__ __launch_bounds__(kThreads) void compact_kernel(const MergeParams P) {
  __shared__ int s_blk, s_prefix;
  __shared__ int s_wave[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0)
    s_blk = static_cast<int>(__hip_atomic_fetch_add(P.ticket, 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT));
  __syncthreads();
  const int blk = s_blk;
  const int n = count_of(P);
  const int i0 = blk * kCompactBlock + kPerThread * tid;
  int flag[kPerThread];
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    flag[j] = i0 + j < n ? P.keep[i0 + j] : 0;
    cnt += flag[j] != 0;
  }
  int incl = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
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
      if (blk == static_cast<int>(gridDim.x) - 1) *P.n_kept = failed ? TG_E_INTERNAL : prefix + total;
    }
  }
  __syncthreads();
  int pos = s_prefix + before + incl - cnt;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j)
    if (flag[j]) P.out[pos++] = P.dets[i0 + j];
}

__global__ void zero_kernel(int32_t *a, int32_t *b) {
  *a = 0;
  *b = 0;
}

int compact_blocks(int32_t n_max) { return (n_max + kCompactBlock - 1) / kCompactBlock; }

// Workspace layout, in bytes from the (8-byte aligned) start.
struct Layout {
  size_t state, counts, cursor, begin, grouped, total;
};
Layout layout(int32_t n_max, int32_t n_frames) {
  Layout L;
  L.state = 0;  // ticket word + one look-back word per compaction workgroup
  L.counts = sizeof(uint64_t) * (1 + static_cast<size_t>(compact_blocks(n_max)));
  L.cursor = L.counts + sizeof(int32_t) * static_cast<size_t>(n_frames);
  L.begin = L.cursor + sizeof(int32_t) * static_cast<size_t>(n_frames);
  L.grouped = L.begin + sizeof(int32_t) * (static_cast<size_t>(n_frames) + 1);
  L.total = L.grouped + sizeof(int32_t) * static_cast<size_t>(n_max);
  return L;
}

}  // namespace

extern "C" size_t tg_merge_workspace_bytes(int32_t n_max, int32_t n_frames) {
  if (n_max <= 0 || n_frames < 0) return 0;
  return layout(n_max, n_frames).total;
}

extern "C" int tg_merge(const tg_merge_args *a, void *stream) {
  if (!a || a->n_max < 0 || a->n_scores < 0 || a->n_frames < 0 || !a->n_kept ||
      !a->n_overflow || !(a->iou_threshold == a->iou_threshold))
    return TG_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (a->n_max == 0) {
    hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(1), 0, s, a->n_kept, a->n_overflow);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  if (!a->dets || !a->n_dets || !a->keep || !a->out || (a->n_scores > 0 && !a->scores))
    return TG_E_INVAL;
  if (int64_t(a->n_frames) + 1 > 0x7FFFFFFF / 2) return TG_E_INVAL;
  const Layout L = layout(a->n_max, a->n_frames);
  if (!a->workspace || a->workspace_bytes < L.total ||
      reinterpret_cast<uintptr_t>(a->workspace) % 8 != 0)
    return TG_E_WORKSPACE;

  uint8_t *ws = static_cast<uint8_t *>(a->workspace);
  MergeParams P;
  P.dets = a->dets;
  P.n_dets = a->n_dets;
  P.n_max = a->n_max;
  P.scores = a->scores;
  P.n_scores = a->n_scores;
  P.n_frames = a->n_frames;
  P.thr = a->iou_threshold;
  P.cross_only = a->cross_only;
  P.keep = a->keep;
  P.out = a->out;
  P.n_kept = a->n_kept;
  P.n_overflow = a->n_overflow;
  P.ticket = reinterpret_cast<uint32_t *>(ws + L.state);
  P.state = reinterpret_cast<uint64_t *>(ws + L.state) + 1;
  P.counts = reinterpret_cast<int32_t *>(ws + L.counts);
  P.cursor = reinterpret_cast<int32_t *>(ws + L.cursor);
  P.frame_begin = reinterpret_cast<int32_t *>(ws + L.begin);
  P.grouped = reinterpret_cast<int32_t *>(ws + L.grouped);

  const int32_t words32 = 2 * a->n_frames;  // counts + cursor
  const int32_t words64 = 1 + compact_blocks(a->n_max);
  const int32_t clear_n = words32 > words64 ? words32 : words64;
  const uint32_t per = static_cast<uint32_t>((a->n_max + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(clear_kernel, dim3((clear_n + kThreads - 1) / kThreads), dim3(kThreads), 0,
                     s, P, words32, words64);
  hipLaunchKernelGGL(count_kernel, dim3(per), dim3(kThreads), 0, s, P);
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kScanThreads), 0, s, P);
  hipLaunchKernelGGL(scatter_kernel, dim3(per), dim3(kThreads), 0, s, P);
  if (a->n_frames > 0)
    hipLaunchKernelGGL(frame_kernel, dim3(static_cast<uint32_t>(a->n_frames)), dim3(kFrameThreads), 0,
                       s, P);
  hipLaunchKernelGGL(compact_kernel, dim3(static_cast<uint32_t>(compact_blocks(a->n_max))),
                     dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
