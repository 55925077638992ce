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
//  5. one 1024-thread workgroup per frame: bitonic sort of 64-bit keys (score, box), then
//     the greedy pass 64 candidates at a time (all threads test the chunk against the
//     detections kept so far and fill the chunk's 64 x 64 suppression bits; one wave walks
//     the chunk). Frames of up to 1024 detections do all of it in LDS. Larger frames sort
//     in the workspace (global bitonic passes for the long strides, LDS tiles of up to 4096
//     keys for the short ones) and index their ranked boxes by a grid of up to 32 x 32 cells
//     over the frame's boxes: a candidate is tested only against the earlier kept
//     detections registered in the cells its box touches, plus a "wide" list (see
//     large_frame for why this finds every suppressor);
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
constexpr int kMaxPerFrame = 1024;  // frames ranked and walked in LDS; larger: workspace
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
  int32_t *counts;       // [n_frames]
  int32_t *cursor;       // [n_frames]
  int32_t *frame_begin;  // [n_frames + 1]
  int32_t *grouped;      // [n_max]
  uint32_t *ticket;
  uint64_t *state;       // [compaction workgroups]
  // Scratch of frames over kMaxPerFrame detections; frame f (first detection lo, n of
  // them) owns [2 lo, 2 (lo + n)) of the key arrays and [lo, lo + n) (times kCellsMax for
  // the cell lists) of the others, so frames never share a word.
  uint64_t *big_key;     // [2 n_max] ranking keys
  int32_t *big_det;      // [2 n_max] detection index of each key
  float4 *rbox;          // [n_max] ranked boxes
  int32_t *rroi;         // [n_max] ranked patch ids
  uint32_t *rcell;       // [n_max] ranked cell ranges (kWide, kEmpty or packed)
  float4 *ebox;          // [kCellsMax n_max] kept boxes listed per cell, then the wide list
  int32_t *eroi;         // [kCellsMax n_max] their patch ids
  float4 *kbox;          // [n_max] all kept boxes, in rank order
  int32_t *kroi;         // [n_max] their patch ids
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
constexpr size_t kOffKey = 0;                                          // u64 [kMaxPerFrame]
constexpr size_t kOffDet = kOffKey + sizeof(uint64_t) * kMaxPerFrame;  // i32 [kMaxPerFrame]
constexpr size_t kOffBox = kOffDet + sizeof(int32_t) * kMaxPerFrame;   // float4 [kMaxPerFrame]
constexpr size_t kOffRoi = kOffBox + sizeof(float4) * kMaxPerFrame;    // i32 [kMaxPerFrame]
constexpr size_t kOffKeptBox = kOffRoi + sizeof(int32_t) * kMaxPerFrame;  // float4 [kMaxPerFrame]
constexpr size_t kOffKeptRoi = kOffKeptBox + sizeof(float4) * kMaxPerFrame;  // i32 [kMaxPerFrame]
constexpr size_t kOffBits = kOffKeptRoi + sizeof(int32_t) * kMaxPerFrame;   // u32 [64][2]
constexpr size_t kOffAlive = kOffBits + sizeof(uint32_t) * 2 * kChunk; // u8 [kMaxPerFrame]
constexpr size_t kLdsBytes = kOffAlive + kMaxPerFrame;


// Step (2) of a chunk (all threads): bit b of row a (bits[2a], bits[2a+1]) is set when
// candidate a suppresses candidate b, for a < b < m; bits must be zero on entry.
__device__ __forceinline__ void chunk_bits(const MergeParams &P, const float4 *box,
                                           const int32_t *roi, int m, uint32_t *bits) {
  constexpr int kCols = kChunk * kChunk / kFrameThreads;  // columns per thread
  const int tid = threadIdx.x;
  const int a = tid / (kChunk / kCols), q = tid % (kChunk / kCols);  // row a, columns
  uint32_t part = 0;                                                 // [kCols q, +kCols)
  if (a < m) {
    const float4 ba = box[a];
    const int ra = roi[a];
    for (int b = max(kCols * q, a + 1); b < min(kCols * q + kCols, m); ++b)
      if ((!P.cross_only || roi[b] != ra) && suppresses(ba, box[b], P.thr))
        part |= 1u << (b & 31);
    if (part) atomicOr(&bits[2 * a + ((kCols * q) >> 5)], part);
  }
}

// Step (3) of a chunk (one wave, row a of the bits in lane a): walks the m candidates in
// rank order, skipping the ones already dead (alive[a] == 0) or removed by a candidate
// kept before them; returns the mask of kept candidates (bit a = candidate a).
__device__ __forceinline__ uint64_t chunk_walk(const uint8_t *alive, const uint32_t *bits,
                                               int m) {
  const int lane = threadIdx.x & 63;
  const uint32_t row_lo = lane < m ? bits[2 * lane] : 0;
  const uint32_t row_hi = lane < m ? bits[2 * lane + 1] : 0;
  uint64_t removed = __ballot(lane < m && !alive[lane]) | (m < 64 ? ~uint64_t(0) << m : 0);
  // only candidates that suppress someone in the chunk can change `removed`: visit those
  // in rank order (a later one's row cannot affect an earlier candidate)
  for (uint64_t rows = __ballot((row_lo | row_hi) != 0); rows != 0; rows &= rows - 1) {
    const int a = __builtin_ctzll(rows);
    if ((removed >> a) & 1) continue;
    // readlane returns int: widen through uint32_t so bit 31 does not sign-extend
    const uint32_t lo32 = static_cast<uint32_t>(__builtin_amdgcn_readlane(row_lo, a));
    const uint32_t hi32 = static_cast<uint32_t>(__builtin_amdgcn_readlane(row_hi, a));
    removed |= (static_cast<uint64_t>(hi32) << 32) | lo32;
  }
  return __ballot(lane < m && !((removed >> lane) & 1));
}

// ---- frames of more than kMaxPerFrame detections ---------------------------------------

constexpr int kTileKeys = 4096;  // keys per LDS tile of the large-frame sort
constexpr int kGridMax = 32;     // cells per axis of the large-frame index
constexpr int kCellsMax = 4;     // cells a box may touch before it goes on the wide list
constexpr uint32_t kWide = 0xFFFFFFFFu;   // tested against every kept detection
constexpr uint32_t kEmpty = 0xFFFFFFFEu;  // x2 < x1 or y2 < y1: overlaps nothing

__device__ __forceinline__ void cmpx(uint64_t *key, int32_t *det, int i, int j, bool up) {
  const uint64_t ki = key[i], kj = key[j];
  if ((ki > kj) == up) {
    key[i] = kj;
    key[j] = ki;
    const int32_t d = det[i];
    det[i] = det[j];
    det[j] = d;
  }
}

// Ascending bitonic sort of gk[0, pw) (payload gd), pw a power of two: the strides of a
// tile (min(pw, kTileKeys) keys) and more are passes over global memory, the shorter ones
// run tile by tile in LDS (tk, td). Each compare-exchange is the one of the plain network.
__device__ __forceinline__ void sort_large(uint64_t *gk, int32_t *gd, int pw, uint64_t *tk,
                                           int32_t *td) {
  const int tid = threadIdx.x;
  const int tile = min(pw, kTileKeys);
  for (int size = tile; size <= pw; size <<= 1) {
    for (int stride = size >> 1; stride >= tile; stride >>= 1) {
      for (int t = tid; t < pw / 2; t += kFrameThreads) {
        const int i = 2 * t - (t & (stride - 1));
        cmpx(gk, gd, i, i + stride, (i & size) == 0);
      }
      __syncthreads();
    }
    // the first round sorts every tile through sizes 2 .. tile; later rounds finish size
    // `size` with the strides below the tile
    for (int base = 0; base < pw; base += tile) {
      for (int k = tid; k < tile; k += kFrameThreads) {
        tk[k] = gk[base + k];
        td[k] = gd[base + k];
      }
      __syncthreads();
      for (int sz = size == tile ? 2 : size; sz <= size; sz <<= 1) {
        for (int stride = min(sz, tile) >> 1; stride > 0; stride >>= 1) {
          for (int t = tid; t < tile / 2; t += kFrameThreads) {
            const int i = 2 * t - (t & (stride - 1));
            cmpx(tk, td, i, i + stride, ((base + i) & sz) == 0);
          }
          __syncthreads();
        }
      }
      for (int k = tid; k < tile; k += kFrameThreads) {
        gk[base + k] = tk[k];
        gd[base + k] = td[k];
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ float wave_minf(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_maxf(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sumf(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Cell of coordinate v (not NaN) on an axis starting at e0 with scale sc (cells per unit,
// finite, >= 0) and g cells: non-decreasing in v, clamped to [0, g).
__device__ __forceinline__ int cell_of(float v, float e0, float sc, int g) {
  const float t = fminf(fmaxf(__fmul_rn(__fsub_rn(v, e0), sc), 0.0f), static_cast<float>(g - 1));
  return static_cast<int>(t);
}

static_assert(kLdsBytes >= (sizeof(uint64_t) + sizeof(int32_t)) * kTileKeys,
              "the large-frame sort tile fits in the frame's LDS");

struct LargeLds {
  float ex0, sx, ey0, sy;
  int gx, gy, all_wide, kept;
  float red[4][kFrameThreads / 64];
  float sum[2][kFrameThreads / 64];
  int off[kGridMax * kGridMax + 2];  // list starts (cells, then the wide list), then the end
  int cur[kGridMax * kGridMax + 1];  // list sizes while counting, then kept entries so far
  float4 cbox[kChunk];
  int32_t croi[kChunk];
  uint32_t crange[kChunk];
  uint8_t calive[kChunk];
  uint32_t bits[2 * kChunk];
  // step (1): candidate q's lists to scan (start in ebox, or -1 for the kept list; length)
  int sstart[kChunk][kCellsMax + 1], slen[kChunk][kCellsMax + 1];
};

// One frame of n > kMaxPerFrame detections (grouped[lo, lo + n)), by one workgroup.
//
// Why the cell index finds every suppressor: with a threshold t >= 0, a suppresses b only
// if inter > t * union >= 0 (the union of two boxes is never negative), so inter > 0 and
// both clipped widths are positive: min(x2a, x2b) > max(x1a, x1b) and likewise in y. The
// point (max(x1a, x1b), max(y1a, y1b)) then lies in both boxes, and since cell_of is
// non-decreasing, its cell lies in the cell ranges of both: a and b share a cell. Boxes
// with a NaN coordinate (where min and max ignore the NaN operand), boxes touching more
// than kCellsMax cells, and every box when t < 0, are "wide": a wide candidate is tested
// against the whole kept list, and every candidate also scans the list of wide boxes.
// Boxes with x2 < x1 or y2 < y1 have no positive width with anything, so when t >= 0
// they neither suppress nor are suppressed and are registered nowhere.
static_assert(sizeof(LargeLds) <= kLdsBytes, "the large-frame state fits in the frame's LDS");

__device__ __forceinline__ void large_frame(const MergeParams &P, int lo, int n, uint8_t *lds) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t *gk = P.big_key + 2 * static_cast<int64_t>(lo);
  int32_t *gd = P.big_det + 2 * static_cast<int64_t>(lo);
  float4 *rbox = P.rbox + lo;
  int32_t *rroi = P.rroi + lo;
  uint32_t *rcell = P.rcell + lo;
  float4 *ebox = P.ebox + static_cast<int64_t>(kCellsMax) * lo;
  int32_t *eroi = P.eroi + static_cast<int64_t>(kCellsMax) * lo;
  float4 *kbox = P.kbox + lo;
  int32_t *kroi = P.kroi + lo;

  // 1. Ranking: keys in the workspace, sorted.
  int pw = 1;
  while (pw < n) pw <<= 1;  // < 2 n
  for (int k = tid; k < pw; k += kFrameThreads) {
    if (k < n) {
      const int i = P.grouped[lo + k];
      const int32_t b = P.dets[i].box;
      const float s = (b >= 0 && b < P.n_scores) ? P.scores[b] : __builtin_nanf("");
      gk[k] = rank_key(s, b);
      gd[k] = i;
    } else {
      gk[k] = ~uint64_t(0);
      gd[k] = -1;
    }
  }
  __syncthreads();
  sort_large(gk, gd, pw, reinterpret_cast<uint64_t *>(lds),
             reinterpret_cast<int32_t *>(lds + sizeof(uint64_t) * kTileKeys));

  // 2. Ranked boxes, and the frame's extent and mean box size for the grid.
  LargeLds &S = *reinterpret_cast<LargeLds *>(lds);
  float xlo = __builtin_inff(), xhi = -__builtin_inff(), ylo = xlo, yhi = xhi;
  float sw = 0.0f, sh = 0.0f;
  for (int r = tid; r < n; r += kFrameThreads) {
    const tg_det d = P.dets[gd[r]];
    rbox[r] = make_float4(d.x1, d.y1, d.x2, d.y2);
    rroi[r] = d.roi;
    if (__builtin_isfinite(d.x1) && __builtin_isfinite(d.x2) && d.x2 >= d.x1) {
      xlo = fminf(xlo, d.x1);
      xhi = fmaxf(xhi, d.x2);
      sw += d.x2 - d.x1;
    }
    if (__builtin_isfinite(d.y1) && __builtin_isfinite(d.y2) && d.y2 >= d.y1) {
      ylo = fminf(ylo, d.y1);
      yhi = fmaxf(yhi, d.y2);
      sh += d.y2 - d.y1;
    }
  }
  xlo = wave_minf(xlo);
  xhi = wave_maxf(xhi);
  ylo = wave_minf(ylo);
  yhi = wave_maxf(yhi);
  sw = wave_sumf(sw);
  sh = wave_sumf(sh);
  if (lane == 0) {
    S.red[0][wave] = xlo;
    S.red[1][wave] = xhi;
    S.red[2][wave] = ylo;
    S.red[3][wave] = yhi;
    S.sum[0][wave] = sw;
    S.sum[1][wave] = sh;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kFrameThreads / 64; ++w) {
      S.red[0][0] = fminf(S.red[0][0], S.red[0][w]);
      S.red[1][0] = fmaxf(S.red[1][0], S.red[1][w]);
      S.red[2][0] = fminf(S.red[2][0], S.red[2][w]);
      S.red[3][0] = fmaxf(S.red[3][0], S.red[3][w]);
      S.sum[0][0] += S.sum[0][w];
      S.sum[1][0] += S.sum[1][w];
    }
    // Cells about twice the mean box size, at most kGridMax per axis. Any finite scale
    // keeps the index exact (only its speed depends on it), so approximate reciprocals
    // do; a degenerate extent just puts everything in one cell.
    const float span_x = S.red[1][0] - S.red[0][0], span_y = S.red[3][0] - S.red[2][0];
    const float inv_n = __builtin_amdgcn_rcpf(static_cast<float>(n));
    const float mw = S.sum[0][0] * inv_n, mh = S.sum[1][0] * inv_n;
    const float fx = span_x * __builtin_amdgcn_rcpf(fmaxf(2.0f * mw, 1e-30f));
    const float fy = span_y * __builtin_amdgcn_rcpf(fmaxf(2.0f * mh, 1e-30f));
    S.gx = fx >= 2.0f ? static_cast<int>(fminf(fx, static_cast<float>(kGridMax))) : 1;
    S.gy = fy >= 2.0f ? static_cast<int>(fminf(fy, static_cast<float>(kGridMax))) : 1;
    const float scx = S.gx * __builtin_amdgcn_rcpf(span_x);
    const float scy = S.gy * __builtin_amdgcn_rcpf(span_y);
    S.ex0 = __builtin_isfinite(S.red[0][0]) ? S.red[0][0] : 0.0f;
    S.ey0 = __builtin_isfinite(S.red[2][0]) ? S.red[2][0] : 0.0f;
    S.sx = (__builtin_isfinite(scx) && scx > 0.0f) ? scx : 0.0f;
    S.sy = (__builtin_isfinite(scy) && scy > 0.0f) ? scy : 0.0f;
    S.all_wide = !(P.thr >= 0.0f);
    S.kept = 0;
  }
  for (int c = tid; c < kGridMax * kGridMax + 1; c += kFrameThreads) S.cur[c] = 0;
  __syncthreads();

  // 3. Cell index: each ranked box's cell range, then counts, offsets and the entries.
  const int gx = S.gx, gy = S.gy, n_cells = gx * gy;
  for (int r = tid; r < n; r += kFrameThreads) {
    const float4 b = rbox[r];
    uint32_t cr;
    if (S.all_wide || b.x != b.x || b.y != b.y || b.z != b.z || b.w != b.w) {
      cr = kWide;
    } else if (b.z < b.x || b.w < b.y) {
      cr = kEmpty;
    } else {
      const int cx0 = cell_of(b.x, S.ex0, S.sx, gx), cx1 = cell_of(b.z, S.ex0, S.sx, gx);
      const int cy0 = cell_of(b.y, S.ey0, S.sy, gy), cy1 = cell_of(b.w, S.ey0, S.sy, gy);
      cr = (cx1 - cx0 + 1) * (cy1 - cy0 + 1) > kCellsMax
               ? kWide
               : static_cast<uint32_t>(cx0 | cx1 << 8 | cy0 << 16 | cy1 << 24);
    }
    rcell[r] = cr;
    if (cr == kWide) {
      atomicAdd(&S.cur[n_cells], 1);
    } else if (cr != kEmpty) {
      for (int cy = (cr >> 16) & 0xFF; cy <= static_cast<int>(cr >> 24); ++cy)
        for (int cx = cr & 0xFF; cx <= static_cast<int>((cr >> 8) & 0xFF); ++cx)
          atomicAdd(&S.cur[cy * gx + cx], 1);
    }
  }
  __syncthreads();
  if (wave == 0) {  // starts of the n_cells + 1 lists: lane l sums a run of them
    constexpr int kRun = (kGridMax * kGridMax + 1 + 63) / 64;
    const int c0 = lane * kRun, c1 = min(c0 + kRun, n_cells + 1);
    int sum = 0;
    for (int c = c0; c < c1; ++c) sum += S.cur[c];
    int incl = sum;
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o);
      if (lane >= o) incl += v;
    }
    int at = incl - sum;
    for (int c = c0; c < c1; ++c) {
      const int k = S.cur[c];
      S.off[c] = at;
      S.cur[c] = 0;  // from here on: kept detections listed so far
      at += k;
    }
    if (lane == 63) S.off[n_cells + 1] = incl;
  }
  __syncthreads();

  // 4. The greedy, kChunk candidates per round as for small frames. A kept detection is
  // appended, box and patch inline, to the lists of the cells its box touches (or to the
  // wide list) -- each list has room for every detection registered in it -- and to the
  // kept list; step (1) scans, for each candidate, only the lists that can hold a
  // suppressor of it, all candidates' entries flattened over the workgroup.
  // the first chunk's candidates; each round loads the next one's while it works
  float4 nb = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  uint32_t ncr = kEmpty;
  int nroi = 0;
  if (tid < min(kChunk, n)) {
    nb = rbox[tid];
    ncr = rcell[tid];
    nroi = rroi[tid];
  }
  for (int c0 = 0; c0 < n; c0 += kChunk) {
    const int m = min(kChunk, n - c0);
    const int K = S.kept;
    if (tid < m) {
      const float4 b = nb;
      const uint32_t cr = ncr;
      S.cbox[tid] = b;
      S.croi[tid] = nroi;
      S.crange[tid] = cr;
      S.calive[tid] = 1;
      int ns = 0;
      if (cr == kWide) {
        S.sstart[tid][0] = -1;
        S.slen[tid][0] = K;
        ns = 1;
      } else if (cr != kEmpty) {
        for (int cy = (cr >> 16) & 0xFF; cy <= static_cast<int>(cr >> 24); ++cy)
          for (int cx = cr & 0xFF; cx <= static_cast<int>((cr >> 8) & 0xFF); ++cx, ++ns) {
            S.sstart[tid][ns] = S.off[cy * gx + cx];
            S.slen[tid][ns] = S.cur[cy * gx + cx];
          }
        S.sstart[tid][ns] = S.off[n_cells];
        S.slen[tid][ns] = S.cur[n_cells];
        ++ns;
      }
      for (; ns <= kCellsMax; ++ns) S.slen[tid][ns] = 0;
    }
    if (tid < 2 * kChunk) S.bits[tid] = 0;
    __syncthreads();
    if (tid < min(kChunk, n - c0 - kChunk)) {  // next round's candidates
      nb = rbox[c0 + kChunk + tid];
      ncr = rcell[c0 + kChunk + tid];
      nroi = rroi[c0 + kChunk + tid];
    }
    // (1) 16 threads per candidate over its lists, up to 8 entries each per pass with the
    // loads issued together
    {
      constexpr int kSub = kFrameThreads / kChunk, kBatch = 8;
      const int q = tid / kSub, sub = tid % kSub;
      if (q < m) {
        int st[kCellsMax + 1], ln[kCellsMax + 1], tq = 0;
#pragma unroll
        for (int k = 0; k <= kCellsMax; ++k) {
          st[k] = S.sstart[q][k];
          ln[k] = S.slen[q][k];
          tq += ln[k];
        }
        const float4 bq = S.cbox[q];
        const int rq = S.croi[q];
        bool dead = false;
        for (int t0 = sub; t0 < tq; t0 += kSub * kBatch) {
          float4 kb[kBatch];
          int kr[kBatch];
#pragma unroll
          for (int u = 0; u < kBatch; ++u) {
            int j = t0 + u * kSub;
            if (j >= tq) continue;
            int at = st[0], k = 0;
#pragma unroll
            for (int kk = 0; kk < kCellsMax; ++kk)  // which list: step over the earlier ones
              if (k == kk && j >= ln[kk]) {
                j -= ln[kk];
                k = kk + 1;
                at = st[kk + 1];
              }
            kb[u] = at < 0 ? kbox[j] : ebox[at + j];
            kr[u] = at < 0 ? kroi[j] : eroi[at + j];
          }
#pragma unroll
          for (int u = 0; u < kBatch; ++u)
            if (t0 + u * kSub < tq && (!P.cross_only || kr[u] != rq) &&
                suppresses(kb[u], bq, P.thr))
              dead = true;
        }
        if (dead) S.calive[q] = 0;  // every writer stores 0
      }
    }
    __syncthreads();
    chunk_bits(P, S.cbox, S.croi, m, S.bits);
    __syncthreads();
    if (tid < 64) {
      const uint64_t kb = chunk_walk(S.calive, S.bits, m);
      const bool keep_me = (kb >> lane) & 1;
      if (lane < m) P.keep[gd[c0 + lane]] = keep_me ? 1 : 0;
      if (keep_me) {
        const float4 b = S.cbox[lane];
        const int roi = S.croi[lane];
        const uint32_t cr = S.crange[lane];
        const int slot = K + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                 static_cast<uint32_t>(kb >> 32),
                                 __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(kb), 0u)));
        kbox[slot] = b;
        kroi[slot] = roi;
        if (cr == kWide) {
          const int at = S.off[n_cells] + atomicAdd(&S.cur[n_cells], 1);
          ebox[at] = b;
          eroi[at] = roi;
        } else if (cr != kEmpty) {
          for (int cy = (cr >> 16) & 0xFF; cy <= static_cast<int>(cr >> 24); ++cy)
            for (int cx = cr & 0xFF; cx <= static_cast<int>((cr >> 8) & 0xFF); ++cx) {
              const int at = S.off[cy * gx + cx] + atomicAdd(&S.cur[cy * gx + cx], 1);
              ebox[at] = b;
              eroi[at] = roi;
            }
        }
      }
      if (lane == 0) S.kept = K + __popcll(kb);
    }
    __syncthreads();
  }
}

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
  if (n > kMaxPerFrame) {
    large_frame(P, lo, n, lds);
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
    chunk_bits(P, box + c0, roi + c0, m, bits);
    __syncthreads();
    if (tid < 64) {
      const uint64_t kb = chunk_walk(alive + c0, bits, m);
      const bool keep_me = (kb >> lane) & 1;
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

__global__ void zero_kernel(int32_t *a) { *a = 0; }

int compact_blocks(int32_t n_max) { return (n_max + kCompactBlock - 1) / kCompactBlock; }

// Workspace layout, in bytes from the (16-byte aligned) start.
struct Layout {
  size_t state, counts, cursor, begin, grouped;
  size_t big_key, big_det, rbox, rroi, rcell, ebox, eroi, kbox, kroi, total;
};
size_t round16(size_t v) { return (v + 15) / 16 * 16; }
Layout layout(int32_t n_max, int32_t n_frames) {
  Layout L;
  const size_t n = static_cast<size_t>(n_max);
  L.state = 0;  // ticket word + one look-back word per compaction workgroup
  L.counts = sizeof(uint64_t) * (1 + static_cast<size_t>(compact_blocks(n_max)));
  L.cursor = L.counts + sizeof(int32_t) * static_cast<size_t>(n_frames);
  L.begin = L.cursor + sizeof(int32_t) * static_cast<size_t>(n_frames);
  L.grouped = L.begin + sizeof(int32_t) * (static_cast<size_t>(n_frames) + 1);
  L.big_key = round16(L.grouped + sizeof(int32_t) * n);
  L.big_det = L.big_key + sizeof(uint64_t) * 2 * n;
  L.rbox = round16(L.big_det + sizeof(int32_t) * 2 * n);
  L.rroi = L.rbox + sizeof(float4) * n;
  L.rcell = L.rroi + sizeof(int32_t) * n;
  L.ebox = round16(L.rcell + sizeof(uint32_t) * n);
  L.eroi = L.ebox + sizeof(float4) * kCellsMax * n;
  L.kbox = round16(L.eroi + sizeof(int32_t) * kCellsMax * n);
  L.kroi = L.kbox + sizeof(float4) * n;
  L.total = L.kroi + sizeof(int32_t) * n;
  return L;
}

}  // namespace

extern "C" size_t tg_merge_workspace_bytes(int32_t n_max, int32_t n_frames) {
  if (n_max <= 0 || n_frames < 0) return 0;
  return layout(n_max, n_frames).total;
}

extern "C" int tg_merge(const tg_merge_args *a, void *stream) {
  if (!a || a->n_max < 0 || a->n_scores < 0 || a->n_frames < 0 || !a->n_kept ||
      !(a->iou_threshold == a->iou_threshold))
    return TG_E_INVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (a->n_max == 0) {
    hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(1), 0, s, a->n_kept);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  if (!a->dets || !a->n_dets || !a->keep || !a->out || (a->n_scores > 0 && !a->scores))
    return TG_E_INVAL;
  if (int64_t(a->n_frames) + 1 > 0x7FFFFFFF / 2) return TG_E_INVAL;
  const Layout L = layout(a->n_max, a->n_frames);
  if (!a->workspace || a->workspace_bytes < L.total ||
      reinterpret_cast<uintptr_t>(a->workspace) % 16 != 0)
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
  P.ticket = reinterpret_cast<uint32_t *>(ws + L.state);
  P.state = reinterpret_cast<uint64_t *>(ws + L.state) + 1;
  P.counts = reinterpret_cast<int32_t *>(ws + L.counts);
  P.cursor = reinterpret_cast<int32_t *>(ws + L.cursor);
  P.frame_begin = reinterpret_cast<int32_t *>(ws + L.begin);
  P.grouped = reinterpret_cast<int32_t *>(ws + L.grouped);
  P.big_key = reinterpret_cast<uint64_t *>(ws + L.big_key);
  P.big_det = reinterpret_cast<int32_t *>(ws + L.big_det);
  P.rbox = reinterpret_cast<float4 *>(ws + L.rbox);
  P.rroi = reinterpret_cast<int32_t *>(ws + L.rroi);
  P.rcell = reinterpret_cast<uint32_t *>(ws + L.rcell);
  P.ebox = reinterpret_cast<float4 *>(ws + L.ebox);
  P.eroi = reinterpret_cast<int32_t *>(ws + L.eroi);
  P.kbox = reinterpret_cast<float4 *>(ws + L.kbox);
  P.kroi = reinterpret_cast<int32_t *>(ws + L.kroi);

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
