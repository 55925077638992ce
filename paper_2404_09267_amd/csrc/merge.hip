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
// Eight launches on the caller's stream, all on device data (the detection count comes from
// tg_unstitch's n_out on the device):
//  1. clear the per-frame counters and look-back words;
//  2. count detections per frame (LDS histograms, one global atomic per frame and
//     workgroup);
//  3. exclusive scan of the counts (one workgroup);
//  4. scatter detection indices into frame groups (ranks inside a workgroup from LDS, one
//     range per frame and workgroup from a global cursor; the order inside a group does
//     not matter, the ranking below is a total order), with each detection's ranking key
//     (score, box), box and patch at its place in the group;
//  5-7. the greedy decided in rounds, with no sort: a spatial index of each frame's boxes
//     (one workgroup per frame), each detection's suppressors ranked above it (over the
//     whole grid), then per frame rounds in which a detection is suppressed once one of
//     them is kept and kept once all of them are suppressed (see "the greedy of a frame"
//     for why this is the greedy walk's result and why the index finds every suppressor);
//     a frame of at most kSmallMax detections is instead decided by its index workgroup
//     in LDS, each pair of its detections tested once;
//  8. stable compaction of the kept detections (decoupled look-back, 1024 per workgroup).
// Inputs of at most kTiny detections (by capacity) take one launch instead (tiny_kernel).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "lookback.h"
#include "tg.h"

// Built with -ffp-contract=off: every binary32 operation here is rounded on its own (no
// multiply-add fusion), so decisions taken in floating point match any plain IEEE
// implementation of the same steps.

namespace {

constexpr int kThreads = 256;
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
  int32_t *counts;       // frame f at [f * cstride]
  int32_t *cursor;       // frame f at [f * cstride]
  int32_t cstride;       // kCounterStride, or 1 for very many frames
  int32_t *frame_begin;  // [n_frames + 1]
  int32_t *grouped;      // [n_max]
  uint32_t *ticket;
  uint32_t *status;      // set when a frame's rounds overrun (cannot happen)
  uint64_t *state;       // [compaction workgroups]
  uint32_t *big;         // set when a frame is too large for its index workgroup alone
  // Per detection, at its position in its frame group: frame f (first detection lo, n of
  // them) owns [lo, lo + n) of these (times kCellsMax for the cell lists), so frames
  // never share a word.
  uint64_t *rkey;        // [n_max] ranking keys
  float4 *rbox;          // [n_max] boxes
  int32_t *rroi;         // [n_max] patch ids
  uint32_t *rcell;       // [n_max] cell ranges (kWide, kEmpty or packed)
  int32_t *rstate;       // [n_max] kUndecided, kKept or kSuppressed
  int32_t *rlist;        // [2 (kCellsMax + 1) n_max] the lists to search: starts, sizes
  int32_t *rpred;        // [kPredSlots n_max] suppressors ranked above (positions)
  int32_t *rnpred;       // [n_max] how many
  int32_t *rovf;         // [n_max] a longer list's start in ovf, or -1: search again
  int32_t *ovf;          // [kOvfPerDet n_max] the whole lists of detections with more
  int64_t ovf_cap;
  unsigned long long *ovf_used;  // entries of ovf handed out
  float4 *ebox;          // [kCellsMax n_max] boxes listed per cell, then the wide list
  int4 *eaux;            // [kCellsMax n_max] their patch ids, keys and positions
};

__device__ __forceinline__ int count_of(const MergeParams &P) {
  return min(max(*P.n_dets, 0), P.n_max);
}

// Frame counters one 256-byte slot apart: the count and scatter passes add to them with
// global atomics (many detections per frame), and counters packed into a few cache lines
// queue on those lines (window_64x30, 1,920 frames: count 20 us, scatter 33 us packed).
constexpr int kCounterStride = 64;      // int32 words
constexpr int kPaddedFramesMax = 16384; // beyond: packed (4 MB of slots at most)

__global__ void clear_kernel(MergeParams P, int32_t n_frames, int32_t n_words64) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_frames) {
    P.counts[static_cast<int64_t>(i) * P.cstride] = 0;
    P.cursor[static_cast<int64_t>(i) * P.cstride] = 0;
  }
  // ticket and status, the overflow cursor, the large-frame flag, the look-back states
  if (i < n_words64) reinterpret_cast<uint64_t *>(P.ticket)[i] = 0;
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
      atomicAdd(local ? &hist[f] : &P.counts[static_cast<int64_t>(f) * P.cstride], 1);
    else
      P.keep[i] = 0;  // no frame to merge in: dropped
  }
  if (!local) return;
  __syncthreads();
  for (int f = tid; f < P.n_frames; f += kThreads)
    if (hist[f]) atomicAdd(&P.counts[static_cast<int64_t>(f) * P.cstride], hist[f]);
}

__global__ __launch_bounds__(kScanThreads) void scan_kernel(const MergeParams P) {
  __shared__ int s_wave[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int carry = 0;
  for (int base = 0; base < P.n_frames; base += kScanThreads) {
    const int f = base + tid;
    const int v = f < P.n_frames ? P.counts[static_cast<int64_t>(f) * P.cstride] : 0;
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

// Ranking key, ascending = higher score first, then lower box index. NaN ranks as -inf;
// -0 and +0 are the same score.
__device__ __forceinline__ uint64_t rank_key(float s, int32_t box) {
  if (s != s) s = -__builtin_inff();
  if (s == 0.0f) s = 0.0f;
  uint32_t b = __float_as_uint(s);
  b ^= (b & 0x80000000u) ? 0xFFFFFFFFu : 0x80000000u;  // ascending order of floats
  return (static_cast<uint64_t>(~b) << 32) | static_cast<uint32_t>(box);
}

// Detection indices into frame groups, with each detection's ranking key, box and patch
// at its position in the group. Up to kHistMax frames a workgroup ranks its detections per
// frame in LDS and reserves one range per non-empty frame.
__global__ __launch_bounds__(kThreads) void scatter_kernel(const MergeParams P) {
  __shared__ int hist[kHistMax];
  const int tid = threadIdx.x;
  const bool local = P.n_frames <= kHistMax;
  if (local)
    for (int f = tid; f < P.n_frames; f += kThreads) hist[f] = 0;
  __syncthreads();
  const int i = blockIdx.x * kThreads + tid;
  int f = -1, rank = 0, pos = -1;
  tg_det d;
  if (i < count_of(P)) {
    d = P.dets[i];
    f = d.frame;
    if (f < 0 || f >= P.n_frames)
      f = -1;
    else if (local)
      rank = atomicAdd(&hist[f], 1);
    else
      pos = P.frame_begin[f] + atomicAdd(&P.cursor[static_cast<int64_t>(f) * P.cstride], 1);
  }
  if (local) {
    __syncthreads();
    for (int g = tid; g < P.n_frames; g += kThreads)  // this workgroup's range of frame g
      if (hist[g])
        hist[g] = P.frame_begin[g] + atomicAdd(&P.cursor[static_cast<int64_t>(g) * P.cstride], hist[g]);
    __syncthreads();
    if (f >= 0) pos = hist[f] + rank;
  }
  if (pos < 0) return;
  P.grouped[pos] = i;
  const float s = (d.box >= 0 && d.box < P.n_scores) ? P.scores[d.box] : __builtin_nanf("");
  P.rkey[pos] = rank_key(s, d.box);
  P.rbox[pos] = make_float4(d.x1, d.y1, d.x2, d.y2);
  P.rroi[pos] = d.roi;
}

// Area of a box (x1, y1, x2, y2 in .x .y .z .w), empty and inverted boxes 0.
__device__ __forceinline__ float box_area(float4 a) {
  return __fmul_rn(fmaxf(0.0f, __fsub_rn(a.z, a.x)), fmaxf(0.0f, __fsub_rn(a.w, a.y)));
}

// Whether boxes a and b, of areas area_a and area_b, overlap by more than thr of their
// union. The result does not depend on the order of a and b: the minima and maxima, the
// product and the sum are commutative, NaN operands included, and a difference of zeros
// differs in sign only, which no comparison sees.
__device__ __forceinline__ bool overlap_above(float4 a, float4 b, float area_a, float area_b,
                                              float thr) {
  const float w = fmaxf(0.0f, __fsub_rn(fminf(a.z, b.z), fmaxf(a.x, b.x)));
  const float h = fmaxf(0.0f, __fsub_rn(fminf(a.w, b.w), fmaxf(a.y, b.y)));
  const float inter = __fmul_rn(w, h);
  const float uni = __fsub_rn(__fadd_rn(area_a, area_b), inter);
  return inter > __fmul_rn(thr, uni);
}

// Whether box a suppresses box b when a is ranked above b.
__device__ __forceinline__ bool suppresses(float4 a, float4 b, float thr) {
  return overlap_above(a, b, box_area(a), box_area(b), thr);
}

// ---- the greedy of a frame, decided in rounds -----------------------------------------
//
// The greedy walk keeps a detection exactly when no detection ranked above it that
// suppresses it is kept (by induction over the ranking). So no sorted ranking is needed:
// given each detection's suppressors ranked above it, rounds decide the frame -- a
// detection is suppressed once one of them is kept, kept once all of them are suppressed.
// The best-ranked undecided detection of a round has only decided suppressors, so every
// round decides at least one: a frame of n detections needs at most n rounds (two to four
// in practice, where chains of boxes suppressing each other are short). Three launches:
//  index:   one workgroup per frame lists every box in a grid of up to kGridMax x kGridMax
//           cells over the frame's boxes (cells two to four times the mean box size) and
//           gives each detection its lists to search;
//  search:  kScanLanes lanes per detection, over all detections at once, find its
//           suppressors ranked above it in those lists (kPredSlots of them are kept; a
//           detection with more is searched again when it is decided);
//  resolve: one workgroup per frame (stepping through the frames when there are more than
//           kGridCap) runs the rounds on the suppressor lists.
// Search and resolve return at once when no frame was too large for the LDS path.
// Why the cells find every suppressor: with a threshold t >= 0, a suppresses b only if
// inter > t * union >= 0 (a union is never negative), so inter > 0 and both clipped widths
// are positive: min(x2a, x2b) > max(x1a, x1b) and likewise in y. The point
// (max(x1a, x1b), max(y1a, y1b)) then lies in both boxes, and since cell_of is
// non-decreasing its cell lies in the cell ranges of both: a and b share a cell. Every box
// is listed in the cells it touches; boxes with a NaN coordinate (where min and max ignore
// the NaN operand), boxes touching more than kCellsMax cells, and every box when t < 0, are
// "wide": listed once in a wide list that every detection searches, and themselves
// searching the whole frame. Boxes with x2 < x1 or y2 < y1 have no positive width with
// anything, so when t >= 0 they neither suppress nor are suppressed: kept from the start
// and listed nowhere.
// index and resolve: workgroups of 1024 threads (index) and 512 (resolve), or of
// kSmallFrame when the frames average at most kSmallFrame detections
constexpr int kSmallFrame = 256;
constexpr int kGridMax = 32;         // cells per axis
constexpr int kCellsMax = 4;         // cells a box may touch before it goes on the wide list
constexpr int kLists = kCellsMax + 1;
constexpr uint32_t kWide = 0xFFFFFFFFu;
constexpr uint32_t kEmpty = 0xFFFFFFFEu;
constexpr int32_t kUndecided = 0, kKept = 1, kSuppressed = 2;
constexpr int kPredSlots = 16;  // suppressors kept in place per detection
constexpr int kOvfPerDet = 16;  // overflow area for longer lists: kOvfPerDet n_max entries
constexpr int kScanLanes = 8;  // lanes per detection in the search
constexpr int kBatch = 8;      // list entries whose loads a lane issues together
constexpr int kSearchDets = kThreads / kScanLanes;  // detections per search workgroup
// Workgroups of the search and of the rounds: they step through detections and frames, so
// that inputs whose frames were all decided in LDS pay for a small launch only.
constexpr int kGridCap = 2048;

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

struct FrameLds {
  float ex0, sx, ey0, sy;
  int gx, gy, all_wide;
  float red[4][1024 / 64];
  float sum[2][1024 / 64];
  float top[2][1024 / 64];  // largest box width and height
  int off[kGridMax * kGridMax + 2];  // list starts (cells, then the wide list), then the end
  int cur[kGridMax * kGridMax + 1];  // list sizes while counting, then while filling
  int cnt[kGridMax * kGridMax + 1];  // list sizes
};
constexpr int kIdx = 4;  // detections per thread and step of the index, loads issued together

// ---- frames that fit one workgroup ------------------------------------------------------
//
// A frame of at most kSmallMax detections is decided by its index workgroup alone, in LDS:
// each thread holds one detection and tests every detection of the frame (four 16-byte
// boxes per step) for the suppressors ranked above it, a row of bits per detection; the
// rounds run on those rows (masks of kept and undecided detections rebuilt from ballots
// each round); the keep flags are written at once. The frame's detections are marked
// kEmpty, so the search passes them by, and the rounds skip the frame; when no frame is
// larger, both return at once.
template <int kN>
struct SmallFrameLds {
  float4 box[kN];
  uint64_t key[kN];
  int32_t roi[kN];
  float area[kN];
  uint32_t sup[kN][kN / 32 + 1];  // odd row stride: rows in distinct banks
  uint32_t kept[kN / 32], open[kN / 32];
};

// Frames of at most kSmallMax detections take the LDS path; the pair tests grow with the
// square of the frame, so larger frames spread their search over the whole grid instead
// (frames of 300-530 detections in one workgroup each: cam20_4k 55 -> 124 us).
constexpr int kSmallMax = 256;
constexpr int kSmallRows = 256;  // row bits (at least kSmallMax, a multiple of 64)
static_assert(kSmallMax <= kSmallRows && kSmallRows <= kSmallFrame, "one detection per thread");

template <int kN>
__device__ void small_frame(const MergeParams &P, int lo, int n, SmallFrameLds<kN> &S) {
  constexpr int kWords = kN / 32;
  const int i = threadIdx.x, lane = i & 63, wave = i >> 6;
  const bool mine = i < n;  // n <= kN <= the workgroup's threads
  float4 box = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  uint64_t key = ~uint64_t(0);
  int roi = 0;
  if (mine) {
    box = P.rbox[lo + i];
    key = P.rkey[lo + i];
    roi = P.rroi[lo + i];
  }
  if (i < kN) {
    S.box[i] = box;
    S.key[i] = key;
    S.roi[i] = roi;
    S.area[i] = box_area(box);
#pragma unroll
    for (int w = 0; w < kWords; ++w) S.sup[i][w] = 0;
  }
  __syncthreads();
  // Each pair once: thread i tests the detections 1 .. n/2 places after it, cyclically (at
  // n/2 exactly, for even n, only the first half of the threads), and the pair's bit goes
  // into the row of whichever of the two is ranked below.
  if (mine) {
    const float area = S.area[i];
    const int last = (n % 2 == 0 && i < n / 2) ? n / 2 : (n - 1) / 2;
    for (int d0 = 1; d0 <= last; d0 += 4) {
      float4 qb[4];
      uint64_t qk[4];
      int qr[4], qj[4];
      float qa[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = i + min(d0 + u, last);  // < 2n
        qj[u] = j >= n ? j - n : j;
        qb[u] = S.box[qj[u]];
        qk[u] = S.key[qj[u]];
        qr[u] = S.roi[qj[u]];
        qa[u] = S.area[qj[u]];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (d0 + u <= last && !(P.cross_only && qr[u] == roi) &&
            overlap_above(qb[u], box, qa[u], area, P.thr)) {
          const int j = qj[u];
          if (qk[u] < key)
            atomicOr(&S.sup[i][j >> 5], 1u << (j & 31));
          else if (key < qk[u])
            atomicOr(&S.sup[j][i >> 5], 1u << (i & 31));
        }
      }
    }
  }
  __syncthreads();
  int st = mine ? kUndecided : kSuppressed;
  bool overrun = false;
  for (int round = 0;; ++round) {
    const uint64_t kb = __ballot(st == kKept), ob = __ballot(st == kUndecided);
    if (lane == 0 && wave < kN / 64) {
      S.kept[2 * wave] = static_cast<uint32_t>(kb);
      S.kept[2 * wave + 1] = static_cast<uint32_t>(kb >> 32);
      S.open[2 * wave] = static_cast<uint32_t>(ob);
      S.open[2 * wave + 1] = static_cast<uint32_t>(ob >> 32);
    }
    if (!__syncthreads_or(st == kUndecided)) break;
    if (round > n) {  // each round decides the best-ranked undecided detection
      overrun = true;
      break;
    }
    if (st == kUndecided) {
      bool any_kept = false, any_open = false;
#pragma unroll
      for (int w = 0; w < kWords; ++w) {
        const uint32_t r = S.sup[i][w];
        any_kept = any_kept || (r & S.kept[w]) != 0;
        any_open = any_open || (r & S.open[w]) != 0;
      }
      st = any_kept ? kSuppressed : (any_open ? kUndecided : kKept);
    }
    __syncthreads();  // every row has been tested before the masks are rewritten
  }
  if (mine) {
    P.keep[P.grouped[lo + i]] = st == kKept ? 1 : 0;
    P.rcell[lo + i] = kEmpty;
  }
  if (overrun && i == 0) *P.status = 1;
}

template <int kFrameThreads>
__global__ __launch_bounds__(kFrameThreads) void index_kernel(const MergeParams P) {
  __shared__ union {
    FrameLds f;
    SmallFrameLds<kSmallRows> s;
  } U;
  FrameLds &S = U.f;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lo = P.frame_begin[blockIdx.x];
  const int n = P.frame_begin[blockIdx.x + 1] - lo;
  if (n <= 0) return;
  if (n <= kSmallMax) {
    small_frame<kSmallRows>(P, lo, n, U.s);
    return;
  }
  if (tid == 0) *P.big = 1;  // the search and the rounds have work
  const int64_t ent0 = static_cast<int64_t>(kCellsMax) * lo;  // the frame's list entries

  // the frame's extent and mean box size
  float xlo = __builtin_inff(), xhi = -__builtin_inff(), ylo = xlo, yhi = xhi;
  float sw = 0.0f, sh = 0.0f, mxw = 0.0f, mxh = 0.0f;
  for (int p0 = tid; p0 < n; p0 += kIdx * kFrameThreads) {
    float4 bb[kIdx];
#pragma unroll
    for (int u = 0; u < kIdx; ++u) {
      const int p = p0 + u * kFrameThreads;
      bb[u] = p < n ? P.rbox[lo + p] : make_float4(0.0f, 0.0f, -1.0f, -1.0f);
    }
#pragma unroll
    for (int u = 0; u < kIdx; ++u) {
      const float4 b = bb[u];
      if (__builtin_isfinite(b.x) && __builtin_isfinite(b.z) && b.z >= b.x) {
        xlo = fminf(xlo, b.x);
        xhi = fmaxf(xhi, b.z);
        sw += b.z - b.x;
        mxw = fmaxf(mxw, b.z - b.x);
      }
      if (__builtin_isfinite(b.y) && __builtin_isfinite(b.w) && b.w >= b.y) {
        ylo = fminf(ylo, b.y);
        yhi = fmaxf(yhi, b.w);
        sh += b.w - b.y;
        mxh = fmaxf(mxh, b.w - b.y);
      }
    }
  }
  xlo = wave_minf(xlo);
  xhi = wave_maxf(xhi);
  ylo = wave_minf(ylo);
  yhi = wave_maxf(yhi);
  sw = wave_sumf(sw);
  sh = wave_sumf(sh);
  mxw = wave_maxf(mxw);
  mxh = wave_maxf(mxh);
  if (lane == 0) {
    S.red[0][wave] = xlo;
    S.red[1][wave] = xhi;
    S.red[2][wave] = ylo;
    S.red[3][wave] = yhi;
    S.sum[0][wave] = sw;
    S.sum[1][wave] = sh;
    S.top[0][wave] = mxw;
    S.top[1][wave] = mxh;
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
      S.top[0][0] = fmaxf(S.top[0][0], S.top[0][w]);
      S.top[1][0] = fmaxf(S.top[1][0], S.top[1][w]);
    }
    // Cells twice the mean box size, or as large as the largest box when that is two to
    // four times the mean, so that no box touches more than 2 x 2 cells (boxes touching
    // more go on the wide list and search their whole frame: on cam20_4k, boxes of
    // 4-256 pixels with a mean of 110, 22 of 8,145 detections did, each searching 400-530
    // entries against a mean of 27, and set the search's time); larger outliers stay
    // wide. At most kGridMax cells per axis. Any finite scale keeps the index exact (only
    // its speed depends on it), so approximate reciprocals do; a degenerate extent just
    // puts everything in one cell.
    const float span_x = S.red[1][0] - S.red[0][0], span_y = S.red[3][0] - S.red[2][0];
    const float inv_n = __builtin_amdgcn_rcpf(static_cast<float>(n));
    const float mw = S.sum[0][0] * inv_n, mh = S.sum[1][0] * inv_n;
    const float tw = S.top[0][0], th = S.top[1][0];
    const float cw = (tw > 2.0f * mw && tw <= 4.0f * mw) ? tw : 2.0f * mw;
    const float ch = (th > 2.0f * mh && th <= 4.0f * mh) ? th : 2.0f * mh;
    const float fx = span_x * __builtin_amdgcn_rcpf(fmaxf(cw, 1e-30f));
    const float fy = span_y * __builtin_amdgcn_rcpf(fmaxf(ch, 1e-30f));
    S.gx = fx >= 2.0f ? static_cast<int>(fminf(fx, static_cast<float>(kGridMax))) : 1;
    S.gy = fy >= 2.0f ? static_cast<int>(fminf(fy, static_cast<float>(kGridMax))) : 1;
    const float scx = S.gx * __builtin_amdgcn_rcpf(span_x);
    const float scy = S.gy * __builtin_amdgcn_rcpf(span_y);
    S.ex0 = __builtin_isfinite(S.red[0][0]) ? S.red[0][0] : 0.0f;
    S.ey0 = __builtin_isfinite(S.red[2][0]) ? S.red[2][0] : 0.0f;
    S.sx = (__builtin_isfinite(scx) && scx > 0.0f) ? scx : 0.0f;
    S.sy = (__builtin_isfinite(scy) && scy > 0.0f) ? scy : 0.0f;
    S.all_wide = !(P.thr >= 0.0f);
  }
  for (int c = tid; c < kGridMax * kGridMax + 1; c += kFrameThreads) S.cur[c] = 0;
  __syncthreads();

  // each box's cell range; the lists' sizes
  const int gx = S.gx, gy = S.gy, n_cells = gx * gy;
  for (int p0 = tid; p0 < n; p0 += kIdx * kFrameThreads) {
    float4 bb[kIdx];
#pragma unroll
    for (int u = 0; u < kIdx; ++u) {
      const int p = p0 + u * kFrameThreads;
      bb[u] = p < n ? P.rbox[lo + p] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
#pragma unroll
    for (int u = 0; u < kIdx; ++u) {
      const int p = p0 + u * kFrameThreads;
      if (p >= n) continue;
      const float4 b = bb[u];
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
      P.rcell[lo + p] = cr;
      P.rstate[lo + p] = cr == kEmpty ? kKept : kUndecided;
        if (cr == kWide) {
        atomicAdd(&S.cur[n_cells], 1);
      } else if (cr != kEmpty) {
        for (int cy = (cr >> 16) & 0xFF; cy <= static_cast<int>(cr >> 24); ++cy)
          for (int cx = cr & 0xFF; cx <= static_cast<int>((cr >> 8) & 0xFF); ++cx)
            atomicAdd(&S.cur[cy * gx + cx], 1);
      }
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
      S.cnt[c] = k;
      S.cur[c] = 0;  // from here on: entries filled so far
      at += k;
    }
    if (lane == 63) S.off[n_cells + 1] = incl;
  }
  __syncthreads();
  // the entries (each listed box, its patch, ranking key and position) and each
  // detection's lists to search: absolute entry starts and sizes (a wide box: the frame's
  // first position and its size, searched as positions)
  for (int p0 = tid; p0 < n; p0 += kIdx * kFrameThreads) {
    uint32_t cc[kIdx];
    float4 bb[kIdx];
    uint64_t kk[kIdx];
    int rr[kIdx];
#pragma unroll
    for (int u = 0; u < kIdx; ++u) {
      const int p = p0 + u * kFrameThreads;
      const bool in = p < n;
      cc[u] = in ? P.rcell[lo + p] : kEmpty;
      bb[u] = in ? P.rbox[lo + p] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      kk[u] = in ? P.rkey[lo + p] : 0;
      rr[u] = in ? P.rroi[lo + p] : 0;
    }
#pragma unroll
    for (int u = 0; u < kIdx; ++u) {
      const int p = p0 + u * kFrameThreads;
      if (p >= n) continue;
      const uint32_t cr = cc[u];
      const int4 aux = make_int4(rr[u], static_cast<int>(static_cast<uint32_t>(kk[u])),
                                 static_cast<int>(static_cast<uint32_t>(kk[u] >> 32)), lo + p);
      int32_t *L = P.rlist + 2 * kLists * static_cast<int64_t>(lo + p);
      int k = 0;
      if (cr == kWide) {
        const int64_t at = ent0 + S.off[n_cells] + atomicAdd(&S.cur[n_cells], 1);
        P.ebox[at] = bb[u];
        P.eaux[at] = aux;
        L[0] = lo;
        L[kLists] = n;
        k = 1;
      } else if (cr != kEmpty) {
        for (int cy = (cr >> 16) & 0xFF; cy <= static_cast<int>(cr >> 24); ++cy)
          for (int cx = cr & 0xFF; cx <= static_cast<int>((cr >> 8) & 0xFF); ++cx, ++k) {
            const int c = cy * gx + cx;
            const int64_t at = ent0 + S.off[c] + atomicAdd(&S.cur[c], 1);
            P.ebox[at] = bb[u];
            P.eaux[at] = aux;
            L[k] = static_cast<int32_t>(ent0) + S.off[c];
            L[kLists + k] = S.cnt[c];
          }
        L[k] = static_cast<int32_t>(ent0) + S.off[n_cells];
        L[kLists + k] = S.cnt[n_cells];
        ++k;
      }
      for (; k < kLists; ++k) {
        L[k] = 0;
        L[kLists + k] = 0;
      }
    }
  }
}

// A detection's lists to search, in registers: starts st[k] and sizes ln[k].
struct Lists {
  int st[kLists], ln[kLists], total;
};
__device__ __forceinline__ Lists lists_of(const MergeParams &P, int a) {
  const int32_t *L = P.rlist + 2 * kLists * static_cast<int64_t>(a);
  Lists l;
  l.total = 0;
#pragma unroll
  for (int k = 0; k < kLists; ++k) {
    l.st[k] = L[k];
    l.ln[k] = L[kLists + k];
    l.total += l.ln[k];
  }
  return l;
}

// One step of a search: candidates t0, t0 + stride, ... (kBatch of them, below l.total) of
// a detection's lists, loaded together; returns a mask of those that are suppressors of
// it (box bp, key kp, patch rp) ranked above it (bit u: candidate t0 + u * stride), and
// their positions in q.
__device__ __forceinline__ uint32_t search_step(const MergeParams &P, const Lists &l, bool wide,
                                                int t0, int stride, float4 bp, uint64_t kp,
                                                int rp, int q[kBatch]) {
  float4 bq[kBatch];
  uint64_t kq[kBatch];
  int rq[kBatch];
  uint32_t hits = 0;
#pragma unroll
  for (int u = 0; u < kBatch; ++u) {
    int t = t0 + u * stride;
    q[u] = -1;
    if (t >= l.total) continue;
    if (wide) {
      q[u] = l.st[0] + t;
      bq[u] = P.rbox[q[u]];
      kq[u] = P.rkey[q[u]];
      rq[u] = P.rroi[q[u]];
    } else {
      int at = l.st[0], k = 0;
#pragma unroll
      for (int kk = 0; kk < kCellsMax; ++kk)  // which list: step over the earlier ones
        if (k == kk && t >= l.ln[kk]) {
          t -= l.ln[kk];
          k = kk + 1;
          at = l.st[kk + 1];
        }
      const int4 e = P.eaux[at + t];
      bq[u] = P.ebox[at + t];
      kq[u] = static_cast<uint64_t>(static_cast<uint32_t>(e.z)) << 32 | static_cast<uint32_t>(e.y);
      rq[u] = e.x;
      q[u] = e.w;
    }
  }
#pragma unroll
  for (int u = 0; u < kBatch; ++u)
    if (q[u] >= 0 && kq[u] < kp && !(P.cross_only && rq[u] == rp) && suppresses(bq[u], bp, P.thr))
      hits |= 1u << u;
  return hits;
}

// The suppressors ranked above each detection: kScanLanes consecutive lanes per detection,
// detections in frame-group order over the whole grid. The first kPredSlots go in place;
// a workgroup whose detections have more reserves room for their whole lists in the
// overflow area (one atomic for all of them) and searches those again to fill it; a
// list that does not fit is left to be searched in the rounds.
__device__ __forceinline__ void search_block(const MergeParams &P, int blk, int n_grouped) {
  __shared__ int s_np[kSearchDets], s_fill[kSearchDets], s_at[kSearchDets];
  const int tid = threadIdx.x, j = tid / kScanLanes, sub = tid % kScanLanes;
  const int a = blk * kSearchDets + j;
  const bool valid = a < n_grouped && P.rcell[a] != kEmpty;
  if (sub == 0) {
    s_np[j] = 0;
    s_fill[j] = 0;
  }
  __syncthreads();
  Lists l;
  float4 bp;
  uint64_t kp = 0;
  int rp = 0;
  bool wide = false;
  if (valid) {
    l = lists_of(P, a);
    bp = P.rbox[a];
    kp = P.rkey[a];
    rp = P.rroi[a];
    wide = P.rcell[a] == kWide;
    for (int t0 = sub; t0 < l.total; t0 += kScanLanes * kBatch) {
      int q[kBatch];
      for (uint32_t h = search_step(P, l, wide, t0, kScanLanes, bp, kp, rp, q); h; h &= h - 1) {
        const int slot = atomicAdd(&s_np[j], 1);
        if (slot < kPredSlots) P.rpred[kPredSlots * static_cast<int64_t>(a) + slot] = q[__builtin_ctz(h)];
      }
    }
  }
  __syncthreads();
  const int np = s_np[j];
  if (valid && sub == 0) P.rnpred[a] = np;
  if (tid == 0) {
    int64_t need = 0;
    for (int k = 0; k < kSearchDets; ++k)
      if (s_np[k] > kPredSlots) need += s_np[k];
    int64_t at = need > 0 ? static_cast<int64_t>(atomicAdd(P.ovf_used, static_cast<unsigned long long>(need)))
                          : 0;
    for (int k = 0; k < kSearchDets; ++k) {
      s_at[k] = -1;
      if (s_np[k] <= kPredSlots) continue;
      if (at + s_np[k] <= P.ovf_cap) s_at[k] = static_cast<int>(at);
      at += s_np[k];
    }
  }
  __syncthreads();
  if (!valid || np <= kPredSlots) return;
  const int at = s_at[j];
  if (sub == 0) P.rovf[a] = at;
  if (at < 0) return;
  for (int t0 = sub; t0 < l.total; t0 += kScanLanes * kBatch) {
    int q[kBatch];
    for (uint32_t h = search_step(P, l, wide, t0, kScanLanes, bp, kp, rp, q); h; h &= h - 1)
      P.ovf[at + atomicAdd(&s_fill[j], 1)] = q[__builtin_ctz(h)];
  }
}

__global__ __launch_bounds__(kThreads) void search_kernel(const MergeParams P) {
  static_assert(kSearchDets * kScanLanes == kThreads, "whole detections per workgroup");
  if (!*P.big) return;  // every frame was decided in its index workgroup
  const int n_grouped = P.frame_begin[P.n_frames];
  const int n_blocks = (n_grouped + kSearchDets - 1) / kSearchDets;
  for (int blk = blockIdx.x; blk < n_blocks; blk += gridDim.x) {
    __syncthreads();  // the previous block's readers of s_np, s_fill and s_at are done
    search_block(P, blk, n_grouped);
  }
}

// This round's decision for an undecided detection a with more suppressors than its
// kPredSlots and no room for them in the overflow area (many boxes crowded on one spot):
// its lists searched again, kBatch candidates at a time -- kSuppressed when one of its
// suppressors is kept, kUndecided when one is still undecided, else kKept.
__device__ __forceinline__ int32_t decide_searching(const MergeParams &P, int a) {
  const Lists l = lists_of(P, a);
  const bool wide = P.rcell[a] == kWide;
  const float4 bp = P.rbox[a];
  const uint64_t kp = P.rkey[a];
  const int rp = P.rroi[a];
  bool pending = false;
  for (int t0 = 0; t0 < l.total; t0 += kBatch) {
    int q[kBatch];
    const uint32_t h = search_step(P, l, wide, t0, 1, bp, kp, rp, q);
    int32_t s[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) s[u] = (h >> u & 1u) ? P.rstate[q[u]] : kSuppressed;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (s[u] == kKept) return kSuppressed;
      pending |= s[u] == kUndecided;
    }
  }
  return pending ? kUndecided : kKept;
}

// The rounds of one frame, then its keep flags.
// (frames of at most kSmallMax detections were decided by index_kernel)
template <int kResolveThreads>
__device__ __forceinline__ void resolve_frame(const MergeParams &P, int lo, int n) {
  const int tid = threadIdx.x;
  constexpr int kRes = 4;  // detections per thread and step, their loads issued together
  for (int round = 0;; ++round) {
    int pending = 0;
    for (int a0 = lo + tid; a0 < lo + n; a0 += kRes * kResolveThreads) {
      int32_t st[kRes], np[kRes];
#pragma unroll
      for (int u = 0; u < kRes; ++u) {
        const int a = a0 + u * kResolveThreads;
        st[u] = a < lo + n ? P.rstate[a] : kKept;
        np[u] = st[u] == kUndecided ? P.rnpred[a] : 0;
      }
      // the states of their first kFirst suppressors, loaded together; the rest one by one
      constexpr int kFirst = 4;
      int32_t ps[kRes][kFirst];
#pragma unroll
      for (int u = 0; u < kRes; ++u)
#pragma unroll
        for (int k = 0; k < kFirst; ++k)
          ps[u][k] = st[u] == kUndecided && k < np[u] && np[u] <= kPredSlots
                         ? P.rstate[P.rpred[kPredSlots * static_cast<int64_t>(a0 + u * kResolveThreads) + k]]
                         : kSuppressed;
      uint32_t search = 0;  // detections with more suppressors than their slots
#pragma unroll
      for (int u = 0; u < kRes; ++u) {
        if (st[u] != kUndecided) continue;
        const int a = a0 + u * kResolveThreads;
        // the list: in place, in the overflow area, or not kept (search again)
        const int32_t *list = P.rpred + kPredSlots * static_cast<int64_t>(a);
        if (np[u] > kPredSlots) {
          const int at = P.rovf[a];
          if (at < 0) {
            search |= 1u << u;
            continue;
          }
          list = P.ovf + at;
        }
        bool kept = false, und = false;
#pragma unroll
        for (int k = 0; k < kFirst; ++k) {
          kept |= ps[u][k] == kKept;
          und |= ps[u][k] == kUndecided;
        }
        for (int k0 = np[u] > kPredSlots ? 0 : kFirst; k0 < np[u] && !kept; k0 += kFirst) {
          int32_t sk[kFirst];
#pragma unroll
          for (int k = 0; k < kFirst; ++k)
            sk[k] = k0 + k < np[u] ? P.rstate[list[k0 + k]] : kSuppressed;
#pragma unroll
          for (int k = 0; k < kFirst; ++k) {
            kept |= sk[k] == kKept;
            und |= sk[k] == kUndecided;
          }
        }
        if (kept || !und)
          P.rstate[a] = kept ? kSuppressed : kKept;
        else
          pending = 1;
      }
      for (; search != 0; search &= search - 1) {
        const int a = a0 + __builtin_ctz(search) * kResolveThreads;
        const int32_t d = decide_searching(P, a);
        if (d != kUndecided)
          P.rstate[a] = d;
        else
          pending = 1;
      }
    }
    __syncthreads();  // this round's decisions are visible to the next
    if (!__syncthreads_or(pending)) break;
    if (round >= n) {  // cannot happen (each round decides one); reported, not spun on
      if (tid == 0) *P.status = 1;
      break;
    }
  }
  for (int a = lo + tid; a < lo + n; a += kResolveThreads)
    P.keep[P.grouped[a]] = P.rstate[a] == kKept ? 1 : 0;
}

template <int kResolveThreads>
__global__ __launch_bounds__(kResolveThreads) void resolve_kernel(const MergeParams P) {
  if (!*P.big) return;  // every frame was decided in its index workgroup
  for (int f = blockIdx.x; f < P.n_frames; f += gridDim.x) {
    const int lo = P.frame_begin[f];
    const int n = P.frame_begin[f + 1] - lo;
    if (n > kSmallMax) resolve_frame<kResolveThreads>(P, lo, n);
  }
}

// ---- small inputs: one workgroup, one launch ------------------------------------------
//
// Up to kTiny detections (n_max <= kTiny) are merged by one workgroup: each thread holds
// one detection, its suppressors (ranked above it in the same frame, with cross_only from
// another patch, and suppressing it) are a kTiny-bit row in LDS found by testing each
// pair once, the rounds above run on those rows (suppressed once a suppressor is kept, kept
// once all are suppressed), and a workgroup prefix sum writes the kept detections in input
// order. On inputs this small the launches of the general path, not their work, are the
// cost.
constexpr int kTiny = 512;
constexpr int kTinyWords = kTiny / 32;

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

// A detection as the pair tests read it: one 32-byte LDS record.
struct alignas(16) TinyDet {
  float4 box;
  uint64_t key;
  int32_t frame, roi;
};

__global__ __launch_bounds__(kTiny) void tiny_kernel(const MergeParams P) {
  __shared__ TinyDet s_det[kTiny];
  __shared__ float s_area[kTiny];
  __shared__ uint32_t s_sup[kTiny][kTinyWords + 1];  // odd row stride: rows in distinct banks
  __shared__ uint32_t s_kept[kTinyWords], s_open[kTinyWords];
  __shared__ int32_t s_wave[kTiny / 64];
  const int i = threadIdx.x, lane = i & 63, wave = i >> 6;
  const int n = count_of(P);
  tg_det d = {0, 0, -1, 0.0f, 0.0f, 0.0f, 0.0f};
  int f = -1;
  uint64_t key = ~uint64_t(0);
  if (i < n) {
    d = P.dets[i];
    if (d.frame >= 0 && d.frame < P.n_frames) f = d.frame;
    const float s = (d.box >= 0 && d.box < P.n_scores) ? P.scores[d.box] : __builtin_nanf("");
    key = rank_key(s, d.box);
  }
  const float4 box = make_float4(d.x1, d.y1, d.x2, d.y2);
  const float area = box_area(box);
  s_det[i] = TinyDet{box, key, f, d.roi};
  s_area[i] = area;
#pragma unroll
  for (int w = 0; w < kTinyWords; ++w) s_sup[i][w] = 0;
  __syncthreads();

  // the suppressor rows, each pair tested once (as in the LDS path of small frames: thread
  // i takes the detections 1 .. n/2 places after it, cyclically, four records per step,
  // and the bit goes into the row of whichever of the two is ranked below); a pair with a
  // detection outside the frames sets no bit, so such a thread skips its share
  if (f >= 0) {
    const int last = (n % 2 == 0 && i < n / 2) ? n / 2 : (n - 1) / 2;
    for (int d0 = 1; d0 <= last; d0 += 4) {
      TinyDet q[4];
      float qa[4];
      int qj[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = i + min(d0 + u, last);  // < 2n
        qj[u] = j >= n ? j - n : j;
        q[u] = s_det[qj[u]];
        qa[u] = s_area[qj[u]];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (d0 + u <= last && q[u].frame == f && !(P.cross_only && q[u].roi == d.roi) &&
            overlap_above(q[u].box, box, qa[u], area, P.thr)) {
          const int j = qj[u];
          if (q[u].key < key)
            atomicOr(&s_sup[i][j >> 5], 1u << (j & 31));
          else if (key < q[u].key)
            atomicOr(&s_sup[j][i >> 5], 1u << (i & 31));
        }
      }
    }
  }
  __syncthreads();

  // rounds; a detection outside the frames is dropped (never kept, never a suppressor)
  int st = f >= 0 ? kUndecided : kSuppressed;
  bool overrun = false;
  for (int round = 0;; ++round) {
    const uint64_t kept = __ballot(st == kKept), open = __ballot(st == kUndecided);
    if (lane == 0) {
      s_kept[2 * wave] = static_cast<uint32_t>(kept);
      s_kept[2 * wave + 1] = static_cast<uint32_t>(kept >> 32);
      s_open[2 * wave] = static_cast<uint32_t>(open);
      s_open[2 * wave + 1] = static_cast<uint32_t>(open >> 32);
    }
    if (!__syncthreads_or(st == kUndecided)) break;
    if (round > n) {  // each round decides the best-ranked undecided detection
      overrun = true;
      break;
    }
    if (st == kUndecided) {
      bool any_kept = false, any_open = false;
#pragma unroll
      for (int w = 0; w < kTinyWords; ++w) {
        const uint32_t r = s_sup[i][w];
        any_kept = any_kept || (r & s_kept[w]) != 0;
        any_open = any_open || (r & s_open[w]) != 0;
      }
      st = any_kept ? kSuppressed : (any_open ? kUndecided : kKept);
    }
    __syncthreads();  // every row has been tested before the masks are rewritten
  }

  const int k = i < n && st == kKept ? 1 : 0;
  if (i < n) P.keep[i] = k;
  const int incl = wave_inclusive_sum(k);
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kTiny / 64; ++w) {
    if (w < wave) before += s_wave[w];
    total += s_wave[w];
  }
  if (k) P.out[before + incl - 1] = d;
  if (i == 0) *P.n_kept = overrun ? TG_E_INTERNAL : total;
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
      if (blk == static_cast<int>(gridDim.x) - 1)
        *P.n_kept = failed || __hip_atomic_load(P.status, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT) != 0
                        ? TG_E_INTERNAL
                        : prefix + total;
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

int counter_stride(int32_t n_frames) { return n_frames <= kPaddedFramesMax ? kCounterStride : 1; }

// Workspace layout, in bytes from the (16-byte aligned) start.
struct Layout {
  size_t state, counts, cursor, begin, grouped;
  size_t rkey, rbox, rroi, rcell, rstate, rlist, rpred, rnpred, rovf, ovf, ebox, eaux, total;
};
size_t round16(size_t v) { return (v + 15) / 16 * 16; }
Layout layout(int32_t n_max, int32_t n_frames) {
  Layout L;
  const size_t n = static_cast<size_t>(n_max);
  // ticket and status word, the overflow area's cursor, one look-back word per compaction
  // workgroup
  L.state = 0;
  L.counts = sizeof(uint64_t) * (3 + static_cast<size_t>(compact_blocks(n_max)));
  const size_t slots = static_cast<size_t>(n_frames) * counter_stride(n_frames);
  L.cursor = L.counts + sizeof(int32_t) * slots;
  L.begin = L.cursor + sizeof(int32_t) * slots;
  L.grouped = L.begin + sizeof(int32_t) * (static_cast<size_t>(n_frames) + 1);
  L.rbox = round16(L.grouped + sizeof(int32_t) * n);
  L.rkey = L.rbox + sizeof(float4) * n;
  L.rroi = L.rkey + sizeof(uint64_t) * n;
  L.rcell = L.rroi + sizeof(int32_t) * n;
  L.rstate = L.rcell + sizeof(uint32_t) * n;
  L.rlist = L.rstate + sizeof(int32_t) * n;
  L.rpred = L.rlist + sizeof(int32_t) * 2 * (kCellsMax + 1) * n;
  L.rnpred = L.rpred + sizeof(int32_t) * kPredSlots * n;
  L.rovf = L.rnpred + sizeof(int32_t) * n;
  L.ovf = L.rovf + sizeof(int32_t) * n;
  L.ebox = round16(L.ovf + sizeof(int32_t) * kOvfPerDet * n);
  L.eaux = L.ebox + sizeof(float4) * kCellsMax * n;
  L.total = L.eaux + sizeof(int4) * kCellsMax * n;
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
  const bool tiny = a->n_max <= kTiny;

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
  P.status = reinterpret_cast<uint32_t *>(ws + L.state) + 1;
  P.ovf_used = reinterpret_cast<unsigned long long *>(ws + L.state) + 1;
  P.big = reinterpret_cast<uint32_t *>(ws + L.state) + 4;
  P.state = reinterpret_cast<uint64_t *>(ws + L.state) + 3;
  P.counts = reinterpret_cast<int32_t *>(ws + L.counts);
  P.cursor = reinterpret_cast<int32_t *>(ws + L.cursor);
  P.cstride = counter_stride(a->n_frames);
  P.frame_begin = reinterpret_cast<int32_t *>(ws + L.begin);
  P.grouped = reinterpret_cast<int32_t *>(ws + L.grouped);
  P.rkey = reinterpret_cast<uint64_t *>(ws + L.rkey);
  P.rbox = reinterpret_cast<float4 *>(ws + L.rbox);
  P.rroi = reinterpret_cast<int32_t *>(ws + L.rroi);
  P.rcell = reinterpret_cast<uint32_t *>(ws + L.rcell);
  P.rstate = reinterpret_cast<int32_t *>(ws + L.rstate);
  P.rlist = reinterpret_cast<int32_t *>(ws + L.rlist);
  P.rpred = reinterpret_cast<int32_t *>(ws + L.rpred);
  P.rnpred = reinterpret_cast<int32_t *>(ws + L.rnpred);
  P.rovf = reinterpret_cast<int32_t *>(ws + L.rovf);
  P.ovf = reinterpret_cast<int32_t *>(ws + L.ovf);
  P.ovf_cap = std::min<int64_t>(int64_t(kOvfPerDet) * a->n_max, 0x7FFFFFFF);
  P.ebox = reinterpret_cast<float4 *>(ws + L.ebox);
  P.eaux = reinterpret_cast<int4 *>(ws + L.eaux);

  if (tiny) {
    hipLaunchKernelGGL(tiny_kernel, dim3(1), dim3(kTiny), 0, s, P);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  const int32_t words64 = 3 + compact_blocks(a->n_max);
  const int32_t clear_n = a->n_frames > words64 ? a->n_frames : words64;
  const uint32_t per = static_cast<uint32_t>((a->n_max + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(clear_kernel, dim3((clear_n + kThreads - 1) / kThreads), dim3(kThreads), 0,
                     s, P, a->n_frames, words64);
  hipLaunchKernelGGL(count_kernel, dim3(per), dim3(kThreads), 0, s, P);
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kScanThreads), 0, s, P);
  hipLaunchKernelGGL(scatter_kernel, dim3(per), dim3(kThreads), 0, s, P);
  if (a->n_frames > 0) {
    const bool small = a->n_max <= int64_t(kSmallFrame) * a->n_frames;
    const dim3 frames(static_cast<uint32_t>(a->n_frames));
    if (small)
      hipLaunchKernelGGL(index_kernel<kSmallFrame>, frames, dim3(kSmallFrame), 0, s, P);
    else
      hipLaunchKernelGGL(index_kernel<1024>, frames, dim3(1024), 0, s, P);
    const int search_blocks = (a->n_max + kSearchDets - 1) / kSearchDets;
    hipLaunchKernelGGL(search_kernel, dim3(static_cast<uint32_t>(std::min(search_blocks, kGridCap))),
                       dim3(kThreads), 0, s, P);
    const dim3 resolve(static_cast<uint32_t>(std::min(a->n_frames, kGridCap)));
    if (small)
      hipLaunchKernelGGL(resolve_kernel<kSmallFrame>, resolve, dim3(kSmallFrame), 0, s, P);
    else
      hipLaunchKernelGGL(resolve_kernel<512>, resolve, dim3(512), 0, s, P);
  }
  hipLaunchKernelGGL(compact_kernel, dim3(static_cast<uint32_t>(compact_blocks(a->n_max))),
                     dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
