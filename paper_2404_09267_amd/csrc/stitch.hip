// tg_stitch: scatter uint8 RGB crops from resident frames into fp16 NCHW canvases.
//
// Tangram stitches unresized patches onto fixed-size canvases so that patches of any
// size batch as one fixed-shape detector input (Sec. I; Sec. III-C). Each canvas
// pixel is either the normalised byte of the one patch that covers it or the
// normalised pad byte.
//
// Design for gfx950 (wave64, 160 KB LDS per CU, HBM-bound, write-dominated):
//  - One 256-thread workgroup per TILE_H x TILE_W canvas tile; grid = tiles x canvases.
//  - The workgroup lists the patches of its canvas that touch the tile with a wave
//    ballot and an mbcnt prefix (at most kSlots per pass; more take extra passes), and
//    paints a one-byte-per-pixel owner map of the tile in LDS, one thread per
//    (patch, row) pair.
//  - Each thread owns four 8-pixel groups of the tile. A group's pixels come from at
//    most two patches or the pad: it reads the 24 source bytes of each patch as one
//    16-byte and one 12-byte load of 4-byte-aligned dwords, realigned in registers,
//    picks each pixel's byte (the pad byte for pad pixels), turns every byte into
//    binary16 through a 3 x 256 table in LDS and writes three 16-byte nontemporal
//    stores.
//  - Groups with three or more patches, or whose window would leave the frame buffer,
//    go to a per-wave queue in LDS that the same wave finishes one pixel per lane.
//  - The table holds the correctly rounded binary16 of (x - mean_k) / std_k for each
//    byte x, computed on the host in double; the kernel is therefore bit-exact for
//    patch pixels and pad alike.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "tg.h"

namespace {

constexpr int kThreads = 256;
constexpr int kTileW = 256;   // pixels; 32 groups of 8
constexpr int kTileH = 32;
constexpr int kGroupsX = kTileW / 8;
constexpr int kGroups = kGroupsX * kTileH;
constexpr int kSlots = 253;   // owner ids 1..253; 0 = not covered yet; 255 = written earlier
constexpr uint8_t kDone = 255;

struct StitchParams {
  const uint8_t *frames;
  int64_t frame_stride;
  int32_t n_frames, frame_w, frame_h, row_pitch;
  const tg_roi *rois;
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin;
  int32_t n_rois, canvas_first, canvas_w, canvas_h;
  int32_t tiles_x;
  uint16_t *out;
  // Highest address at which a 28-byte source window may start: the last dword holding
  // a valid frame byte ends 28 bytes later. Windows are clamped to it so that no load
  // touches a dword without a valid byte.
  const uint8_t *window_limit;
  const uint8_t *window_base;  // first dword holding a frame byte
  int32_t window_ok;
  uint32_t pad2[3];    // pad value of each channel, replicated in both halves
  uint32_t pad_byte[3];
  uint32_t lut[384];   // channel k, byte x -> half bits at lut16[k * 256 + x]
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x3a4 __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

__device__ __forceinline__ uint32_t lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Paint owner bytes [a, b) of one tile row with `id`: single bytes up to 16-byte
// alignment, then 16-byte stores, then the tail.
__device__ __forceinline__ void paint(uint8_t *row, int a, int b, uint32_t id) {
  const uint32_t v = id * 0x01010101u;
  while (a < b && (a & 15)) row[a++] = static_cast<uint8_t>(id);
  for (; a + 16 <= b; a += 16) *reinterpret_cast<u32x4 *>(row + a) = u32x4{v, v, v, v};
  while (a < b) row[a++] = static_cast<uint8_t>(id);
}

// The 24 source bytes of eight pixels starting at `src`, realigned into e[0..5]. They
// lie in the 7 dwords from the one holding the first byte, read as one 16-byte and one
// 12-byte load. Near the end of the frame buffer the window slides back one dword (only
// possible when the start is aligned). A window whose dwords would not all hold frame
// bytes is refused (returns false); windows of pixels that all lie in one patch are
// never refused.
__device__ __forceinline__ bool load_window(const StitchParams &P, const uint8_t *src,
                                            uint32_t e[6]) {
  const uint32_t sh = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(src) & 3u);
  const uint8_t *a0 = src - sh;  // pointer arithmetic keeps the global address space
  const bool slid = a0 > P.window_limit;
  if (a0 < P.window_base || (slid && (sh != 0 || a0 > P.window_limit + 4))) return false;
  const uint32_t *q = reinterpret_cast<const uint32_t *>(slid ? a0 - 4 : a0);
  const u32x4a4 v0 = *reinterpret_cast<const u32x4a4 *>(q);
  const u32x3a4 v1 = *reinterpret_cast<const u32x3a4 *>(q + 4);
  const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, 0u};
  // Blend with a mask rather than `slid ? w[j + 1] : w[j]`, which the compiler turns
  // into an indexed private array (scratch memory).
  const uint32_t m = slid ? ~0u : 0u;
  uint32_t d[7];
#pragma unroll
  for (int j = 0; j < 7; ++j) d[j] = (w[j] & ~m) | (w[j + 1] & m);
#pragma unroll
  for (int j = 0; j < 6; ++j) e[j] = __builtin_amdgcn_alignbyte(d[j + 1], d[j], sh);
  return true;
}

__device__ __forceinline__ uint32_t byte_of(const uint32_t e[6], int b) {
  return (e[b >> 2] >> (8 * (b & 3))) & 0xFFu;
}

// One group of 8 pixels: the three planes' eight halves packed two per dword.
struct Group {
  uint32_t p[3][4];
};

template <bool kVec>
__device__ __forceinline__ void store_group(const StitchParams &P, int c_local, int Y, int X0,
                                            const Group &g, uint32_t mask) {
  const int64_t plane = static_cast<int64_t>(P.canvas_h) * P.canvas_w;
  uint16_t *base = P.out + (static_cast<int64_t>(c_local) * 3) * plane +
                   static_cast<int64_t>(Y) * P.canvas_w + X0;
  if (kVec && mask == 0xFFu) {
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      u32x4 v = {g.p[k][0], g.p[k][1], g.p[k][2], g.p[k][3]};
      __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(base + k * plane));
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (!(mask & (1u << i)) || X0 + i >= P.canvas_w) continue;
#pragma unroll
    for (int k = 0; k < 3; ++k)
      base[k * plane + i] = static_cast<uint16_t>(g.p[k][i >> 1] >> ((i & 1) * 16));
  }
}

template <bool kVec>
__global__ __launch_bounds__(kThreads) void stitch_kernel(const StitchParams P) {
  __shared__ uint16_t s_lut[3 * 256];
  __shared__ __attribute__((aligned(16))) uint8_t s_owner[kTileH * kTileW];
  __shared__ int64_t s_base[kSlots];
  __shared__ int16_t s_rect[kSlots][4];  // tile-local x0, y0, x1, y1 (half-open)
  __shared__ int32_t s_wave_hits[kThreads / 64];
  __shared__ int32_t s_resume;
  __shared__ int16_t s_wq[kThreads / 64][kGroups / (kThreads / 64)];  // per-wave queues

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c_local = blockIdx.y;
  const int canvas = P.canvas_first + c_local;
  const int tx = blockIdx.x % P.tiles_x;
  const int ty = blockIdx.x / P.tiles_x;
  const int X_t = tx * kTileW, Y_t = ty * kTileH;
  const int tw = min(kTileW, P.canvas_w - X_t);
  const int th = min(kTileH, P.canvas_h - Y_t);

  for (int i = tid; i < 384; i += kThreads) reinterpret_cast<uint32_t *>(s_lut)[i] = P.lut[i];

  // Clamp the canvas's segment of `order` so a corrupt plan cannot index outside it.
  const int k_lo = min(max(P.canvas_begin[canvas], 0), P.n_rois);
  const int k_hi = min(max(P.canvas_begin[canvas + 1], k_lo), P.n_rois);

  int scan = k_lo;
  bool first_pass = true;
  for (;;) {
    // ---- list the patches touching this tile (up to kSlots) -------------------
    int n_slots = 0;
    bool overflow = false;
    while (scan < k_hi && !overflow) {
      const int k = scan + tid;
      bool hit = false;
      int64_t base = 0;
      int x0 = 0, y0 = 0, x1 = 0, y1 = 0;
      if (k < k_hi) {
        const int id = P.order[k];
        if (id >= 0 && id < P.n_rois) {
          const tg_roi r = P.rois[id];
          const tg_place pl = P.place[id];
          const bool sane = pl.canvas == canvas && r.w > 0 && r.h > 0 && pl.x >= 0 &&
                            pl.y >= 0 && pl.x <= P.canvas_w - r.w &&
                            pl.y <= P.canvas_h - r.h && r.frame >= 0 &&
                            r.frame < P.n_frames && r.x >= 0 && r.y >= 0 &&
                            r.x <= P.frame_w - r.w && r.y <= P.frame_h - r.h;
          if (sane) {
            x0 = max(pl.x, X_t) - X_t;
            y0 = max(pl.y, Y_t) - Y_t;
            x1 = min(pl.x + r.w, X_t + tw) - X_t;
            y1 = min(pl.y + r.h, Y_t + th) - Y_t;
            hit = x0 < x1 && y0 < y1;
            base = static_cast<int64_t>(r.frame) * P.frame_stride +
                   static_cast<int64_t>(r.y - pl.y) * P.row_pitch +
                   3 * static_cast<int64_t>(r.x - pl.x);
          }
        }
      }
      const uint64_t ballot = __ballot(hit);
      if (lane == 0) s_wave_hits[wave] = __popcll(ballot);
      if (tid == 0) s_resume = -1;
      __syncthreads();
      int before = n_slots, total = 0;
      for (int w = 0; w < kThreads / 64; ++w) {
        if (w < wave) before += s_wave_hits[w];
        total += s_wave_hits[w];
      }
      if (hit) {
        const int slot = before + static_cast<int>(lane_rank(ballot));
        if (slot < kSlots) {
          s_base[slot] = base;
          s_rect[slot][0] = static_cast<int16_t>(x0);
          s_rect[slot][1] = static_cast<int16_t>(y0);
          s_rect[slot][2] = static_cast<int16_t>(x1);
          s_rect[slot][3] = static_cast<int16_t>(y1);
        } else if (slot == kSlots) {
          s_resume = k;  // first patch that did not fit: the next pass starts here
        }
      }
      __syncthreads();
      if (n_slots + total > kSlots) {
        overflow = true;
        n_slots = kSlots;
        scan = s_resume;
      } else {
        n_slots += total;
        scan += kThreads;
      }
      __syncthreads();  // s_wave_hits / s_resume are rewritten by the next round
    }
    const bool final_pass = scan >= k_hi;

    // ---- owner map: 0 = pad so far, 1..kSlots = slot + 1, kDone = written -------
    uint32_t *own32 = reinterpret_cast<uint32_t *>(s_owner);
    for (int i = tid; i < kTileH * kTileW / 4; i += kThreads) {
      uint32_t v = 0;
      if (!first_pass) {  // mark every byte painted in an earlier pass as done
        const uint32_t o = own32[i];
#pragma unroll
        for (int b = 0; b < 4; ++b)
          if ((o >> (8 * b)) & 0xFFu) v |= uint32_t(kDone) << (8 * b);
      }
      own32[i] = v;
    }
    __syncthreads();
    for (int t = tid; t < n_slots * kTileH; t += kThreads) {
      const int sl = t / kTileH, y = t % kTileH;
      if (y < s_rect[sl][1] || y >= s_rect[sl][3]) continue;
      paint(s_owner + y * kTileW, s_rect[sl][0], s_rect[sl][2], static_cast<uint32_t>(sl + 1));
    }
    __syncthreads();

    // ---- write the tile ------------------------------------------------------------
    // Each lane takes its 8-pixel groups in turn. A group's pixels come from at most two
    // patches (A, B) or the pad value: one source window per patch, then per pixel the
    // byte of its owner (the pad byte for pad pixels: the table maps it to the pad
    // value). Groups with three or more patches, or whose window would leave the frame
    // buffer, go to the wave's own queue and are finished by the same wave one pixel
    // per lane.
    int n_queued = 0;
#pragma unroll 1
    for (int g = tid; g < kGroups; g += kThreads) {
      const int r = g / kGroupsX;
      const int X0l = (g % kGroupsX) * 8;
      // Groups outside the canvas read as all done; every lane still reaches the ballot
      // below, which keeps the queue count wave-uniform.
      const bool inside = r < th && X0l < tw;
      const uint64_t own =
          inside ? *reinterpret_cast<const uint64_t *>(s_owner + r * kTileW + X0l) : ~uint64_t(0);
      const int Y = Y_t + r, X0 = X_t + X0l;
      uint32_t wmask = 0, A = 0, B = 0, from_b = 0, is_pad = 0;
      bool queue = false;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t o = static_cast<uint32_t>(own >> (8 * i)) & 0xFFu;
        if (o == kDone) continue;
        if (o == 0) {
          if (final_pass) {
            wmask |= 1u << i;
            is_pad |= 1u << i;
          }
          continue;
        }
        wmask |= 1u << i;
        if (A == 0 || o == A) {
          A = o;
        } else if (B == 0 || o == B) {
          B = o;
          from_b |= 1u << i;
        } else {
          queue = true;
        }
      }
      if (!kVec && X0 + 8 > P.canvas_w) wmask &= (1u << (P.canvas_w - X0)) - 1u;
      uint32_t eA[6] = {0, 0, 0, 0, 0, 0}, eB[6] = {0, 0, 0, 0, 0, 0};
      const int64_t row_off = static_cast<int64_t>(Y) * P.row_pitch + 3 * X0;
      if (!queue && A) queue = !load_window(P, P.frames + s_base[A - 1] + row_off, eA);
      if (!queue && B) queue = !load_window(P, P.frames + s_base[B - 1] + row_off, eB);
      if (!P.window_ok && (A || B)) queue = true;
      const uint64_t qb = __ballot(queue && wmask);
      if (queue && wmask)
        s_wq[wave][n_queued + static_cast<int>(lane_rank(qb))] = static_cast<int16_t>(g);
      n_queued += __popcll(qb);
      if (queue || !wmask) continue;
      Group G;
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        const uint32_t pk = P.pad_byte[k];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          uint32_t x[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int i = 2 * j + h, b = 3 * i + k;
            const uint32_t xa = byte_of(eA, b), xb = byte_of(eB, b);
            x[h] = (is_pad >> i) & 1u ? pk : ((from_b >> i) & 1u ? xb : xa);
          }
          G.p[k][j] = uint32_t(s_lut[k * 256 + x[0]]) | (uint32_t(s_lut[k * 256 + x[1]]) << 16);
        }
      }
      store_group<kVec>(P, c_local, Y, X0, G, wmask);
    }
    // The wave's queue: one pixel per lane, eight consecutive lanes per group, so the
    // 2-byte stores of a group form one contiguous 16-byte run per plane.
    if (n_queued) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int64_t plane = static_cast<int64_t>(P.canvas_h) * P.canvas_w;
      uint16_t *obase = P.out + static_cast<int64_t>(c_local) * 3 * plane;
      for (int u = lane; u < n_queued * 8; u += 64) {
        const int g = s_wq[wave][u >> 3], i = u & 7;
        const int r = g / kGroupsX, x = (g % kGroupsX) * 8 + i;
        if (x >= tw) continue;
        const uint32_t o = s_owner[r * kTileW + x];
        if (o == kDone || (o == 0 && !final_pass)) continue;
        const int Y = Y_t + r, X = X_t + x;
        uint32_t h[3];
        if (o == 0) {
#pragma unroll
          for (int k = 0; k < 3; ++k) h[k] = P.pad2[k] & 0xFFFFu;
        } else {
          const uint8_t *px = P.frames + s_base[o - 1] + static_cast<int64_t>(Y) * P.row_pitch +
                              3 * static_cast<int64_t>(X);
#pragma unroll
          for (int k = 0; k < 3; ++k) h[k] = s_lut[k * 256 + px[k]];
        }
        uint16_t *dst = obase + static_cast<int64_t>(Y) * P.canvas_w + X;
#pragma unroll
        for (int k = 0; k < 3; ++k) dst[k * plane] = static_cast<uint16_t>(h[k]);
      }
    }
    if (final_pass) break;
    first_pass = false;
    __syncthreads();  // the next pass rewrites slots and the owner map
  }
}

// Correctly rounded binary16 of a double (round to nearest, ties to even), from the
// double's fields: 1 sign, 11 exponent (bias 1023), 52 fraction bits.
uint16_t half_bits_rne(double v) {
  uint64_t b;
  std::memcpy(&b, &v, sizeof b);
  const uint16_t sign = static_cast<uint16_t>((b >> 48) & 0x8000u);
  const int biased = static_cast<int>((b >> 52) & 0x7FFu);
  const uint64_t frac = b & ((uint64_t(1) << 52) - 1);
  if (biased == 0x7FF) return sign | (frac ? 0x7E00u : 0x7C00u);
  if (biased == 0) return sign;  // below 2^-1022: far under half's smallest subnormal
  const int e = biased - 1023;
  if (e > 15) return sign | 0x7C00u;
  const uint64_t sig = frac | (uint64_t(1) << 52);  // value = sig * 2^(e - 52)
  // Normal halves keep 10 fraction bits (drop 42); subnormals count units of 2^-24.
  const int drop = e >= -14 ? 42 : 28 - e;
  if (drop > 53) return sign;  // below 2^-25: rounds to zero
  uint64_t q = sig >> drop;
  const uint64_t rest = sig & ((uint64_t(1) << drop) - 1);
  const uint64_t halfway = uint64_t(1) << (drop - 1);
  if (rest > halfway || (rest == halfway && (q & 1))) ++q;
  // Normal: exponent field (e + 15) plus q - 1024; a carry to q == 2048 bumps the
  // exponent (and at e == 15 lands exactly on infinity). Subnormal: q itself, where
  // q == 1024 is the smallest normal's encoding.
  const uint32_t bits = e >= -14 ? (uint32_t(e + 15) << 10) + uint32_t(q - 1024) : uint32_t(q);
  return static_cast<uint16_t>(sign | bits);
}

}  // namespace

extern "C" int tg_stitch(const tg_stitch_args *a, void *stream) {
  if (!a) return TG_E_INVAL;
  if (a->canvas_count < 0 || a->canvas_first < 0 || a->n_canvases < 0 || a->n_rois < 0)
    return TG_E_INVAL;
  if (a->canvas_w < 1 || a->canvas_h < 1 || a->frame_w < 1 || a->frame_h < 1 ||
      a->n_frames < 0 || a->row_pitch < 3 * int64_t(a->frame_w) ||
      a->frame_stride < int64_t(a->frame_h) * a->row_pitch)
    return TG_E_INVAL;
  for (int k = 0; k < 3; ++k)
    if (!std::isfinite(a->mean[k]) || !std::isfinite(a->std[k]) || !(a->std[k] > 0.0f))
      return TG_E_INVAL;
  if (int64_t(a->canvas_first) + a->canvas_count > a->n_canvases) return TG_E_RANGE;
  if (a->canvas_count == 0) return TG_OK;
  if (!a->frames || !a->rois || !a->place || !a->order || !a->canvas_begin || !a->out)
    return TG_E_INVAL;

  StitchParams P;
  P.frames = a->frames;
  P.frame_stride = a->frame_stride;
  P.n_frames = a->n_frames;
  P.frame_w = a->frame_w;
  P.frame_h = a->frame_h;
  P.row_pitch = a->row_pitch;
  P.rois = a->rois;
  P.place = a->place;
  P.order = a->order;
  P.canvas_begin = a->canvas_begin;
  P.n_rois = a->n_rois;
  P.canvas_first = a->canvas_first;
  P.canvas_w = a->canvas_w;
  P.canvas_h = a->canvas_h;
  P.tiles_x = (a->canvas_w + kTileW - 1) / kTileW;
  P.out = a->out;
  // One past the last valid frame byte, rounded up to a dword; windows start at most
  // 28 bytes before it. Frame buffers too small for one window take the per-pixel path.
  const int64_t valid_end = int64_t(a->n_frames - 1) * a->frame_stride +
                            int64_t(a->frame_h - 1) * a->row_pitch + 3 * int64_t(a->frame_w);
  const uintptr_t end4 = (reinterpret_cast<uintptr_t>(a->frames) + uintptr_t(valid_end) + 3) &
                         ~uintptr_t(3);
  const uintptr_t begin4 = reinterpret_cast<uintptr_t>(a->frames) & ~uintptr_t(3);
  P.window_limit = a->frames + (int64_t(end4 - 28) - int64_t(reinterpret_cast<uintptr_t>(a->frames)));
  P.window_base = a->frames - (reinterpret_cast<uintptr_t>(a->frames) - begin4);
  P.window_ok = a->n_frames > 0 && end4 >= begin4 + 32;
  uint16_t lut16[768];
  for (int k = 0; k < 3; ++k)
    for (int x = 0; x < 256; ++x)
      lut16[k * 256 + x] = half_bits_rne((double(x) - double(a->mean[k])) / double(a->std[k]));
  std::memcpy(P.lut, lut16, sizeof lut16);
  for (int k = 0; k < 3; ++k) {
    const uint32_t pv = lut16[k * 256 + a->pad[k]];
    P.pad2[k] = pv | (pv << 16);
    P.pad_byte[k] = a->pad[k];
  }
  const int tiles_y = (a->canvas_h + kTileH - 1) / kTileH;
  const int64_t tiles = int64_t(P.tiles_x) * tiles_y;
  if (tiles > 0x7FFFFFFF || a->canvas_count > 65535) return TG_E_INVAL;
  const dim3 grid(static_cast<uint32_t>(tiles), static_cast<uint32_t>(a->canvas_count));
  const bool vec = (a->canvas_w % 8 == 0) && (reinterpret_cast<uintptr_t>(a->out) % 16 == 0);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (vec)
    hipLaunchKernelGGL(stitch_kernel<true>, grid, dim3(kThreads), 0, s, P);
  else
    hipLaunchKernelGGL(stitch_kernel<false>, grid, dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
