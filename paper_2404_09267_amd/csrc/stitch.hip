// tg_stitch: scatter uint8 RGB crops from resident frames into fp16 NCHW canvases.
//
// Tangram stitches unresized patches onto fixed-size canvases so that patches of any
// size batch as one fixed-shape detector input (Sec. I; Sec. III-C). Each canvas
// pixel is either the normalised byte of the one patch that covers it or the
// normalised pad byte.
//
// Design for gfx950 (wave64, 160 KB LDS per CU, 8 XCDs, HBM-bound, write-dominated):
//  - One 256-thread workgroup per TILE_H x TILE_W canvas tile. Workgroup ids are
//    remapped so that each XCD (which takes every eighth workgroup) works through a
//    contiguous range of tiles: horizontally adjacent tiles read the two halves of the
//    same source lines, which then meet in one L2.
//  - The tile's pixels are staged in LDS as u8 RGB rows, prefilled with the pad bytes.
//  - The workgroup lists its canvas's patches that meet the tile with a wave ballot and
//    an mbcnt prefix (kRecs at a time), and enumerates every (patch, tile row, 16-byte
//    LDS chunk) triple with a block-wide prefix sum. Each lane copies its chunks: one
//    16-byte + one 4-byte load of aligned dwords per chunk, realigned with v_alignbyte,
//    several chunks in flight per lane; chunks at a patch's left or right edge write
//    only their own bytes.
//  - Every lane then converts 8-pixel groups from LDS: each byte goes through a 3 x 256
//    binary16 table in LDS (RGB interleaved in, planar out) and the group leaves as
//    three 16-byte nontemporal stores, one per plane.
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
constexpr int kWaves = kThreads / 64;
constexpr int kTileW = 256;            // pixels
constexpr int kTileH = 32;
constexpr int kRowBytes = 3 * kTileW;  // one staged tile row, u8 RGB
constexpr int kChunksPerRow = kRowBytes / 16;
constexpr int kGroupsX = kTileW / 8;
constexpr int kGroups = kGroupsX * kTileH;
constexpr int kRecs = 256;             // patches listed per round
constexpr int kInFlight = 4;           // chunks whose loads a lane issues before writing
constexpr int kXcds = 8;

struct StitchParams {
  const uint8_t *frames;
  int64_t frame_stride;
  int32_t n_frames, frame_w, frame_h, row_pitch;
  const tg_roi *rois;
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin;
  int32_t n_rois, canvas_first, canvas_count, canvas_w, canvas_h;
  int32_t tiles_x, tiles_per_canvas, n_tiles;
  uint16_t *out;
  // 20-byte source windows start on a dword at or after window_base and at or before
  // window_limit, so that every dword they touch holds a frame byte. Chunks whose
  // window would not fit (only at the two ends of the frame buffer) copy byte by byte.
  const uint8_t *window_base;
  const uint8_t *window_limit;
  uint32_t pad_dw[3];  // the pad bytes repeated over 12 bytes (4 pixels), as 3 dwords
  uint32_t lut[384];   // channel k, byte x -> half bits at lut16[k * 256 + x]
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

__device__ __forceinline__ uint32_t lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d, 64);
    if (lane >= d) v += u;
  }
  return v;
}

// One group of 8 pixels: the three planes' eight halves packed two per dword.
struct Group {
  uint32_t p[3][4];
};

template <bool kVec>
__device__ __forceinline__ void store_group(const StitchParams &P, int c_local, int Y, int X0,
                                            const Group &g) {
  const int64_t plane = static_cast<int64_t>(P.canvas_h) * P.canvas_w;
  uint16_t *base = P.out + (static_cast<int64_t>(c_local) * 3) * plane +
                   static_cast<int64_t>(Y) * P.canvas_w + X0;
  if (kVec) {  // canvas_w % 8 == 0 and a 16-byte aligned output: whole groups only
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      u32x4 v = {g.p[k][0], g.p[k][1], g.p[k][2], g.p[k][3]};
      __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(base + k * plane));
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (X0 + i >= P.canvas_w) continue;
#pragma unroll
    for (int k = 0; k < 3; ++k)
      base[k * plane + i] = static_cast<uint16_t>(g.p[k][i >> 1] >> ((i & 1) * 16));
  }
}

struct Shared {
  uint16_t lut[3 * 256];
  int64_t src[kRecs];        // frame offset of the patch's bytes for tile pixel (0, 0)
  int32_t start[kRecs + 1];  // exclusive prefix of the records' chunk counts
  int16_t rect[kRecs][4];    // tile-local byte range [b0, b1) of a row; rows [y0, y1)
  int32_t wave_sum[kWaves];
  int32_t resume;
};

template <bool kVec>
__global__ __launch_bounds__(kThreads) void stitch_kernel(const StitchParams P) {
  __shared__ __attribute__((aligned(16))) uint8_t s_px[kTileH * kRowBytes];
  __shared__ Shared S;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // XCD-aware order: the workgroups of XCD x (ids x, x + 8, ...) take consecutive tiles.
  const int w = blockIdx.x;
  const int per = P.n_tiles / kXcds, extra = P.n_tiles % kXcds;
  const int xcd = w % kXcds;
  const int L = xcd * per + min(xcd, extra) + w / kXcds;
  const int c_local = L / P.tiles_per_canvas;
  const int t_in = L % P.tiles_per_canvas;
  const int canvas = P.canvas_first + c_local;
  const int X_t = (t_in % P.tiles_x) * kTileW, Y_t = (t_in / P.tiles_x) * kTileH;
  const int tw = min(kTileW, P.canvas_w - X_t);
  const int th = min(kTileH, P.canvas_h - Y_t);

  for (int i = tid; i < 384; i += kThreads) reinterpret_cast<uint32_t *>(S.lut)[i] = P.lut[i];
  // Pad prefill: 16-byte chunk j of a row starts at dword 4j, whose phase in the 3-dword
  // pad pattern is (4j) mod 3 = j mod 3.
  for (int i = tid; i < kTileH * kChunksPerRow; i += kThreads) {
    const int ph = (i % kChunksPerRow) % 3;
    const u32x4 v = {P.pad_dw[ph], P.pad_dw[(ph + 1) % 3], P.pad_dw[(ph + 2) % 3], P.pad_dw[ph]};
    *reinterpret_cast<u32x4 *>(s_px + 16 * i) = v;
  }

  // Clamp the canvas's segment of `order` so a corrupt plan cannot index outside it.
  const int k_lo = min(max(P.canvas_begin[canvas], 0), P.n_rois);
  const int k_hi = min(max(P.canvas_begin[canvas + 1], k_lo), P.n_rois);

  for (int scan = k_lo; scan < k_hi;) {
    // ---- list up to kRecs patches that meet the tile, in plan order -----------------
    int n = 0;
    int resume = k_hi;
    while (scan < k_hi) {
      const int k = scan + tid;
      bool hit = false;
      int64_t src = 0;
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
            // canvas pixel (X, Y) of this patch, channel k, is frame byte
            // src + (Y - Y_t) * row_pitch + 3 * (X - X_t) + k
            src = static_cast<int64_t>(r.frame) * P.frame_stride +
                  static_cast<int64_t>(r.y - pl.y + Y_t) * P.row_pitch +
                  3 * static_cast<int64_t>(r.x - pl.x + X_t);
          }
        }
      }
      const uint64_t ballot = __ballot(hit);
      if (lane == 0) S.wave_sum[wave] = __popcll(ballot);
      if (tid == 0) S.resume = k_hi;
      __syncthreads();
      int before = n, total = 0;
#pragma unroll
      for (int v = 0; v < kWaves; ++v) {
        if (v < wave) before += S.wave_sum[v];
        total += S.wave_sum[v];
      }
      if (hit) {
        const int slot = before + static_cast<int>(lane_rank(ballot));
        if (slot < kRecs) {
          S.src[slot] = src;
          S.rect[slot][0] = static_cast<int16_t>(3 * x0);
          S.rect[slot][1] = static_cast<int16_t>(3 * x1);
          S.rect[slot][2] = static_cast<int16_t>(y0);
          S.rect[slot][3] = static_cast<int16_t>(y1);
        } else if (slot == kRecs) {
          S.resume = k;  // first patch that did not fit: the next round starts here
        }
      }
      __syncthreads();
      const bool full = n + total > kRecs;
      resume = S.resume;
      __syncthreads();  // wave_sum / resume are rewritten by the next round
      if (full) {
        n = kRecs;
        break;
      }
      n += total;
      scan += kThreads;
    }
    scan = resume;  // k_hi unless the list filled up

    // ---- chunk counts and their block-wide exclusive prefix -------------------------
    int cnt = 0;
    if (tid < n) {
      const int b0 = S.rect[tid][0], b1 = S.rect[tid][1];
      cnt = (S.rect[tid][3] - S.rect[tid][2]) * (((b1 - 1) >> 4) - (b0 >> 4) + 1);
    }
    const int incl = wave_inclusive_sum(cnt);
    if (lane == 63) S.wave_sum[wave] = incl;
    __syncthreads();
    int offset = 0, total = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      if (v < wave) offset += S.wave_sum[v];
      total += S.wave_sum[v];
    }
    if (tid < n) S.start[tid] = offset + incl - cnt;
    if (tid == 0) S.start[n] = total;
    __syncthreads();

    // ---- copy the patches' rows into the staged tile ---------------------------------
    for (int base = 0; base < total; base += kThreads * kInFlight) {
      uint32_t win[kInFlight][5];
      int dst[kInFlight], lo[kInFlight], hi[kInFlight];
      const uint8_t *sp[kInFlight];
      bool fast[kInFlight];
#pragma unroll
      for (int j = 0; j < kInFlight; ++j) {
        const int i = base + j * kThreads + tid;
        dst[j] = -1;
        lo[j] = hi[j] = 0;
        sp[j] = P.frames;
        fast[j] = false;
        if (i < total) {
          // the record whose chunk range holds i: the largest r with start[r] <= i
          int a = 0, b = n - 1;
          while (a < b) {
            const int m = (a + b + 1) >> 1;
            if (S.start[m] <= i)
              a = m;
            else
              b = m - 1;
          }
          const int b0 = S.rect[a][0], b1 = S.rect[a][1];
          const int q0 = b0 >> 4, nq = ((b1 - 1) >> 4) - q0 + 1;
          const int local = i - S.start[a];
          const int row = S.rect[a][2] + local / nq;
          const int q = q0 + local % nq;
          dst[j] = row * kRowBytes + 16 * q;
          lo[j] = max(b0 - 16 * q, 0);
          hi[j] = min(b1 - 16 * q, 16);
          // staged byte 16q + t of this row comes from frame byte sp + t
          sp[j] = P.frames + S.src[a] + static_cast<int64_t>(row) * P.row_pitch + 16 * q;
          const uint8_t *a0 = sp[j] - (reinterpret_cast<uintptr_t>(sp[j]) & 3u);
          fast[j] = a0 >= P.window_base && a0 <= P.window_limit;
          if (fast[j]) {
            const u32x4a4 v = *reinterpret_cast<const u32x4a4 *>(a0);
            win[j][0] = v.x;
            win[j][1] = v.y;
            win[j][2] = v.z;
            win[j][3] = v.w;
            win[j][4] = *reinterpret_cast<const uint32_t *>(a0 + 16);
          }
        }
      }
#pragma unroll
      for (int j = 0; j < kInFlight; ++j) {
        if (dst[j] < 0) continue;
        uint8_t *d = s_px + dst[j];
        if (fast[j]) {
          const uint32_t sh = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(sp[j]) & 3u);
          uint32_t e[4];
#pragma unroll
          for (int t = 0; t < 4; ++t)
            e[t] = __builtin_amdgcn_alignbyte(win[j][t + 1], win[j][t], sh);
          if (lo[j] == 0 && hi[j] == 16) {
            *reinterpret_cast<u32x4 *>(d) = u32x4{e[0], e[1], e[2], e[3]};
          } else {
#pragma unroll
            for (int t = 0; t < 16; ++t)
              if (t >= lo[j] && t < hi[j]) d[t] = static_cast<uint8_t>(e[t >> 2] >> (8 * (t & 3)));
          }
        } else {
          for (int t = lo[j]; t < hi[j]; ++t) d[t] = sp[j][t];
        }
      }
    }
    __syncthreads();  // records are rewritten by the next round; staging is complete
  }
  __syncthreads();  // the prefill is complete when the canvas has no patch at all

  // ---- convert and store: RGB interleaved in LDS -> three fp16 planes -----------------
#pragma unroll 2
  for (int g = tid; g < kGroups; g += kThreads) {
    const int r = g / kGroupsX, X0l = (g % kGroupsX) * 8;
    if (r >= th || X0l >= tw) continue;
    const u32x2 *p = reinterpret_cast<const u32x2 *>(s_px + r * kRowBytes + 3 * X0l);
    const u32x2 v0 = p[0], v1 = p[1], v2 = p[2];
    const uint32_t e[6] = {v0.x, v0.y, v1.x, v1.y, v2.x, v2.y};
    Group G;
#pragma unroll
    for (int k = 0; k < 3; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int b0 = 3 * (2 * j) + k, b1 = 3 * (2 * j + 1) + k;
        const uint32_t x0 = (e[b0 >> 2] >> (8 * (b0 & 3))) & 0xFFu;
        const uint32_t x1 = (e[b1 >> 2] >> (8 * (b1 & 3))) & 0xFFu;
        G.p[k][j] = uint32_t(S.lut[k * 256 + x0]) | (uint32_t(S.lut[k * 256 + x1]) << 16);
      }
    store_group<kVec>(P, c_local, Y_t + r, X_t + X0l, G);
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
  P.canvas_count = a->canvas_count;
  P.canvas_w = a->canvas_w;
  P.canvas_h = a->canvas_h;
  P.tiles_x = (a->canvas_w + kTileW - 1) / kTileW;
  const int64_t tiles_pc = int64_t(P.tiles_x) * ((a->canvas_h + kTileH - 1) / kTileH);
  const int64_t n_tiles = tiles_pc * a->canvas_count;
  if (n_tiles > 0x7FFFFFFF) return TG_E_INVAL;
  P.tiles_per_canvas = static_cast<int32_t>(tiles_pc);
  P.n_tiles = static_cast<int32_t>(n_tiles);
  P.out = a->out;
  // A 20-byte window may start on any dword from the one holding the first frame byte
  // up to the one 20 bytes before the end of the dword holding the last valid byte.
  // With n_frames == 0 no patch is sane and no window is formed.
  const int64_t valid_end = a->n_frames > 0 ? int64_t(a->n_frames - 1) * a->frame_stride +
                                                  int64_t(a->frame_h - 1) * a->row_pitch +
                                                  3 * int64_t(a->frame_w)
                                            : 0;
  const uintptr_t f0 = reinterpret_cast<uintptr_t>(a->frames);
  const uintptr_t begin4 = f0 & ~uintptr_t(3);
  const uintptr_t end4 = (f0 + uintptr_t(valid_end) + 3) & ~uintptr_t(3);
  P.window_base = a->frames - (f0 - begin4);
  // below window_base (no fast window at all) when the buffer holds under 20 bytes
  P.window_limit = a->frames + (int64_t(end4) - 20 - int64_t(f0));
  uint16_t lut16[768];
  for (int k = 0; k < 3; ++k)
    for (int x = 0; x < 256; ++x)
      lut16[k * 256 + x] = half_bits_rne((double(x) - double(a->mean[k])) / double(a->std[k]));
  std::memcpy(P.lut, lut16, sizeof lut16);
  uint8_t pat[12];
  for (int i = 0; i < 12; ++i) pat[i] = a->pad[i % 3];
  std::memcpy(P.pad_dw, pat, sizeof pat);

  const bool vec = (a->canvas_w % 8 == 0) && (reinterpret_cast<uintptr_t>(a->out) % 16 == 0);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<uint32_t>(n_tiles));
  if (vec)
    hipLaunchKernelGGL(stitch_kernel<true>, grid, dim3(kThreads), 0, s, P);
  else
    hipLaunchKernelGGL(stitch_kernel<false>, grid, dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
