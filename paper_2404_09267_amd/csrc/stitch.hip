// tg_stitch: scatter uint8 RGB crops from resident frames into fp16 NCHW canvases.
//
// Tangram stitches unresized patches onto fixed-size canvases so that patches of any
// size batch as one fixed-shape detector input (Sec. I; Sec. III-C). Each canvas pixel
// is either the normalised byte of the one patch that covers it or the normalised pad
// byte.
//
// Design for gfx950 (wave64, HBM-bound, write-dominated: 6 bytes written per canvas
// pixel, 3 bytes read per covered pixel):
//  - Work units (stitch_units.h): runs of 6144 canvas pixels in raster order, one
//    256-thread workgroup each, launched in address order. A run is three whole 4 KB
//    pages of each fp16 plane, so the workgroups resident on the chip write a compact
//    window of whole pages that sweeps through the output; HBM absorbs writes fastest
//    that way. (Runs of 2048 pixels on 128 threads were 6-15 % slower: the per-unit plan
//    scan, list and barriers are then paid three times as often.)
//  - A workgroup makes one pass over its run: it prefills its LDS staging row with the
//    pad pixel (4 bytes per pixel: R, G, B and an unused byte, so that every patch edge
//    falls on a dword boundary and no two patches ever share a staged dword); lists the
//    canvas's patches meeting the run's rows (plan entries read through L2; a wave
//    ballot and a DPP prefix of each patch's piece count give list slots and piece
//    numbers together); each lane then loads a piece -- up to 16 pixels of one patch
//    row, on the run's 4-pixel grid -- as 13 dwords from the dword at or below its first
//    source byte, realigns them with v_alignbyte, spreads the 3-byte pixels over dwords
//    with v_perm and writes whole 4-pixel blocks (partial blocks at patch edges pixel by
//    pixel); finally each lane converts two 8-pixel groups into three 16-byte fp16
//    stores each, one per plane, nontemporal.
//  - The footprint is small (under 10 KB of LDS, under 64 VGPRs), so sixteen workgroups
//    are resident per CU and one workgroup's plan and frame round trips overlap the
//    others' stores. Every wave loads before it stores, so no wait for a load ever waits
//    on a store. Lane-dependent choices are selects, not branches.
//  - Normalisation: binary16((x - mean) / std) correctly rounded (the quotient in
//    double). The host searches fp32 constants (a, c) near (1/std, -mean/std) for which
//    binary16(fma(x, a, c)) equals that for all 256 bytes of a channel -- under both
//    single rounding and rounding through fp32 -- and the kernel then uses one
//    v_fma_mix per value. When no such pair exists the kernel reads a 3 x 256 binary16
//    table from LDS instead. Both are bit-exact.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "norm.h"
#include "stitch_units.h"
#include "tg.h"

namespace {

using tg_detail::StitchGeometry;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kRun = tg_detail::kStitchRun;  // pixels per unit
constexpr int kGroups = kRun / 8 / kThreads; // 8-pixel groups per thread
constexpr int kRecs = 40;                    // patches one list holds (more: further lists)
constexpr int kPx = 16;                      // pixels per piece (four 4-pixel blocks)
static_assert(kRun == 8 * kThreads * kGroups, "whole 8-pixel groups per thread");

struct StitchParams {
  const uint8_t *frames;
  int64_t frame_stride;
  int32_t n_frames, frame_w, frame_h, row_pitch;
  const tg_roi *rois;
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin;
  int32_t n_rois, canvas_first, canvas_w, canvas_h;
  int64_t plane;  // canvas_w * canvas_h
  int32_t runs, n_units;
  const int32_t *unit_order;  // device, or null for units in index order
  uint16_t *out;
  // Every 13-dword window a piece loads starts at or after load_base and ends at or
  // before load_end, so that all of its dwords hold frame bytes; pieces that would not
  // fit (only at the two ends of the frame buffer) are copied byte by byte.
  const uint8_t *load_base;
  const uint8_t *load_end;
  uint32_t pad_px;     // the pad pixel as staged: R | G << 8 | B << 16
  float fa[3], fc[3];  // per channel: binary16(fma(x, fa, fc)) is the normalised byte
  uint32_t lut[384];   // channel k, byte x -> binary16 bits at lut16[k * 256 + x]
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

// The run a workgroup stitches: canvas pixels [p0, p0 + np) of the plane in raster
// order, i.e. row Y0 from column X0, whole rows up to Y1, row Y1 up to column X1e.
// Staged pixel (run pixel) of canvas pixel (x, y): (y - Y0) * W + x - X0.
struct Run {
  int64_t p0;
  int32_t np, W;
  int32_t Y0, X0, Y1, X1e;
};

__device__ __forceinline__ uint32_t lane_rank(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Inclusive prefix sum over the 64 lanes of a wave: DPP row shifts inside each row of 16
// lanes, then row broadcasts across rows. Lanes whose DPP source is out of range (or
// whose row is masked off) add the `old` operand, 0.
__device__ __forceinline__ int wave_inclusive_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
  return v;
}

// Workgroup barrier that orders LDS only (no wait for outstanding global memory).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

struct Shared {
  // The listed patches: frame offset of channel 0 of the source pixel under canvas pixel
  // (0, 0) (so canvas pixel (x, y) reads src + y * row_pitch + 3 * x), the patch's
  // columns [x0, x1) and first row inside the run ya; its pieces by row class (see
  // Layout): the first-row pieces end at piece f_end, the middle rows' at m_end, pm per
  // middle row; st is the exclusive prefix of the patches' piece counts.
  int64_t src[kRecs];
  int32_t x0[kRecs], x1[kRecs], ya[kRecs];
  int32_t f_end[kRecs], m_end[kRecs], pm[kRecs];
  int32_t st[kRecs + 1];
  int32_t wave_cnt[kWaves], wave_pcs[kWaves];
  int32_t resume;
};

// The run pixels [u0, u1) of the row-y segment of columns [x0, x1): the part inside the
// run's window of that row (empty: u0 = u1 = 0); rowbase is the run pixel of column 0.
__device__ __forceinline__ void row_segment(const Run &R, int y, int x0, int x1, int &u0,
                                            int &u1, int64_t &rowbase) {
  const int a = y == R.Y0 ? R.X0 : 0, b = y == R.Y1 ? R.X1e : R.W;
  const int xa = max(x0, a), xb = min(x1, b);
  rowbase = static_cast<int64_t>(y - R.Y0) * R.W - R.X0;
  u0 = xa < xb ? static_cast<int>(rowbase + xa) : 0;
  u1 = xa < xb ? static_cast<int>(rowbase + xb) : 0;
}

// Pieces of a segment: kPx-pixel windows on the run's 4-pixel grid from the block
// holding u0.
__device__ __forceinline__ int pieces_of(int u0, int u1) {
  return u0 < u1 ? (u1 - (u0 & ~3) + kPx - 1) / kPx : 0;
}

// A listed patch's pieces, row class by row class: its first-row segment (when it meets
// the run's first row, whose window starts at X0), its middle rows (whole patch width;
// the same count for every such row, the most w pixels can need from any block offset,
// so a row's last piece may be empty) and its last-row segment (the run's last row,
// whose window ends at X1e).
struct Layout {
  int nf, pf, nm, pm, nl, pl;
};

__device__ __forceinline__ Layout layout_of(const Run &R, int x0, int x1, int ya, int yb) {
  Layout L;
  L.nf = ya == R.Y0;
  L.nl = yb == R.Y1 && R.Y1 > R.Y0;
  L.nm = yb - ya + 1 - L.nf - L.nl;
  int u0, u1;
  int64_t rb;
  row_segment(R, R.Y0, x0, x1, u0, u1, rb);
  L.pf = L.nf ? pieces_of(u0, u1) : 0;
  row_segment(R, R.Y1, x0, x1, u0, u1, rb);
  L.pl = L.nl ? pieces_of(u0, u1) : 0;
  L.pm = L.nm > 0 ? (x1 - x0 + 3 + kPx - 1) / kPx : 0;
  return L;
}

// Lists, in plan order, up to kRecs patches of `canvas` that have pieces in run R, from
// plan position `scan`; *total gets their piece count. Returns the position the next
// list starts from (k_hi when everything fit). Plan entries that are out of range or
// inconsistent are skipped, so a corrupt plan cannot lead to out-of-bounds accesses.
__device__ __forceinline__ int build_list(const StitchParams &P, Shared &S, int canvas,
                                          const Run &R, int scan, int k_hi, int &n_out,
                                          int &total_out) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int n = 0, total = 0;
  int resume = k_hi;
  while (scan < k_hi) {
    const int k = scan + tid;
    int pcs = 0;
    int64_t src = 0;
    int x0 = 0, x1 = 0, ya = 0, f_end = 0, m_end = 0, pm = 0;
    if (k < k_hi) {
      const int id = P.order[k];
      if (id >= 0 && id < P.n_rois) {
        const tg_roi r = P.rois[id];
        const tg_place pl = P.place[id];
        const bool sane = pl.canvas == canvas && r.w > 0 && r.h > 0 && pl.x >= 0 &&
                          pl.y >= 0 && pl.x <= P.canvas_w - r.w && pl.y <= P.canvas_h - r.h &&
                          r.frame >= 0 && r.frame < P.n_frames && r.x >= 0 && r.y >= 0 &&
                          r.x <= P.frame_w - r.w && r.y <= P.frame_h - r.h;
        const int yb = sane ? min(pl.y + r.h - 1, R.Y1) : -1;
        ya = max(pl.y, R.Y0);
        if (sane && ya <= yb) {
          x0 = pl.x;
          x1 = pl.x + r.w;
          const Layout L = layout_of(R, x0, x1, ya, yb);
          f_end = L.nf * L.pf;
          m_end = f_end + L.nm * L.pm;
          pm = L.pm;
          pcs = m_end + L.nl * L.pl;
          src = static_cast<int64_t>(r.frame) * P.frame_stride +
                static_cast<int64_t>(r.y - pl.y) * P.row_pitch + 3 * static_cast<int64_t>(r.x - pl.x);
        }
      }
    }
    const bool hit = pcs > 0;
    const uint64_t ballot = __ballot(hit);
    const int incl = wave_inclusive_sum(pcs);
    if (lane == 63) {
      S.wave_cnt[wave] = __popcll(ballot);
      S.wave_pcs[wave] = incl;
    }
    if (tid == 0) S.resume = k_hi;
    lds_barrier();
    int before = n, before_p = total, round_n = 0, round_p = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      const int c = S.wave_cnt[v], q = S.wave_pcs[v];
      if (v < wave) {
        before += c;
        before_p += q;
      }
      round_n += c;
      round_p += q;
    }
    if (hit) {
      const int slot = before + static_cast<int>(lane_rank(ballot));
      const int st = before_p + incl - pcs;
      if (slot < kRecs) {
        S.src[slot] = src;
        S.x0[slot] = x0;
        S.x1[slot] = x1;
        S.ya[slot] = ya;
        S.f_end[slot] = f_end;
        S.m_end[slot] = m_end;
        S.pm[slot] = pm;
        S.st[slot] = st;
      } else if (slot == kRecs) {
        S.resume = k;  // the first patch that did not fit starts the next list
        S.st[kRecs] = st;
      }
    }
    lds_barrier();
    if (n + round_n > kRecs) {
      n = kRecs;
      total = S.st[kRecs];
      resume = S.resume;
      break;
    }
    n += round_n;
    total += round_p;
    scan += kThreads;
    if (scan < k_hi) lds_barrier();  // wave sums and resume are rewritten by the next round
  }
  n_out = n;
  total_out = total;
  return resume;
}

// The record holding piece p: the largest a < n with st[a] <= p.
__device__ __forceinline__ int find_record(const Shared &S, int n, int p) {
  int a = 0;
  for (int step = n > 1 ? (1 << (31 - __clz(n - 1))) : 0; step > 0; step >>= 1) {
    const int m = a + step;
    if (m < n && S.st[m] <= p) a = m;
  }
  return a;
}

// Piece p: run pixels [u0, u1) (empty for an empty piece or a lane without one), inside
// the window [v, v + kPx) with v on the 4-pixel grid; the frame byte of channel 0 of run
// pixel v.
struct Piece {
  int v, u0, u1;
  const uint8_t *sp;
};

__device__ __forceinline__ Piece piece_of(const StitchParams &P, const Shared &S, const Run &R,
                                          int n, int total, int p) {
  Piece pc;
  pc.v = pc.u0 = pc.u1 = 0;
  pc.sp = P.frames;
  if (p >= total) return pc;
  const int a = find_record(S, n, p);
  const int j = p - S.st[a], f = S.f_end[a], me = S.m_end[a], pm = S.pm[a];
  const int ya = S.ya[a];
  // middle-row index: pm <= ceil((W + 3) / 16) and the quotient below W; the +0.5
  // keeps the float quotient inside the right integer interval
  const int jj = j - f;
  const int r = static_cast<int>((static_cast<float>(jj) + 0.5f) *
                                 __builtin_amdgcn_rcpf(static_cast<float>(max(pm, 1))));
  const bool first = j < f, mid = !first && j < me;
  const int y = first ? R.Y0 : (mid ? ya + (ya == R.Y0) + r : R.Y1);
  const int k = first ? j : (mid ? jj - r * pm : j - me);
  int u0, u1;
  int64_t rowbase;
  row_segment(R, y, S.x0[a], S.x1[a], u0, u1, rowbase);
  pc.v = (u0 & ~3) + kPx * k;
  pc.u0 = max(u0, pc.v);
  pc.u1 = min(u1, pc.v + kPx);
  // frame byte of run pixel u on row y: src + y * row_pitch + 3 * (u - rowbase)
  pc.sp = P.frames + S.src[a] + static_cast<int64_t>(y) * P.row_pitch + 3 * (pc.v - rowbase);
  return pc;
}

// What lanes without a piece, and windows near the frame buffer's ends, read instead.
__device__ uint32_t g_dummy[16];

// The 13 dwords from the one at or below piece pc's first source byte (3 * kPx bytes
// and the misalignment); unconditional, so that the batch of loads is straight-line.
__device__ __forceinline__ bool issue(const StitchParams &P, const Piece &pc, uint32_t w[13]) {
  const uint8_t *a0 = pc.sp - (reinterpret_cast<uintptr_t>(pc.sp) & 3u);
  const bool fast = pc.u0 < pc.u1 && a0 >= P.load_base && a0 + 52 <= P.load_end;
  const uint8_t *ad = fast ? a0 : reinterpret_cast<const uint8_t *>(g_dummy);
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const u32x4a4 v = *reinterpret_cast<const u32x4a4 *>(ad + 16 * c);
    w[4 * c] = v.x;
    w[4 * c + 1] = v.y;
    w[4 * c + 2] = v.z;
    w[4 * c + 3] = v.w;
  }
  w[12] = *reinterpret_cast<const uint32_t *>(ad + 48);
  return fast;
}

// Spreads the landed piece over staged pixels [u0, u1): whole 4-pixel blocks with one
// 16-byte write, pixels of blocks a patch edge cuts one by one. Writes that are not
// wanted go to the dummy slot, so the code has no lane-dependent branch.
__device__ __forceinline__ void land(const Piece &pc, const uint32_t w[13], uint32_t *stage,
                                     uint32_t *dummy) {
  const uint32_t sh = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(pc.sp) & 3u);
  uint32_t a[12];
#pragma unroll
  for (int i = 0; i < 12; ++i) a[i] = __builtin_amdgcn_alignbyte(w[i + 1], w[i], sh);
  // pixel i: bytes 3i .. 3i + 2 of a[] -> one dword (byte 3 unused)
  uint32_t px[kPx];
#pragma unroll
  for (int i = 0; i < kPx; ++i) {
    const int b = 3 * i, d = b >> 2, o = b & 3;
    // v_perm selects from {hi = first operand, lo = second}: selector bytes 0-3 name
    // bytes of lo, 4-7 bytes of hi
    const uint32_t sel = o == 0 ? 0x0C020100u : (o == 1 ? 0x0C030201u : (o == 2 ? 0x0C040302u : 0x0C050403u));
    px[i] = __builtin_amdgcn_perm(d + 1 < 12 ? a[d + 1] : 0u, a[d], sel);
  }
#pragma unroll
  for (int j = 0; j < kPx / 4; ++j) {
    const int b = pc.v + 4 * j;
    const bool whole = b >= pc.u0 && b + 4 <= pc.u1;
    *reinterpret_cast<u32x4 *>(whole ? stage + b : dummy) =
        u32x4{px[4 * j], px[4 * j + 1], px[4 * j + 2], px[4 * j + 3]};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = b + i;
      const bool one = !whole && u >= pc.u0 && u < pc.u1;
      *(one ? stage + u : dummy + 4 + i) = px[4 * j + i];
    }
  }
}

// A piece near the frame buffer's ends: byte by byte.
__device__ __forceinline__ void land_bytes(const Piece &pc, uint32_t *stage) {
  for (int u = pc.u0; u < pc.u1; ++u) {
    const uint8_t *b = pc.sp + 3 * (u - pc.v);
    stage[u] = uint32_t(b[0]) | (uint32_t(b[1]) << 8) | (uint32_t(b[2]) << 16);
  }
}

// binary16 of fma(x, a, c) for two bytes, packed low then high (v_fma_mix takes fp32
// operands and writes one half of the destination).
__device__ __forceinline__ uint32_t norm2(uint32_t x0, uint32_t x1, float a, float c) {
  uint32_t r;
  const float f0 = static_cast<float>(x0), f1 = static_cast<float>(x1);
  asm("v_fma_mixlo_f16 %0, %1, %2, %3" : "=v"(r) : "v"(f0), "v"(a), "v"(c));
  asm("v_fma_mixhi_f16 %0, %1, %2, %3" : "+v"(r) : "v"(f1), "v"(a), "v"(c));
  return r;
}

template <bool kVec, bool kLut>
__global__ __launch_bounds__(kThreads) void stitch_kernel(const StitchParams P) {
  __shared__ __attribute__((aligned(16))) uint32_t s_px[kRun + 8];  // + 8: dummy slot
  __shared__ Shared S;
  __shared__ uint16_t s_lut[kLut ? 3 * 256 : 2];

  const int tid = threadIdx.x;
  const int L = P.unit_order ? P.unit_order[blockIdx.x] : static_cast<int>(blockIdx.x);
  if (L < 0 || L >= P.n_units) return;  // not a unit: the whole workgroup leaves
  const int c_local = L / P.runs;
  const int canvas = P.canvas_first + c_local;
  Run R;
  R.W = P.canvas_w;
  R.p0 = static_cast<int64_t>(L - c_local * P.runs) * kRun;
  R.np = static_cast<int>(min(static_cast<int64_t>(kRun), P.plane - R.p0));
  const int64_t pe = R.p0 + R.np - 1;
  if (P.plane <= 0x7FFFFFFF) {  // 32-bit division when the plane allows it
    const uint32_t p0 = static_cast<uint32_t>(R.p0), p1 = static_cast<uint32_t>(pe);
    const uint32_t W = static_cast<uint32_t>(R.W);
    R.Y0 = static_cast<int>(p0 / W);
    R.Y1 = static_cast<int>(p1 / W);
  } else {
    R.Y0 = static_cast<int>(R.p0 / R.W);
    R.Y1 = static_cast<int>(pe / R.W);
  }
  R.X0 = static_cast<int>(R.p0 - static_cast<int64_t>(R.Y0) * R.W);
  R.X1e = static_cast<int>(pe - static_cast<int64_t>(R.Y1) * R.W) + 1;

  if (kLut)
    for (int i = tid; i < 384; i += kThreads) reinterpret_cast<uint32_t *>(s_lut)[i] = P.lut[i];
  // Pad prefill, ordered before the pieces land by the list's barriers and before the
  // conversion by the barrier after landing.
#pragma unroll
  for (int i = 0; i < kRun / 4 / kThreads; ++i)
    reinterpret_cast<u32x4 *>(s_px)[tid + i * kThreads] = u32x4{P.pad_px, P.pad_px, P.pad_px, P.pad_px};

  // The canvas's segment of `order`, clamped so a corrupt plan cannot index outside it.
  const int k_lo = min(max(P.canvas_begin[canvas], 0), P.n_rois);
  const int k_hi = min(max(P.canvas_begin[canvas + 1], k_lo), P.n_rois);
  int scan = k_lo;
  do {
    int n, total;
    const int next = build_list(P, S, canvas, R, scan, k_hi, n, total);
    for (int p = tid; p < total; p += kThreads) {
      const Piece pc = piece_of(P, S, R, n, total, p);
      uint32_t w[13];
      if (issue(P, pc, w))
        land(pc, w, s_px, s_px + kRun);
      else
        land_bytes(pc, s_px);
    }
    lds_barrier();  // staged pixels complete; the list may be rebuilt
    scan = next;
  } while (scan < k_hi);

  // 8-pixel groups tid, tid + kThreads: three 16-byte fp16 runs each, one per plane.
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    const int g = tid + gi * kThreads;
    const int g0 = 8 * g;
    if (g0 >= R.np) break;
    const u32x4 q0 = reinterpret_cast<const u32x4 *>(s_px)[2 * g];
    const u32x4 q1 = reinterpret_cast<const u32x4 *>(s_px)[2 * g + 1];
    const uint32_t e[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
    uint32_t o[3][4];
#pragma unroll
    for (int k = 0; k < 3; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t x0 = (e[2 * j] >> (8 * k)) & 0xFFu;
        const uint32_t x1 = (e[2 * j + 1] >> (8 * k)) & 0xFFu;
        if (kLut)
          o[k][j] = uint32_t(s_lut[k * 256 + x0]) | (uint32_t(s_lut[k * 256 + x1]) << 16);
        else
          o[k][j] = norm2(x0, x1, P.fa[k], P.fc[k]);
      }
    uint16_t *base = P.out + static_cast<int64_t>(c_local) * 3 * P.plane + R.p0 + g0;
    if (kVec) {  // plane % 8 == 0 and a 16-byte aligned output: whole groups only
#pragma unroll
      for (int k = 0; k < 3; ++k)
        __builtin_nontemporal_store(u32x4{o[k][0], o[k][1], o[k][2], o[k][3]},
                                    reinterpret_cast<u32x4 *>(base + k * P.plane));
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (g0 + i >= R.np) continue;
#pragma unroll
        for (int k = 0; k < 3; ++k)
          base[k * P.plane + i] = static_cast<uint16_t>(o[k][i >> 1] >> ((i & 1) * 16));
      }
    }
  }
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
  StitchGeometry g;
  if (!tg_detail::stitch_geometry(a->canvas_w, a->canvas_h, a->canvas_count, &g))
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
  P.plane = g.plane;
  P.runs = g.runs;
  P.n_units = g.n_units;
  P.unit_order = a->unit_order;
  P.out = a->out;
  // A piece's window of dwords must lie between the dword holding the first frame byte
  // and the end of the dword holding the last valid byte. With n_frames == 0 no patch is
  // sane and no load is formed.
  const int64_t valid_end = a->n_frames > 0 ? int64_t(a->n_frames - 1) * a->frame_stride +
                                                  int64_t(a->frame_h - 1) * a->row_pitch +
                                                  3 * int64_t(a->frame_w)
                                            : 0;
  const uintptr_t f0 = reinterpret_cast<uintptr_t>(a->frames);
  const uintptr_t begin4 = f0 & ~uintptr_t(3);
  const uintptr_t end4 = (f0 + uintptr_t(valid_end) + 3) & ~uintptr_t(3);
  P.load_base = a->frames - (f0 - begin4);
  P.load_end = a->frames + (int64_t(end4) - int64_t(f0));

  const tg_detail::NormConsts &nm = tg_detail::norm_consts(a->mean, a->std);
  std::memcpy(P.lut, nm.lut16, sizeof nm.lut16);
  for (int k = 0; k < 3; ++k) {
    P.fa[k] = nm.fa[k];
    P.fc[k] = nm.fc[k];
  }
  P.pad_px = uint32_t(a->pad[0]) | (uint32_t(a->pad[1]) << 8) | (uint32_t(a->pad[2]) << 16);

  const bool vec = (g.plane % 8 == 0) && (reinterpret_cast<uintptr_t>(a->out) % 16 == 0);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<uint32_t>(g.n_units));
  if (vec && nm.affine)
    hipLaunchKernelGGL((stitch_kernel<true, false>), grid, dim3(kThreads), 0, s, P);
  else if (vec)
    hipLaunchKernelGGL((stitch_kernel<true, true>), grid, dim3(kThreads), 0, s, P);
  else if (nm.affine)
    hipLaunchKernelGGL((stitch_kernel<false, false>), grid, dim3(kThreads), 0, s, P);
  else
    hipLaunchKernelGGL((stitch_kernel<false, true>), grid, dim3(kThreads), 0, s, P);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
