// tg_stitch: scatter uint8 RGB crops from resident frames into fp16 NCHW canvases.
//
// Tangram stitches unresized patches onto fixed-size canvases so that patches of any
// size batch as one fixed-shape detector input (Sec. I; Sec. III-C). Each canvas pixel
// is either the normalised byte of the one patch that covers it or the normalised pad
// byte.
//
// Design for gfx950 (wave64, 160 KB LDS per CU, HBM-bound, write-dominated):
//  - Work units (stitch_units.h): a band of canvas rows across a tile of up to 1280
//    columns -- a whole canvas row for the canvases used here. One 256-thread
//    workgroup per unit; units are launched in the order the caller's schedule gives
//    (heaviest first, from tg_stitch_schedule) so that the last units to run are short.
//  - The workgroup lists the patches meeting its band once (wave ballot + mbcnt
//    compaction into LDS) and walks the band in steps of 3 rows through two LDS
//    staging buffers of u8 RGB rows, prefilled with the pad bytes.
//  - Waves are specialised. Two loader waves only read: each lane takes a "piece" of up
//    to 7 consecutive 16-byte chunks of one patch row, reads it as one straight-line
//    batch of 16-byte loads from the dword-aligned address below it and realigns it with
//    v_alignbyte into the staged row. The loads of step s + 1 are issued before step s
//    lands, and every wait is an explicit vmcnt the compiler can count. Two converter
//    waves only write: each lane turns 8 staged pixels into three 16-byte fp16 planes
//    (one nontemporal store each) and restores the pad bytes it consumed. A wave that
//    stores never waits for loads, and a wave that loads never waits for stores; the
//    two meet at LDS-only barriers, one per step.
//  - Normalisation: binary16((x - mean) / std) correctly rounded (the quotient in
//    double). The host searches fp32 constants (a, c) near (1/std, -mean/std) for which
//    binary16(fma(x, a, c)) equals that for all 256 bytes of a channel -- under both
//    single rounding and rounding through fp32 -- and the converters then use one
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
constexpr int kLoadWaves = 2;
constexpr int kLoadThreads = 64 * kLoadWaves;
constexpr int kConvThreads = kThreads - kLoadThreads;
constexpr int kTileW = tg_detail::kStitchTileW;      // widest staged row, pixels
constexpr int kRowBytes = 3 * kTileW;                // one staged row, u8 RGB
constexpr int kStepRows = tg_detail::kStitchStepRows;
constexpr int kBufBytes = kStepRows * kRowBytes;     // one staging buffer
constexpr int kRecs = 192;                           // patches listed per band (more: slow path)
constexpr int kPiece = 7;                            // 16-byte chunks per piece
static_assert(kRowBytes % 48 == 0, "pad prefill works in 48-byte chunk triples");
static_assert(kBufBytes < (1 << 15), "piece destination field");

struct StitchParams {
  const uint8_t *frames;
  int64_t frame_stride;
  int32_t n_frames, frame_w, frame_h, row_pitch;
  const tg_roi *rois;
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin;
  int32_t n_rois, canvas_first, canvas_count, canvas_w, canvas_h;
  int32_t tiles_x, bands_y, band_steps, n_units;
  const int32_t *unit_order;  // device, or null for units in index order
  uint16_t *out;
  // Every 16-byte load of a piece starts at or after load_base and at or before
  // load_limit, so that all of its dwords hold frame bytes; pieces that would not fit
  // (only at the two ends of the frame buffer) are copied byte by byte.
  const uint8_t *load_base;
  const uint8_t *load_limit;
  uint32_t pad_dw[3];  // the pad bytes repeated over 12 bytes (4 pixels), as 3 dwords
  float fa[3], fc[3];  // per channel: binary16(fma(x, fa, fc)) is the normalised byte
  uint32_t lut[384];   // channel k, byte x -> binary16 bits at lut16[k * 256 + x]
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

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

// Workgroup barrier that orders LDS only: outstanding global loads and stores are not
// waited for (converters keep their stores, loaders their next step's loads, in flight).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Makes this wave's LDS writes visible to its own later LDS reads from other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Waits until at most N vector memory operations of this wave are outstanding (loads
// complete in issue order). s_waitcnt fields: vmcnt bits [3:0] and [15:14], expcnt
// [6:4], lgkmcnt [11:8]; expcnt and lgkmcnt are left at their maxima (no wait).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

struct Shared {
  // The band's patches: frame offset of the patch byte that would land on staged row 0,
  // staged byte 0; the staged byte range [b0, b1) and band row range [y0, y1) it covers.
  int64_t src[kRecs];
  int16_t rect[kRecs][4];
  // Exclusive piece-count prefixes: loader wave w uses tables 2w and 2w + 1 for the two
  // steps it has in flight; on the slow path wave w uses table w.
  int32_t start[2 * kLoadWaves > kWaves ? 2 * kLoadWaves : kWaves][kRecs + 1];
  int32_t wave_sum[kWaves];
  int32_t resume;
};

// Lists, in plan order, up to kRecs patches of `canvas` that meet columns [X_t, X_t + tw)
// and rows [Y0, Y0 + rows), from plan position `scan`. Returns the position the next
// list starts from (k_hi when everything fit). Plan entries that are out of range or
// inconsistent are skipped, so a corrupt plan cannot lead to out-of-bounds accesses.
__device__ __forceinline__ int build_list(const StitchParams &P, Shared &S, int canvas, int X_t,
                                          int tw, int Y0, int rows, int scan, int k_hi,
                                          int &n_out) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
                          pl.y >= 0 && pl.x <= P.canvas_w - r.w && pl.y <= P.canvas_h - r.h &&
                          r.frame >= 0 && r.frame < P.n_frames && r.x >= 0 && r.y >= 0 &&
                          r.x <= P.frame_w - r.w && r.y <= P.frame_h - r.h;
        if (sane) {
          x0 = max(pl.x, X_t) - X_t;
          y0 = max(pl.y, Y0) - Y0;
          x1 = min(pl.x + r.w, X_t + tw) - X_t;
          y1 = min(pl.y + r.h, Y0 + rows) - Y0;
          hit = x0 < x1 && y0 < y1;
          // canvas pixel (X, Y) of this patch, channel k, is frame byte
          // src + (Y - Y0) * row_pitch + 3 * (X - X_t) + k
          src = static_cast<int64_t>(r.frame) * P.frame_stride +
                static_cast<int64_t>(r.y - pl.y + Y0) * P.row_pitch +
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
        S.resume = k;  // the first patch that did not fit starts the next list
      }
    }
    __syncthreads();
    const bool full = n + total > kRecs;
    resume = S.resume;
    __syncthreads();  // wave_sum and resume are rewritten by the next round
    if (full) {
      n = kRecs;
      break;
    }
    n += total;
    scan += kThreads;
  }
  n_out = n;
  return resume;
}

__device__ __forceinline__ int pieces_per_row(int b0, int b1) {
  const int nq = ((b1 - 1) >> 4) - (b0 >> 4) + 1;  // 16-byte staged chunks the row spans
  return (nq + kPiece - 1) / kPiece;
}

// This wave's exclusive prefix (into st) of the piece counts of records [0, n) over
// band rows [r0, r1); returns the total.
__device__ __forceinline__ int prefix_pieces(const Shared &S, int32_t *st, int n, int r0,
                                             int r1) {
  const int lane = threadIdx.x & 63;
  int carry = 0;
  for (int b = 0; b < n; b += 64) {
    const int r = b + lane;
    int cnt = 0;
    if (r < n) {
      const int y0 = max(static_cast<int>(S.rect[r][2]), r0);
      const int y1 = min(static_cast<int>(S.rect[r][3]), r1);
      if (y0 < y1) cnt = (y1 - y0) * pieces_per_row(S.rect[r][0], S.rect[r][1]);
    }
    const int incl = wave_inclusive_sum(cnt);
    if (r < n) st[r] = carry + incl - cnt;
    carry += __builtin_amdgcn_readlane(incl, 63);
  }
  if (lane == 0) st[n] = carry;
  wave_lds_sync();
  return carry;
}

// The record holding piece p: the largest a < n with st[a] <= p.
__device__ __forceinline__ int find_record(const int32_t *st, int n, int p) {
  int a = 0;
  for (int step = n > 1 ? (1 << (31 - __clz(n - 1))) : 0; step > 0; step >>= 1) {
    const int m = a + step;
    if (m < n && st[m] <= p) a = m;
  }
  return a;
}

struct Piece {
  int dst;            // staged byte (in the step's buffer) of chunk 0
  int m;              // chunks, 1..kPiece
  int lo, hi;         // chunk 0 starts at its byte lo; chunk m - 1 ends before its byte hi
  const uint8_t *sp;  // frame byte landing on staged byte dst
};

__device__ __forceinline__ Piece piece_of(const StitchParams &P, const Shared &S,
                                          const int32_t *st, int a, int p, int r0) {
  const int b0 = S.rect[a][0], b1 = S.rect[a][1];
  const int y0 = max(static_cast<int>(S.rect[a][2]), r0);
  const int q0 = b0 >> 4, nq = ((b1 - 1) >> 4) - q0 + 1;
  const int ppr = (nq + kPiece - 1) / kPiece;
  const int local = p - st[a];
  const int rl = local / ppr;
  const int k = local - rl * ppr;
  const int row = y0 + rl;
  const int qf = q0 + k * kPiece;
  Piece pc;
  pc.m = min(kPiece, q0 + nq - qf);
  pc.dst = (row - r0) * kRowBytes + 16 * qf;
  pc.lo = max(b0 - 16 * qf, 0);
  pc.hi = min(b1 - 16 * (qf + pc.m - 1), 16);
  pc.sp = P.frames + S.src[a] + static_cast<int64_t>(row) * P.row_pitch + 16 * qf;
  return pc;
}

// One lane's piece in flight: its source run read from the dword at or below its first
// byte as kPiece 16-byte loads plus one dword; chunk c uses dwords [4c, 4c + 5).
struct Flight {
  uint32_t meta;  // dst | (m-1) << 15 | lo << 19 | hi << 23 | sh << 28 | slow << 30 | valid << 31
  uint32_t w[4 * kPiece + 1];
};

// What lanes without a piece, and chunks past a piece's end, read instead.
__device__ uint32_t g_dummy[8];

// Decodes piece p (if p < total) and issues its loads. The loads are unconditional so
// that each call is one straight-line batch of kPiece + 1 loads whose waits the
// compiler can count.
__device__ __forceinline__ void issue(const StitchParams &P, const Shared &S, const int32_t *st,
                                      int n, int total, int r0, int p, Flight &F) {
  F.meta = 0;
  const uint8_t *run = nullptr;
  int m = 0;
  if (p < total) {
    const Piece pc = piece_of(P, S, st, find_record(st, n, p), p, r0);
    const uint32_t sh = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(pc.sp) & 3u);
    const uint8_t *a0 = pc.sp - sh;
    m = pc.m;
    F.meta = uint32_t(pc.dst) | (uint32_t(pc.m - 1) << 15) | (uint32_t(pc.lo) << 19) |
             (uint32_t(pc.hi) << 23) | (sh << 28) | (1u << 31);
    // loads [a0, a0 + 16 (m + 1)) must stay inside the frame buffer's dwords
    if (a0 >= P.load_base && a0 + 16 * pc.m <= P.load_limit)
      run = a0;
    else
      F.meta |= 1u << 30;
  }
  const uint8_t *dummy = reinterpret_cast<const uint8_t *>(g_dummy);
#pragma unroll
  for (int c = 0; c < kPiece; ++c) {
    const uint8_t *ad = (run != nullptr && c <= m) ? run + 16 * c : dummy;
    const u32x4a4 v = *reinterpret_cast<const u32x4a4 *>(ad);
    F.w[4 * c] = v.x;
    F.w[4 * c + 1] = v.y;
    F.w[4 * c + 2] = v.z;
    F.w[4 * c + 3] = v.w;
  }
  F.w[4 * kPiece] = *reinterpret_cast<const uint32_t *>(
      (run != nullptr && m == kPiece) ? run + 16 * kPiece : dummy);
  // keep the scheduler from hoisting later work (the landing of the other flight, whose
  // loads were issued earlier) above these loads
  __builtin_amdgcn_sched_barrier(0);
}

// Writes bytes [lo, hi) of a 16-byte-aligned LDS chunk: whole dwords by plain stores,
// dwords shared with a neighbouring patch (or pad) by an atomic and-then-or of this
// chunk's bytes only, so lanes writing other bytes of the same dword do not collide.
__device__ __forceinline__ void write_bytes(uint8_t *d, const uint32_t e[4], int lo, int hi) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int a = max(lo, 4 * q), b = min(hi, 4 * q + 4);
    if (a >= b) continue;
    uint32_t *p = reinterpret_cast<uint32_t *>(d + 4 * q);
    if (b - a == 4) {
      *p = e[q];
    } else {
      const uint32_t mask = (0xFFFFFFFFu >> (32 - 8 * (b - a))) << (8 * (a - 4 * q));
      __hip_atomic_fetch_and(p, ~mask, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __hip_atomic_fetch_or(p, e[q] & mask, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
}

// Realigns a landed piece and writes it into the staged rows.
__device__ __forceinline__ void land(const StitchParams &P, const Shared &S, const int32_t *st,
                                     uint8_t *buf, int n, int r0, int p, const Flight &F) {
  const uint32_t kind = F.meta >> 30;
  if (kind == 0x3u) {  // near the frame buffer's ends: byte by byte
    const Piece pc = piece_of(P, S, st, find_record(st, n, p), p, r0);
    for (int c = 0; c < pc.m; ++c) {
      const int lo = c == 0 ? pc.lo : 0, hi = c == pc.m - 1 ? pc.hi : 16;
      for (int q = lo; q < hi; ++q) buf[pc.dst + 16 * c + q] = pc.sp[16 * c + q];
    }
    return;
  }
  if (kind != 0x2u) return;
  const int m = static_cast<int>((F.meta >> 15) & 15) + 1;
  const int lo0 = (F.meta >> 19) & 15, hi1 = (F.meta >> 23) & 31;
  const uint32_t sh = (F.meta >> 28) & 3;
  uint8_t *d = buf + (F.meta & 0x7FFF);
#pragma unroll
  for (int c = 0; c < kPiece; ++c) {
    const bool whole = c < m && (c > 0 || lo0 == 0) && (c < m - 1 || hi1 == 16);
    if (!whole) continue;
    u32x4 e;
    e.x = __builtin_amdgcn_alignbyte(F.w[4 * c + 1], F.w[4 * c], sh);
    e.y = __builtin_amdgcn_alignbyte(F.w[4 * c + 2], F.w[4 * c + 1], sh);
    e.z = __builtin_amdgcn_alignbyte(F.w[4 * c + 3], F.w[4 * c + 2], sh);
    e.w = __builtin_amdgcn_alignbyte(F.w[4 * c + 4], F.w[4 * c + 3], sh);
    *reinterpret_cast<u32x4 *>(d + 16 * c) = e;
  }
  if (lo0 > 0 || (m == 1 && hi1 < 16)) {  // first chunk starts inside (or single, cut)
    uint32_t e[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) e[q] = __builtin_amdgcn_alignbyte(F.w[q + 1], F.w[q], sh);
    write_bytes(d, e, lo0, m == 1 ? hi1 : 16);
  }
  if (m > 1 && hi1 < 16) {  // last chunk (not also the first) ends inside
    uint32_t r[5];
#pragma unroll
    for (int q = 0; q < 5; ++q) r[q] = F.w[4 + q];
#pragma unroll
    for (int c = 2; c < kPiece; ++c)
      if (c == m - 1) {
#pragma unroll
        for (int q = 0; q < 5; ++q) r[q] = F.w[4 * c + q];
      }
    uint32_t e[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) e[q] = __builtin_amdgcn_alignbyte(r[q + 1], r[q], sh);
    write_bytes(d + 16 * (m - 1), e, 0, hi1);
  }
}

// Pieces from, from + nt, ... (< total) of a step, batch after batch, each landed
// before the next is issued.
__device__ __forceinline__ void copy_rest(const StitchParams &P, const Shared &S, const int32_t *st,
                                          uint8_t *buf, int n, int total, int r0, int from,
                                          int nt) {
  for (int p = from; p < total; p += nt) {
    Flight F;
    issue(P, S, st, n, total, r0, p, F);
    wait_vm<0>();
    land(P, S, st, buf, n, r0, p, F);
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

// Converts `rows` staged rows (8-pixel groups g = t, t + nt, ...) into the three fp16
// planes of canvas c_local at canvas row Y, columns from X_t, and restores the pad
// bytes of every group it read.
template <bool kVec, bool kLut, int kNt>
__device__ __forceinline__ void convert_rows(const StitchParams &P, const uint16_t *lut,
                                             uint8_t *buf, int c_local, int Y, int rows,
                                             int X_t, int tw, int t) {
  const int gx = (tw + 7) >> 3;
  const int ng = rows * gx;
  const int64_t plane = static_cast<int64_t>(P.canvas_h) * P.canvas_w;
  const uint32_t p0 = P.pad_dw[0], p1 = P.pad_dw[1], p2 = P.pad_dw[2];
  // A fixed trip count: the loop is unrolled, so no loop preheader makes the wave wait
  // for its earlier stores.
  constexpr int kIt = (kStepRows * (kTileW / 8) + kNt - 1) / kNt;
#pragma unroll
  for (int it = 0; it < kIt; ++it) {
    const int g = t + it * kNt;
    if (g >= ng) continue;
    const int rr = g / gx, col = g - rr * gx;
    u32x2 *p = reinterpret_cast<u32x2 *>(buf + rr * kRowBytes + 24 * col);
    const u32x2 v0 = p[0], v1 = p[1], v2 = p[2];
    // 24 staged bytes start at a multiple of 3: pattern phase 0
    p[0] = u32x2{p0, p1};
    p[1] = u32x2{p2, p0};
    p[2] = u32x2{p1, p2};
    const uint32_t e[6] = {v0.x, v0.y, v1.x, v1.y, v2.x, v2.y};
    uint32_t o[3][4];
#pragma unroll
    for (int k = 0; k < 3; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int b0 = 3 * (2 * j) + k, b1 = 3 * (2 * j + 1) + k;
        const uint32_t x0 = (e[b0 >> 2] >> (8 * (b0 & 3))) & 0xFFu;
        const uint32_t x1 = (e[b1 >> 2] >> (8 * (b1 & 3))) & 0xFFu;
        if (kLut)
          o[k][j] = uint32_t(lut[k * 256 + x0]) | (uint32_t(lut[k * 256 + x1]) << 16);
        else
          o[k][j] = norm2(x0, x1, P.fa[k], P.fc[k]);
      }
    const int X0 = X_t + 8 * col;
    uint16_t *base = P.out + (static_cast<int64_t>(c_local) * 3) * plane +
                     static_cast<int64_t>(Y + rr) * P.canvas_w + X0;
    if (kVec) {  // canvas_w % 8 == 0 and a 16-byte aligned output: whole groups only
#pragma unroll
      for (int k = 0; k < 3; ++k)
        __builtin_nontemporal_store(u32x4{o[k][0], o[k][1], o[k][2], o[k][3]},
                                    reinterpret_cast<u32x4 *>(base + k * plane));
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (X0 + i >= P.canvas_w) continue;
#pragma unroll
        for (int k = 0; k < 3; ++k)
          base[k * plane + i] = static_cast<uint16_t>(o[k][i >> 1] >> ((i & 1) * 16));
      }
    }
  }
}

template <bool kVec, bool kLut>
__global__ __launch_bounds__(kThreads) void stitch_kernel(const StitchParams P) {
  __shared__ __attribute__((aligned(16))) uint8_t s_px[2 * kBufBytes];
  __shared__ Shared S;
  __shared__ uint16_t s_lut[kLut ? 3 * 256 : 2];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int L = P.unit_order ? P.unit_order[blockIdx.x] : static_cast<int>(blockIdx.x);
  if (L < 0 || L >= P.n_units) return;  // not a unit: the whole workgroup leaves
  const int per_canvas = P.tiles_x * P.bands_y;
  const int c_local = L / per_canvas;
  const int rem = L - c_local * per_canvas;
  const int band = rem / P.tiles_x;
  const int tx = rem - band * P.tiles_x;
  const int canvas = P.canvas_first + c_local;
  const int X_t = tx * kTileW;
  const int tw = min(kTileW, P.canvas_w - X_t);
  const int Y_b = band * P.band_steps * kStepRows;
  const int bh = min(P.band_steps * kStepRows, P.canvas_h - Y_b);
  const int ns = (bh + kStepRows - 1) / kStepRows;

  if (kLut)
    for (int i = tid; i < 384; i += kThreads) reinterpret_cast<uint32_t *>(s_lut)[i] = P.lut[i];
  {
    // A staged row is a whole number of 48-byte chunk triples, each repeating the 12-byte
    // pad pattern from phase 0.
    const uint32_t p0 = P.pad_dw[0], p1 = P.pad_dw[1], p2 = P.pad_dw[2];
    for (int i = tid; i < 2 * kBufBytes / 48; i += kThreads) {
      u32x4 *d = reinterpret_cast<u32x4 *>(s_px + 48 * i);
      d[0] = u32x4{p0, p1, p2, p0};
      d[1] = u32x4{p1, p2, p0, p1};
      d[2] = u32x4{p2, p0, p1, p2};
    }
  }
  lds_barrier();  // the prefill is complete even when no list round runs below

  // The canvas's segment of `order`, clamped so a corrupt plan cannot index outside it.
  const int k_lo = min(max(P.canvas_begin[canvas], 0), P.n_rois);
  const int k_hi = min(max(P.canvas_begin[canvas + 1], k_lo), P.n_rois);

  int n;
  if (build_list(P, S, canvas, X_t, tw, Y_b, bh, k_lo, k_hi, n) == k_hi) {
    // Step s of the band (rows [3s, 3s + 3)) is staged in buffer s % 2 by the loaders
    // while the converters turn step s - 1 into fp16; one barrier per step.
    if (wave < kLoadWaves) {
      int32_t *st0 = S.start[2 * wave], *st1 = S.start[2 * wave + 1];
      for (int s = 0; s < ns; s += 2) {
        // Steps s and s + 1: both first flights are issued before either lands.
        const int r0 = s * kStepRows, r1 = r0 + kStepRows;
        const bool two = s + 1 < ns;
        Flight A, B;
        const int tot0 = prefix_pieces(S, st0, n, r0, min(r1, bh));
        issue(P, S, st0, n, tot0, r0, tid, A);
        int tot1 = 0;
        if (two) {
          tot1 = prefix_pieces(S, st1, n, r1, min(r1 + kStepRows, bh));
          issue(P, S, st1, n, tot1, r1, tid, B);
          wait_vm<kPiece + 1>();  // A's loads; B's stay in flight
        } else {
          wait_vm<0>();
        }
        land(P, S, st0, s_px, n, r0, tid, A);
        copy_rest(P, S, st0, s_px, n, tot0, r0, tid + kLoadThreads, kLoadThreads);
        lds_barrier();
        if (!two) break;
        wait_vm<0>();
        land(P, S, st1, s_px + kBufBytes, n, r1, tid, B);
        copy_rest(P, S, st1, s_px + kBufBytes, n, tot1, r1, tid + kLoadThreads, kLoadThreads);
        lds_barrier();
      }
      lds_barrier();  // the converters' last step
    } else {
      for (int s = 0; s <= ns; ++s) {
        if (s >= 1) {
          const int r0 = (s - 1) * kStepRows;
          convert_rows<kVec, kLut, kConvThreads>(P, s_lut, s_px + ((s - 1) & 1) * kBufBytes,
                                                 c_local, Y_b + r0, min(kStepRows, bh - r0),
                                                 X_t, tw, tid - kLoadThreads);
        }
        lds_barrier();
      }
    }
  } else {
    // More patches meet the band than one list holds: each step takes as many lists as
    // it needs, every wave copying, then every wave converting.
    for (int s = 0; s < ns; ++s) {
      const int r0 = s * kStepRows, rows = min(kStepRows, bh - r0);
      for (int scan = k_lo; scan < k_hi;) {
        __syncthreads();  // the previous list is no longer read
        const int next = build_list(P, S, canvas, X_t, tw, Y_b + r0, rows, scan, k_hi, n);
        int32_t *st = S.start[wave];
        const int total = prefix_pieces(S, st, n, 0, rows);
        copy_rest(P, S, st, s_px, n, total, 0, tid, kThreads);
        scan = next;
      }
      lds_barrier();
      convert_rows<kVec, kLut, kThreads>(P, s_lut, s_px, c_local, Y_b + r0, rows, X_t, tw,
                                         tid);
      lds_barrier();
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
  P.canvas_count = a->canvas_count;
  P.canvas_w = a->canvas_w;
  P.canvas_h = a->canvas_h;
  P.tiles_x = g.tiles_x;
  P.bands_y = g.bands_y;
  P.band_steps = g.band_steps;
  P.n_units = g.n_units;
  P.unit_order = a->unit_order;
  P.out = a->out;
  // A 16-byte load may start on any dword from the one holding the first frame byte up
  // to the one 16 bytes before the end of the dword holding the last valid byte. With
  // n_frames == 0 no patch is sane and no load is formed.
  const int64_t valid_end = a->n_frames > 0 ? int64_t(a->n_frames - 1) * a->frame_stride +
                                                  int64_t(a->frame_h - 1) * a->row_pitch +
                                                  3 * int64_t(a->frame_w)
                                            : 0;
  const uintptr_t f0 = reinterpret_cast<uintptr_t>(a->frames);
  const uintptr_t begin4 = f0 & ~uintptr_t(3);
  const uintptr_t end4 = (f0 + uintptr_t(valid_end) + 3) & ~uintptr_t(3);
  P.load_base = a->frames - (f0 - begin4);
  // below load_base (no fast load at all) when the buffer holds under 16 bytes
  P.load_limit = a->frames + (int64_t(end4) - 16 - int64_t(f0));

  const tg_detail::NormConsts &nm = tg_detail::norm_consts(a->mean, a->std);
  std::memcpy(P.lut, nm.lut16, sizeof nm.lut16);
  for (int k = 0; k < 3; ++k) {
    P.fa[k] = nm.fa[k];
    P.fc[k] = nm.fc[k];
  }
  uint8_t pat[12];
  for (int i = 0; i < 12; ++i) pat[i] = a->pad[i % 3];
  std::memcpy(P.pad_dw, pat, sizeof pat);

  const bool vec = (a->canvas_w % 8 == 0) && (reinterpret_cast<uintptr_t>(a->out) % 16 == 0);
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
