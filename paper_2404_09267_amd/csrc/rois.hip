// tg_mask_rois: RoIs from a foreground mask, as the bounding boxes of 8-connected
// components (the paper cuts its RoIs from the background model's foreground,
// Sec. III-A, step 1).
//
// Connected components by union-find with atomic-min linking (a root always points to
// the smallest index of its set, so every set ends rooted at its first pixel in raster
// order) -- the GPU union-find labelling of D. P. Playne and K. A. Hawick (IEEE TPDS 29(6),
// 2018), tile-local first and merged along tile borders as in the block-based labelling of
// S. Allegretti, F. Bolelli and C. Grana (IEEE TPDS 31(2), 2020) -- in seven launches on
// the caller's stream. Foreground masks are sparse, so only the scan reads the mask; the
// other passes visit the 32x32 tiles that hold foreground, through per-tile records
// (row masks, local-root masks, the tile-local roots of the border pixels) indexed by
// tile id. Same-address global atomics serialize across the chip, so no pass counts or
// takes tickets on one word per workgroup of a large grid.
//  1. scan:   one 256-thread workgroup per 16 tiles side by side streams the mask (16-byte
//             loads where it can), stores a bit per tile (set: foreground) and writes the
//             32 row masks of the tiles with foreground; it also zeroes the tickets,
//             counters and look-back words of the later passes.
//  2. list:   compacts the bitmap into the list of non-empty tiles (increasing ids), a
//             few large workgroups with a decoupled look-back.
//  3. local:  one wave per listed tile, a grid of resident one-wave workgroups walking
//             the list: union-find in LDS over the tile's row runs (one union per pair
//             of touching runs); each tile-local root's label word gets its own frame
//             index, the tile's local roots and border roots go to its record, and each
//             local component's box and pixel count, folded in LDS, to one of the tile's
//             256 entry slots, and the tile's count of local roots is added to its
//             band's. No other label word is written or read.
//  4. merge:  per listed tile, four 16-pixel items (its top row in two halves, its left
//             column in two halves) join each foreground pixel with its foreground
//             neighbours across the border, reading the records of the tile and of the
//             tiles around it, with global atomics on the label array; an item whose
//             neighbouring tiles are all empty is skipped. Every 8-neighbour pair across a
//             tile border is seen from the tile below or to the right of it. A root that
//             gets linked leaves its band's count, which then counts components.
//  5. number: per band of 32 rows (a tile row of a frame), the recorded local roots still
//             their own parent (the components) are numbered in raster order, each
//             component's record is initialised and its root marked with its number. The
//             band's first number is the sum of the earlier bands' counts, read by the
//             band's workgroup (over kDirectBands bands, a one-workgroup scan launched
//             before it puts it in place).
//  6. boxes:  each local component (its entry) follows the union-find from its root to
//             its component's number and folds its box and count into the record with
//             one set of global atomics.
//  7. filter: components of at least min_area pixels, compacted in number order with a
//             look-back, written as tg_roi rows; each frame's first row (frame_begin) is
//             the compacted position of the frame's first component.
// Every union-find walk checks the invariant it relies on (unionfind.h); a walk that meets a
// link that does not point to a smaller index ends, sets the workspace's status word, and
// the call reports *n_rois = *n_components = TG_E_INTERNAL instead of RoIs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <map>
#include <mutex>
#include <tuple>

#include "lookback.h"
#include "tg.h"
#include "unionfind.h"

namespace {

constexpr int kTile = 32;
constexpr int kEntryThreads = 256;  // boxes pass: one wave per listed tile
constexpr int kScanTiles = 16;     // tiles side by side per workgroup of the scan pass
constexpr int kScanThreads = 256;  // 8 threads per row of 16 tiles, 64 pixels each
constexpr int kListGroups = 2048;  // list-walking grid when the occupancy query fails
constexpr int kListThreads = 256;  // list pass: kListPer bitmap words per thread
constexpr int kListPer = 4;
constexpr int kListChunk = kListThreads * kListPer;  // bitmap words per list workgroup
constexpr int kBorderThreads = 256;
// Labels: only the words of tile-local roots are used. Such a word holds kRootFlag | its
// parent in the union-find over roots (itself at first), and becomes -(component + 1)
// once it is numbered. Frames have fewer than 2^30 pixels, so the flag bit is free.
constexpr int32_t kRootFlag = 1 << 30;
constexpr int32_t kIndex = kRootFlag - 1;
constexpr int kBandThreads = 256;  // numbering passes: 8 threads per row of a 32-row band
constexpr int kBandBatch = 16;     // wide bands: tiles whose loads a thread issues together
constexpr int kBandTiles = 256;    // widest band (in tiles) whose non-empty tiles go to LDS
constexpr int kPairBatch = 4;      // (row, tile) pairs whose loads a thread issues together
constexpr int kBandScanThreads = 1024;  // the scan over the bands' counts: one workgroup
constexpr int kDirectBands = 4096;  // up to this many bands, numbering sums the counts itself
constexpr int kFilterBlock = 1024;  // components per workgroup of the filter pass
constexpr int kFilterThreads = 256;

struct Comp {
  int32_t frame, root, x0, y0, x1, y1, area, unused;
};
static_assert(sizeof(Comp) == 32, "component record is 32 bytes");

// Tiles of all frames, numbered frame by frame, tile rows top to bottom, tiles left to
// right: tile (f, ty, tx) is (f * tiles_y + ty) * tiles_x + tx; band f * tiles_y + ty is
// that tile row. The tile bitmap gives each band wpb = ceil(tiles_x / 32) words of its
// own: tile tx of band b is bit tx % 32 of word b * wpb + tx / 32.
struct Tiles {
  int tiles_x, tiles_y, wpb;
  int64_t n;
};

struct Layout {
  // [0]: list ticket, [1]: filter ticket, [2]: status, [3]: non-empty tiles listed,
  // [4]: unused, then the look-back words of the list and filter passes and the bands'
  // counts of components (32-bit); all cleared by the scan
  uint64_t *words;
  uint64_t *list_state, *filter_state;
  // the tile bitmap (bit set: the tile holds foreground), band by band (Tiles), every
  // word written by the scan
  uint32_t *tile_bits;
  // per band: its count of components (tile-local roots added by the local pass, linked
  // roots removed by the merge), then its first component's number
  int32_t *band_first;
  int32_t *tile_list;  // ids of the non-empty tiles, in increasing order
  // Record of non-empty tile t: fg[32 t + r], row r's foreground as a 32-bit mask;
  // roots[32 t + r], row r's tile-local roots; border[128 t + e], the tile-local root (a
  // frame index) of border pixel e -- row 0 (e < 32), row 31, column 0, column 31
  // (e - 96) -- or -1 for background.
  uint32_t *rec_fg, *rec_roots;
  int32_t *rec_border;
  // One entry per tile-local component, at most 256 per tile (8-connected, 32x32):
  // entries[256 t + j], j < n_ent[t]: local root << 26 | x0 << 21 | x1 << 16 | y1 << 11 |
  // pixel count, the box in tile coordinates (its top row is the root's).
  uint64_t *entries;
  int32_t *n_ent;
  Comp *comp;
  int32_t *label;
  int64_t n_words;
  size_t bytes;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int64_t list_chunks(int64_t n_bit_words) { return (n_bit_words + kListChunk - 1) / kListChunk; }

Layout layout(void *base, int64_t n_px, int64_t n_bands, int64_t n_tiles,
              int64_t n_bit_words, int32_t max_components) {
  Layout L;
  const int64_t n_chunks = list_chunks(n_bit_words);
  const int64_t n_filter = (max_components + kFilterBlock - 1) / kFilterBlock;
  L.n_words = 5 + n_chunks + n_filter + (n_bands + 1) / 2;
  const size_t nt = static_cast<size_t>(n_tiles);
  const size_t o_bits = round_up(8 * static_cast<size_t>(L.n_words), 256);
  const size_t o_list = round_up(o_bits + 4 * static_cast<size_t>(n_bit_words), 256);
  const size_t o_fg = round_up(o_list + 4 * nt, 256);
  const size_t o_roots = round_up(o_fg + 128 * nt, 256);
  const size_t o_border = round_up(o_roots + 128 * nt, 256);
  const size_t o_entries = round_up(o_border + 512 * nt, 256);
  const size_t o_nent = round_up(o_entries + 8 * 256 * nt, 256);
  const size_t o_comp = round_up(o_nent + 4 * nt, 256);
  const size_t o_label = round_up(o_comp + sizeof(Comp) * static_cast<size_t>(max_components), 256);
  L.bytes = round_up(o_label + 4 * static_cast<size_t>(n_px), 256);
  char *b = static_cast<char *>(base);
  L.words = b ? reinterpret_cast<uint64_t *>(b) : nullptr;
  L.list_state = b ? L.words + 5 : nullptr;
  L.filter_state = b ? L.list_state + n_chunks : nullptr;
  L.band_first = b ? reinterpret_cast<int32_t *>(L.filter_state + n_filter) : nullptr;
  L.tile_bits = b ? reinterpret_cast<uint32_t *>(b + o_bits) : nullptr;
  L.tile_list = b ? reinterpret_cast<int32_t *>(b + o_list) : nullptr;
  L.rec_fg = b ? reinterpret_cast<uint32_t *>(b + o_fg) : nullptr;
  L.rec_roots = b ? reinterpret_cast<uint32_t *>(b + o_roots) : nullptr;
  L.rec_border = b ? reinterpret_cast<int32_t *>(b + o_border) : nullptr;
  L.entries = b ? reinterpret_cast<uint64_t *>(b + o_entries) : nullptr;
  L.n_ent = b ? reinterpret_cast<int32_t *>(b + o_nent) : nullptr;
  L.comp = b ? reinterpret_cast<Comp *>(b + o_comp) : nullptr;
  L.label = b ? reinterpret_cast<int32_t *>(b + o_label) : nullptr;
  return L;
}

// ---- union-find ---------------------------------------------------------------------

__device__ __forceinline__ int lds_load(int *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ int g_load(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Union-find over a tile's labels in LDS (unionfind.h).
struct LdsLabels {
  int *L;
  __device__ int parent(int i) const { return lds_load(&L[i]); }
  __device__ int link(int i, int p) { return atomicMin(&L[i], p); }
};

// Union-find over the flagged words of tile-local roots in global memory (one frame's
// labels, W pixels a row). Links only lower a word, so a root that is linked (to a
// smaller index) stops being a root for good; that link is the one that removes it from
// its band's count of components (band_count: the frame's bands). The removals are
// collected for up to two bands and applied by flush(), so that no atomic on a count
// sits between the loads of a union-find walk; a third band is applied at once.
struct RootLabels {
  int32_t *L;
  int32_t *band_count;
  int W;
  int band0 = -1, n0 = 0, band1 = -1, n1 = 0;
  __device__ int parent(int i) const { return g_load(&L[i]) & kIndex; }
  __device__ int link(int i, int p) {
    const int old = __hip_atomic_fetch_min(&L[i], p | kRootFlag, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT) & kIndex;
    if (old == i && p < i) {
      const int band = (i / W) / kTile;
      if (band == band0 || band0 < 0) {
        band0 = band;
        ++n0;
      } else if (band == band1 || band1 < 0) {
        band1 = band;
        ++n1;
      } else {
        atomicSub(&band_count[band], 1);
      }
    }
    return old;
  }
  __device__ void flush() {
    if (n0) atomicSub(&band_count[band0], n0);
    if (n1) atomicSub(&band_count[band1], n1);
  }
};

// Records in the workspace's status word that a union-find walk met a link that breaks
// the invariant (tg_mask_rois then reports TG_E_INTERNAL instead of RoIs).
__device__ __forceinline__ void fail(uint32_t *status) {
  __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Workgroup barrier that orders LDS only: no wait for the workgroup's outstanding global
// stores, which a plain __syncthreads() would drain first.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Whether tile tx of band `band` holds foreground.
__device__ __forceinline__ bool tile_set(const uint32_t *bits, const Tiles &T, int band, int tx) {
  return (bits[static_cast<int64_t>(band) * T.wpb + (tx >> 5)] >> (tx & 31)) & 1u;
}

// Frame, tile row and tile column of tile id t.
struct TileAt {
  int f, ty, tx;
};
__device__ __forceinline__ TileAt tile_at(const Tiles &T, int t) {
  const int ft = t / T.tiles_x;
  TileAt a;
  a.tx = t - ft * T.tiles_x;
  a.f = ft / T.tiles_y;
  a.ty = ft - a.f * T.tiles_y;
  return a;
}

// Run-based labelling of one 32x32 tile by one wave. A row's foreground is a 32-bit
// word; its runs (maximal horizontal segments) are the union-find nodes, run j of row r
// being node 16 r + j (a row holds at most 16 runs), so node order is raster order of the
// runs' first pixels and every set ends rooted at the run holding its first pixel. A run
// of row r touches, 8-connected, the runs of row r - 1 that meet columns s - 1 .. e + 1
// of its span s .. e: consecutive runs of that row, from the one holding the lowest
// foreground column of the window to the one holding the highest.
constexpr int kLocalThreads = 64;  // one wave per tile: lane l on row l % 32
constexpr int kRunNodes = kTile * 16;

struct RunTile {
  int L[kRunNodes];                    // union-find links over the runs
  unsigned long long span[kRunNodes];  // per root: row bits << 32 | column bits
  int count[kRunNodes];                // per root: pixels
  uint8_t col[kRunNodes];              // first column of each run
};

// Ordinal of the run of row word `starts` (its runs' first columns as bits) that holds
// column c, c being foreground.
__device__ __forceinline__ int run_ordinal(uint32_t starts, int c) {
  return __popc(starts & (0xFFFFFFFFu >> (31 - c))) - 1;
}

// Last column of the run that starts at column s of a row whose runs end at the bits of
// `ends`.
__device__ __forceinline__ int run_end(uint32_t ends, int s) {
  return __builtin_ctz(ends & (0xFFFFFFFFu << s));
}

// Columns lo .. hi as bits (0 <= lo <= hi <= 31).
__device__ __forceinline__ uint32_t col_span(int lo, int hi) {
  return (0xFFFFFFFFu >> (31 - hi)) & (0xFFFFFFFFu << lo);
}

// ---- kernels ------------------------------------------------------------------------

// Which tiles hold foreground: one workgroup per 16 tiles side by side (a 512 x 32 block
// of one frame), thread t reading row t / 8 of the block, pixels 64 (t % 8) .. + 63 (the
// row segments of two tiles) with 16-byte loads (kMode 2: mask 16-byte aligned and rows a
// multiple of 16 bytes), dwords (kMode 1) or bytes (kMode 0), all issued before any is
// used. Every block stores its 16 tiles' bits (half a bitmap word; the grid has
// 2 wpb blocks per band, the last ones past the frame's width storing zeros) and writes
// the 32 row masks of each tile with foreground to its record. Nothing is counted here:
// the same-address atomics of a global list counter would serialize the workgroups. The
// blocks also zero the n_clear counter words that the later passes use.
template <int kMode>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const uint8_t *mask, int W, int H,
                                                            int64_t frame_px, Tiles T,
                                                            uint32_t *tile_bits,
                                                            uint32_t *rec_fg, uint64_t *words,
                                                            int64_t n_clear) {
  __shared__ uint32_t s_bits;
  const int t = threadIdx.x, r = t >> 3, q = t & 7;
  const int64_t f = blockIdx.z;
  const int64_t g = (static_cast<int64_t>(blockIdx.z) * gridDim.y + blockIdx.y) * gridDim.x +
                    blockIdx.x;
  const int64_t all = static_cast<int64_t>(gridDim.x) * gridDim.y * gridDim.z * kScanThreads;
  for (int64_t i = g * kScanThreads + t; i < n_clear; i += all) words[i] = 0;
  const int tx0 = blockIdx.x * kScanTiles, ty = blockIdx.y;
  const int y = ty * kTile + r, x = tx0 * kTile + 64 * q;
  if (t == 0) s_bits = 0;
  uint32_t m0 = 0, m1 = 0;  // row y: foreground of pixels x + c and x + 32 + c as bit c
  if (y < H && x < W) {
    const uint8_t *row = mask + f * frame_px + static_cast<int64_t>(y) * W;
    if (kMode == 2) {  // rows a multiple of 16 bytes: a chunk is wholly inside or outside
      typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
      u32x4 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        v[i] = x + 16 * i < W ? *reinterpret_cast<const u32x4 *>(row + x + 16 * i) : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const uint32_t bit = ((v[i][j >> 2] >> (8 * (j & 3))) & 0xFFu) ? 1u << (16 * (i & 1) + j) : 0u;
          if (i < 2)
            m0 |= bit;
          else
            m1 |= bit;
        }
    } else if (kMode == 1) {  // rows a multiple of 4 bytes
      uint32_t v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i)
        v[i] = x + 4 * i < W ? *reinterpret_cast<const uint32_t *>(row + x + 4 * i) : 0u;
#pragma unroll
      for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t bit = ((v[i] >> (8 * k)) & 0xFFu) ? 1u << (4 * (i & 7) + k) : 0u;
          if (i < 8)
            m0 |= bit;
          else
            m1 |= bit;
        }
    } else {
#pragma unroll 8
      for (int i = 0; i < 32; ++i) {
        m0 |= (x + i < W && row[x + i]) ? 1u << i : 0u;
        m1 |= (x + 32 + i < W && row[x + 32 + i]) ? 1u << i : 0u;
      }
    }
  }
  // lane l of a wave is row l / 8, tile pair l % 8: a tile holds foreground when any of
  // the wave's rows does
  const uint64_t b0 = __ballot(m0 != 0), b1 = __ballot(m1 != 0);
  if ((t & 63) == 0) {
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      m |= ((b0 >> k) & 0x0101010101010101ull) ? 1u << (2 * k) : 0u;
      m |= ((b1 >> k) & 0x0101010101010101ull) ? 1u << (2 * k + 1) : 0u;
    }
    if (m) atomicOr(&s_bits, m);
  }
  __syncthreads();
  const uint32_t m = s_bits;
  const int64_t band = f * T.tiles_y + ty;
  if (t == 0)
    reinterpret_cast<uint16_t *>(tile_bits)[band * 2 * T.wpb + blockIdx.x] =
        static_cast<uint16_t>(m);
  if (m == 0) return;  // uniform
  const int id0 = static_cast<int>(band * T.tiles_x + tx0);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int j = 2 * q + h;
    if (m >> j & 1u) rec_fg[32 * static_cast<int64_t>(id0 + j) + r] = h ? m1 : m0;
  }
}

// Lists the non-empty tiles in increasing order (bands in order, each band's tiles left to
// right): workgroup c (in ticket order) takes kListChunk words of the tile bitmap, kListPer
// per thread; a block-wide scan of their
// counts and a decoupled look-back over the workgroups place each set bit. The last
// workgroup writes the count (0, with the status word set, if the look-back failed).
__global__ __launch_bounds__(kListThreads) void list_kernel(const uint32_t *tile_bits,
                                                            int64_t n_bit_words, Tiles T,
                                                            int32_t *tile_list,
                                                            uint64_t *words, uint64_t *state,
                                                            int32_t n_chunks, uint32_t *n_list,
                                                            uint32_t *status) {
  __shared__ int s_chunk;
  __shared__ int s_wave[kListThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0)
    s_chunk = static_cast<int>(__hip_atomic_fetch_add(reinterpret_cast<uint32_t *>(words), 1u,
                                                      __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT));
  __syncthreads();
  const int c = s_chunk;  // < n_chunks: exactly n_chunks workgroups take tickets
  const int64_t w0 = static_cast<int64_t>(c) * kListChunk + tid * kListPer;
  uint32_t bits[kListPer];
  int cnt = 0;
#pragma unroll
  for (int i = 0; i < kListPer; ++i) {
    bits[i] = w0 + i < n_bit_words ? tile_bits[w0 + i] : 0u;
    cnt += __popc(bits[i]);
  }
  int incl = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kListThreads / 64; ++w) {
    if (w < wave) before += s_wave[w];
    total += s_wave[w];
  }
  bool failed;
  const int prefix = tg_detail::lookback_prefix_block<kListThreads, 1>(state, c, total, &failed);
  if (failed) {
    if (tid == 0) fail(status);
  } else {
    int at = prefix + before + incl - cnt;
#pragma unroll
    for (int i = 0; i < kListPer; ++i) {
      const int64_t band = (w0 + i) / T.wpb;
      const int tx0 = static_cast<int>(w0 + i - band * T.wpb) * 32;
      for (uint32_t m = bits[i]; m != 0; m &= m - 1)
        tile_list[at++] = static_cast<int32_t>(band * T.tiles_x + tx0 + __builtin_ctz(m));
    }
  }
  if (c == n_chunks - 1 && tid == 0)
    *n_list = failed ? 0u : static_cast<uint32_t>(prefix + total);
}

// Labels the listed tiles, one wave per tile, a grid of resident one-wave workgroups
// walking the list (each tile's list entry and row mask loaded one tile ahead). Lane l
// holds row l % 32; the row's runs are shared between the two halves of the wave by the
// parity of their ordinal. Per tile: union-find over the runs in LDS (one union per pair
// of touching runs of adjacent rows), each run resolved to its root, and the root's rows,
// columns and pixel count folded in LDS. Written: the frame index of each tile-local root
// (flagged) in the label array -- the only label words any later pass reads --, the
// tile's local-root row masks and border roots in its record, and one entry per local
// component (its box in tile coordinates and its pixel count) in the tile's slots; the
// number of local roots is added to the band's count of components.
__global__ __launch_bounds__(kLocalThreads) void local_kernel(int W, int64_t frame_px, Tiles T,
                                                              const int32_t *tile_list,
                                                              const uint32_t *n_list,
                                                              const uint32_t *rec_fg,
                                                              uint32_t *rec_roots,
                                                              int32_t *rec_border,
                                                              uint64_t *entries, int32_t *n_ent,
                                                              int32_t *label, int32_t *band_count,
                                                              uint32_t *status) {
  __shared__ RunTile S;
  const int n = static_cast<int>(*n_list);
  const int lane = threadIdx.x, r = lane & 31, half = lane >> 5;
  int next_id = 0;
  uint32_t next_row = 0;
  if (static_cast<int>(blockIdx.x) < n) {
    next_id = tile_list[blockIdx.x];
    next_row = rec_fg[32 * static_cast<int64_t>(next_id) + r];
  }
  for (int it = blockIdx.x; it < n; it += gridDim.x) {
    const int id = next_id;
    const TileAt a = tile_at(T, id);
    const uint32_t w = next_row;
    if (it + static_cast<int>(gridDim.x) < n) {
      next_id = tile_list[it + gridDim.x];
      next_row = rec_fg[32 * static_cast<int64_t>(next_id) + r];
    }
    const int tx0 = a.tx * kTile, ty0 = a.ty * kTile;
    int32_t *lf = label + a.f * frame_px;
    const uint32_t up = __shfl(w, (lane + 63) & 63);  // row r - 1 (used for r > 0)
    const uint32_t st = w & ~(w << 1), en = w & ~(w >> 1), ust = up & ~(up << 1);
    // the runs of even ordinal go to half 0, odd to half 1: bit s of the prefix parity
    // of st is set when the run starting at s has an even ordinal
    uint32_t par = st;
    par ^= par << 1;
    par ^= par << 2;
    par ^= par << 4;
    par ^= par << 8;
    par ^= par << 16;
    const uint32_t mine = half ? st & ~par : st & par;
    lds_barrier();  // the previous tile's reads of S are over
    for (uint32_t m = mine; m; m &= m - 1) {
      const int s = __builtin_ctz(m), node = 16 * r + run_ordinal(st, s);
      S.L[node] = node;
      S.span[node] = 0;
      S.count[node] = 0;
      S.col[node] = static_cast<uint8_t>(s);
    }
    lds_barrier();
    LdsLabels lab{S.L};
    bool ok = true;
    if (r > 0) {
      for (uint32_t m = mine; m; m &= m - 1) {
        const int s = __builtin_ctz(m), e = run_end(en, s);
        const uint32_t x = up & col_span(s > 0 ? s - 1 : 0, e < kTile - 1 ? e + 1 : kTile - 1);
        if (!x) continue;
        const int node = 16 * r + run_ordinal(st, s);
        const int kb = run_ordinal(ust, __builtin_ctz(x)), ke = run_ordinal(ust, 31 - __builtin_clz(x));
        for (int k = kb; k <= ke; ++k) ok &= tg_detail::uf_unite(lab, node, 16 * (r - 1) + k);
      }
    }
    if (!ok) fail(status);
    lds_barrier();  // every union is in
    // each run to its root (left in L, so that after the barrier L maps a run to its root),
    // folded into the root's rows, columns and count; the roots written to the label array
    uint32_t roots = 0;
    for (uint32_t m = mine; m; m &= m - 1) {
      const int s = __builtin_ctz(m), e = run_end(en, s), node = 16 * r + run_ordinal(st, s);
      int R = tg_detail::uf_find(lab, node);
      if (R < 0) {
        fail(status);
        R = node;
      }
      if (R != node) lab.link(node, R);
      atomicOr(&S.span[R], static_cast<unsigned long long>(1u << r) << 32 | col_span(s, e));
      atomicAdd(&S.count[R], e - s + 1);
      if (R == node) {
        roots |= 1u << s;
        const int P = (ty0 + r) * W + tx0 + s;
        lf[P] = P | kRootFlag;
      }
    }
    roots |= __shfl_xor(roots, 32);
    if (half == 0) rec_roots[32 * static_cast<int64_t>(id) + r] = roots;
    lds_barrier();  // L resolved, the folds complete
    // border roots: lane l takes entry l (row 0 / row 31, column l % 32), then entry 64 + l
    // (column 0 / column 31, row l % 32); background entries are -1
    int32_t *border = rec_border + 128 * static_cast<int64_t>(id);
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int row = pass ? r : (half ? kTile - 1 : 0), c = pass ? (half ? kTile - 1 : 0) : r;
      const uint32_t rw = pass ? w : __shfl(w, half ? kTile - 1 : 0);
      int32_t v = -1;
      if (rw >> c & 1u) {
        const int R = S.L[16 * row + run_ordinal(rw & ~(rw << 1), c)];
        v = (ty0 + (R >> 4)) * W + tx0 + S.col[R];
      }
      border[64 * pass + lane] = v;
    }
    // one entry per local component, in the tile's own 256 entries, in row order
    const int mine_roots = half ? 0 : __popc(roots);
    int incl = mine_roots;
    for (int o = 1; o < 32; o <<= 1) {
      const int v = __shfl_up(incl, o);
      if (r >= o) incl += v;
    }
    const int total = __shfl(incl, kTile - 1);
    if (lane == 0) {
      n_ent[id] = total;
      atomicAdd(&band_count[a.f * T.tiles_y + a.ty], total);
    }
    uint64_t *ent = entries + 256 * static_cast<int64_t>(id) + (incl - mine_roots);
    if (half == 0) {
      for (uint32_t m = roots; m; m &= m - 1) {
        const int s = __builtin_ctz(m), node = 16 * r + run_ordinal(st, s);
        const unsigned long long sp = S.span[node];
        const uint32_t cols = static_cast<uint32_t>(sp), rows = static_cast<uint32_t>(sp >> 32);
        *ent++ = static_cast<uint64_t>(r * kTile + s) << 26 |
                 static_cast<uint64_t>(__builtin_ctz(cols)) << 21 |
                 static_cast<uint64_t>(31 - __builtin_clz(cols)) << 16 |
                 static_cast<uint64_t>(31 - __builtin_clz(rows)) << 11 |
                 static_cast<uint64_t>(S.count[node]);
      }
    }
  }
}

// Four items per listed tile, walked by a grid of resident workgroups: its top row in
// two halves of 16 pixels against the row above, then its left column in two halves
// against the column to its left. Every 8-neighbour pair across a tile border is seen
// from the tile below or to the right of it. Foreground bits and tile-local roots come
// from the tiles' records (the tile itself and the up to three tiles holding the
// neighbours); an item whose neighbouring tiles are all empty is skipped.
//
// Along a border, the pixels of a run (adjacent foreground pixels of one tile) share
// their tile-local root, so an item joins runs, not pixels: the item's 16 pixels (bits of
// fg) meet the 18 neighbours at offsets -1 .. 16 along the border (bits of nb), pixel k
// meeting neighbours k .. k + 2; neighbour runs also break where the neighbours change
// tile (between offsets 0 and 1 of the first half, 16 and 17 of the second). Each pair of
// touching runs is one union, the two roots loaded from the records only then -- a lane
// has one or two pairs where a pixel-by-pixel walk had up to 48 positions, which a wave
// would step through one union at a time.
__global__ __launch_bounds__(kBorderThreads) void merge_kernel(
    int W, int64_t frame_px, Tiles T, const uint32_t *tile_bits, const int32_t *tile_list,
    const uint32_t *n_list, const uint32_t *rec_fg, const int32_t *rec_border, int32_t *label,
    int32_t *band_count, uint32_t *status) {
  const int n4 = 4 * static_cast<int>(*n_list);
  for (int i = blockIdx.x * kBorderThreads + threadIdx.x; i < n4;
       i += gridDim.x * kBorderThreads) {
    const int s = i >> 2, k = i & 3, h = k & 1, id = tile_list[s];
    const TileAt a = tile_at(T, id);
    const int band = a.f * T.tiles_y + a.ty;
    const uint32_t *fs = rec_fg + 32 * static_cast<int64_t>(id);
    uint32_t fg = 0, nb = 0;
    // record index of the item's own border pixel 0; of neighbour offset j (main tile:
    // main + j; the corner tiles before offset 0 / after offset 16: corner_lo, corner_hi)
    int64_t own = 0, main = 0, corner_lo = 0, corner_hi = 0;
    if (k < 2) {  // top row, pixels 16 h .. 16 h + 15, against row 31 of the tiles above
      const int up = id - T.tiles_x;
      if (a.ty == 0) continue;
      const bool u = tile_set(tile_bits, T, band - 1, a.tx);
      const bool ul = h == 0 && a.tx > 0 && tile_set(tile_bits, T, band - 1, a.tx - 1);
      const bool ur = h == 1 && a.tx + 1 < T.tiles_x && tile_set(tile_bits, T, band - 1, a.tx + 1);
      if (!(u || ul || ur)) continue;
      fg = (fs[0] >> (16 * h)) & 0xFFFFu;
      if (fg == 0) continue;
      own = 128 * static_cast<int64_t>(id) + 16 * h;
      main = 128 * static_cast<int64_t>(up) + 32 + 16 * h - 1;  // row 31, column 16 h - 1 + j
      corner_lo = 128 * static_cast<int64_t>(up - 1) + 32 + 31;
      corner_hi = 128 * static_cast<int64_t>(up + 1) + 32;
      if (u) {  // neighbour j is column 16 h - 1 + j of the tile above
        const uint32_t row = rec_fg[32 * static_cast<int64_t>(up) + 31];
        nb = h ? (row >> 15) & 0x1FFFFu : (row & 0x1FFFFu) << 1;
      }
      if (ul) nb |= rec_fg[32 * static_cast<int64_t>(up - 1) + 31] >> 31;
      if (ur) nb |= (rec_fg[32 * static_cast<int64_t>(up + 1) + 31] & 1u) << 17;
    } else {  // left column, rows 16 h .. 16 h + 15, against column 31 of the tiles left
      const int left = id - 1;
      if (a.tx == 0) continue;
      const bool l = tile_set(tile_bits, T, band, a.tx - 1);
      const bool lu = h == 0 && a.ty > 0 && tile_set(tile_bits, T, band - 1, a.tx - 1);
      const bool ld = h == 1 && a.ty + 1 < T.tiles_y && tile_set(tile_bits, T, band + 1, a.tx - 1);
      if (!(l || lu || ld)) continue;
#pragma unroll
      for (int j = 0; j < 16; ++j) fg |= (fs[16 * h + j] & 1u) << j;
      if (fg == 0) continue;
      own = 128 * static_cast<int64_t>(id) + 64 + 16 * h;
      main = 128 * static_cast<int64_t>(left) + 96 + 16 * h - 1;  // column 31, row 16 h - 1 + j
      corner_lo = 128 * static_cast<int64_t>(left - T.tiles_x) + 96 + 31;
      corner_hi = 128 * static_cast<int64_t>(left + T.tiles_x) + 96;
      if (l) {  // neighbour j is row 16 h - 1 + j of the tile to the left
        const uint32_t *f = rec_fg + 32 * static_cast<int64_t>(left);
#pragma unroll
        for (int j = 0; j < 18; ++j) {
          const int rr = 16 * h - 1 + j;
          if (rr < 0 || rr >= kTile) continue;
          nb |= (f[rr] >> 31) << j;
        }
      }
      if (lu) nb |= rec_fg[32 * static_cast<int64_t>(left - T.tiles_x) + 31] >> 31;
      if (ld) nb |= (rec_fg[32 * static_cast<int64_t>(left + T.tiles_x)] >> 31) << 17;
    }
    // runs: own ones start at the bits of fst; neighbour ones at those of nst, which also
    // break where the neighbours change tile
    const uint32_t fst = fg & ~(fg << 1);
    const uint32_t nst = (nb & ~(nb << 1)) | (nb & (h ? 1u << 17 : 1u << 1));
    RootLabels roots{label + a.f * frame_px, band_count + a.f * T.tiles_y, W};
    bool ok = true;
    for (uint32_t m = fst; m != 0; m &= m - 1) {
      const int s0 = __builtin_ctz(m), e = s0 + __builtin_ctz(~(fg >> s0)) - 1;
      const uint32_t x = nb & col_span(s0, e + 2);  // the neighbours of pixels s0 .. e
      if (x == 0) continue;
      const int lo = __builtin_ctz(x), hi = 31 - __builtin_clz(x);
      const int first = 31 - __builtin_clz(nst & (0xFFFFFFFFu >> (31 - lo)));  // run holding lo
      const int ra = rec_border[own + s0];
      for (uint32_t q = nst & col_span(first, hi); q != 0; q &= q - 1) {
        const int j = __builtin_ctz(q);
        const int64_t at = h == 0 && j == 0 ? corner_lo : h == 1 && j == 17 ? corner_hi : main + j;
        ok &= tg_detail::uf_unite(roots, ra, rec_border[at]);
      }
    }
    roots.flush();
    if (!ok) fail(status);
  }
}

// Numbers the components in raster order over the bands of 32 rows (a tile row of a
// frame: band b is frame b / tiles_y, tile row b % tiles_y), none of whose workgroups
// waits for another. The bands' counts of components are already known: the local pass
// adds each tile's local roots, the merge removes each root it links.
//  scan:   (over kDirectBands bands only) one workgroup turns the counts into each band's
//          first number and writes the number of components.
//  number: one workgroup per band, which (up to kDirectBands bands) sums the earlier
//          bands' counts itself; its threads take the band's (row, tile) pairs in
//          raster order, so that a block-wide scan of their counts places each component.
//          A pair's candidates are the tile's recorded local roots in that row; a
//          candidate is a component when it is still its own parent (label = own frame
//          index, flagged). Each component's record is initialised and its root marked
//          with its number. Bands up to kBandTiles tiles wide list their non-empty tiles
//          in LDS and deal the pairs out (number_kernel); wider ones give thread t row
//          t / 8 and the t % 8-th eighth of the tiles (number_wide_kernel).
// One batch of a thread's tiles (b0 .. b0 + kBandBatch - 1, below tx_hi) in row y (row rr
// of the band; band_bits: the band's bitmap words): comps[u] gets the bits of tile
// b0 + u's recorded local roots in that row
// that are still their own parent (the components). Each level of loads (bitmap,
// records, labels) is issued for the whole batch before any is used. Returns how many.
__device__ __forceinline__ int batch_roots(int W, const uint32_t *band_bits,
                                           const uint32_t *rec_roots, const int32_t *lf,
                                           int base, int y, int b0, int tx_hi, int rr,
                                           uint32_t comps[kBandBatch]) {
  uint32_t cand[kBandBatch];
#pragma unroll
  for (int u = 0; u < kBandBatch; ++u) {
    const int tile = base + b0 + u, tx = b0 + u;
    cand[u] = tx < tx_hi && ((band_bits[tx >> 5] >> (tx & 31)) & 1u)
                  ? rec_roots[32 * static_cast<int64_t>(tile) + rr]
                  : 0u;
  }
  // the label of each tile's first candidate, all loaded together; further candidates in
  // the same row of a tile (a second local root there is rare) one by one
  int first[kBandBatch];
#pragma unroll
  for (int u = 0; u < kBandBatch; ++u) {
    const int P = y * W + (b0 + u) * kTile + __builtin_ctz(cand[u] | 0x80000000u);
    first[u] = cand[u] ? lf[P] : 0;
  }
  int cnt = 0;
#pragma unroll
  for (int u = 0; u < kBandBatch; ++u) {
    comps[u] = 0;
    if (cand[u] == 0) continue;
    const int P = y * W + (b0 + u) * kTile + __builtin_ctz(cand[u]);
    if (first[u] == (P | kRootFlag)) comps[u] = cand[u] & (0u - cand[u]);
    for (uint32_t m = cand[u] & (cand[u] - 1); m != 0; m &= m - 1) {
      const int Q = y * W + (b0 + u) * kTile + __builtin_ctz(m);
      if (lf[Q] == (Q | kRootFlag)) comps[u] |= m & (0u - m);
    }
    cnt += __popc(comps[u]);
  }
  return cnt;
}

// Numbers the components of one batch (as found by batch_roots) from id on: initialises
// each one's record (below max_components) and marks its root with its number.
__device__ __forceinline__ int batch_assign(int W, int32_t *lf, int y, int b0,
                                            const uint32_t comps[kBandBatch], Comp *comp,
                                            int f, int id, int32_t max_components) {
#pragma unroll
  for (int u = 0; u < kBandBatch; ++u) {
    for (uint32_t m = comps[u]; m != 0; m &= m - 1) {
      const int P = y * W + (b0 + u) * kTile + __builtin_ctz(m);
      if (id >= 0 && id < max_components) {
        comp[id] = Comp{f, P, INT_MAX, y, INT_MIN, INT_MIN, 0, 0};
        lf[P] = -(id + 1);
      }
      ++id;
    }
  }
  return id;
}

// This thread's share of a band: frame, first tile id of the band, pixel row, tile range.
struct BandPart {
  int f, base, y, tx_lo, tx_hi, rr;
  bool rows_in;
};
__device__ __forceinline__ BandPart band_part(const Tiles &T, int H, int band) {
  BandPart p;
  const int tid = threadIdx.x;
  p.f = band / T.tiles_y;
  const int ty = band - p.f * T.tiles_y;
  p.rr = tid >> 3;
  p.y = ty * kTile + p.rr;
  const int q = tid & 7, chunk = (T.tiles_x + 7) / 8;
  p.tx_lo = min(q * chunk, T.tiles_x);
  p.tx_hi = min(p.tx_lo + chunk, T.tiles_x);
  p.base = (p.f * T.tiles_y + ty) * T.tiles_x;
  p.rows_in = p.y < H;
  return p;
}

// Exclusive scan of v over a workgroup of kThreads threads (s_wave: kThreads / 64 ints of
// LDS); *total gets the sum.
template <int kThreads>
__device__ __forceinline__ int block_exclusive(int v, int *s_wave, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o);
    if (lane >= o) incl += u;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) {
    if (w < wave) before += s_wave[w];
    sum += s_wave[w];
  }
  *total = sum;
  return before + incl - v;
}

__global__ __launch_bounds__(kBandScanThreads) void band_scan_kernel(int32_t *band_first,
                                                                     int64_t n_bands,
                                                                     int32_t *n_components,
                                                                     uint32_t *status) {
  __shared__ int s_wave[kBandScanThreads / 64];
  constexpr int kPer = 4;
  int carry = 0;
  for (int64_t b0 = 0; b0 < n_bands; b0 += kBandScanThreads * kPer) {
    const int64_t i0 = b0 + threadIdx.x * kPer;
    int v[kPer], cnt = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      v[k] = i0 + k < n_bands ? band_first[i0 + k] : 0;
      if (v[k] < 0) {  // only a broken union-find could remove more roots than there were
        fail(status);
        v[k] = 0;
      }
      cnt += v[k];
    }
    int total;
    int at = carry + block_exclusive<kBandScanThreads>(cnt, s_wave, &total);
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      if (i0 + k < n_bands) band_first[i0 + k] = at;
      at += v[k];
    }
    carry += total;
    __syncthreads();  // s_wave is written again by the next step
  }
  if (threadIdx.x == 0) *n_components = carry;
}

// The number of the band's first component. With `direct` (at most kDirectBands bands)
// the workgroup sums the earlier bands' counts itself -- each band checks its own count,
// and the last one writes the number of components; otherwise the scan pass has already
// put it in place of the band's count. Called by every thread of the workgroup.
__device__ __forceinline__ int band_start(const int32_t *band_count, int band, int n_bands,
                                          bool direct, int32_t *n_components,
                                          uint32_t *status) {
  __shared__ int s_sum[kBandThreads / 64];
  if (!direct) return band_count[band];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int v = 0;
  for (int b = tid; b < band; b += kBandThreads) v += max(band_count[b], 0);
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) s_sum[wave] = v;
  __syncthreads();
  int sum = 0;
#pragma unroll
  for (int w = 0; w < kBandThreads / 64; ++w) sum += s_sum[w];
  if (tid == 0) {
    const int own = band_count[band];
    if (own < 0) fail(status);  // only a broken union-find removes more roots than there were
    if (band == n_bands - 1) *n_components = sum + max(own, 0);
  }
  return sum;
}

__global__ __launch_bounds__(kBandThreads) void number_wide_kernel(
    int W, int H, int64_t frame_px, Tiles T, const uint32_t *tile_bits,
    const uint32_t *rec_roots, int32_t *label, const int32_t *band_count, int direct,
    int32_t n_bands, int32_t *n_components, Comp *comp, int32_t max_components,
    uint32_t *status) {
  __shared__ int s_wave[kBandThreads / 64];
  const int band = blockIdx.x;
  const BandPart p = band_part(T, H, band);
  int32_t *lf = label + static_cast<int64_t>(p.f) * frame_px;
  const uint32_t *band_bits = tile_bits + static_cast<int64_t>(band) * T.wpb;
  // a thread's tiles fit one batch for frames up to 8 * kBandBatch tiles wide: its
  // components are then kept in registers between the count and the numbering
  const bool one = (T.tiles_x + 7) / 8 <= kBandBatch;
  uint32_t comps[kBandBatch];
  int cnt = 0;
  if (p.rows_in)
    for (int b0 = p.tx_lo; b0 < p.tx_hi; b0 += kBandBatch)
      cnt += batch_roots(W, band_bits, rec_roots, lf, p.base, p.y, b0, p.tx_hi, p.rr, comps);
  int total;
  const int start = band_start(band_count, band, n_bands, direct, n_components, status);
  int id = start + block_exclusive<kBandThreads>(cnt, s_wave, &total);
  if (cnt == 0) return;
  if (one) {
    batch_assign(W, lf, p.y, p.tx_lo, comps, comp, p.f, id, max_components);
    return;
  }
  for (int b0 = p.tx_lo; b0 < p.tx_hi; b0 += kBandBatch) {  // again, the loads now in cache
    batch_roots(W, band_bits, rec_roots, lf, p.base, p.y, b0, p.tx_hi, p.rr, comps);
    id = batch_assign(W, lf, p.y, b0, comps, comp, p.f, id, max_components);
  }
}

// Numbering of one band when it is at most kBandTiles tiles wide: its non-empty tiles,
// left to right, are listed in LDS from the bitmap, and the band's (row, listed tile)
// pairs in raster order (row-major over the listed tiles) are dealt out in consecutive
// runs of c = ceil(32 nl / kBandThreads) to the threads, so that thread order is raster
// order and a thread usually has one pair. A pair's candidates are the tile's recorded
// local roots in that row; the label loads of up to kPairBatch pairs are issued together.
__global__ __launch_bounds__(kBandThreads) void number_kernel(
    int W, int64_t frame_px, Tiles T, const uint32_t *tile_bits, const uint32_t *rec_roots,
    int32_t *label, const int32_t *band_count, int direct, int32_t n_bands,
    int32_t *n_components, Comp *comp, int32_t max_components, uint32_t *status) {
  __shared__ int s_tx[kBandTiles];
  __shared__ int s_nl;
  __shared__ int s_wave[kBandThreads / 64];
  const int tid = threadIdx.x, band = blockIdx.x;
  const int f = band / T.tiles_y, ty = band - f * T.tiles_y;
  const int base = band * T.tiles_x;  // tile id of the band's first tile
  int32_t *lf = label + static_cast<int64_t>(f) * frame_px;
  if (tid < 64) {  // the band's bitmap words, one per lane (tiles_x <= kBandTiles: <= 8)
    const uint32_t bits = tid < T.wpb ? tile_bits[static_cast<int64_t>(band) * T.wpb + tid] : 0u;
    const int cnt = __popc(bits);
    int incl = cnt;
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o);
      if (tid >= o) incl += v;
    }
    int at = incl - cnt;
    for (uint32_t m = bits; m != 0; m &= m - 1) s_tx[at++] = tid * 32 + __builtin_ctz(m);
    if (tid == 63) s_nl = incl;
  }
  __syncthreads();
  const int nl = s_nl, n_pairs = kTile * nl;
  const int c = (n_pairs + kBandThreads - 1) / kBandThreads;
  const int p0 = min(tid * c, n_pairs), p1 = min(p0 + c, n_pairs);
  // the components among the candidates of pairs g .. g + kPairBatch - 1 (below p1)
  auto batch = [&](int g, uint32_t comps[kPairBatch], int yx[kPairBatch]) {
    uint32_t cand[kPairBatch];
    int first[kPairBatch];
#pragma unroll
    for (int u = 0; u < kPairBatch; ++u) {
      const int p = g + u, rr = p / max(nl, 1), j = p - rr * max(nl, 1);
      const int tx = p < p1 ? s_tx[j] : 0;
      yx[u] = (ty * kTile + rr) * W + tx * kTile;  // frame index of the pair's row start
      cand[u] = p < p1 ? rec_roots[32 * static_cast<int64_t>(base + tx) + rr] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kPairBatch; ++u)
      first[u] = cand[u] ? lf[yx[u] + __builtin_ctz(cand[u])] : 0;
    int n = 0;
#pragma unroll
    for (int u = 0; u < kPairBatch; ++u) {
      comps[u] = 0;
      if (cand[u] == 0) continue;
      const int P = yx[u] + __builtin_ctz(cand[u]);
      if (first[u] == (P | kRootFlag)) comps[u] = cand[u] & (0u - cand[u]);
      for (uint32_t m = cand[u] & (cand[u] - 1); m != 0; m &= m - 1) {
        const int Q = yx[u] + __builtin_ctz(m);
        if (lf[Q] == (Q | kRootFlag)) comps[u] |= m & (0u - m);
      }
      n += __popc(comps[u]);
    }
    return n;
  };
  auto number = [&](const uint32_t comps[kPairBatch], const int yx[kPairBatch], int id) {
#pragma unroll
    for (int u = 0; u < kPairBatch; ++u)
      for (uint32_t m = comps[u]; m != 0; m &= m - 1) {
        const int P = yx[u] + __builtin_ctz(m);
        if (id >= 0 && id < max_components) {
          comp[id] = Comp{f, P, INT_MAX, P / W, INT_MIN, INT_MIN, 0, 0};
          lf[P] = -(id + 1);
        }
        ++id;
      }
    return id;
  };
  uint32_t comps[kPairBatch];
  int yx[kPairBatch];
  int cnt = 0;
  for (int g = p0; g < p1; g += kPairBatch) cnt += batch(g, comps, yx);
  int total;
  const int start = band_start(band_count, band, n_bands, direct, n_components, status);
  int id = start + block_exclusive<kBandThreads>(cnt, s_wave, &total);
  if (cnt == 0) return;
  if (p1 - p0 <= kPairBatch) {  // one batch: its components are still in registers
    number(comps, yx, id);
    return;
  }
  for (int g = p0; g < p1; g += kPairBatch) {  // again, the loads now in cache
    batch(g, comps, yx);
    id = number(comps, yx, id);
  }
}

// Folds each tile-local component (its entry) into its component's record: up the
// union-find from its local root to the numbered root, then one set of global atomics
// (the record's top row is its root's, set when it was numbered). One wave per listed
// tile, the waves of a grid of resident workgroups walking the list; lane l takes the
// tile's entries l, l + 64, ...
__global__ __launch_bounds__(kEntryThreads) void boxes_kernel(int W, int64_t frame_px, Tiles T,
                                                              const int32_t *tile_list,
                                                              const uint32_t *n_list,
                                                              const uint64_t *entries,
                                                              const int32_t *n_ent,
                                                              const int32_t *label, Comp *comp,
                                                              uint32_t *status) {
  const int n = static_cast<int>(*n_list);
  const int lane = threadIdx.x & 63;
  const int waves = static_cast<int>(gridDim.x) * (kEntryThreads / 64);
  for (int s = (blockIdx.x * kEntryThreads + threadIdx.x) >> 6; s < n; s += waves) {
    const int id = tile_list[s];
    const int ne = n_ent[id];
    const TileAt a = tile_at(T, id);
    const int x0 = a.tx * kTile, y0 = a.ty * kTile;
    const int32_t *lf = label + a.f * frame_px;
    for (int j = lane; j < ne; j += 64) {
      const uint64_t v64 = entries[256 * static_cast<int64_t>(id) + j];
      const int i = static_cast<int>(v64 >> 26) & 1023;
      const int ex0 = static_cast<int>(v64 >> 21) & 31, ex1 = static_cast<int>(v64 >> 16) & 31;
      const int ey1 = static_cast<int>(v64 >> 11) & 31, cnt = static_cast<int>(v64 & 2047);
      // up the union-find over local roots to the numbered root; every link points to a
      // smaller index (unionfind.h), so the walk ends -- a link that does not is reported
      int cur = (y0 + (i >> 5)) * W + x0 + (i & 31);
      int v = lf[cur];
      while (v >= 0) {
        const int nx = v & kIndex;
        if (nx == cur) break;
        if (nx > cur) {
          fail(status);
          break;
        }
        cur = nx;
        v = lf[cur];
      }
      if (v >= 0) continue;  // a component past max_components (or a broken link): not measured
      Comp *c = comp + (-v - 1);
      atomicMin(&c->x0, x0 + ex0);
      atomicMax(&c->x1, x0 + ex1);
      atomicMax(&c->y1, y0 + ey1);
      atomicAdd(&c->area, cnt);
    }
  }
}

// Components of at least min_area pixels, in number order: workgroup k (in ticket order)
// takes kFilterBlock components, kPer per thread, places its kept ones with a block-wide
// scan and a decoupled look-back, and writes them as rows. Components are numbered frame
// by frame, so frame f's first row is the compacted position of the first component
// numbered in a frame >= f: the thread holding component c writes frame_begin for the
// frames after component c - 1's up to its own, and the last component's thread for the
// frames after its own.
__global__ __launch_bounds__(kFilterThreads) void filter_kernel(
    const Comp *comp, int32_t *n_components, int32_t max_components, int32_t min_area,
    tg_roi *rois, int32_t *areas, int32_t max_rois, int32_t n_frames, int32_t *frame_begin,
    uint64_t *words, uint64_t *state, int32_t *n_rois) {
  __shared__ int s_blk, s_base;
  __shared__ int s_wave[kFilterThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // A failure of an earlier pass (a union-find link that broke the invariant, or a
  // look-back that could not complete) makes the call report TG_E_INTERNAL, no RoIs.
  const uint32_t status = __hip_atomic_load(reinterpret_cast<const uint32_t *>(words + 2),
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (status != 0 || *n_components < 0) {
    for (int64_t f = blockIdx.x * static_cast<int64_t>(kFilterThreads) + tid; f <= n_frames;
         f += static_cast<int64_t>(gridDim.x) * kFilterThreads)
      frame_begin[f] = 0;
    if (blockIdx.x == 0 && tid == 0) {
      *n_rois = TG_E_INTERNAL;
      *n_components = TG_E_INTERNAL;
    }
    return;
  }
  // The grid is sized for max_components; only the first max(1, ceil(n / kFilterBlock))
  // workgroups take a ticket, so the ticket counter sees no more atomics than there are
  // blocks of components (at least one workgroup runs, to write n_rois when n == 0).
  const int n = min(*n_components, max_components);
  const int need = n > 0 ? (n + kFilterBlock - 1) / kFilterBlock : 1;
  if (static_cast<int>(blockIdx.x) >= need) return;
  if (tid == 0)
    s_blk = static_cast<int>(__hip_atomic_fetch_add(reinterpret_cast<uint32_t *>(words + 1), 1u,
                                                    __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  __syncthreads();
  const int blk = s_blk;  // < need: exactly `need` workgroups take tickets
  const int start = blk * kFilterBlock;

  constexpr int kPer = kFilterBlock / kFilterThreads;
  bool keep[kPer];
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int id = start + tid * kPer + k;
    keep[k] = id < n && comp[id].area >= min_area;
    cnt += keep[k];
  }
  int incl = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kFilterThreads / 64; ++w) {
    if (w < wave) before += s_wave[w];
    total += s_wave[w];
  }
  if (wave == 0) {
    bool failed;
    const int prefix = tg_detail::lookback_prefix(state, blk, total, &failed);
    if (lane == 0) {
      s_base = prefix;
      if ((start < n && n <= start + kFilterBlock) || n == 0)
        *n_rois = failed ? TG_E_INTERNAL : prefix + total;
    }
  }
  __syncthreads();
  if (n == 0) {  // no components: every frame begins at row 0
    for (int f = tid; f <= n_frames; f += kFilterThreads) frame_begin[f] = 0;
    return;
  }
  int k_out = s_base + before + incl - cnt;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int id = start + tid * kPer + k;
    if (id >= n) break;
    const Comp c = comp[id];
    for (int f = id > 0 ? comp[id - 1].frame + 1 : 0; f <= c.frame; ++f) frame_begin[f] = k_out;
    if (keep[k]) {
      if (k_out < max_rois) {
        rois[k_out] = tg_roi{c.frame, c.x0, c.y0, c.x1 - c.x0 + 1, c.y1 - c.y0 + 1};
        if (areas) areas[k_out] = c.area;
      }
      ++k_out;
    }
    if (id == n - 1)
      for (int f = c.frame + 1; f <= n_frames; ++f) frame_begin[f] = k_out;
  }
}

__global__ void empty_kernel(int32_t *n_rois, int32_t *n_components, int32_t *frame_begin) {
  *n_rois = 0;
  *n_components = 0;
  frame_begin[0] = 0;
}

// Workgroups of `kernel` (`threads` each) resident on the current device at once, at
// least 1: the grid of a pass that walks a list, so that no workgroup waits for a slot
// while others walk their share. Asked of the runtime once per device and kernel.
int resident_groups(const void *kernel, int threads) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return kListGroups;
  static std::mutex mu;
  static std::map<std::tuple<int, const void *, int>, int> known;
  const auto key = std::make_tuple(dev, kernel, threads);
  {
    std::lock_guard<std::mutex> lock(mu);
    const auto it = known.find(key);
    if (it != known.end()) return it->second;
  }
  int cus = 0, per = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, 0) != hipSuccess)
    return kListGroups;
  const int groups = std::max(1, cus * per);
  std::lock_guard<std::mutex> lock(mu);
  known[key] = groups;
  return groups;
}

Tiles tiles_of(int32_t n_frames, int32_t width, int32_t height) {
  Tiles T;
  T.tiles_x = (width + kTile - 1) / kTile;
  T.tiles_y = (height + kTile - 1) / kTile;
  T.wpb = (T.tiles_x + 31) / 32;
  T.n = int64_t(n_frames) * T.tiles_x * T.tiles_y;
  return T;
}

bool sizes_ok(int32_t n_frames, int32_t width, int32_t height, int32_t max_components) {
  if (n_frames < 0 || n_frames > 65535 || width < 1 || height < 1 || max_components < 1)
    return false;
  if (int64_t(width) * height >= (int64_t(1) << 30)) return false;  // the label flag bit
  if ((int64_t(height) + kTile - 1) / kTile > 65535) return false;
  const Tiles T = tiles_of(n_frames, width, height);
  if (T.n >= (int64_t(1) << 28)) return false;  // tile slots fit 28 bits of an entry
  return true;
}

}  // namespace

extern "C" size_t tg_mask_rois_workspace_bytes(int32_t n_frames, int32_t width, int32_t height,
                                               int32_t max_components) {
  if (!sizes_ok(n_frames, width, height, max_components)) return 0;
  const Tiles T = tiles_of(n_frames, width, height);
  const int64_t n_bands = int64_t(n_frames) * T.tiles_y;
  return layout(nullptr, int64_t(n_frames) * width * height, n_bands, T.n, n_bands * T.wpb,
                max_components)
      .bytes;
}

extern "C" int tg_mask_rois(const tg_mask_rois_args *a, void *stream) {
  if (!a || !sizes_ok(a->n_frames, a->width, a->height, a->max_components) || a->max_rois < 0 ||
      !a->frame_begin || !a->n_rois || !a->n_components)
    return TG_E_INVAL;
  if (a->n_frames > 0 && !a->mask) return TG_E_INVAL;
  if (a->max_rois > 0 && !a->rois) return TG_E_INVAL;
  const int64_t frame_px = int64_t(a->width) * a->height, n_px = a->n_frames * frame_px;
  const Tiles T = tiles_of(a->n_frames, a->width, a->height);
  const int64_t n_bands = int64_t(a->n_frames) * T.tiles_y;
  const Layout L = layout(a->workspace, n_px, n_bands, T.n, n_bands * T.wpb, a->max_components);
  if (!a->workspace || a->workspace_bytes < L.bytes ||
      reinterpret_cast<uintptr_t>(a->workspace) % 16 != 0)
    return TG_E_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int W = a->width, H = a->height;
  const dim3 scan_groups(static_cast<uint32_t>(2 * T.wpb),
                         static_cast<uint32_t>(T.tiles_y), static_cast<uint32_t>(a->n_frames));
  const dim3 local_groups(static_cast<uint32_t>(std::min<int64_t>(
      T.n, resident_groups(reinterpret_cast<const void *>(local_kernel), kLocalThreads))));
  const dim3 border_groups(static_cast<uint32_t>(std::min<int64_t>(
      (4 * T.n + kBorderThreads - 1) / kBorderThreads,
      resident_groups(reinterpret_cast<const void *>(merge_kernel), kBorderThreads))));
  const dim3 entry_groups(static_cast<uint32_t>(std::min<int64_t>(
      (64 * T.n + kEntryThreads - 1) / kEntryThreads,
      resident_groups(reinterpret_cast<const void *>(boxes_kernel), kEntryThreads))));
  // dword mask reads need every row start dword-aligned; 16-byte reads need the mask
  // itself 16-byte aligned (and, for whole rows, rows a multiple of 16 bytes)
  const uintptr_t mp = reinterpret_cast<uintptr_t>(a->mask);
  const bool word = mp % 4 == 0 && W % 4 == 0, vec = mp % 16 == 0;
  const int64_t n_filter = (a->max_components + kFilterBlock - 1) / kFilterBlock;

  if (n_px == 0) {  // no frames: no components, no rows
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(1), 0, s, a->n_rois, a->n_components,
                       a->frame_begin);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  uint32_t *status = reinterpret_cast<uint32_t *>(L.words + 2);
  uint32_t *n_list = reinterpret_cast<uint32_t *>(L.words + 3);
  if (vec && W % 16 == 0)
    hipLaunchKernelGGL(scan_kernel<2>, scan_groups, dim3(kScanThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_bits, L.rec_fg, L.words, L.n_words);
  else if (word)
    hipLaunchKernelGGL(scan_kernel<1>, scan_groups, dim3(kScanThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_bits, L.rec_fg, L.words, L.n_words);
  else
    hipLaunchKernelGGL(scan_kernel<0>, scan_groups, dim3(kScanThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_bits, L.rec_fg, L.words, L.n_words);
  const int64_t n_bit_words = n_bands * T.wpb, n_chunks = list_chunks(n_bit_words);
  hipLaunchKernelGGL(list_kernel, dim3(static_cast<uint32_t>(n_chunks)), dim3(kListThreads), 0,
                     s, L.tile_bits, n_bit_words, T, L.tile_list, L.words, L.list_state,
                     static_cast<int32_t>(n_chunks), n_list, status);
  hipLaunchKernelGGL(local_kernel, local_groups, dim3(kLocalThreads), 0, s, W, frame_px, T,
                     L.tile_list, n_list, L.rec_fg, L.rec_roots, L.rec_border, L.entries,
                     L.n_ent, L.label, L.band_first, status);
  hipLaunchKernelGGL(merge_kernel, border_groups, dim3(kBorderThreads), 0, s, W, frame_px, T,
                     L.tile_bits, L.tile_list, n_list, L.rec_fg, L.rec_border, L.label,
                     L.band_first, status);
  const int direct = n_bands <= kDirectBands;
  if (!direct)
    hipLaunchKernelGGL(band_scan_kernel, dim3(1), dim3(kBandScanThreads), 0, s, L.band_first,
                       n_bands, a->n_components, status);
  const dim3 bands(static_cast<uint32_t>(n_bands));
  const int32_t nb = static_cast<int32_t>(n_bands);
  if (T.tiles_x <= kBandTiles)
    hipLaunchKernelGGL(number_kernel, bands, dim3(kBandThreads), 0, s, W, frame_px, T,
                       L.tile_bits, L.rec_roots, L.label, L.band_first, direct, nb,
                       a->n_components, L.comp, a->max_components, status);
  else
    hipLaunchKernelGGL(number_wide_kernel, bands, dim3(kBandThreads), 0, s, W, H, frame_px, T,
                       L.tile_bits, L.rec_roots, L.label, L.band_first, direct, nb,
                       a->n_components, L.comp, a->max_components, status);
  hipLaunchKernelGGL(boxes_kernel, entry_groups, dim3(kEntryThreads), 0, s, W, frame_px, T,
                     L.tile_list, n_list, L.entries, L.n_ent, L.label, L.comp, status);
  hipLaunchKernelGGL(filter_kernel, dim3(static_cast<uint32_t>(n_filter)), dim3(kFilterThreads),
                     0, s, L.comp, a->n_components, a->max_components, a->min_area, a->rois,
                     a->areas, a->max_rois, a->n_frames, a->frame_begin, L.words,
                     L.filter_state, a->n_rois);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
