// tg_mask_rois: RoIs from a foreground mask, as the bounding boxes of 8-connected
// components (the paper cuts its RoIs from the background model's foreground,
// Sec. III-A, step 1).
//
// Connected components by union-find with atomic-min linking (a root always points to
// the smallest index of its set, so every set ends rooted at its first pixel in raster
// order) -- the GPU union-find labelling of D. P. Playne and K. A. Hawick (IEEE TPDS 29(6),
// 2018), tile-local first and merged along tile borders as in the block-based labelling of
// S. Allegretti, F. Bolelli and C. Grana (IEEE TPDS 31(2), 2020) -- in eight launches on
// the caller's stream. Foreground masks are sparse, so only one pass reads every mask
// byte; the others visit the 32x32 tiles that hold foreground.
//  1. clear:  zeroes the tickets, counters, look-back words and the tile bitmap.
//  2. scan:   one 256-thread workgroup per 16 tiles side by side streams the mask (16-byte
//             loads where it can), sets a bit per tile with foreground and appends those
//             tiles to a list.
//  3. local:  a fixed grid walks the list: each tile is labelled in LDS and every
//             foreground pixel gets the frame index of its tile-local root.
//  4. merge:  per listed tile, four 16-pixel items (its top row in two halves, its left
//             column in two halves) join each foreground pixel with its foreground
//             neighbours across the border, with global atomics on the label array; an
//             item whose neighbouring tiles are all empty is skipped. Every 8-neighbour
//             pair across a tile border is seen from the tile below or to the right of it.
//  5. roots:  65536-pixel raster spans in ticket order (each thread's 256 mask bytes as
//             sixteen 16-byte loads, skipping 32-pixel words of empty tiles when rows are
//             a multiple of 32 pixels) find the tile-local roots still their own parent
//             (the components), number them in raster order with a decoupled look-back,
//             initialise each component's record and mark the root with its number.
//  6. boxes:  the grid walks the list again: each tile's local components, read off the
//             labels the local pass left, fold their pixels' extent and count in LDS; each
//             local component then follows the union-find to its component number and
//             folds its totals into the record with global atomics.
//  7. filter: components of at least min_area pixels, compacted in number order with a
//             look-back, written as tg_roi rows.
//  8. begin:  frame_begin by binary search over the kept rows' frames.
// Every union-find walk checks the invariant it relies on (unionfind.h); a walk that meets a
// link that does not point to a smaller index ends, sets the workspace's status word, and
// the call reports *n_rois = *n_components = TG_E_INTERNAL instead of RoIs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>

#include "lookback.h"
#include "tg.h"
#include "unionfind.h"

namespace {

constexpr int kTile = 32;
constexpr int kTileThreads = 256;  // 8 threads per tile row, 4 pixels each
constexpr int kScanTiles = 16;     // tiles side by side per workgroup of the scan pass
constexpr int kScanThreads = 256;  // 8 threads per row of 16 tiles, 64 pixels each
constexpr int kListGroups = 2048;  // workgroups walking the list of non-empty tiles
constexpr int kBorderThreads = 256;
// Labels: a foreground pixel's word holds its tile-local root (a frame index) once the
// local pass is done, and never changes afterwards unless the pixel is a tile-local root.
// A tile-local root's word holds kRootFlag | its parent in the union-find over roots
// (itself at first), and becomes -(component + 1) once it is numbered. Frames have fewer
// than 2^30 pixels, so the flag bit is free.
constexpr int32_t kRootFlag = 1 << 30;
constexpr int32_t kIndex = kRootFlag - 1;
constexpr int kSpan = 65536;       // pixels per workgroup of the roots pass
constexpr int kSpanThreads = 256;  // 256 pixels per thread: sixteen 16-byte loads
constexpr int kSpanPix = kSpan / kSpanThreads;
constexpr int kSpanWords = kSpanPix / 32;  // foreground / root bit words per thread
constexpr int kFilterBlock = 1024;  // components per workgroup of the filter pass
constexpr int kFilterThreads = 256;

struct Comp {
  int32_t frame, root, x0, y0, x1, y1, area, unused;
};
static_assert(sizeof(Comp) == 32, "component record is 32 bytes");

// Tiles of all frames, numbered frame by frame, tile rows top to bottom, tiles left to
// right: tile (f, ty, tx) is (f * tiles_y + ty) * tiles_x + tx.
struct Tiles {
  int tiles_x, tiles_y;
  int64_t n;
};

struct Layout {
  // [0]: roots ticket, [1]: filter ticket, [2]: status, [3]: non-empty tiles listed, then
  // the look-back words of the roots and filter passes, then the tile bitmap (bit t of
  // 32-bit word t / 32: tile t holds foreground); all cleared by the first launch
  uint64_t *words;
  uint64_t *root_state, *filter_state;
  uint32_t *tile_bits;
  int32_t *tile_list;  // ids of the non-empty tiles, in no particular order
  Comp *comp;
  int32_t *kept_frame;
  int32_t *label;
  int64_t n_words;
  size_t bytes;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

Layout layout(void *base, int64_t n_px, int64_t n_tiles, int32_t max_components) {
  Layout L;
  const int64_t n_spans = (n_px + kSpan - 1) / kSpan;
  const int64_t n_filter = (max_components + kFilterBlock - 1) / kFilterBlock;
  const int64_t bit_words64 = (n_tiles + 63) / 64;
  L.n_words = 4 + n_spans + n_filter + bit_words64;
  const size_t o_list = round_up(8 * static_cast<size_t>(L.n_words), 256);
  const size_t o_comp = round_up(o_list + 4 * static_cast<size_t>(n_tiles), 256);
  const size_t o_kept = round_up(o_comp + sizeof(Comp) * static_cast<size_t>(max_components), 256);
  const size_t o_label = round_up(o_kept + 4 * static_cast<size_t>(max_components), 256);
  L.bytes = round_up(o_label + 4 * static_cast<size_t>(n_px), 256);
  char *b = static_cast<char *>(base);
  L.words = b ? reinterpret_cast<uint64_t *>(b) : nullptr;
  L.root_state = b ? L.words + 4 : nullptr;
  L.filter_state = b ? L.root_state + n_spans : nullptr;
  L.tile_bits = b ? reinterpret_cast<uint32_t *>(L.filter_state + n_filter) : nullptr;
  L.tile_list = b ? reinterpret_cast<int32_t *>(b + o_list) : nullptr;
  L.comp = b ? reinterpret_cast<Comp *>(b + o_comp) : nullptr;
  L.kept_frame = b ? reinterpret_cast<int32_t *>(b + o_kept) : nullptr;
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

// Union-find over the flagged words of tile-local roots in global memory.
struct RootLabels {
  int32_t *L;
  __device__ int parent(int i) const { return g_load(&L[i]) & kIndex; }
  __device__ int link(int i, int p) {
    return __hip_atomic_fetch_min(&L[i], p | kRootFlag, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT) & kIndex;
  }
};

// Records in the workspace's status word that a union-find walk met a link that breaks
// the invariant (tg_mask_rois then reports TG_E_INTERNAL instead of RoIs).
__device__ __forceinline__ void fail(uint32_t *status) {
  __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Foreground bits of this thread's 4 pixels of the tile at column tx0, row ty0: thread t
// holds row t / 8, columns 4 (t % 8) .. + 3, read from addresses clamped into the frame
// (pixels outside it are masked off): one dword when every row start is dword-aligned
// (kWord), else four bytes.
template <bool kWord>
__device__ __forceinline__ uint32_t load_tile_fg(const uint8_t *mf, int W, int H, int tx0,
                                                 int ty0) {
  const int t = threadIdx.x, r = t >> 3, c0 = (t & 7) * 4, y = ty0 + r;
  const uint8_t *row = mf + static_cast<int64_t>(min(y, H - 1)) * W;
  const int x0 = tx0 + c0;
  uint32_t raw[4];
  if (kWord) {
    raw[0] = *reinterpret_cast<const uint32_t *>(row + min(x0, W - 4));
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) raw[k] = row[min(x0 + k, W - 1)];
  }
  uint32_t bits = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t v = kWord ? (raw[0] >> (8 * k)) & 0xFFu : raw[k];
    bits |= (v != 0 && x0 + k < W) ? 1u << k : 0u;
  }
  return y < H ? bits : 0u;
}

__device__ __forceinline__ bool tile_set(const uint32_t *bits, int t) {
  return (bits[t >> 5] >> (t & 31)) & 1u;
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

// Labels one 32x32 tile in LDS (L: 1024 ints, -1 for background, else a parent index
// within the tile; rows: 32 words of scratch) from this thread's foreground bits
// (load_tile_fg). Returns false, uniformly, when the tile has no foreground. Starts with a
// barrier, so the caller's previous use of L (and of any other LDS) is over before L is
// rewritten.
//
// A pixel starts linked to the first pixel of its horizontal run among the thread's four,
// so runs inside a thread cost no union. Each pixel p then joins the neighbours that a
// raster-scan decision tree for 8-connectivity requires -- with a the upper-left, b the
// upper, c the upper-right and d the left neighbour: b alone when b is foreground (a and c
// touch b, and d touches b diagonally, through their own joins); otherwise d (when it lies
// in another thread) and c; otherwise a and c -- and skips b when the previous pixel of its
// run has already joined a, which touches b. That reaches the same sets as joining every
// foreground neighbour, with about one union per run instead of four per pixel.
__device__ __forceinline__ bool label_tile(uint32_t fg, int *L, uint32_t *rows,
                                           uint32_t *status) {
  const int t = threadIdx.x, r = t >> 3, c0 = (t & 7) * 4;
  if (!__syncthreads_or(fg != 0)) return false;
  if (__syncthreads_and(fg == 0xFu)) {  // a solid tile is one set rooted at its pixel 0
#pragma unroll
    for (int k = 0; k < 4; ++k) L[r * kTile + c0 + k] = 0;
    __syncthreads();
    return true;
  }
  // this row's foreground as one word (the 8 threads of a row are 8 consecutive lanes)
  uint32_t row = fg << c0;
  row |= __shfl_xor(row, 1);
  row |= __shfl_xor(row, 2);
  row |= __shfl_xor(row, 4);
  if ((t & 7) == 0) rows[r] = row;
  int start = -1;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int i = r * kTile + c0 + k;
    start = (fg >> k & 1u) ? (start >= 0 ? start : i) : -1;
    L[i] = start;
  }
  __syncthreads();
  const uint32_t up = r > 0 ? rows[r - 1] : 0u;
  LdsLabels m{L};
  bool ok = true;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (!(fg >> k & 1u)) continue;
    const int c = c0 + k, i = r * kTile + c;
    const bool a = c > 0 && (up >> (c - 1) & 1u), b = up >> c & 1u;
    const bool cc = c + 1 < kTile && (up >> (c + 1) & 1u);
    const bool d = c > 0 && (row >> (c - 1) & 1u);
    if (b) {
      if (!(k > 0 && d && a)) ok &= tg_detail::uf_unite(m, i, i - kTile);
    } else if (d) {
      if (k == 0) ok &= tg_detail::uf_unite(m, i, i - 1);
      if (cc) ok &= tg_detail::uf_unite(m, i, i - kTile + 1);
    } else {
      if (a) ok &= tg_detail::uf_unite(m, i, i - kTile - 1);
      if (cc) ok &= tg_detail::uf_unite(m, i, i - kTile + 1);
    }
  }
  if (!ok) fail(status);
  __syncthreads();
  return true;
}

// ---- kernels ------------------------------------------------------------------------

__global__ void clear_kernel(uint64_t *words, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) words[i] = 0;
}

// Which tiles hold foreground: one workgroup per 16 tiles side by side (a 512 x 32 block
// of one frame), thread t reading row t / 8 of the block, pixels 64 (t % 8) .. + 63 (the
// row segments of two tiles) with 16-byte loads (kMode 2: mask 16-byte aligned and rows a
// multiple of 16 bytes), dwords (kMode 1) or bytes (kMode 0), all issued before any is
// used. A block with foreground sets its tiles' bits and appends their ids to the list.
template <int kMode>
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const uint8_t *mask, int W, int H,
                                                            int64_t frame_px, Tiles T,
                                                            uint32_t *tile_bits,
                                                            int32_t *tile_list,
                                                            uint32_t *n_list) {
  __shared__ uint32_t s_bits;
  const int t = threadIdx.x, r = t >> 3, q = t & 7;
  const int64_t f = blockIdx.z;
  const int tx0 = blockIdx.x * kScanTiles, ty = blockIdx.y;
  const int y = ty * kTile + r, x = tx0 * kTile + 64 * q;
  if (t == 0) s_bits = 0;
  bool nz0 = false, nz1 = false;  // pixels x .. x + 31, x + 32 .. x + 63 of row y
  if (y < H && x < W) {
    const uint8_t *row = mask + f * frame_px + static_cast<int64_t>(y) * W;
    if (kMode == 2) {  // rows a multiple of 16 bytes: a chunk is wholly inside or outside
      typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
      u32x4 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        v[i] = x + 16 * i < W ? *reinterpret_cast<const u32x4 *>(row + x + 16 * i) : u32x4{0, 0, 0, 0};
      const u32x4 a = v[0] | v[1], b = v[2] | v[3];
      nz0 = (a.x | a.y | a.z | a.w) != 0;
      nz1 = (b.x | b.y | b.z | b.w) != 0;
    } else if (kMode == 1) {  // rows a multiple of 4 bytes
      uint32_t v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i)
        v[i] = x + 4 * i < W ? *reinterpret_cast<const uint32_t *>(row + x + 4 * i) : 0u;
      uint32_t a = 0, b = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        a |= v[i];
        b |= v[i + 8];
      }
      nz0 = a != 0;
      nz1 = b != 0;
    } else {
      uint32_t a = 0, b = 0;
#pragma unroll 8
      for (int i = 0; i < 32; ++i) {
        a |= x + i < W ? row[x + i] : 0u;
        b |= x + 32 + i < W ? row[x + 32 + i] : 0u;
      }
      nz0 = a != 0;
      nz1 = b != 0;
    }
  }
  // lane l of a wave is row l / 8, tile pair l % 8: a tile holds foreground when any of
  // the wave's rows does
  const uint64_t b0 = __ballot(nz0), b1 = __ballot(nz1);
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
  if (m == 0 || t != 0) return;
  const int id0 = static_cast<int>((f * T.tiles_y + ty) * T.tiles_x + tx0);
  const int sh = id0 & 31;
  atomicOr(&tile_bits[id0 >> 5], m << sh);
  if (sh > 16 && (m >> (32 - sh)) != 0)  // only words that hold existing tiles
    atomicOr(&tile_bits[(id0 >> 5) + 1], m >> (32 - sh));
  int at = static_cast<int>(atomicAdd(n_list, static_cast<uint32_t>(__popc(m))));
  for (uint32_t k = m; k != 0; k &= k - 1) tile_list[at++] = id0 + __builtin_ctz(k);
}

// Labels the listed tiles, a grid of kListGroups workgroups walking the list: for each
// foreground pixel, the frame index of its tile-local root (flagged on the roots).
template <bool kWord>
__global__ __launch_bounds__(kTileThreads) void local_kernel(const uint8_t *mask, int W, int H,
                                                             int64_t frame_px, Tiles T,
                                                             const int32_t *tile_list,
                                                             const uint32_t *n_list,
                                                             int32_t *label, uint32_t *status) {
  __shared__ int L[kTile * kTile];
  __shared__ uint32_t rows[kTile];
  const int n = static_cast<int>(*n_list);
  const int t = threadIdx.x, r = t >> 3, c0 = (t & 7) * 4;
  for (int it = blockIdx.x; it < n; it += gridDim.x) {
    const TileAt a = tile_at(T, tile_list[it]);
    const int tx0 = a.tx * kTile, ty0 = a.ty * kTile;
    const uint32_t fg = load_tile_fg<kWord>(mask + a.f * frame_px, W, H, tx0, ty0);
    if (!label_tile(fg, L, rows, status)) continue;  // (a listed tile always holds foreground)
    int32_t *lf = label + a.f * frame_px;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (!(fg >> k & 1u)) continue;
      const int i = r * kTile + c0 + k;
      LdsLabels m{L};
      int root = tg_detail::uf_find(m, i);
      if (root < 0) {
        fail(status);
        root = i;
      }
      const int gr = (ty0 + (root >> 5)) * W + tx0 + (root & (kTile - 1));
      lf[static_cast<int64_t>(ty0 + r) * W + tx0 + c0 + k] = root == i ? gr | kRootFlag : gr;
    }
  }
}

// Joins the foreground pixels of a 16-pixel run along a tile border (bits of `fg`) with
// their foreground neighbours across it. Along the border the run covers coordinates
// start .. start + 15 of [0, lim); pixel k is frame index own0 + k ostep, and the 18
// pixels across the border at coordinates start - 1 .. start + 16 are nb0 + k' nstep.
// Neighbour bytes and all labels are read first (addresses clamped into the frame), then
// each pixel joins neighbours k, k + 1, k + 2 through their current labels (members of
// their sets), skipping a pair equal to the one just joined: along a border most repeat.
__device__ __forceinline__ void join_border(const uint8_t *mf, int32_t *lf, uint32_t fg, int own0,
                                            int ostep, int nb0, int nstep, int start, int lim,
                                            uint32_t *status) {
  if (fg == 0) return;
  uint32_t m[18];
  int32_t ln[18], lo[16];
#pragma unroll
  for (int k = 0; k < 18; ++k) {
    const int c = min(max(start - 1 + k, 0), lim - 1);
    const int idx = nb0 + (c - (start - 1)) * nstep;
    m[k] = mf[idx];
    ln[k] = g_load(&lf[idx]) & kIndex;
  }
#pragma unroll
  for (int k = 0; k < 16; ++k)
    lo[k] = g_load(&lf[own0 + (min(start + k, lim - 1) - start) * ostep]) & kIndex;
  uint32_t nb = 0;
#pragma unroll
  for (int k = 0; k < 18; ++k)
    nb |= (m[k] != 0 && start - 1 + k >= 0 && start - 1 + k < lim) ? 1u << k : 0u;
  int pa = -1, pb = -1;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (!(fg >> k & 1u)) continue;
#pragma unroll
    for (int d = 0; d < 3; ++d) {
      if (!(nb >> (k + d) & 1u)) continue;
      const int a = lo[k], b = ln[k + d];
      if (a == pa && b == pb) continue;
      RootLabels m{lf};
      if (!tg_detail::uf_unite(m, a, b)) fail(status);
      pa = a;
      pb = b;
    }
  }
}

// Four items per listed tile, walked by a grid of kListGroups workgroups: its top row in
// two halves of 16 pixels against the row above (one 16-byte load where the row is
// 16-byte aligned), then its left column in two halves against the column to its left.
// Every 8-neighbour pair across a tile border is seen from the tile below or to the right
// of it, and needs foreground on both sides: an item runs only when its own tile is listed
// and one of the three tiles holding its neighbours is non-empty.
__global__ __launch_bounds__(kBorderThreads) void merge_kernel(const uint8_t *mask, int W, int H,
                                                               int64_t frame_px, Tiles T,
                                                               const uint32_t *tile_bits,
                                                               const int32_t *tile_list,
                                                               const uint32_t *n_list, bool vec,
                                                               int32_t *label, uint32_t *status) {
  const int n4 = 4 * static_cast<int>(*n_list);
  for (int i = blockIdx.x * kBorderThreads + threadIdx.x; i < n4;
       i += gridDim.x * kBorderThreads) {
    const int id = tile_list[i >> 2], k = i & 3;
    const TileAt a = tile_at(T, id);
    const uint8_t *mf = mask + a.f * frame_px;
    int32_t *lf = label + a.f * frame_px;
    uint32_t fg = 0;
    if (k < 2) {  // top row of the tile against the row above
      if (a.ty == 0) continue;
      const int x0 = a.tx * kTile + 16 * k, y = a.ty * kTile;
      const int up = id - T.tiles_x;
      if (x0 >= W || !(tile_set(tile_bits, up) || (a.tx > 0 && tile_set(tile_bits, up - 1)) ||
                       (a.tx + 1 < T.tiles_x && tile_set(tile_bits, up + 1))))
        continue;
      const uint8_t *p = mf + y * W + x0;
      if (vec && x0 + 16 <= W) {
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = *reinterpret_cast<const u32x4 *>(p);
#pragma unroll
        for (int j = 0; j < 16; ++j) fg |= ((v[j >> 2] >> (8 * (j & 3))) & 0xFFu) ? 1u << j : 0u;
      } else {
        const uint8_t *rowp = mf + y * W;
        uint32_t v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = rowp[min(x0 + j, W - 1)];
#pragma unroll
        for (int j = 0; j < 16; ++j) fg |= (v[j] != 0 && x0 + j < W) ? 1u << j : 0u;
      }
      join_border(mf, lf, fg, y * W + x0, 1, (y - 1) * W + x0 - 1, 1, x0, W, status);
    } else {  // left column of the tile against the column to its left
      if (a.tx == 0) continue;
      const int y0 = a.ty * kTile + 16 * (k - 2), x = a.tx * kTile;
      const int left = id - 1;
      if (y0 >= H ||
          !(tile_set(tile_bits, left) || (a.ty > 0 && tile_set(tile_bits, left - T.tiles_x)) ||
            (a.ty + 1 < T.tiles_y && tile_set(tile_bits, left + T.tiles_x))))
        continue;
      uint32_t v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) v[j] = mf[min(y0 + j, H - 1) * W + x];
#pragma unroll
      for (int j = 0; j < 16; ++j) fg |= (v[j] != 0 && y0 + j < H) ? 1u << j : 0u;
      join_border(mf, lf, fg, y0 * W + x, W, (y0 - 1) * W + x - 1, W, y0, H, status);
    }
  }
}

__global__ __launch_bounds__(kSpanThreads) void roots_kernel(
    const uint8_t *mask, bool vec, int64_t n_px, int64_t frame_px, int64_t n_spans, int W,
    Tiles T, const uint32_t *tile_bits, bool skip, int32_t *label, Comp *comp,
    int32_t max_components, uint64_t *words, uint64_t *state, int32_t *n_components) {
  __shared__ int s_span, s_base;
  __shared__ int s_wave[kSpanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0)
    s_span = static_cast<int>(__hip_atomic_fetch_add(reinterpret_cast<uint32_t *>(words), 1u,
                                                     __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT));
  __syncthreads();
  const int64_t span = s_span;
  const int64_t p0 = span * kSpan + static_cast<int64_t>(tid) * kSpanPix;

  // Which of this thread's eight 32-pixel words can hold foreground: with rows a multiple
  // of 32 pixels (`skip`) every word lies in one tile, and only words of non-empty tiles
  // are read; otherwise all are.
  uint32_t need = 0xFFu;
  if (skip && p0 < n_px) {
    need = 0;
    int64_t f = p0 / frame_px, loc = p0 - f * frame_px;
    for (int w = 0; w < kSpanWords && p0 + 32 * w < n_px; ++w) {
      const int l = static_cast<int>(loc), y = l / W, x = l - y * W;
      if (tile_set(tile_bits, static_cast<int>((f * T.tiles_y + (y >> 5)) * T.tiles_x + (x >> 5))))
        need |= 1u << w;
      loc += 32;
      if (loc >= frame_px) {
        loc -= frame_px;
        ++f;
      }
    }
  }
  // Which of this thread's 256 pixels are foreground (16-byte loads when the mask is
  // 16-byte aligned and the bytes are inside it), then which of those are roots.
  uint32_t fgm[kSpanWords] = {};
  if (p0 < n_px && need != 0) {
    if (vec && p0 + kSpanPix <= n_px) {
      typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
      u32x4 v[kSpanPix / 16];
#pragma unroll
      for (int q = 0; q < kSpanPix / 16; ++q)
        v[q] = (need >> (q >> 1)) & 1u ? *reinterpret_cast<const u32x4 *>(mask + p0 + 16 * q)
                                       : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int q = 0; q < kSpanPix / 16; ++q)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          fgm[q >> 1] |= ((v[q][j >> 2] >> (8 * (j & 3))) & 0xFFu) ? 1u << (16 * (q & 1) + j) : 0u;
    } else {
      for (int j = 0; j < kSpanPix; ++j)
        fgm[j >> 5] |= ((need >> (j >> 5)) & 1u && p0 + j < n_px && mask[min(p0 + j, n_px - 1)])
                           ? 1u << (j & 31) : 0u;
    }
  }
  // A foreground pixel is a root when its label is its own frame index, flagged (a
  // tile-local root still its own parent). The 32 labels of a
  // word with any foreground are read as eight 16-byte loads issued together (one round
  // trip per word, not one per pixel); a word that would leave the label array, or frames
  // of under 32 pixels, go pixel by pixel.
  uint32_t roots[kSpanWords] = {};
  int cnt = 0;
#pragma unroll
  for (int w = 0; w < kSpanWords; ++w) {
    if (fgm[w] == 0) continue;
    const int64_t P0 = p0 + 32 * w;
    if (P0 + 32 <= n_px && frame_px >= 32) {
      typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
      i32x4 lv[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) lv[q] = *reinterpret_cast<const i32x4 *>(label + P0 + 4 * q);
      int64_t local = P0 % frame_px;
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        if (local == frame_px) local = 0;
        if ((fgm[w] >> j & 1u) && lv[j >> 2][j & 3] == (static_cast<int32_t>(local) | kRootFlag))
          roots[w] |= 1u << j;
        ++local;
      }
    } else {
      for (uint32_t m = fgm[w]; m != 0; m &= m - 1) {
        const int j = __builtin_ctz(m);
        const int64_t P = P0 + j;
        if (label[P] == (static_cast<int32_t>(P % frame_px) | kRootFlag)) roots[w] |= 1u << j;
      }
    }
    cnt += __popc(roots[w]);
  }

  // Exclusive scan of the counts over the workgroup, then the look-back over spans.
  int incl = cnt;
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o);
    if (lane >= o) incl += v;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kSpanThreads / 64; ++w) {
    if (w < wave) before += s_wave[w];
    total += s_wave[w];
  }
  if (wave == 0) {
    bool failed;
    const int prefix = tg_detail::lookback_prefix(state, static_cast<int>(span), total, &failed);
    if (lane == 0) {
      s_base = prefix;
      if (span == n_spans - 1) *n_components = failed ? TG_E_INTERNAL : prefix + total;
    }
  }
  __syncthreads();

  int id = s_base + before + incl - cnt;
#pragma unroll
  for (int w = 0; w < kSpanWords; ++w) {
    for (uint32_t m = roots[w]; m != 0; m &= m - 1, ++id) {
      if (id >= max_components) continue;
      const int64_t P = p0 + 32 * w + __builtin_ctz(m);
      const int64_t f = P / frame_px;
      comp[id] = Comp{static_cast<int32_t>(f), static_cast<int32_t>(P - f * frame_px), INT_MAX,
                      INT_MAX, INT_MIN, INT_MIN, 0, 0};
      label[P] = -(id + 1);
    }
  }
}

__device__ __forceinline__ int wave_min(int v) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_sum(int v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Folds the listed tiles' pixels into their components' records, a grid of kListGroups
// workgroups walking the list.
template <bool kWord>
__global__ __launch_bounds__(kTileThreads) void boxes_kernel(const uint8_t *mask, int W, int H,
                                                             int64_t frame_px, Tiles T,
                                                             const int32_t *tile_list,
                                                             const uint32_t *n_list,
                                                             const int32_t *label,
                                                             Comp *comp, uint32_t *status) {
  __shared__ int bx0[kTile * kTile], by0[kTile * kTile], bx1[kTile * kTile],
      by1[kTile * kTile], bn[kTile * kTile];
  const int n_tiles = static_cast<int>(*n_list);
  const int t = threadIdx.x, r = t >> 3, c0 = (t & 7) * 4;
  for (int it = blockIdx.x; it < n_tiles; it += gridDim.x) {
    const TileAt a = tile_at(T, tile_list[it]);
    const int tx0 = a.tx * kTile, ty0 = a.ty * kTile, y = ty0 + r;
    const uint32_t fgw = load_tile_fg<kWord>(mask + a.f * frame_px, W, H, tx0, ty0);
    const int32_t *lf = label + a.f * frame_px;
    const int32_t *row = lf + static_cast<int64_t>(min(y, H - 1)) * W;
    // (also the barrier between this tile's use of the LDS sums and the previous one's)
    if (!__syncthreads_or(fgw != 0)) continue;
    // The tile-local components come from the labels the local pass left: a foreground
    // pixel's word is its local root, unless the pixel is a local root itself (flagged or
    // already numbered).
    int32_t lv[4];
    if (kWord) {
      typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
      const i32x4 v = *reinterpret_cast<const i32x4 *>(row + min(tx0 + c0, W - 4));
#pragma unroll
      for (int k = 0; k < 4; ++k) lv[k] = v[k];
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) lv[k] = row[min(tx0 + c0 + k, W - 1)];
    }
    bool fg[4];
    int root[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = r * kTile + c0 + k;
      fg[k] = fgw >> k & 1u;
      root[k] = -1;
      if (fg[k]) {
        const int v = lv[k];
        if (v < 0 || (v & kRootFlag)) {
          root[k] = i;
        } else {
          const int vy = v / W;
          root[k] = (vy - ty0) * kTile + (v - vy * W - tx0);
        }
      }
      if (root[k] == i) {
        bx0[i] = INT_MAX;
        by0[i] = INT_MAX;
        bx1[i] = INT_MIN;
        by1[i] = INT_MIN;
        bn[i] = 0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int x = tx0 + c0 + k;
      // When every foreground lane of the wave is in one local component, reduce across
      // the wave first and fold once.
      const uint64_t fgm = __ballot(fg[k]);
      if (!fgm) continue;
      const int lead = __shfl(root[k], __builtin_ctzll(fgm));
      if (__ballot(fg[k] && root[k] != lead) == 0) {
        const int mx0 = wave_min(fg[k] ? x : INT_MAX), my0 = wave_min(fg[k] ? y : INT_MAX);
        const int mx1 = wave_max(fg[k] ? x : INT_MIN), my1 = wave_max(fg[k] ? y : INT_MIN);
        const int n = wave_sum(fg[k] ? 1 : 0);
        if ((threadIdx.x & 63) == 0) {
          atomicMin(&bx0[lead], mx0);
          atomicMin(&by0[lead], my0);
          atomicMax(&bx1[lead], mx1);
          atomicMax(&by1[lead], my1);
          atomicAdd(&bn[lead], n);
        }
      } else if (fg[k]) {
        atomicMin(&bx0[root[k]], x);
        atomicMin(&by0[root[k]], y);
        atomicMax(&bx1[root[k]], x);
        atomicMax(&by1[root[k]], y);
        atomicAdd(&bn[root[k]], 1);
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = r * kTile + c0 + k;
      if (root[k] != i) continue;
      // up the union-find over local roots to the numbered root; every link points to a
      // smaller index (unionfind.h), so the walk ends -- a link that does not is reported
      int cur = y * W + tx0 + c0 + k;
      int v = lv[k];
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
      atomicMin(&c->x0, bx0[i]);
      atomicMin(&c->y0, by0[i]);
      atomicMax(&c->x1, bx1[i]);
      atomicMax(&c->y1, by1[i]);
      atomicAdd(&c->area, bn[i]);
    }
  }
}

__global__ __launch_bounds__(kFilterThreads) void filter_kernel(
    const Comp *comp, int32_t *n_components, int32_t max_components, int32_t min_area,
    tg_roi *rois, int32_t *areas, int32_t max_rois, int32_t *kept_frame, uint64_t *words,
    uint64_t *state, int32_t *n_rois) {
  __shared__ int s_blk, s_base;
  __shared__ int s_wave[kFilterThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // A failure of an earlier pass (a union-find link that broke the invariant, or a
  // look-back that could not complete) makes the call report TG_E_INTERNAL, no RoIs.
  const uint32_t status = __hip_atomic_load(reinterpret_cast<const uint32_t *>(words + 2),
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (status != 0 || *n_components < 0) {
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
  int k_out = s_base + before + incl - cnt;
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    if (!keep[k]) continue;
    const Comp c = comp[start + tid * kPer + k];
    kept_frame[k_out] = c.frame;
    if (k_out < max_rois) {
      rois[k_out] = tg_roi{c.frame, c.x0, c.y0, c.x1 - c.x0 + 1, c.y1 - c.y0 + 1};
      if (areas) areas[k_out] = c.area;
    }
    ++k_out;
  }
}

__global__ void begin_kernel(const int32_t *kept_frame, const int32_t *n_rois, int32_t n_frames,
                             int32_t *frame_begin) {
  const int f = blockIdx.x * blockDim.x + threadIdx.x;
  if (f > n_frames) return;
  int lo = 0, hi = *n_rois;  // first kept row whose frame is >= f
  while (lo < hi) {
    const int mid = lo + (hi - lo) / 2;
    if (kept_frame[mid] < f)
      lo = mid + 1;
    else
      hi = mid;
  }
  frame_begin[f] = lo;
}

__global__ void empty_kernel(int32_t *n_rois, int32_t *n_components, int32_t *frame_begin) {
  *n_rois = 0;
  *n_components = 0;
  frame_begin[0] = 0;
}

Tiles tiles_of(int32_t n_frames, int32_t width, int32_t height) {
  Tiles T;
  T.tiles_x = (width + kTile - 1) / kTile;
  T.tiles_y = (height + kTile - 1) / kTile;
  T.n = int64_t(n_frames) * T.tiles_x * T.tiles_y;
  return T;
}

bool sizes_ok(int32_t n_frames, int32_t width, int32_t height, int32_t max_components) {
  if (n_frames < 0 || n_frames > 65535 || width < 1 || height < 1 || max_components < 1)
    return false;
  if (int64_t(width) * height >= (int64_t(1) << 30)) return false;  // the label flag bit
  if ((int64_t(height) + kTile - 1) / kTile > 65535) return false;
  const Tiles T = tiles_of(n_frames, width, height);
  if (T.n >= (int64_t(1) << 31)) return false;  // tile ids are int32
  return true;
}

}  // namespace

extern "C" size_t tg_mask_rois_workspace_bytes(int32_t n_frames, int32_t width, int32_t height,
                                               int32_t max_components) {
  if (!sizes_ok(n_frames, width, height, max_components)) return 0;
  return layout(nullptr, int64_t(n_frames) * width * height,
                tiles_of(n_frames, width, height).n, max_components).bytes;
}

extern "C" int tg_mask_rois(const tg_mask_rois_args *a, void *stream) {
  if (!a || !sizes_ok(a->n_frames, a->width, a->height, a->max_components) || a->max_rois < 0 ||
      !a->frame_begin || !a->n_rois || !a->n_components)
    return TG_E_INVAL;
  if (a->n_frames > 0 && !a->mask) return TG_E_INVAL;
  if (a->max_rois > 0 && !a->rois) return TG_E_INVAL;
  const int64_t frame_px = int64_t(a->width) * a->height, n_px = a->n_frames * frame_px;
  const Tiles T = tiles_of(a->n_frames, a->width, a->height);
  const Layout L = layout(a->workspace, n_px, T.n, a->max_components);
  if (!a->workspace || a->workspace_bytes < L.bytes ||
      reinterpret_cast<uintptr_t>(a->workspace) % 16 != 0)
    return TG_E_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int W = a->width, H = a->height;
  const dim3 scan_groups(static_cast<uint32_t>((T.tiles_x + kScanTiles - 1) / kScanTiles),
                         static_cast<uint32_t>(T.tiles_y), static_cast<uint32_t>(a->n_frames));
  const dim3 list_groups(static_cast<uint32_t>(std::min<int64_t>(T.n, kListGroups)));
  const dim3 border_groups(static_cast<uint32_t>(
      std::min<int64_t>((4 * T.n + kBorderThreads - 1) / kBorderThreads, kListGroups)));
  // dword mask reads need every row start dword-aligned; 16-byte reads need the mask
  // itself 16-byte aligned (and, for whole rows, rows a multiple of 16 bytes)
  const uintptr_t mp = reinterpret_cast<uintptr_t>(a->mask);
  const bool word = mp % 4 == 0 && W % 4 == 0, vec = mp % 16 == 0;
  const int64_t n_spans = (n_px + kSpan - 1) / kSpan;
  const int64_t n_filter = (a->max_components + kFilterBlock - 1) / kFilterBlock;

  if (n_px == 0) {  // no frames: no components, no rows
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(1), 0, s, a->n_rois, a->n_components,
                       a->frame_begin);
    return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
  }
  uint32_t *status = reinterpret_cast<uint32_t *>(L.words + 2);
  hipLaunchKernelGGL(clear_kernel, dim3(static_cast<uint32_t>((L.n_words + 255) / 256)),
                     dim3(256), 0, s, L.words, L.n_words);
  uint32_t *n_list = reinterpret_cast<uint32_t *>(L.words + 3);
  if (vec && W % 16 == 0)
    hipLaunchKernelGGL(scan_kernel<2>, scan_groups, dim3(kScanThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_bits, L.tile_list, n_list);
  else if (word)
    hipLaunchKernelGGL(scan_kernel<1>, scan_groups, dim3(kScanThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_bits, L.tile_list, n_list);
  else
    hipLaunchKernelGGL(scan_kernel<0>, scan_groups, dim3(kScanThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_bits, L.tile_list, n_list);
  if (word)
    hipLaunchKernelGGL(local_kernel<true>, list_groups, dim3(kTileThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_list, n_list, L.label, status);
  else
    hipLaunchKernelGGL(local_kernel<false>, list_groups, dim3(kTileThreads), 0, s, a->mask, W,
                       H, frame_px, T, L.tile_list, n_list, L.label, status);
  hipLaunchKernelGGL(merge_kernel, border_groups, dim3(kBorderThreads), 0, s, a->mask, W, H,
                     frame_px, T, L.tile_bits, L.tile_list, n_list, vec && W % 16 == 0, L.label,
                     status);
  hipLaunchKernelGGL(roots_kernel, dim3(static_cast<uint32_t>(n_spans)), dim3(kSpanThreads), 0,
                     s, a->mask, vec, n_px, frame_px, n_spans, W, T, L.tile_bits, W % 32 == 0,
                     L.label, L.comp, a->max_components, L.words, L.root_state,
                     a->n_components);
  if (word)
    hipLaunchKernelGGL(boxes_kernel<true>, list_groups, dim3(kTileThreads), 0, s, a->mask, W, H,
                       frame_px, T, L.tile_list, n_list, L.label, L.comp, status);
  else
    hipLaunchKernelGGL(boxes_kernel<false>, list_groups, dim3(kTileThreads), 0, s, a->mask, W,
                       H, frame_px, T, L.tile_list, n_list, L.label, L.comp, status);
  hipLaunchKernelGGL(filter_kernel, dim3(static_cast<uint32_t>(n_filter)), dim3(kFilterThreads),
                     0, s, L.comp, a->n_components, a->max_components, a->min_area, a->rois,
                     a->areas, a->max_rois, L.kept_frame, L.words, L.filter_state, a->n_rois);
  hipLaunchKernelGGL(begin_kernel, dim3(static_cast<uint32_t>((a->n_frames + 1 + 255) / 256)),
                     dim3(256), 0, s, L.kept_frame, a->n_rois, a->n_frames, a->frame_begin);
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
