// Host-side packing of RoI rectangles onto fixed-size canvases (tg_plan_pack).
//
// Tangram stitches unresized patches onto M x N canvases and opens a new canvas when
// the current one cannot take the next patch (Sec. III-B; Sec. III-C, Patch-stitching
// Solver and Alg. 2). Two families are offered: shelf packing (first-fit decreasing
// height, or arrival order) and the paper's guillotine solver with best short-side
// fit. This translation unit makes no HIP call, so the planner runs and is tested on
// machines without a GPU.
#include <algorithm>
#include <cstdint>
#include <new>
#include <numeric>
#include <vector>

#include "packers.h"
#include "stitch_units.h"
#include "tg.h"

namespace {

using tg_detail::GuillotinePacker;
using tg_detail::ShelfPacker;

int check_rois(const tg_roi *rois, int32_t n, const tg_pack_params &p, int32_t *bad) {
  for (int32_t i = 0; i < n; ++i) {
    const tg_roi &r = rois[i];
    int code = TG_OK;
    if (r.w < 1 || r.h < 1)
      code = TG_E_INVAL;
    else if (r.frame < 0 || r.frame >= p.n_frames || r.x < 0 || r.y < 0 ||
             int64_t(r.x) + r.w > p.frame_w || int64_t(r.y) + r.h > p.frame_h)
      code = TG_E_ROI_OOB;
    else if (r.w > p.canvas_w || r.h > p.canvas_h)
      code = TG_E_ROI_TOO_LARGE;
    if (code != TG_OK) {
      *bad = i;
      return code;
    }
  }
  return TG_OK;
}

template <class Packer>
void run(Packer &packer, const tg_roi *rois, const std::vector<int32_t> &seq, tg_place *place,
         int32_t *order, int32_t *canvas_begin, int32_t *n_canvases) {
  int32_t canvas = -1;
  for (size_t t = 0; t < seq.size(); ++t) {
    const int32_t i = seq[t];
    int32_t x, y;
    const bool fresh = packer.put(rois[i].w, rois[i].h, &x, &y);
    if (fresh || canvas < 0) {
      ++canvas;
      canvas_begin[canvas] = static_cast<int32_t>(t);
    }
    place[i] = tg_place{canvas, x, y};
    order[t] = i;
  }
  *n_canvases = canvas + 1;
  canvas_begin[canvas + 1] = static_cast<int32_t>(seq.size());
}

}  // namespace

extern "C" int tg_plan_pack(const tg_roi *rois, int32_t n, const tg_pack_params *params,
                            tg_place *place, int32_t *order, int32_t *canvas_begin,
                            int32_t *n_canvases, int32_t *bad_index) {
  if (!params || !canvas_begin || !n_canvases || !bad_index || n < 0) return TG_E_INVAL;
  if (n > 0 && (!rois || !place || !order)) return TG_E_INVAL;
  const tg_pack_params p = *params;
  if (p.canvas_w < 1 || p.canvas_h < 1 || p.frame_w < 1 || p.frame_h < 1 || p.n_frames < 0)
    return TG_E_INVAL;
  if (p.policy != TG_PACK_SHELF_FFDH && p.policy != TG_PACK_SHELF_ARRIVAL &&
      p.policy != TG_PACK_GUILLOTINE_BSSF)
    return TG_E_INVAL;
  *bad_index = -1;
  try {
    if (int rc = check_rois(rois, n, p, bad_index); rc != TG_OK) return rc;
    std::vector<int32_t> seq(static_cast<size_t>(n));
    std::iota(seq.begin(), seq.end(), 0);
    if (p.policy == TG_PACK_SHELF_FFDH) {
      // stable counting sort by height, tallest first (heights are in [1, canvas_h])
      std::vector<int32_t> count(static_cast<size_t>(p.canvas_h) + 2, 0);
      for (int32_t i = 0; i < n; ++i) ++count[static_cast<size_t>(p.canvas_h - rois[i].h + 1)];
      for (size_t b = 1; b < count.size(); ++b) count[b] += count[b - 1];
      for (int32_t i = 0; i < n; ++i)
        seq[static_cast<size_t>(count[static_cast<size_t>(p.canvas_h - rois[i].h)]++)] = i;
    }
    if (p.policy == TG_PACK_GUILLOTINE_BSSF) {
      GuillotinePacker g(p.canvas_w, p.canvas_h);
      run(g, rois, seq, place, order, canvas_begin, n_canvases);
    } else {
      ShelfPacker s(p.canvas_w, p.canvas_h);
      run(s, rois, seq, place, order, canvas_begin, n_canvases);
    }
    return TG_OK;
  } catch (const std::bad_alloc &) {
    return TG_E_INTERNAL;
  } catch (...) {
    return TG_E_INTERNAL;
  }
}

extern "C" int32_t tg_batch_count(int32_t n_canvases, int32_t batch_cap) {
  if (n_canvases <= 0) return 0;
  if (batch_cap <= 0) return 1;
  return static_cast<int32_t>((int64_t(n_canvases) + batch_cap - 1) / batch_cap);
}

extern "C" int tg_batch_range(int32_t n_canvases, int32_t batch_cap, int32_t k, int32_t *first,
                              int32_t *count) {
  if (!first || !count) return TG_E_INVAL;
  if (k < 0 || k >= tg_batch_count(n_canvases, batch_cap)) return TG_E_RANGE;
  const int64_t cap = batch_cap <= 0 ? n_canvases : batch_cap;
  const int64_t lo = int64_t(k) * cap;
  *first = static_cast<int32_t>(lo);
  *count = static_cast<int32_t>(std::min<int64_t>(cap, n_canvases - lo));
  return TG_OK;
}

extern "C" const char *tg_strerror(int code) {
  switch (code) {
    case TG_OK: return "ok";
    case TG_E_INVAL: return "invalid argument";
    case TG_E_ROI_TOO_LARGE: return "RoI larger than the canvas";
    case TG_E_ROI_OOB: return "RoI outside its frame";
    case TG_E_RANGE: return "canvas or batch range outside the plan";
    case TG_E_WORKSPACE: return "workspace missing or too small";
    case TG_E_HIP: return "HIP launch failed";
    case TG_E_INTERNAL: return "internal error";
    default: return "unknown status";
  }
}

extern "C" int32_t tg_stitch_units(int32_t canvas_w, int32_t canvas_h, int32_t canvas_count) {
  if (canvas_w < 1 || canvas_h < 1 || canvas_count < 0) return TG_E_INVAL;
  if (canvas_count == 0) return 0;
  tg_detail::StitchGeometry g;
  if (!tg_detail::stitch_geometry(canvas_w, canvas_h, canvas_count, &g)) return TG_E_INVAL;
  return g.n_units;
}

extern "C" int tg_stitch_schedule(const tg_roi *rois, const tg_place *place,
                                  const int32_t *order, const int32_t *canvas_begin,
                                  int32_t n_rois, int32_t n_canvases, int32_t canvas_first,
                                  int32_t canvas_count, int32_t canvas_w, int32_t canvas_h,
                                  int32_t *unit_order) {
  if (n_rois < 0 || n_canvases < 0 || canvas_first < 0 || canvas_count < 0 || canvas_w < 1 ||
      canvas_h < 1)
    return TG_E_INVAL;
  if (int64_t(canvas_first) + canvas_count > n_canvases) return TG_E_RANGE;
  if (canvas_count == 0) return TG_OK;
  if (!canvas_begin || !unit_order || (n_rois > 0 && (!rois || !place || !order)))
    return TG_E_INVAL;
  tg_detail::StitchGeometry g;
  if (!tg_detail::stitch_geometry(canvas_w, canvas_h, canvas_count, &g)) return TG_E_INVAL;
  try {
    const int64_t band_rows = int64_t(g.band_steps) * tg_detail::kStitchStepRows;
    const int64_t tile_w = tg_detail::kStitchTileW;
    const int64_t per_canvas = int64_t(g.bands_y) * g.tiles_x;
    // weight: pixels of a patch's first and last band, added directly; full[]: a
    // difference array over bands (per tile) for the full bands in between.
    std::vector<int64_t> weight(static_cast<size_t>(g.n_units), 0);
    std::vector<int64_t> full(static_cast<size_t>(per_canvas + g.tiles_x), 0);
    for (int32_t c = 0; c < canvas_count; ++c) {
      std::fill(full.begin(), full.end(), 0);
      int64_t *wc = weight.data() + static_cast<size_t>(int64_t(c) * per_canvas);
      const int32_t j = canvas_first + c;
      const int64_t lo = std::clamp<int64_t>(canvas_begin[j], 0, n_rois);
      const int64_t hi = std::clamp<int64_t>(canvas_begin[j + 1], lo, n_rois);
      for (int64_t k = lo; k < hi; ++k) {
        const int32_t id = order[k];
        if (id < 0 || id >= n_rois) continue;
        const tg_roi &r = rois[id];
        const tg_place &pl = place[id];
        if (pl.canvas != j || r.w < 1 || r.h < 1 || pl.x < 0 || pl.y < 0 ||
            int64_t(pl.x) + r.w > canvas_w || int64_t(pl.y) + r.h > canvas_h)
          continue;
        const int64_t y0 = pl.y, y1 = int64_t(pl.y) + r.h;
        const int64_t b0 = y0 / band_rows, b1 = (y1 - 1) / band_rows;
        for (int64_t tx = pl.x / tile_w; tx * tile_w < int64_t(pl.x) + r.w; ++tx) {
          const int64_t cols = std::min<int64_t>(pl.x + r.w, (tx + 1) * tile_w) -
                               std::max<int64_t>(pl.x, tx * tile_w);
          if (b0 == b1) {
            wc[b0 * g.tiles_x + tx] += cols * (y1 - y0);
            continue;
          }
          wc[b0 * g.tiles_x + tx] += cols * ((b0 + 1) * band_rows - y0);
          wc[b1 * g.tiles_x + tx] += cols * (y1 - b1 * band_rows);
          full[(b0 + 1) * g.tiles_x + tx] += cols * band_rows;
          full[b1 * g.tiles_x + tx] -= cols * band_rows;
        }
      }
      for (int32_t tx = 0; tx < g.tiles_x; ++tx) {
        int64_t run = 0;
        for (int64_t b = 0; b < g.bands_y; ++b) {
          run += full[b * g.tiles_x + tx];
          wc[b * g.tiles_x + tx] += run;
        }
      }
    }
    // Heaviest first, ties in unit order: a stable counting sort on key (max - weight).
    // A unit's weight is at most its area, below 2^22 (band rows <= 3072, tile columns <=
    // 1280); keys below 2^16 take one pass over max + 1 buckets, larger ones an LSD radix
    // sort of 11 bits per pass.
    int64_t wmax = 0;
    for (int64_t v : weight) wmax = std::max(wmax, v);
    const size_t n = static_cast<size_t>(g.n_units);
    if (wmax < (int64_t(1) << 16)) {
      std::vector<int32_t> count(static_cast<size_t>(wmax) + 2, 0);
      for (size_t u = 0; u < n; ++u) ++count[static_cast<size_t>(wmax - weight[u]) + 1];
      for (int64_t b = 0; b < wmax; ++b) count[b + 1] += count[b];
      for (size_t u = 0; u < n; ++u)
        unit_order[count[static_cast<size_t>(wmax - weight[u])]++] = static_cast<int32_t>(u);
      return TG_OK;
    }
    std::vector<int32_t> ids(n), tmp(n);
    std::iota(ids.begin(), ids.end(), 0);
    for (int shift = 0; (wmax >> shift) > 0; shift += 11) {
      size_t count[2049] = {};
      for (int32_t u : ids) ++count[((wmax - weight[static_cast<size_t>(u)]) >> shift & 2047) + 1];
      for (int b = 0; b < 2048; ++b) count[b + 1] += count[b];
      for (int32_t u : ids) tmp[count[(wmax - weight[static_cast<size_t>(u)]) >> shift & 2047]++] = u;
      ids.swap(tmp);
    }
    std::copy(ids.begin(), ids.end(), unit_order);
    return TG_OK;
  } catch (...) {
    return TG_E_INTERNAL;
  }
}

extern "C" int32_t tg_abi_version(void) { return 5; }
