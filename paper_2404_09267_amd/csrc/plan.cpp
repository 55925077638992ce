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

extern "C" int32_t tg_abi_version(void) { return 8; }
