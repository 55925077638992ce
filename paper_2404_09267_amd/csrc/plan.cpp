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

#include "tg.h"

namespace {

struct Shelf {
  int32_t top;    // y of the shelf on its canvas
  int32_t height; // height of the RoI that opened it
  int32_t fill;   // x where the next RoI on this shelf would go
};

// Shelves of the open canvas. First fit: the earliest-created shelf that is tall
// enough and has room on its right. Otherwise a new shelf under the lowest one;
// otherwise the canvas is closed and never revisited.
class ShelfPacker {
 public:
  ShelfPacker(int32_t cw, int32_t ch) : cw_(cw), ch_(ch) {}

  // Returns true when the RoI needed a fresh canvas.
  bool put(int32_t w, int32_t h, int32_t *x, int32_t *y) {
    for (Shelf &s : shelves_) {
      if (h > s.height || w > cw_ - s.fill) continue;
      *x = s.fill;
      *y = s.top;
      s.fill += w;
      return false;
    }
    bool fresh = false;
    if (h > ch_ - depth_) {
      shelves_.clear();
      depth_ = 0;
      fresh = true;
    }
    shelves_.push_back(Shelf{depth_, h, w});
    *x = 0;
    *y = depth_;
    depth_ += h;
    return fresh;
  }

 private:
  int32_t cw_, ch_;
  int32_t depth_ = 0; // bottom of the lowest shelf
  std::vector<Shelf> shelves_;
};

struct Free {
  int32_t x, y, w, h;
};

// The Patch-stitching Solver of Alg. 2 for one open canvas at a time.
class GuillotinePacker {
 public:
  GuillotinePacker(int32_t cw, int32_t ch) : cw_(cw), ch_(ch) { reset(); }

  bool put(int32_t w, int32_t h, int32_t *x, int32_t *y) {
    bool fresh = false;
    size_t pick = pick_for(w, h);
    if (pick == kNone) {
      reset();
      pick = 0;
      fresh = true;
    }
    const Free c = free_[pick];
    *x = c.x;
    *y = c.y;
    // Split the leftover of c along c's shorter side into a piece right of the RoI
    // and a piece below it.
    Free right{c.x + w, c.y, c.w - w, c.h};
    Free below{c.x, c.y + h, c.w, c.h - h};
    if (c.w <= c.h)
      right.h = h;  // cut spans c's full width: the right piece is only as tall as the RoI
    else
      below.w = w;  // cut spans c's full height: the lower piece is only as wide as the RoI
    free_.erase(free_.begin() + static_cast<std::ptrdiff_t>(pick));
    if (right.w > 0 && right.h > 0) free_.push_back(right);
    if (below.w > 0 && below.h > 0) free_.push_back(below);
    return fresh;
  }

 private:
  static constexpr size_t kNone = static_cast<size_t>(-1);

  void reset() {
    free_.clear();
    free_.push_back(Free{0, 0, cw_, ch_});
  }

  // Smallest short-side leftover; ties to the smaller long-side leftover, then to the
  // earlier rectangle.
  size_t pick_for(int32_t w, int32_t h) const {
    size_t best = kNone;
    int64_t best_key = 0;
    for (size_t k = 0; k < free_.size(); ++k) {
      const Free &f = free_[k];
      if (f.w < w || f.h < h) continue;
      const int64_t a = f.w - w, b = f.h - h;
      const int64_t key = (std::min(a, b) << 32) | std::max(a, b);
      if (best == kNone || key < best_key) {
        best = k;
        best_key = key;
      }
    }
    return best;
  }

  int32_t cw_, ch_;
  std::vector<Free> free_;
};

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
    if (p.policy == TG_PACK_SHELF_FFDH)
      std::stable_sort(seq.begin(), seq.end(),
                       [rois](int32_t a, int32_t b) { return rois[a].h > rois[b].h; });
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

extern "C" int32_t tg_abi_version(void) { return 1; }
