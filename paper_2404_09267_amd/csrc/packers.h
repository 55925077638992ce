// Incremental rectangle packers shared by the planner (plan.cpp) and the SLO-aware
// invoker (invoker.cpp). Both place one rectangle at a time on the open canvas and
// open a new canvas (next-fit: the old one is never revisited) when it cannot take the
// rectangle (Sec. III-C, Patch-stitching Solver and Alg. 2). A placement depends only on
// the rectangles placed before it, so placing a queue one arrival at a time gives the
// same result as packing the whole queue at once in that order.
#ifndef TG_PACKERS_H
#define TG_PACKERS_H

#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <vector>

namespace tg_detail {

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

}  // namespace tg_detail

#endif  // TG_PACKERS_H
