// Work units of one tg_stitch launch, shared by the kernel launcher (stitch.hip) and the
// host-side unit count (plan.cpp).
//
// A canvas plane is cut, in raster order, into runs of kStitchRun pixels (the last run
// of a canvas may be shorter); one unit = one run of one canvas, processed by one
// workgroup, which writes the run in all three fp16 planes. 6144 pixels are three 4 KB
// pages of one plane: when a plane starts on a 4 KB boundary, every unit writes whole
// pages, and the units of a launch, numbered in address order, sweep the output.
#ifndef TG_STITCH_UNITS_H
#define TG_STITCH_UNITS_H

#include <cstdint>

namespace tg_detail {

constexpr int32_t kStitchRun = 6144;

struct StitchGeometry {
  int64_t plane;   // canvas_w * canvas_h pixels
  int32_t runs;    // units per canvas
  int32_t n_units; // canvas_count * runs
};

// Unit k is run (k % runs) of canvas (k / runs): pixels [6144 r, min(6144 (r + 1), plane))
// in raster order. False when the sizes are not positive or the count overflows int32.
inline bool stitch_geometry(int32_t canvas_w, int32_t canvas_h, int32_t canvas_count,
                            StitchGeometry *g) {
  if (canvas_w < 1 || canvas_h < 1 || canvas_count < 1) return false;
  const int64_t plane = int64_t(canvas_w) * canvas_h;
  const int64_t runs = (plane + kStitchRun - 1) / kStitchRun;
  const int64_t n_units = runs * canvas_count;
  if (n_units > 0x7FFFFFFF) return false;
  g->plane = plane;
  g->runs = static_cast<int32_t>(runs);
  g->n_units = static_cast<int32_t>(n_units);
  return true;
}

}  // namespace tg_detail

#endif  // TG_STITCH_UNITS_H
