// Work units of one tg_stitch launch, shared by the kernel launcher (stitch.hip) and the
// host scheduler (plan.cpp) so that both cut canvases the same way.
//
// A canvas is cut into tiles of at most kStitchTileW columns (one tile when the canvas
// is at most that wide) and each tile into bands of whole steps; a step is
// kStitchStepRows canvas rows, the rows one staging buffer holds. One unit = one band of
// one tile of one canvas, processed by one workgroup. The band height is chosen so that
// a launch has about kStitchUnitTarget units: enough workgroups for several rounds over
// the chip, few enough that each amortises its patch-list setup.
#ifndef TG_STITCH_UNITS_H
#define TG_STITCH_UNITS_H

#include <cstdint>

namespace tg_detail {

constexpr int32_t kStitchTileW = 1280;
constexpr int32_t kStitchStepRows = 3;
constexpr int64_t kStitchUnitTarget = 6144;
constexpr int64_t kStitchMaxSteps = 1024;  // steps per band at most

struct StitchGeometry {
  int32_t tiles_x;     // tiles across a canvas
  int32_t band_steps;  // steps per band
  int32_t bands_y;     // bands down a canvas
  int32_t n_units;     // canvas_count * bands_y * tiles_x
};

// Unit k is canvas (k / (bands_y * tiles_x)), band ((k / tiles_x) % bands_y), tile
// (k % tiles_x). False when the sizes are not positive or the count overflows int32.
inline bool stitch_geometry(int32_t canvas_w, int32_t canvas_h, int32_t canvas_count,
                            StitchGeometry *g) {
  if (canvas_w < 1 || canvas_h < 1 || canvas_count < 1) return false;
  const int64_t tiles_x = (int64_t(canvas_w) + kStitchTileW - 1) / kStitchTileW;
  const int64_t steps = (int64_t(canvas_h) + kStitchStepRows - 1) / kStitchStepRows;
  int64_t band_steps = (steps * tiles_x * canvas_count + kStitchUnitTarget - 1) / kStitchUnitTarget;
  band_steps = band_steps < 1 ? 1 : (band_steps > kStitchMaxSteps ? kStitchMaxSteps : band_steps);
  const int64_t bands_y = (steps + band_steps - 1) / band_steps;
  const int64_t n_units = bands_y * tiles_x * canvas_count;
  if (n_units > 0x7FFFFFFF) return false;
  g->tiles_x = static_cast<int32_t>(tiles_x);
  g->band_steps = static_cast<int32_t>(band_steps);
  g->bands_y = static_cast<int32_t>(bands_y);
  g->n_units = static_cast<int32_t>(n_units);
  return true;
}

}  // namespace tg_detail

#endif  // TG_STITCH_UNITS_H
