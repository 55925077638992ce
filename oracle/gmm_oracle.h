/*
 * Test infrastructure only: per-pixel adaptive Gaussian-mixture background model and
 * the RoIs it yields, as plain C loops. Only tests/, the package smoke check and the
 * bench's CPU-baseline leg may call it; the product path never links it.
 *
 * The paper obtains its RoIs from a Gaussian-mixture background model (Sec. III-A,
 * step 1 of Adaptive Frame Partitioning, citing Stauffer and Grimson's adaptive
 * mixture; Sec. V runs a MOG2-style subtractor). The update here is the adaptive
 * mixture with the number of components chosen online (Zivkovic, ICPR 2004): every
 * component is an isotropic RGB Gaussian with weight w, mean mu and variance v; the
 * ownership of a sample goes to the heaviest close component; rho = alpha / w replaces
 * the density-scaled rate of Stauffer and Grimson. All arithmetic is binary32 with every
 * operation rounded on its own (built with -ffp-contract=off), in the order spelt out
 * at oracle_gmm_pixel, because the foreground decisions it makes must be taken in the
 * same precision by any implementation compared with it.
 *
 * Layouts:
 *   frames uint8 [n_px][3]            RGB samples, one per pixel
 *   state  float [n_px][n_mix][5]     {w, mu_r, mu_g, mu_b, v} per component, heaviest
 *                                     first; only the first modes[p] are meaningful
 *   modes  uint8 [n_px]               components in use (0 = fresh pixel)
 *   mask   uint8 [n_px]               1 = foreground, 0 = background
 */
#ifndef TG_GMM_ORACLE_H
#define TG_GMM_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_GMM_MAX_MIX = 8 };

typedef struct {
  int32_t n_mix;              /* K, the most components a pixel may hold */
  float alpha;                /* learning rate of this frame, (0, 1] */
  float var_threshold;        /* background test: |x - mu|^2 < var_threshold * v */
  float var_threshold_gen;    /* ownership test: |x - mu|^2 < var_threshold_gen * v */
  float var_init, var_min, var_max;
  float background_ratio;     /* 1 - c_f: weight the background components cover */
  float complexity_reduction; /* c_T, in [0, 1) */
} orc_gmm_params;

/* One pixel, one sample. Returns the foreground flag. */
int oracle_gmm_pixel(const uint8_t x[3], float *state, uint8_t *modes,
                     const orc_gmm_params *p);

/* Every pixel of one frame set. Returns 0, or 1 for bad parameters. */
int oracle_gmm_update(const uint8_t *frames, int64_t n_px, float *state, uint8_t *modes,
                      uint8_t *mask, const orc_gmm_params *p);

/* Foreground components of each frame's mask, 8-connected, found by flood fill;
 * components of fewer than min_area pixels are dropped. Writes the kept components'
 * bounding boxes as rows {frame, x, y, w, h} (frames in order, each frame's components
 * in raster order of their first pixel) up to `cap` rows, frame_begin[n_frames + 1]
 * and, per row, the pixel count. Returns the number of kept components (which may
 * exceed cap), or -1 for bad arguments. */
int64_t oracle_mask_rois(const uint8_t *mask, int32_t n_frames, int32_t width,
                         int32_t height, int32_t min_area, int32_t *rows, int64_t *areas,
                         int64_t cap, int32_t *frame_begin);

#ifdef __cplusplus
}
#endif

#endif /* TG_GMM_ORACLE_H */
