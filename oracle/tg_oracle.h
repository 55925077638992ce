/*
 * Test infrastructure only: a plain, slow CPU oracle for Tangram's patch-stitching
 * batch assembly (arXiv 2404.09267). Only tests/, the package smoke check and the
 * bench's CPU-baseline leg may call it; the product path never links it.
 *
 * It shares no source, header, table or constant with the GPU library. Arrays are
 * plain int32/float/uint8/uint16 so that ctypes can hand numpy buffers straight in.
 *
 * Layouts (all row-major, contiguous):
 *   rois   int32 [n][5]  = {frame, x, y, w, h}   source rect, pixels, y down
 *   place  int32 [n][3]  = {canvas, x, y}        top-left of the RoI on its canvas
 *   order  int32 [n]                              RoI ids in placement sequence
 *   cbeg   int32 [J+1]                            order[cbeg[j]..cbeg[j+1]) lie on canvas j
 *   frames uint8 [F][H][pitch]                    HWC RGB, pixel (x,y) channel k at
 *                                                 f*fstride + y*pitch + 3*x + k
 *   out    uint16 [count][3][Hc][Wc]              IEEE binary16 bit patterns (NCHW)
 *   boxes  float [n][4] = {x1, y1, x2, y2}        canvas pixels, continuous
 *   dets   orc_det [n]                            kept boxes, input order
 */
#ifndef TG_ORACLE_H
#define TG_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORC_OK = 0,
  ORC_E_INVAL = 1,        /* bad argument, or an RoI with w < 1 or h < 1 */
  ORC_E_ROI_OOB = 2,      /* RoI not inside its frame, or frame id out of range */
  ORC_E_ROI_TOO_LARGE = 3,/* RoI wider or taller than the canvas */
  ORC_E_RANGE = 4         /* canvas range outside the plan */
};

enum { ORC_SHELF_FFDH = 0, ORC_SHELF_ARRIVAL = 1, ORC_GUILLOTINE_BSSF = 2 };

typedef struct {
  int32_t box, roi, frame;
  float x1, y1, x2, y2;
} orc_det;

/* IEEE-754 binary16, round to nearest with ties to even, from a double. */
uint16_t oracle_half_from_double(double v);

/* R_k(x) = half(((double)x - mean_k) / std_k) for k in 0..2, x in 0..255,
 * written to table[k*256 + x]. */
void oracle_norm_table(const float mean[3], const float stdv[3], uint16_t *table);

/* Packing (Sec. III-C and Alg. 2's solver; shelf policies by the readings of the
 * build's design notes). Returns an ORC_* code; on a per-RoI error *bad holds the
 * first offending RoI. */
int oracle_pack(const int32_t *rois, int32_t n, int32_t canvas_w, int32_t canvas_h,
                int32_t frame_w, int32_t frame_h, int32_t n_frames, int32_t policy,
                int32_t *place, int32_t *order, int32_t *cbeg, int32_t *n_canvases,
                int32_t *bad);

/* The guillotine solver's final free-rectangle list of every canvas, {canvas,x,y,w,h}
 * per row, canvas-major and in list order; returns the row count, or a negative
 * value if the rows do not fit in `cap` or the input is invalid. */
int32_t oracle_guillotine_free(const int32_t *rois, int32_t n, int32_t canvas_w,
                               int32_t canvas_h, int32_t *rects, int32_t cap);

/* Invariant checker for any plan; 0 when every invariant holds, else a code naming
 * the first one that fails (see the source). */
int oracle_check_plan(const int32_t *rois, int32_t n, int32_t canvas_w, int32_t canvas_h,
                      int32_t policy, const int32_t *place, const int32_t *order,
                      const int32_t *cbeg, int32_t n_canvases);

/* Canvas pixels for canvases [first, first+count) of a plan. */
int oracle_stitch(const uint8_t *frames, int64_t fstride, int32_t pitch,
                  const int32_t *rois, const int32_t *place, const int32_t *order,
                  const int32_t *cbeg, int32_t n_canvases, int32_t first, int32_t count,
                  int32_t canvas_w, int32_t canvas_h, const float mean[3],
                  const float stdv[3], const uint8_t pad[3], uint16_t *out);

/* Source byte offset (into frames) of canvas pixel (c, X, Y), channel 0, or -1 for
 * pad, for `m` sample points given as int32 [m][3] = {canvas, X, Y}. */
void oracle_pixel_sources(const int32_t *rois, const int32_t *place, const int32_t *order,
                          const int32_t *cbeg, int32_t n_canvases, int64_t fstride,
                          int32_t pitch, const int32_t *pts, int32_t m, int64_t *src);

/* Box remapping; returns ORC_OK. rule 0: the patch holding the box centre; rule 1: the
 * patch the box overlaps most (area > 0, ties to the lower RoI id, NaN matches nothing). */
int oracle_unstitch(const float *boxes, const int32_t *box_canvas, int32_t n,
                    const int32_t *rois, const int32_t *place, const int32_t *order,
                    const int32_t *cbeg, int32_t n_canvases, int32_t clip, int32_t rule,
                    int32_t *roi_of_box, orc_det *dets, int32_t *n_out);

/* Threads OpenMP would use for the stitch/unstitch loops. */
int32_t oracle_threads(void);
/* Threads for later OpenMP loops (n > 0). */
void oracle_set_threads(int32_t n);

#ifdef __cplusplus
}
#endif
#endif
