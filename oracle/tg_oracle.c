/*
 * Test infrastructure only (see tg_oracle.h): the plain CPU oracle of the
 * patch-stitching path of Tangram (arXiv 2404.09267). Written for a reader who
 * checks it against the paper by eye, not for speed: scalar loops, fp64 where the
 * definition is real-valued, no blocking, no tables beyond what a definition needs.
 *
 * Build: gcc -std=c11 -O2 -ffp-contract=off -fopenmp -shared -fPIC.
 * -ffp-contract=off keeps every float expression rounded operation by operation.
 */
#include "tg_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------- */
/* binary16 rounding                                                          */
/* ------------------------------------------------------------------------- */

/* IEEE-754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Normal numbers are (1 + f/1024) * 2^(E) for E in -14..15; subnormals are
 * f * 2^-24. Rounding is to nearest, ties to even: rint() in the default
 * rounding mode does exactly that on an exactly scaled double. */
uint16_t oracle_half_from_double(double v) {
  uint16_t sign = signbit(v) ? 0x8000u : 0u;
  if (isnan(v)) return (uint16_t)(sign | 0x7E00u);
  double a = fabs(v);
  if (isinf(a)) return (uint16_t)(sign | 0x7C00u);
  if (a < ldexp(1.0, -14)) {
    /* subnormal range: a = m * 2^-24; m == 1024 after rounding is the smallest
     * normal, whose encoding (exponent field 1, fraction 0) is also 1024. */
    double m = rint(ldexp(a, 24));
    return (uint16_t)(sign | (uint16_t)m);
  }
  int e;
  (void)frexp(a, &e); /* a in [2^(e-1), 2^e) */
  int E = e - 1;
  double m = rint(ldexp(a, 10 - E)); /* significand scaled to [1024, 2048] */
  if (m == 2048.0) {
    m = 1024.0;
    E += 1;
  }
  if (E > 15) return (uint16_t)(sign | 0x7C00u); /* rounds past 65504: infinity */
  return (uint16_t)(sign | (uint16_t)((E + 15) << 10) | (uint16_t)((int)m - 1024));
}

/* Detector-input normalisation: per channel (x - mean_k) / std_k in fp64, then
 * one rounding to binary16. The paper does not specify it; the build adopts it
 * as the detector's input transform (see the design notes' readings). */
static uint16_t norm_value(int x, int k, const float mean[3], const float stdv[3]) {
  double q = ((double)x - (double)mean[k]) / (double)stdv[k];
  return oracle_half_from_double(q);
}

void oracle_norm_table(const float mean[3], const float stdv[3], uint16_t *table) {
  for (int k = 0; k < 3; ++k)
    for (int x = 0; x < 256; ++x) table[k * 256 + x] = norm_value(x, k, mean, stdv);
}

/* ------------------------------------------------------------------------- */
/* Packing                                                                    */
/* ------------------------------------------------------------------------- */

#define R_FRAME(i) rois[5 * (i) + 0]
#define R_X(i) rois[5 * (i) + 1]
#define R_Y(i) rois[5 * (i) + 2]
#define R_W(i) rois[5 * (i) + 3]
#define R_H(i) rois[5 * (i) + 4]

/* Checks every RoI in index order. A patch may not be resized (Sec. III-C), so one
 * larger than the canvas cannot be placed at all. */
static int validate(const int32_t *rois, int32_t n, int32_t cw, int32_t ch, int32_t fw,
                    int32_t fh, int32_t nf, int32_t *bad) {
  for (int32_t i = 0; i < n; ++i) {
    int64_t f = R_FRAME(i), x = R_X(i), y = R_Y(i), w = R_W(i), h = R_H(i);
    if (w < 1 || h < 1) {
      *bad = i;
      return ORC_E_INVAL;
    }
    if (f < 0 || f >= nf || x < 0 || y < 0 || x + w > fw || y + h > fh) {
      *bad = i;
      return ORC_E_ROI_OOB;
    }
    if (w > cw || h > ch) {
      *bad = i;
      return ORC_E_ROI_TOO_LARGE;
    }
  }
  return ORC_OK;
}

/* Sort key for first-fit decreasing height: taller first, equal heights keep their
 * input order (the index comparison makes the order total, so qsort acts stably). */
static const int32_t *g_sort_rois;
static int by_height_desc(const void *pa, const void *pb) {
  int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
  const int32_t *rois = g_sort_rois;
  if (R_H(a) != R_H(b)) return R_H(a) > R_H(b) ? -1 : 1;
  return (a > b) - (a < b);
}

typedef struct {
  int32_t y, height, used;
} shelf_t;

/* Shelf packing: each canvas is cut into horizontal shelves stacked from the top.
 * An RoI goes on the first shelf (in creation order) that is tall enough and has
 * room left on its right; otherwise a new shelf as tall as the RoI is opened under
 * the last one; if that would pass the canvas bottom, the canvas is closed and a
 * new blank one opened (Alg. 2 re-initialises a new canvas when nothing fits). */
static void pack_shelf(const int32_t *rois, const int32_t *seq, int32_t n, int32_t cw,
                       int32_t ch, int32_t *place, int32_t *order, int32_t *cbeg,
                       int32_t *n_canvases) {
  shelf_t *shelves = (shelf_t *)malloc(sizeof(shelf_t) * (size_t)(ch > 0 ? ch : 1));
  int32_t ns = 0, top = 0, canvas = 0;
  cbeg[0] = 0;
  for (int32_t t = 0; t < n; ++t) {
    int32_t i = seq[t], w = R_W(i), h = R_H(i);
    int32_t px = -1, py = -1;
    for (int32_t s = 0; s < ns; ++s) {
      if (h <= shelves[s].height && shelves[s].used + w <= cw) {
        px = shelves[s].used;
        py = shelves[s].y;
        shelves[s].used += w;
        break;
      }
    }
    if (px < 0) {
      if (top + h > ch) { /* close this canvas; open the next one */
        canvas += 1;
        cbeg[canvas] = t;
        ns = 0;
        top = 0;
      }
      shelves[ns].y = top;
      shelves[ns].height = h;
      shelves[ns].used = w;
      ns += 1;
      px = 0;
      py = top;
      top += h;
    }
    place[3 * i + 0] = canvas;
    place[3 * i + 1] = px;
    place[3 * i + 2] = py;
    order[t] = i;
  }
  *n_canvases = n > 0 ? canvas + 1 : 0;
  cbeg[*n_canvases] = n;
  free(shelves);
}

typedef struct {
  int32_t x, y, w, h;
} rect_t;

/* Alg. 2, Patch_stitching_solver, patches taken in queue order:
 *  - candidates are the free rectangles c with w_c >= w_i and h_c >= h_i;
 *  - the chosen one minimises min(w_c - w_i, h_c - h_i) (ties: the smaller
 *    max(w_c - w_i, h_c - h_i), then the earlier rectangle in the list);
 *  - the patch goes to the corner of c nearest the canvas origin;
 *  - c is replaced by the two leftover rectangles, split along c's shorter side:
 *    c no wider than tall -> the cut runs across the full width under the patch,
 *    otherwise the cut runs down the full height to the right of the patch;
 *  - with no candidate, a new blank canvas is started and the patch placed on it.
 * If `free_out` is given, each canvas's final free list is appended to it. */
static int32_t pack_guillotine(const int32_t *rois, int32_t n, int32_t cw, int32_t ch,
                               int32_t *place, int32_t *order, int32_t *cbeg,
                               int32_t *n_canvases, int32_t *free_out, int32_t free_cap) {
  rect_t *F = (rect_t *)malloc(sizeof(rect_t) * (size_t)(2 * n + 2));
  int32_t nF = 0, canvas = 0, n_free_out = 0;
  if (n > 0) {
    F[0].x = 0;
    F[0].y = 0;
    F[0].w = cw;
    F[0].h = ch;
    nF = 1;
  }
  if (cbeg) cbeg[0] = 0;
  for (int32_t i = 0; i < n; ++i) {
    int32_t w = R_W(i), h = R_H(i);
    int32_t best = -1, best_short = 0, best_long = 0;
    for (int32_t f = 0; f < nF; ++f) {
      if (F[f].w < w || F[f].h < h) continue;
      int32_t dw = F[f].w - w, dh = F[f].h - h;
      int32_t s = dw < dh ? dw : dh, l = dw < dh ? dh : dw;
      if (best < 0 || s < best_short || (s == best_short && l < best_long)) {
        best = f;
        best_short = s;
        best_long = l;
      }
    }
    if (best < 0) { /* nothing fits: close this canvas and start a blank one */
      if (free_out) {
        for (int32_t f = 0; f < nF; ++f) {
          if (n_free_out >= free_cap) {
            free(F);
            return -1;
          }
          int32_t *r = free_out + 5 * n_free_out++;
          r[0] = canvas; r[1] = F[f].x; r[2] = F[f].y; r[3] = F[f].w; r[4] = F[f].h;
        }
      }
      canvas += 1;
      if (cbeg) cbeg[canvas] = i;
      F[0].x = 0;
      F[0].y = 0;
      F[0].w = cw;
      F[0].h = ch;
      nF = 1;
      best = 0;
    }
    rect_t c = F[best];
    if (place) {
      place[3 * i + 0] = canvas;
      place[3 * i + 1] = c.x;
      place[3 * i + 2] = c.y;
    }
    if (order) order[i] = i;
    rect_t right, below;
    if (c.w <= c.h) { /* cut across the full width of c */
      right.x = c.x + w; right.y = c.y; right.w = c.w - w; right.h = h;
      below.x = c.x; below.y = c.y + h; below.w = c.w; below.h = c.h - h;
    } else { /* cut down the full height of c */
      right.x = c.x + w; right.y = c.y; right.w = c.w - w; right.h = c.h;
      below.x = c.x; below.y = c.y + h; below.w = w; below.h = c.h - h;
    }
    for (int32_t f = best; f + 1 < nF; ++f) F[f] = F[f + 1];
    nF -= 1;
    if (right.w > 0 && right.h > 0) F[nF++] = right;
    if (below.w > 0 && below.h > 0) F[nF++] = below;
  }
  if (free_out && n > 0) {
    for (int32_t f = 0; f < nF; ++f) {
      if (n_free_out >= free_cap) {
        free(F);
        return -1;
      }
      int32_t *r = free_out + 5 * n_free_out++;
      r[0] = canvas; r[1] = F[f].x; r[2] = F[f].y; r[3] = F[f].w; r[4] = F[f].h;
    }
  }
  if (n_canvases) *n_canvases = n > 0 ? canvas + 1 : 0;
  if (cbeg) cbeg[n > 0 ? canvas + 1 : 0] = n;
  free(F);
  return n_free_out;
}

int oracle_pack(const int32_t *rois, int32_t n, int32_t cw, int32_t ch, int32_t fw,
                int32_t fh, int32_t nf, int32_t policy, int32_t *place, int32_t *order,
                int32_t *cbeg, int32_t *n_canvases, int32_t *bad) {
  if (n < 0 || cw < 1 || ch < 1 || fw < 1 || fh < 1 || nf < 0) return ORC_E_INVAL;
  if (policy < ORC_SHELF_FFDH || policy > ORC_GUILLOTINE_BSSF) return ORC_E_INVAL;
  *bad = -1;
  int rc = validate(rois, n, cw, ch, fw, fh, nf, bad);
  if (rc != ORC_OK) return rc;
  if (policy == ORC_GUILLOTINE_BSSF) {
    pack_guillotine(rois, n, cw, ch, place, order, cbeg, n_canvases, NULL, 0);
    return ORC_OK;
  }
  int32_t *seq = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
  for (int32_t i = 0; i < n; ++i) seq[i] = i;
  if (policy == ORC_SHELF_FFDH) {
    g_sort_rois = rois;
    qsort(seq, (size_t)n, sizeof(int32_t), by_height_desc);
  }
  pack_shelf(rois, seq, n, cw, ch, place, order, cbeg, n_canvases);
  free(seq);
  return ORC_OK;
}

int32_t oracle_guillotine_free(const int32_t *rois, int32_t n, int32_t cw, int32_t ch,
                               int32_t *rects, int32_t cap) {
  if (n < 0 || cw < 1 || ch < 1) return -1;
  for (int32_t i = 0; i < n; ++i)
    if (R_W(i) < 1 || R_H(i) < 1 || R_W(i) > cw || R_H(i) > ch) return -1;
  return pack_guillotine(rois, n, cw, ch, NULL, NULL, NULL, NULL, rects, cap);
}

/* ------------------------------------------------------------------------- */
/* Plan invariants                                                            */
/* ------------------------------------------------------------------------- */

/* Return codes:
 *  1 order is not a permutation of 0..n-1
 *  2 cbeg is not a monotone CSR from 0 to n over n_canvases canvases
 *  3 an RoI's place.canvas disagrees with the canvas segment holding it in order
 *  4 a placed rect leaves the canvas
 *  5 two rects on one canvas overlap (an occupancy count exceeds 1)
 *  6 summed RoI area on a canvas exceeds the canvas area (constraint (4))
 *  7 shelf structure broken (shelf policies): an RoI taller than its shelf, shelves
 *    not stacked from the top without gaps, or RoIs on a shelf not packed left to right
 *  8 placement sequence broken: FFDH not in height-descending stable order, or the
 *    arrival-order policies not in input order
 *  9 next-fit broken (shelf policies): the first RoI of a canvas would still have
 *    fitted the previous canvas's final shelves or under its last shelf
 * 10 an empty canvas */
int oracle_check_plan(const int32_t *rois, int32_t n, int32_t cw, int32_t ch, int32_t policy,
                      const int32_t *place, const int32_t *order, const int32_t *cbeg,
                      int32_t J) {
  if (n == 0) return (J == 0 && cbeg[0] == 0) ? 0 : 2;
  char *seen = (char *)calloc((size_t)n, 1);
  for (int32_t t = 0; t < n; ++t) {
    int32_t i = order[t];
    if (i < 0 || i >= n || seen[i]) {
      free(seen);
      return 1;
    }
    seen[i] = 1;
  }
  free(seen);
  if (J < 1 || cbeg[0] != 0 || cbeg[J] != n) return 2;
  for (int32_t j = 0; j < J; ++j) {
    if (cbeg[j + 1] < cbeg[j]) return 2;
    if (cbeg[j + 1] == cbeg[j]) return 10;
  }
  for (int32_t j = 0; j < J; ++j)
    for (int32_t t = cbeg[j]; t < cbeg[j + 1]; ++t)
      if (place[3 * order[t]] != j) return 3;
  for (int32_t i = 0; i < n; ++i) {
    int64_t x = place[3 * i + 1], y = place[3 * i + 2];
    if (x < 0 || y < 0 || x + R_W(i) > cw || y + R_H(i) > ch) return 4;
  }
  /* occupancy count map, one canvas at a time */
  unsigned char *occ = (unsigned char *)malloc((size_t)cw * (size_t)ch);
  for (int32_t j = 0; j < J; ++j) {
    memset(occ, 0, (size_t)cw * (size_t)ch);
    int64_t area = 0;
    for (int32_t t = cbeg[j]; t < cbeg[j + 1]; ++t) {
      int32_t i = order[t];
      area += (int64_t)R_W(i) * R_H(i);
      for (int32_t yy = 0; yy < R_H(i); ++yy)
        for (int32_t xx = 0; xx < R_W(i); ++xx) {
          size_t at = (size_t)(place[3 * i + 2] + yy) * (size_t)cw + (size_t)(place[3 * i + 1] + xx);
          if (occ[at]) {
            free(occ);
            return 5;
          }
          occ[at] = 1;
        }
    }
    if (area > (int64_t)cw * ch) {
      free(occ);
      return 6;
    }
  }
  free(occ);
  /* placement sequence */
  for (int32_t t = 0; t + 1 < n; ++t) {
    int32_t a = order[t], b = order[t + 1];
    if (policy == ORC_SHELF_FFDH) {
      if (R_H(a) < R_H(b) || (R_H(a) == R_H(b) && a > b)) return 8;
    } else if (a + 1 != b) {
      return 8;
    }
  }
  if (policy == ORC_GUILLOTINE_BSSF) return 0;
  /* shelves: on each canvas the shelves are the RoIs in placement sequence that sit
   * at x == 0; each later RoI sits on the most recent shelf opened before it or an
   * earlier one, flush right of the RoIs already on that shelf. */
  shelf_t *sh = (shelf_t *)malloc(sizeof(shelf_t) * (size_t)n);
  for (int32_t j = 0; j < J; ++j) {
    int32_t ns = 0, top = 0;
    for (int32_t t = cbeg[j]; t < cbeg[j + 1]; ++t) {
      int32_t i = order[t], x = place[3 * i + 1], y = place[3 * i + 2];
      if (x == 0) {
        if (y != top) { free(sh); return 7; }
        sh[ns].y = y; sh[ns].height = R_H(i); sh[ns].used = R_W(i);
        ns += 1;
        top += R_H(i);
        if (top > ch) { free(sh); return 7; }
        continue;
      }
      int32_t s = 0;
      while (s < ns && sh[s].y != y) ++s;
      if (s == ns || R_H(i) > sh[s].height || x != sh[s].used) { free(sh); return 7; }
      sh[s].used += R_W(i);
    }
    if (j + 1 < J) { /* the next canvas's first RoI must not fit this one */
      int32_t i = order[cbeg[j + 1]];
      for (int32_t s = 0; s < ns; ++s)
        if (R_H(i) <= sh[s].height && sh[s].used + R_W(i) <= cw) { free(sh); return 9; }
      if (top + R_H(i) <= ch) { free(sh); return 9; }
    }
  }
  free(sh);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Stitch                                                                     */
/* ------------------------------------------------------------------------- */

/* Patches are copied onto the canvas without resizing (Sec. I, III-B, III-C);
 * every canvas pixel outside all patches takes the normalised pad value. The
 * output is the detector's NCHW binary16 input. */
int oracle_stitch(const uint8_t *frames, int64_t fstride, int32_t pitch, const int32_t *rois,
                  const int32_t *place, const int32_t *order, const int32_t *cbeg, int32_t J,
                  int32_t first, int32_t count, int32_t cw, int32_t ch, const float mean[3],
                  const float stdv[3], const uint8_t pad[3], uint16_t *out) {
  if (first < 0 || count < 0 || (int64_t)first + count > J) return ORC_E_RANGE;
  const int64_t plane = (int64_t)cw * ch;
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t c = 0; c < count; ++c) {
    uint16_t *o = out + (int64_t)c * 3 * plane;
    for (int k = 0; k < 3; ++k) {
      uint16_t pv = norm_value(pad[k], k, mean, stdv);
      for (int64_t p = 0; p < plane; ++p) o[k * plane + p] = pv;
    }
    int32_t j = first + c;
    for (int32_t t = cbeg[j]; t < cbeg[j + 1]; ++t) {
      int32_t i = order[t];
      int32_t dx = place[3 * i + 1], dy = place[3 * i + 2];
      for (int32_t yy = 0; yy < R_H(i); ++yy) {
        const uint8_t *src = frames + (int64_t)R_FRAME(i) * fstride +
                             (int64_t)(R_Y(i) + yy) * pitch + 3 * (int64_t)R_X(i);
        for (int32_t xx = 0; xx < R_W(i); ++xx)
          for (int k = 0; k < 3; ++k)
            o[k * plane + (int64_t)(dy + yy) * cw + (dx + xx)] =
                norm_value(src[3 * xx + k], k, mean, stdv);
      }
    }
  }
  return ORC_OK;
}

void oracle_pixel_sources(const int32_t *rois, const int32_t *place, const int32_t *order,
                          const int32_t *cbeg, int32_t J, int64_t fstride, int32_t pitch,
                          const int32_t *pts, int32_t m, int64_t *src) {
#pragma omp parallel for schedule(static)
  for (int32_t q = 0; q < m; ++q) {
    int32_t c = pts[3 * q], X = pts[3 * q + 1], Y = pts[3 * q + 2];
    src[q] = -1;
    if (c < 0 || c >= J) continue;
    for (int32_t t = cbeg[c]; t < cbeg[c + 1]; ++t) {
      int32_t i = order[t];
      int32_t dx = place[3 * i + 1], dy = place[3 * i + 2];
      if (X >= dx && X < dx + R_W(i) && Y >= dy && Y < dy + R_H(i)) {
        src[q] = (int64_t)R_FRAME(i) * fstride + (int64_t)(R_Y(i) + Y - dy) * pitch +
                 3 * (int64_t)(R_X(i) + X - dx);
        break;
      }
    }
  }
}

/* ------------------------------------------------------------------------- */
/* Unstitch                                                                   */
/* ------------------------------------------------------------------------- */

/* A detection belongs to the patch that contains its centre (half-open on the right
 * and bottom edges); it is clipped to that patch when asked and moved back by the
 * patch's offset between canvas and frame. Boxes whose centre lies on pad, whose
 * canvas id is out of range, or that hold a NaN are dropped (roi_of_box = -1). The
 * paper evaluates per-frame detection accuracy (Sec. V-D) without stating this
 * mapping; this is the build's reading. */
/* Length of [lo, hi] inside [p0, p1], at least 0 (binary32, one rounding). */
static float overlap_1d(float lo, float hi, float p0, float p1) {
  float a = (hi < p1 ? hi : p1) - (lo > p0 ? lo : p0);
  return a > 0.0f ? a : 0.0f;
}

int oracle_unstitch(const float *boxes, const int32_t *box_canvas, int32_t n,
                    const int32_t *rois, const int32_t *place, const int32_t *order,
                    const int32_t *cbeg, int32_t J, int32_t clip, int32_t rule,
                    int32_t *roi_of_box, orc_det *dets, int32_t *n_out) {
#pragma omp parallel for schedule(static)
  for (int32_t b = 0; b < n; ++b) {
    roi_of_box[b] = -1;
    int32_t c = box_canvas[b];
    if (c < 0 || c >= J) continue;
    if (rule == 1) {
      /* the patch of the canvas that the box overlaps most (area > 0); ties to the lower
         RoI id; a NaN coordinate matches nothing */
      const float *bx = boxes + 4 * b;
      if (bx[0] != bx[0] || bx[1] != bx[1] || bx[2] != bx[2] || bx[3] != bx[3]) continue;
      float best = 0.0f;
      for (int32_t t = cbeg[c]; t < cbeg[c + 1]; ++t) {
        int32_t i = order[t];
        float x0 = (float)place[3 * i + 1], y0 = (float)place[3 * i + 2];
        float x1 = (float)(place[3 * i + 1] + R_W(i)), y1 = (float)(place[3 * i + 2] + R_H(i));
        float area = overlap_1d(bx[0], bx[2], x0, x1) * overlap_1d(bx[1], bx[3], y0, y1);
        if (area > best || (area == best && area > 0.0f && i < roi_of_box[b])) {
          best = area;
          roi_of_box[b] = i;
        }
      }
      continue;
    }
    float cx = (boxes[4 * b + 0] + boxes[4 * b + 2]) * 0.5f;
    float cy = (boxes[4 * b + 1] + boxes[4 * b + 3]) * 0.5f;
    for (int32_t t = cbeg[c]; t < cbeg[c + 1]; ++t) {
      int32_t i = order[t];
      float x0 = (float)place[3 * i + 1], y0 = (float)place[3 * i + 2];
      float x1 = (float)(place[3 * i + 1] + R_W(i)), y1 = (float)(place[3 * i + 2] + R_H(i));
      if (x0 <= cx && cx < x1 && y0 <= cy && cy < y1) {
        roi_of_box[b] = i;
        break;
      }
    }
  }
  int32_t k = 0;
  for (int32_t b = 0; b < n; ++b) {
    int32_t i = roi_of_box[b];
    if (i < 0) continue;
    int32_t dx = place[3 * i + 1], dy = place[3 * i + 2];
    float lo_x = (float)dx, hi_x = (float)(dx + R_W(i));
    float lo_y = (float)dy, hi_y = (float)(dy + R_H(i));
    float v[4] = {boxes[4 * b + 0], boxes[4 * b + 1], boxes[4 * b + 2], boxes[4 * b + 3]};
    if (clip) {
      for (int q = 0; q < 4; ++q) {
        float lo = (q % 2 == 0) ? lo_x : lo_y, hi = (q % 2 == 0) ? hi_x : hi_y;
        if (v[q] < lo) v[q] = lo;
        if (v[q] > hi) v[q] = hi;
      }
    }
    float sx = (float)(R_X(i) - dx), sy = (float)(R_Y(i) - dy);
    dets[k].box = b;
    dets[k].roi = i;
    dets[k].frame = R_FRAME(i);
    dets[k].x1 = v[0] + sx;
    dets[k].y1 = v[1] + sy;
    dets[k].x2 = v[2] + sx;
    dets[k].y2 = v[3] + sy;
    ++k;
  }
  *n_out = k;
  return ORC_OK;
}

void oracle_set_threads(int32_t n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

int32_t oracle_threads(void) {
#ifdef _OPENMP
  return (int32_t)omp_get_max_threads();
#else
  return 1;
#endif
}
