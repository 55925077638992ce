/*
 * Test infrastructure only: adaptive Gaussian-mixture background model and the
 * bounding boxes of its foreground components (declarations and layouts in
 * gmm_oracle.h). Plain loops; nothing here is shared with the GPU library.
 */
#include "gmm_oracle.h"

#include <stdlib.h>
#include <string.h>

enum { W_ = 0, MR = 1, MG = 2, MB = 3, V_ = 4, NF = 5 };

static int params_ok(const orc_gmm_params *p) {
  return p && p->n_mix >= 1 && p->n_mix <= ORC_GMM_MAX_MIX && p->alpha > 0.0f &&
         p->alpha <= 1.0f && p->var_min > 0.0f && p->var_min <= p->var_max &&
         p->var_init >= p->var_min && p->var_init <= p->var_max &&
         p->complexity_reduction >= 0.0f && p->complexity_reduction < 1.0f &&
         p->var_threshold >= 0.0f && p->var_threshold_gen >= 0.0f;
}

/*
 * One sample x of one pixel, in this order (the adaptive mixture of Zivkovic 2004 with
 * the background set of Stauffer and Grimson):
 *  1. For the components in order (heaviest first) take d2 = |x - mu|^2, summed r, g, b
 *     left to right. The sample is owned by the first component with
 *     d2 < var_threshold_gen * v. It is background if some component whose predecessors'
 *     weights sum to at most background_ratio (the background set: the heaviest
 *     components up to and including the first that takes the running sum past the
 *     ratio) has d2 < var_threshold * v.
 *  2. Every component's weight becomes (w + alpha * (o - w)) - alpha * c_T, o = 1 for
 *     the owner and 0 otherwise. The owner then moves towards the sample with
 *     rho = alpha / w (its new weight): mu += rho * (x - mu) per channel and
 *     v += rho * (d2 - v), v clamped to [var_min, var_max].
 *  3. Components whose weight fell below zero are removed, the rest keep their order.
 *  4. With no owner a component is created with weight alpha, mean x and variance
 *     var_init: appended, or replacing the last (lightest) one when K are in use.
 *  5. The weights are divided by their sum (taken in list order).
 *  6. The list is sorted by weight, heaviest first, equal weights keeping their order.
 */
int oracle_gmm_pixel(const uint8_t px[3], float *st, uint8_t *modes,
                     const orc_gmm_params *p) {
  const int K = p->n_mix;
  int M = *modes;
  if (M > K) M = K;
  const float x[3] = {(float)px[0], (float)px[1], (float)px[2]};
  float d2[ORC_GMM_MAX_MIX];

  /* 1 */
  int owner = -1, background = 0;
  float before = 0.0f;
  for (int m = 0; m < M; ++m) {
    const float *c = st + NF * m;
    const float dr = x[0] - c[MR], dg = x[1] - c[MG], db = x[2] - c[MB];
    float d = dr * dr;
    d = d + dg * dg;
    d = d + db * db;
    d2[m] = d;
    if (owner < 0 && d < p->var_threshold_gen * c[V_]) owner = m;
    if (before <= p->background_ratio && d < p->var_threshold * c[V_]) background = 1;
    before = before + c[W_];
  }

  /* 2 */
  const float decay = p->alpha * p->complexity_reduction;
  for (int m = 0; m < M; ++m) {
    float *c = st + NF * m;
    const float o = m == owner ? 1.0f : 0.0f;
    c[W_] = (c[W_] + p->alpha * (o - c[W_])) - decay;
  }
  if (owner >= 0) {
    float *c = st + NF * owner;
    const float rho = p->alpha / c[W_];
    c[MR] = c[MR] + rho * (x[0] - c[MR]);
    c[MG] = c[MG] + rho * (x[1] - c[MG]);
    c[MB] = c[MB] + rho * (x[2] - c[MB]);
    float v = c[V_] + rho * (d2[owner] - c[V_]);
    if (v < p->var_min) v = p->var_min;
    if (v > p->var_max) v = p->var_max;
    c[V_] = v;
  }

  /* 3 */
  int kept = 0;
  for (int m = 0; m < M; ++m) {
    if (st[NF * m + W_] < 0.0f) continue;
    if (kept != m) memcpy(st + NF * kept, st + NF * m, sizeof(float) * NF);
    ++kept;
  }
  M = kept;

  /* 4 */
  if (owner < 0) {
    const int at = M < K ? M : K - 1;
    float *c = st + NF * at;
    c[W_] = p->alpha;
    c[MR] = x[0];
    c[MG] = x[1];
    c[MB] = x[2];
    c[V_] = p->var_init;
    M = at + 1;
  }

  /* 5 */
  float sum = 0.0f;
  for (int m = 0; m < M; ++m) sum = sum + st[NF * m + W_];
  for (int m = 0; m < M; ++m) st[NF * m + W_] = st[NF * m + W_] / sum;

  /* 6: insertion sort, stable */
  for (int m = 1; m < M; ++m) {
    float tmp[NF];
    memcpy(tmp, st + NF * m, sizeof tmp);
    int j = m;
    while (j > 0 && st[NF * (j - 1) + W_] < tmp[W_]) {
      memcpy(st + NF * j, st + NF * (j - 1), sizeof tmp);
      --j;
    }
    memcpy(st + NF * j, tmp, sizeof tmp);
  }

  *modes = (uint8_t)M;
  return !background;
}

int oracle_gmm_update(const uint8_t *frames, int64_t n_px, float *state, uint8_t *modes,
                      uint8_t *mask, const orc_gmm_params *p) {
  if (!params_ok(p) || n_px < 0 || (n_px > 0 && (!frames || !state || !modes || !mask)))
    return 1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n_px; ++i)
    mask[i] = (uint8_t)oracle_gmm_pixel(frames + 3 * i, state + (int64_t)NF * p->n_mix * i,
                                        modes + i, p);
  return 0;
}

/*
 * Connected components by flood fill: pixels are visited in raster order, and each
 * foreground pixel not yet reached starts a component, which a stack-based fill grows
 * through the eight neighbours of every pixel it takes. The component's bounding box
 * and pixel count are kept if the count reaches min_area.
 */
int64_t oracle_mask_rois(const uint8_t *mask, int32_t n_frames, int32_t width,
                         int32_t height, int32_t min_area, int32_t *rows, int64_t *areas,
                         int64_t cap, int32_t *frame_begin) {
  if (n_frames < 0 || width < 1 || height < 1 || cap < 0 || !frame_begin ||
      (n_frames > 0 && !mask) || (cap > 0 && (!rows || !areas)))
    return -1;
  const int64_t n = (int64_t)width * height;
  uint8_t *seen = malloc(n > 0 ? (size_t)n : 1);
  int64_t *stack = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
  if (!seen || !stack) {
    free(seen);
    free(stack);
    return -1;
  }
  int64_t count = 0;
  for (int32_t f = 0; f < n_frames; ++f) {
    frame_begin[f] = (int32_t)count;
    const uint8_t *m = mask + (int64_t)f * n;
    memset(seen, 0, (size_t)n);
    for (int64_t start = 0; start < n; ++start) {
      if (!m[start] || seen[start]) continue;
      int64_t top = 0, area = 0;
      int32_t x0 = width, y0 = height, x1 = -1, y1 = -1;
      stack[top++] = start;
      seen[start] = 1;
      while (top > 0) {
        const int64_t q = stack[--top];
        const int32_t qx = (int32_t)(q % width), qy = (int32_t)(q / width);
        ++area;
        if (qx < x0) x0 = qx;
        if (qx > x1) x1 = qx;
        if (qy < y0) y0 = qy;
        if (qy > y1) y1 = qy;
        for (int dy = -1; dy <= 1; ++dy)
          for (int dx = -1; dx <= 1; ++dx) {
            const int32_t nx = qx + dx, ny = qy + dy;
            if (nx < 0 || ny < 0 || nx >= width || ny >= height) continue;
            const int64_t r = (int64_t)ny * width + nx;
            if (m[r] && !seen[r]) {
              seen[r] = 1;
              stack[top++] = r;
            }
          }
      }
      if (area < min_area) continue;
      if (count < cap) {
        int32_t *row = rows + 5 * count;
        row[0] = f;
        row[1] = x0;
        row[2] = y0;
        row[3] = x1 - x0 + 1;
        row[4] = y1 - y0 + 1;
        areas[count] = area;
      }
      ++count;
    }
  }
  frame_begin[n_frames] = (int32_t)count;
  free(seen);
  free(stack);
  return count;
}
