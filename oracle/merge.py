"""Test infrastructure only: per-frame merge of detections mapped back from patches.

The paper evaluates detections per source frame after stitching (Sec. V-D) and, when a
frame is cut into zone patches (Sec. III-A, Alg. 1), patches of one frame can overlap, so
one object can come back from two patches. This greedy per-frame suppression is the
library's reading (the paper does not spell one out):
  - a frame's detections are ranked by score, higher first; equal scores by box index,
    lower first; a NaN score ranks as -infinity;
  - walking that ranking, a detection is kept unless a detection kept before it in the same
    frame overlaps it by IoU > threshold (with `cross_only`, only one from another patch);
  - IoU > t is decided as inter > t * union in binary32, each operation rounded on its own:
    w = max(0, min(x2) - max(x1)), likewise h, inter = w * h, area = max(0, x2 - x1) *
    max(0, y2 - y1), union = (area_a + area_b) - inter;
  - detections whose frame id is outside [0, n_frames) are dropped;
  - kept detections are listed in their input order.
Plain loops over numpy float32 scalars; nothing here imports the library.
"""
from __future__ import annotations

import numpy as np

f32 = np.float32


def suppresses(a, b, thr):
    """Whether box a = (x1, y1, x2, y2) suppresses box b at IoU threshold thr."""
    zero = f32(0)
    w = max(zero, f32(min(a[2], b[2]) - max(a[0], b[0])))
    h = max(zero, f32(min(a[3], b[3]) - max(a[1], b[1])))
    inter = f32(w * h)
    area_a = f32(max(zero, f32(a[2] - a[0])) * max(zero, f32(a[3] - a[1])))
    area_b = f32(max(zero, f32(b[2] - b[0])) * max(zero, f32(b[3] - b[1])))
    union = f32(f32(area_a + area_b) - inter)
    return bool(inter > f32(f32(thr) * union))


def merge(dets, scores, n_frames, thr, cross_only=True):
    """dets: structured array with box, roi, frame, x1, y1, x2, y2 (tg_det); scores:
    float32 per input box. Returns (keep flag per detection, kept detections)."""
    n = len(dets)
    keep = np.zeros(n, dtype=bool)
    box = [tuple(f32(dets[k][c]) for c in ("x1", "y1", "x2", "y2")) for k in range(n)]

    def rank(k):
        s = f32(scores[int(dets[k]["box"])])
        return (-(s if s == s else f32(-np.inf)), int(dets[k]["box"]))

    for f in range(n_frames):
        ranked = sorted((k for k in range(n) if int(dets[k]["frame"]) == f), key=rank)
        kept = []
        for k in ranked:
            if not any(suppresses(box[j], box[k], thr)
                       for j in kept if not cross_only or dets[j]["roi"] != dets[k]["roi"]):
                keep[k] = True
                kept.append(k)
    return keep, dets[keep]
