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
Plain loops over numpy float32 scalars, and the same test applied to a frame's kept list
at once with numpy float32 arrays (`suppressed_by_any`, operation for operation the scalar
`suppresses`, including how Python's min and max treat NaN); nothing here imports the
library.
"""
from __future__ import annotations

import numpy as np

f32 = np.float32


def suppresses(a, b, thr):
    """Whether box a = (x1, y1, x2, y2) suppresses box b at IoU threshold thr."""
    with np.errstate(over="ignore", invalid="ignore"):  # IEEE infinities and NaN are inputs
        return _suppresses(a, b, thr)


def _suppresses(a, b, thr):
    zero = f32(0)
    w = max(zero, f32(min(a[2], b[2]) - max(a[0], b[0])))
    h = max(zero, f32(min(a[3], b[3]) - max(a[1], b[1])))
    inter = f32(w * h)
    area_a = f32(max(zero, f32(a[2] - a[0])) * max(zero, f32(a[3] - a[1])))
    area_b = f32(max(zero, f32(b[2] - b[0])) * max(zero, f32(b[3] - b[1])))
    union = f32(f32(area_a + area_b) - inter)
    return bool(inter > f32(f32(thr) * union))


def _pmin(a, b):
    """Python's min(a, b) elementwise: a unless b < a (so a NaN a stays, a NaN b is
    ignored)."""
    return np.where(b < a, b, a)


def _pmax(a, b):
    """Python's max(a, b) elementwise: a unless b > a."""
    return np.where(b > a, b, a)


def suppressed_by_any(kept, b, thr, kept_roi=None, roi_b=None):
    """Whether any box of kept (float32 [K, 4], x1 y1 x2 y2) suppresses box b, i.e.
    any(suppresses(kept[j], b, thr)) over the rows j whose kept_roi differs from roi_b
    (all rows when kept_roi is None), with the same binary32 operations as suppresses."""
    if len(kept) == 0:
        return False
    with np.errstate(over="ignore", invalid="ignore"):
        return _suppressed_by_any(kept, b, thr, kept_roi, roi_b)


def _suppressed_by_any(kept, b, thr, kept_roi, roi_b):
    zero = f32(0)
    a0, a1, a2, a3 = (kept[:, c] for c in range(4))
    b0, b1, b2, b3 = (f32(v) for v in b)
    w = _pmax(zero, (_pmin(a2, b2) - _pmax(a0, b0)).astype(f32))
    h = _pmax(zero, (_pmin(a3, b3) - _pmax(a1, b1)).astype(f32))
    inter = (w * h).astype(f32)
    area_a = (_pmax(zero, (a2 - a0).astype(f32)) * _pmax(zero, (a3 - a1).astype(f32))).astype(f32)
    area_b = f32(max(zero, f32(b2 - b0)) * max(zero, f32(b3 - b1)))
    union = ((area_a + area_b).astype(f32) - inter).astype(f32)
    hit = inter > (f32(thr) * union).astype(f32)
    if kept_roi is not None:
        hit &= kept_roi != roi_b
    return bool(hit.any())


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
        kept_box = np.empty((len(ranked), 4), dtype=f32)
        kept_roi = np.empty(len(ranked), dtype=np.int64)
        K = 0
        for k in ranked:
            roi = int(dets[k]["roi"])
            if not suppressed_by_any(kept_box[:K], box[k], thr,
                                     kept_roi[:K] if cross_only else None, roi):
                keep[k] = True
                kept_box[K] = box[k]
                kept_roi[K] = roi
                K += 1
    return keep, dets[keep]
