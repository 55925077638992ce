"""Test infrastructure only: brute-force checkers for tiny inputs.

These use a different formulation from the C oracle so that the two can pin each
other: every canvas pixel searches *all* RoIs (not the plan's canvas lists), values
are rounded to binary16 by numpy's own float64 -> float16 conversion, and box
centres and offsets use numpy float32 arithmetic.
"""
from __future__ import annotations

import numpy as np


def norm_half_bits(x, k, mean, std) -> int:
    """binary16 bits of (x - mean_k) / std_k, rounded once from float64 by numpy."""
    q = (np.float64(x) - np.float64(np.float32(mean[k]))) / np.float64(np.float32(std[k]))
    return int(np.array(q, dtype=np.float64).astype(np.float16).view(np.uint16))


def stitch(frames, rois, place, first, count, canvas_w, canvas_h, mean, std, pad):
    """Per-pixel search over every RoI. frames uint8 [F,H,W,3]."""
    rois = np.asarray(rois).reshape(-1, 5)
    place = np.asarray(place).reshape(-1, 3)
    out = np.empty((count, 3, canvas_h, canvas_w), dtype=np.uint16)
    padv = [norm_half_bits(int(pad[k]), k, mean, std) for k in range(3)]
    for c in range(count):
        cid = first + c
        for Y in range(canvas_h):
            for X in range(canvas_w):
                owner = [i for i in range(rois.shape[0])
                         if place[i, 0] == cid
                         and place[i, 1] <= X < place[i, 1] + rois[i, 3]
                         and place[i, 2] <= Y < place[i, 2] + rois[i, 4]]
                assert len(owner) <= 1, "overlapping patches"
                for k in range(3):
                    if owner:
                        i = owner[0]
                        f, sx, sy = rois[i, 0], rois[i, 1], rois[i, 2]
                        v = frames[f, sy + Y - place[i, 2], sx + X - place[i, 1], k]
                        out[c, k, Y, X] = norm_half_bits(int(v), k, mean, std)
                    else:
                        out[c, k, Y, X] = padv[k]
    return out


def overlap_area(box, rect):
    """binary32 area of box (x1, y1, x2, y2) inside rect (x0, y0, x1, y1), one rounding per
    operation, 0 when they do not overlap."""
    f32 = np.float32
    w = f32(min(box[2], rect[2]) - max(box[0], rect[0]))
    h = f32(min(box[3], rect[3]) - max(box[1], rect[1]))
    return f32(max(w, f32(0)) * max(h, f32(0)))


def unstitch(boxes, box_canvas, rois, place, n_canvases, clip=True, rule=0):
    """Per-box search over every RoI; returns (roi_of_box, list of det tuples). rule 0:
    the RoI holding the centre; rule 1: the RoI overlapped most (ties: lower id)."""
    rois = np.asarray(rois).reshape(-1, 5)
    place = np.asarray(place).reshape(-1, 3)
    boxes = np.asarray(boxes, dtype=np.float32).reshape(-1, 4)
    f32 = np.float32
    rob = np.full(boxes.shape[0], -1, dtype=np.int32)
    dets = []
    for b in range(boxes.shape[0]):
        c = int(box_canvas[b])
        if not 0 <= c < n_canvases:
            continue
        x1, y1, x2, y2 = (f32(v) for v in boxes[b])
        if rule == 1:
            if np.isnan([x1, y1, x2, y2]).any():
                continue
            best, hits = f32(0), []
            for i in range(rois.shape[0]):
                if place[i, 0] != c:
                    continue
                with np.errstate(invalid="ignore", over="ignore"):
                    a = overlap_area((x1, y1, x2, y2),
                                     (f32(place[i, 1]), f32(place[i, 2]),
                                      f32(place[i, 1] + rois[i, 3]), f32(place[i, 2] + rois[i, 4])))
                if a > best:  # ascending ids: the first maximum is the lowest id
                    best, hits = a, [i]
        else:
            with np.errstate(invalid="ignore", over="ignore"):
                cx = f32(f32(x1 + x2) * f32(0.5))
                cy = f32(f32(y1 + y2) * f32(0.5))
            hits = [i for i in range(rois.shape[0])
                    if place[i, 0] == c
                    and f32(place[i, 1]) <= cx < f32(place[i, 1] + rois[i, 3])
                    and f32(place[i, 2]) <= cy < f32(place[i, 2] + rois[i, 4])]
        assert len(hits) <= 1
        if not hits:
            continue
        i = hits[0]
        rob[b] = i
        dx, dy, w, h = int(place[i, 1]), int(place[i, 2]), int(rois[i, 3]), int(rois[i, 4])
        v = [x1, y1, x2, y2]
        if clip:
            lo = [f32(dx), f32(dy), f32(dx), f32(dy)]
            hi = [f32(dx + w), f32(dy + h), f32(dx + w), f32(dy + h)]
            v = [min(max(v[q], lo[q]), hi[q]) for q in range(4)]
        ox, oy = f32(int(rois[i, 1]) - dx), f32(int(rois[i, 2]) - dy)
        with np.errstate(over="ignore"):
            dets.append((b, i, int(rois[i, 0]), f32(v[0] + ox), f32(v[1] + oy),
                         f32(v[2] + ox), f32(v[3] + oy)))
    return rob, dets
