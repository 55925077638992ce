"""Test infrastructure only: adaptive frame partitioning, written out literally.

Follows Alg. 1 and its description (Sec. III-A, Adaptive Frame Partitioning): the frame is
divided into X x Y zones of equal size; every RoI goes to the zone it overlaps most;
every zone that received RoIs becomes one patch, the minimum rectangle enclosing them.
Readings where the paper is silent:
  - zone i of X spans columns [floor(i W / X), floor((i + 1) W / X)) (likewise rows), so
    the zones tile the frame exactly even when X does not divide W;
  - zones are numbered row-major (r = j X + i) and an overlap tie goes to the lower r;
  - the patch is the enclosing rectangle itself, not clipped to its zone;
  - patches are listed frame by frame, zones in row-major order (the algorithm's loop
    over zones).
Nothing here imports the library.
"""
from __future__ import annotations


def zone_bounds(k, n, size):
    """[start, end) of zone k of n along an axis of `size` pixels."""
    return (k * size) // n, ((k + 1) * size) // n


def overlap_area(box, rect):
    """Area of the intersection of two [x0, x1) x [y0, y1) rectangles."""
    w = min(box[2], rect[2]) - max(box[0], rect[0])
    h = min(box[3], rect[3]) - max(box[1], rect[1])
    return max(w, 0) * max(h, 0)


def partition_frame(boxes, frame_w, frame_h, zones_x, zones_y):
    """boxes: list of (x, y, w, h) of one frame. Returns (zone of each box, patches as
    (x, y, w, h) in zone order)."""
    zones = []
    for j in range(zones_y):
        y0, y1 = zone_bounds(j, zones_y, frame_h)
        for i in range(zones_x):
            x0, x1 = zone_bounds(i, zones_x, frame_w)
            zones.append((x0, y0, x1, y1))
    lists = [[] for _ in zones]
    zone_of = []
    for (x, y, w, h) in boxes:
        b = (x, y, x + w, y + h)
        areas = [overlap_area(b, z) for z in zones]
        best = max(range(len(zones)), key=lambda r: (areas[r], -r))  # first maximum
        lists[best].append(b)
        zone_of.append(best)
    patches = []
    for members in lists:
        if members:
            x0 = min(b[0] for b in members)
            y0 = min(b[1] for b in members)
            x1 = max(b[2] for b in members)
            y1 = max(b[3] for b in members)
            patches.append((x0, y0, x1 - x0, y1 - y0))
    return zone_of, patches


def partition(boxes, frame_begin, frame_w, frame_h, zones_x, zones_y):
    """boxes: rows (frame, x, y, w, h) grouped by frame through frame_begin. Returns
    (zone of each box, patches as rows (frame, x, y, w, h))."""
    zone_of, patches = [], []
    for f in range(len(frame_begin) - 1):
        rows = boxes[frame_begin[f]:frame_begin[f + 1]]
        z, p = partition_frame([tuple(int(v) for v in r[1:5]) for r in rows], frame_w, frame_h,
                               zones_x, zones_y)
        zone_of += z
        patches += [(f,) + q for q in p]
    return zone_of, patches
