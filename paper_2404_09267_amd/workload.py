"""Seeded synthetic workloads for the patch-stitching path.

This module is shared by the GPU path's tests/bench and by the oracle's tests, so it
holds input recipes only: RoI rectangles, frame pixels, detector boxes and the
constants of each workload. No packing, normalisation or box remapping happens here.

The paper measures on PANDA4K (gigapixel scenes resized to 3840x2160, Sec. V-A),
which is not available; these workloads stand in for it with the frame sizes,
camera counts and RoI-size ranges of the five named scenarios below.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# ImageNet statistics in uint8 units, RGB order, and the letterbox grey pad value.
MEAN = (123.675, 116.28, 103.53)
STD = (58.395, 57.12, 57.375)
PAD = (114, 114, 114)


@dataclass(frozen=True)
class Workload:
    name: str
    index: int              # seeds derive from it: RoIs 1000+i, pixels 2000+i, boxes 3000+i
    cameras: int
    frames_per_camera: int
    frame_w: int
    frame_h: int
    rois_per_frame: int
    roi_dist: str           # "uniform" | "loguniform" | "loguniform_aspect"
    roi_lo: int
    roi_hi: int
    canvas: int             # square canvas side
    batch_cap: int          # canvases per batch; 0 = all canvases in one batch
    n_boxes: int
    box_mode: str           # "inside" (box fully inside the canvas) | "centre"
    box_lo: float
    box_hi: float

    @property
    def n_frames(self) -> int:
        return self.cameras * self.frames_per_camera

    @property
    def n_rois(self) -> int:
        return self.n_frames * self.rois_per_frame

    @property
    def frame_bytes(self) -> int:
        return self.frame_w * self.frame_h * 3


WORKLOADS = {
    "cam1_1080p": Workload("cam1_1080p", 0, 1, 1, 1920, 1080, 16, "uniform", 32, 256,
                           1024, 0, 200, "inside", 4.0, 256.0),
    "cam5_4k": Workload("cam5_4k", 1, 5, 1, 3840, 2160, 40, "loguniform_aspect", 32, 512,
                        1024, 0, 2000, "inside", 4.0, 256.0),
    "cam20_4k": Workload("cam20_4k", 2, 20, 1, 3840, 2160, 100, "loguniform", 32, 640,
                         1280, 32, 10000, "centre", 4.0, 256.0),
    "small_roi_8cam": Workload("small_roi_8cam", 3, 8, 1, 3840, 2160, 2000, "uniform", 8, 64,
                               640, 0, 50000, "centre", 4.0, 48.0),
    "window_64x30": Workload("window_64x30", 4, 64, 30, 3840, 2160, 60, "loguniform", 32, 512,
                             1024, 64, 200000, "centre", 4.0, 256.0),
}
ORDERED = ["cam1_1080p", "cam5_4k", "cam20_4k", "small_roi_8cam", "window_64x30"]


def _sides(rng: np.random.Generator, wl: Workload, n: int):
    lo, hi = wl.roi_lo, wl.roi_hi
    if wl.roi_dist == "uniform":
        return rng.integers(lo, hi + 1, size=n), rng.integers(lo, hi + 1, size=n)
    if wl.roi_dist == "loguniform":
        w = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=n)))
        h = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=n)))
        return w.astype(np.int64), h.astype(np.int64)
    if wl.roi_dist == "loguniform_aspect":
        # draw both sides log-uniformly and redraw the pair until 0.5 <= h/w <= 2
        ws, hs = [], []
        got = 0
        while got < n:
            w = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=2 * n)))
            h = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=2 * n)))
            keep = (h >= 0.5 * w) & (h <= 2.0 * w)
            ws.append(w[keep]); hs.append(h[keep])
            got += int(keep.sum())
        return (np.concatenate(ws)[:n].astype(np.int64),
                np.concatenate(hs)[:n].astype(np.int64))
    raise ValueError(wl.roi_dist)


def make_rois(wl: Workload, seed: int | None = None) -> np.ndarray:
    """int32 [n, 5] = {frame, x, y, w, h} in arrival order: time-major, then camera,
    then RoI. Frame id = t * cameras + camera. Positions uniform inside the frame."""
    rng = np.random.default_rng(1000 + wl.index if seed is None else seed)
    n = wl.n_rois
    w, h = _sides(rng, wl, n)
    x = rng.integers(0, wl.frame_w - w + 1)
    y = rng.integers(0, wl.frame_h - h + 1)
    frame = np.repeat(np.arange(wl.n_frames, dtype=np.int64), wl.rois_per_frame)
    return np.stack([frame, x, y, w, h], axis=1).astype(np.int32)


def make_boxes(wl: Workload, n_canvases: int, seed: int | None = None):
    """(boxes float32 [n, 4] = x1,y1,x2,y2 in canvas pixels, canvas int32 [n])."""
    rng = np.random.default_rng(3000 + wl.index if seed is None else seed)
    n, C = wl.n_boxes, wl.canvas
    bw = rng.uniform(wl.box_lo, wl.box_hi, size=n)
    bh = rng.uniform(wl.box_lo, wl.box_hi, size=n)
    if wl.box_mode == "inside":
        x1 = rng.uniform(0.0, C - bw)
        y1 = rng.uniform(0.0, C - bh)
        x2, y2 = x1 + bw, y1 + bh
    else:
        cx = rng.uniform(0.0, C, size=n)
        cy = rng.uniform(0.0, C, size=n)
        x1, x2 = cx - 0.5 * bw, cx + 0.5 * bw
        y1, y2 = cy - 0.5 * bh, cy + 0.5 * bh
    canvas = rng.integers(0, max(n_canvases, 1), size=n)
    boxes = np.stack([x1, y1, x2, y2], axis=1).astype(np.float32)
    return boxes, canvas.astype(np.int32)


def make_frames(wl: Workload, device, seed: int | None = None, n_frames: int | None = None):
    """uint8 [F, H, W, 3] uniform random pixels, generated where they will live."""
    import torch

    F = wl.n_frames if n_frames is None else n_frames
    g = torch.Generator(device=device)
    g.manual_seed(2000 + wl.index if seed is None else seed)
    return torch.randint(0, 256, (F, wl.frame_h, wl.frame_w, 3), dtype=torch.uint8,
                         device=device, generator=g)


def random_frames_np(n_frames: int, h: int, w: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(n_frames, h, w, 3), dtype=np.uint8)


def random_rois(rng: np.random.Generator, n: int, n_frames: int, frame_w: int, frame_h: int,
                lo: int, hi_w: int, hi_h: int) -> np.ndarray:
    """Small random RoI tables for tests: sides uniform in [lo, hi], inside the frame."""
    w = rng.integers(lo, min(hi_w, frame_w) + 1, size=n)
    h = rng.integers(lo, min(hi_h, frame_h) + 1, size=n)
    x = rng.integers(0, frame_w - w + 1)
    y = rng.integers(0, frame_h - h + 1)
    f = rng.integers(0, n_frames, size=n)
    return np.stack([f, x, y, w, h], axis=1).astype(np.int32)


def camera_arrival_trace(wl: Workload, rounds=((0.0, 0.5), (0.3, 0.25)), fps: float = 30.0,
                         cap: int = 32, seed: int = 5):
    """An arrival trace for the SLO-aware invoker: the workload's RoIs as patches, frame
    f of the round sent at offset + f / (fps * n_frames) plus up to 4 ms of jitter, with
    deadline = arrival + the round's SLO; `rounds` lists (offset s, SLO s). Also returns a
    synthetic latency table (mean, std per batch of 1..cap canvases) that grows with the
    batch. Returns (w, h, t_arrive, t_ddl, lat_mean, lat_std) as numpy arrays."""
    rois = make_rois(wl)
    rng = np.random.default_rng(seed)
    per = len(rois) // wl.n_frames
    t = np.repeat(np.arange(wl.n_frames) * (1.0 / fps / wl.n_frames), per)
    t = np.sort(t + rng.uniform(0, 0.004, len(t)))
    w = np.concatenate([rois[: len(t), 3]] * len(rounds))
    h = np.concatenate([rois[: len(t), 4]] * len(rounds))
    t_arrive = np.concatenate([t + off for off, _ in rounds])
    t_ddl = np.concatenate([t + off + slo for off, slo in rounds])
    b = np.arange(1, cap + 1)
    return w, h, t_arrive, t_ddl, 0.02 + 0.012 * b, 0.002 + 0.0005 * b


def make_gmm_boxes(n_frames: int, per_frame: int, frame_w: int, frame_h: int, seed: int,
                   lo: int = 8, hi: int = 160, clusters: int = 4):
    """Synthetic background-model RoIs (the input of adaptive frame partitioning), grouped
    by frame: per frame a count uniform in [0, 2 * per_frame], sides log-uniform in
    [lo, hi], 70 % of the boxes scattered around one of `clusters` centres (normal,
    sigma = frame_w / 12) and the rest uniform, every box clamped inside the frame.
    Returns (boxes int32 [n, 5] as (frame, x, y, w, h), frame_begin int32 [n_frames + 1])."""
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 2 * per_frame + 1, n_frames)
    frame_begin = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    n = int(frame_begin[-1])
    frame = np.repeat(np.arange(n_frames), counts)
    w = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), n))).astype(np.int64)
    h = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), n))).astype(np.int64)
    w = np.clip(w, 1, frame_w)
    h = np.clip(h, 1, frame_h)
    cx = rng.uniform(0, frame_w, (n_frames, clusters))
    cy = rng.uniform(0, frame_h, (n_frames, clusters))
    pick = rng.integers(0, clusters, n)
    near = rng.random(n) < 0.7
    sd = frame_w / 12.0
    x = np.where(near, cx[frame, pick] + rng.normal(0, sd, n), rng.uniform(0, frame_w, n))
    y = np.where(near, cy[frame, pick] + rng.normal(0, sd, n), rng.uniform(0, frame_h, n))
    x = np.clip(np.rint(x - w / 2), 0, frame_w - w).astype(np.int64)
    y = np.clip(np.rint(y - h / 2), 0, frame_h - h).astype(np.int64)
    boxes = np.stack([frame, x, y, w, h], 1).astype(np.int32)
    return boxes, frame_begin


class SyntheticVideo:
    """Seeded stand-in for the paper's fixed high-resolution cameras (PANDA4K video is not
    available), the input of the background model. Per camera: a static background of
    16 x 16-pixel cells of random RGB levels in [40, 200), integer sensor noise in [-noise, noise]
    (random bytes spread evenly over the range) redrawn every frame (slices of one seeded bank), and `objects` solid
    RGB rectangles with log-uniform sides in [lo, hi] moving at constant velocity (each
    axis uniform in [-max_speed, max_speed] px per frame) and bouncing off the frame edges.
    frame(t) returns uint8 [cameras, height, width, 3]."""

    def __init__(self, cameras: int, width: int, height: int, objects: int = 40, lo: int = 16,
                 hi: int = 256, max_speed: float = 8.0, noise: int = 3, seed: int = 0):
        rng = np.random.default_rng(seed)
        self.cameras, self.width, self.height, self.noise = cameras, width, height, noise
        cell = 16
        gh, gw = -(-height // cell), -(-width // cell)
        coarse = rng.integers(40, 200, (cameras, gh, gw, 3), dtype=np.uint8)
        # stored lowered by `noise`, so that adding a bank value in [0, 2 noise] stays in uint8
        bg = np.repeat(np.repeat(coarse - np.uint8(noise), cell, axis=1), cell, axis=2)
        self.bg = np.ascontiguousarray(bg[:, :height, :width])
        self.n = cameras * height * width * 3
        self.bank_slack = 1 << 20
        # random bytes mapped onto [0, 2 noise] by (b * (2 noise + 1)) >> 8
        lut = ((np.arange(256) * (2 * noise + 1)) >> 8).astype(np.uint8)
        self.bank = lut[np.frombuffer(rng.bytes(self.n + self.bank_slack), dtype=np.uint8)]
        k = cameras * objects
        self.obj_cam = np.repeat(np.arange(cameras), objects)
        self.obj_w = np.clip(np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), k))), 1, width).astype(np.int64)
        self.obj_h = np.clip(np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), k))), 1, height).astype(np.int64)
        self.obj_x = rng.uniform(0, 1, k) * (width - self.obj_w)
        self.obj_y = rng.uniform(0, 1, k) * (height - self.obj_h)
        self.obj_vx = rng.uniform(-max_speed, max_speed, k)
        self.obj_vy = rng.uniform(-max_speed, max_speed, k)
        self.obj_rgb = rng.integers(0, 256, (k, 3), dtype=np.uint8)

    @staticmethod
    def _bounce(p0, v, t, span):
        if span <= 0:
            return 0
        m = (p0 + v * t) % (2 * span)
        return int(m if m <= span else 2 * span - m)

    def frame(self, t: int) -> np.ndarray:
        off = (t * 1_000_003) % self.bank_slack
        f = self.bg + self.bank[off: off + self.n].reshape(self.bg.shape)
        for i in range(len(self.obj_cam)):
            w, h = int(self.obj_w[i]), int(self.obj_h[i])
            x = self._bounce(self.obj_x[i], self.obj_vx[i], t, self.width - w)
            y = self._bounce(self.obj_y[i], self.obj_vy[i], t, self.height - h)
            f[self.obj_cam[i], y: y + h, x: x + w] = self.obj_rgb[i]
        return f


def gmm_alpha(t: int, history: int = 500) -> float:
    """Learning rate handed to the background model for frame t: 1 / (t + 1) while the
    model warms up, then 1 / history (a running mean of the first frames, then an
    exponential window of `history` frames)."""
    return 1.0 / min(t + 1, history)


# The background-model workload of the bench: the 20 cameras of cam20_4k, 5 components.
GMM_BENCH = dict(cameras=20, width=3840, height=2160, n_mix=5, objects=40, seed=7)
