"""Host side of tg_stitch's launch: unit geometry (tg_stitch_units), the heaviest-first
unit order (tg_stitch_schedule) and which exact normalisation path a mean/std takes
(tg_stitch_norm_uses_table). No GPU needed."""
import ctypes
import math

import numpy as np
import pytest

from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

from stitch_geometry import TILE_W, geometry


def unit_weights(rois, plan, first, count, cw, ch):
    """Canvas pixels covered by patches in each unit, pixel by pixel (small canvases)."""
    tiles, band_rows, bands, n_units = geometry(cw, ch, count)
    w = np.zeros(n_units, np.int64)
    for c in range(count):
        cov = np.zeros((ch, cw), np.int64)
        j = first + c
        for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]:
            _, x, y = plan.place[i]
            cov[y:y + rois[i, 4], x:x + rois[i, 3]] += 1
        for by in range(bands):
            for tx in range(tiles):
                w[(c * bands + by) * tiles + tx] = cov[by * band_rows:(by + 1) * band_rows,
                                                       tx * TILE_W:(tx + 1) * TILE_W].sum()
    return w


@pytest.mark.parametrize("cw,ch,count", [(1280, 1280, 32), (1280, 1280, 31), (1024, 1024, 9),
                                         (640, 640, 53), (1024, 1024, 1), (1920, 1080, 5),
                                         (1, 1, 1), (2561, 7, 3), (64, 50000, 1)])
def test_unit_count_matches_geometry(cw, ch, count):
    assert tg.stitch_units(cw, ch, count) == geometry(cw, ch, count)[3]


def test_unit_count_edges():
    assert tg.stitch_units(1280, 1280, 0) == 0
    for bad in [(0, 10, 1), (10, 0, 1), (10, 10, -1)]:
        assert tg.lib().tg_stitch_units(*bad) == tg.E_INVAL


@pytest.mark.parametrize("policy", [0, 1, 2])
def test_schedule_is_heaviest_first_permutation(policy):
    rng = np.random.default_rng(40 + policy)
    rois = W.random_rois(rng, 300, 3, 700, 500, 4, 200, 200)
    cw = ch = 320
    plan = tg.plan_pack(rois, cw, ch, 700, 500, 3, policy)
    J = plan.n_canvases
    assert J >= 4
    for first, count in [(0, J), (1, J - 2), (J - 1, 1)]:
        order = tg.stitch_schedule(rois, plan, first, count, cw, ch)
        n_units = geometry(cw, ch, count)[3]
        assert sorted(order.tolist()) == list(range(n_units))
        w = unit_weights(rois, plan, first, count, cw, ch)[order]
        assert np.all(np.diff(w) <= 0), "not heaviest first"
        # equal weights keep unit order (stable)
        for i in range(len(order) - 1):
            if w[i] == w[i + 1]:
                assert order[i] < order[i + 1]


def test_schedule_with_tall_units():
    """Units of more than 2^16 pixels (a 1280 x 600000 canvas): weights as the summed
    intersection areas of unit and patch rectangles."""
    cw, ch = 1280, 600000
    tiles, band_rows, bands, n_units = geometry(cw, ch, 1)
    assert band_rows * TILE_W >= 1 << 16
    rng = np.random.default_rng(7)
    k = 400
    w = rng.integers(1, 600, k)
    h = rng.integers(1, 4 * band_rows, k)
    x = rng.integers(0, cw - w + 1)
    y = rng.integers(0, ch - h + 1)
    rois = np.stack([np.zeros(k), np.zeros(k), np.zeros(k), w, h], 1).astype(np.int32)
    place = np.stack([np.zeros(k), x, y], 1).astype(np.int32)
    plan = tg.Plan(place, np.arange(k, dtype=np.int32), np.array([0, k], np.int32), 1)
    order = tg.stitch_schedule(rois, plan, 0, 1, cw, ch)
    assert sorted(order.tolist()) == list(range(n_units))
    ub = np.arange(n_units) // tiles
    ut = np.arange(n_units) % tiles
    ox = (np.minimum(x + w, (ut[:, None] + 1) * TILE_W) - np.maximum(x, ut[:, None] * TILE_W))
    oy = (np.minimum(y + h, (ub[:, None] + 1) * band_rows) - np.maximum(y, ub[:, None] * band_rows))
    weight = (np.clip(ox, 0, None) * np.clip(oy, 0, None)).sum(1)
    assert weight.max() >= 1 << 16
    ws = weight[order]
    assert np.all(np.diff(ws) <= 0)
    tie = ws[:-1] == ws[1:]
    assert np.all(order[:-1][tie] < order[1:][tie])


def test_schedule_on_cam20_batches():
    wl = W.WORKLOADS["cam20_4k"]
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    for k in range(tg.batch_count(plan.n_canvases, wl.batch_cap)):
        first, count = tg.batch_range(plan.n_canvases, wl.batch_cap, k)
        order = tg.stitch_schedule(rois, plan, first, count, wl.canvas, wl.canvas)
        assert np.array_equal(np.sort(order), np.arange(tg.stitch_units(wl.canvas, wl.canvas,
                                                                         count)))


def test_schedule_skips_corrupt_entries_and_checks_arguments():
    rois = np.array([[0, 0, 0, 10, 10], [0, 5, 5, 10, 10], [0, 0, 0, 4, 4]], np.int32)
    place = np.array([[0, 0, 0], [0, 0, 20], [1, 0, 0]], np.int32)
    plan = tg.Plan(place, np.array([0, 1, 2], np.int32), np.array([0, 2, 3], np.int32), 2)
    good = tg.stitch_schedule(rois, plan, 0, 2, 32, 32)
    bad = tg.Plan(place.copy(), np.array([0, 7, 2], np.int32), plan.canvas_begin, 2)
    bad.place[0] = [1, 0, 0]  # claims another canvas than its order segment
    order = tg.stitch_schedule(rois, bad, 0, 2, 32, 32)
    assert sorted(order.tolist()) == sorted(good.tolist())
    # canvas 0 now has no valid patch, canvas 1 keeps its 4 x 4 one: its unit is first
    tiles, band_rows, bands, _ = geometry(32, 32, 2)
    assert order[0] == (1 * bands + 0) * tiles + 0
    out = np.zeros(64, np.int32)
    L = tg.lib()
    r = np.ascontiguousarray(rois)

    def call(first, count, cw=32, ch=32, o=out, n_canvases=2):
        return L.tg_stitch_schedule(r.ctypes.data, place.ctypes.data, plan.order.ctypes.data,
                                    plan.canvas_begin.ctypes.data, 3, n_canvases, first,
                                    count, cw, ch, o.ctypes.data if o is not None else None)

    assert call(1, 2) == tg.E_RANGE
    assert call(0, 0) == tg.OK
    assert call(0, 1, cw=0) == tg.E_INVAL
    assert call(-1, 1) == tg.E_INVAL
    assert call(0, 1, o=None) == tg.E_INVAL


# Triples for which no fp32 (a, c) reproduces every correctly rounded byte exactly
# (found by a search over random mean/std); ImageNet's statistics have such pairs.
TABLE_CASES = [((174.00369262695312, 189.9988250732422, 150.99696350097656),
                (0.031708136200904846, 1.5641870498657227, 1.5637657642364502))]


def test_norm_path_selection():
    assert tg.stitch_norm_uses_table(W.MEAN, W.STD) is False
    assert tg.stitch_norm_uses_table((0, 0, 0), (255, 255, 255)) is False
    assert tg.stitch_norm_uses_table((10.5, 300.0, -7.25), (0.01, 1000.0, 3.5)) is False
    for mean, std in TABLE_CASES:
        assert tg.stitch_norm_uses_table(mean, std) is True
    for mean, std in [((0, 0, 0), (1, 0, 1)), ((0, float("nan"), 0), (1, 1, 1)),
                      ((0, 0, 0), (1, 1, float("inf")))]:
        with pytest.raises(tg.TgError):
            tg.stitch_norm_uses_table(mean, std)
    f3 = ctypes.c_float * 3
    assert tg.lib().tg_stitch_norm_uses_table(None, f3(1, 1, 1)) == tg.E_INVAL
