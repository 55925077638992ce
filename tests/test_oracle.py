"""Pins for the CPU oracle, against what the paper and the mathematics fix.

Every check here is independent of the oracle's own code paths: hand-traced
examples (tests/golden), IEEE-754 values derived by hand, numpy's float16
conversion as the library routine for rounding, closed forms for equal squares,
geometric invariants, and per-pixel / per-box brute force over every RoI.
"""
import itertools

import numpy as np
import pytest

from conftest import load_golden
from paper_2404_09267_amd import workload as W

POLICIES = {"shelf_ffdh": 0, "shelf_arrival": 1, "guillotine_bssf": 2}


def np_half_bits(v):
    with np.errstate(over="ignore"):
        return int(np.array(v, dtype=np.float64).astype(np.float16).view(np.uint16))


# --------------------------------------------------------------------------- rounding

def test_half_golden(orc):
    g = load_golden("half_values.json")
    for e in g["rounding"]:
        assert orc.half_from_double(e["v"]) == int(e["bits"], 16), e


def test_half_matches_numpy_conversion(orc):
    """numpy's float64 -> float16 cast is correctly rounded (ties to even); the
    oracle must agree on random values, on every finite half, and on every exact
    midpoint between neighbouring halves (the tie cases)."""
    rng = np.random.default_rng(7)
    vals = list(rng.standard_normal(2000) * 10.0 ** rng.integers(-9, 6, size=2000))
    halves = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    vals += list(halves[::7]) + list(-halves[::11])
    mids = (halves[:-1] + halves[1:]) / 2.0  # exact in float64
    vals += list(mids[::3]) + list(-mids[::5])
    vals += [70000.0, -70000.0, 1e-30, -1e-30, float("inf"), -float("inf")]
    for v in vals:
        assert orc.half_from_double(v) == np_half_bits(v), v


def test_half_nan(orc):
    assert orc.half_from_double(float("nan")) & 0x7FFF == 0x7E00


def test_norm_golden(orc):
    for e in load_golden("half_values.json")["normalise"]:
        t = orc.norm_table(e["mean"], e["std"])
        for k in range(3):
            assert t[k, e["x"]] == int(e["bits"], 16), e


@pytest.mark.parametrize("mean,std", [(W.MEAN, W.STD), ((0, 0, 0), (255, 255, 255)),
                                      ((10.5, 200.25, 0.125), (0.75, 3.0, 1e-3))])
def test_norm_table_matches_numpy(orc, mean, std):
    t = orc.norm_table(mean, std)
    m32 = np.asarray(mean, dtype=np.float32).astype(np.float64)
    s32 = np.asarray(std, dtype=np.float32).astype(np.float64)
    x = np.arange(256, dtype=np.float64)
    for k in range(3):
        with np.errstate(over="ignore"):
            ref = ((x - m32[k]) / s32[k]).astype(np.float16).view(np.uint16)
        np.testing.assert_array_equal(t[k], ref)


# --------------------------------------------------------------------------- packing

def _pack(orc, ex, policy):
    cw, ch = ex["canvas"]
    fw, fh, nf = ex["frame"]
    return orc.pack(np.array(ex["rois"]), cw, ch, fw, fh, nf, POLICIES[policy])


@pytest.mark.parametrize("policy", list(POLICIES))
def test_pack_golden(orc, policy):
    n_checked = 0
    for ex in load_golden("pack_examples.json")["examples"]:
        if policy not in ex:
            continue
        want = ex[policy]
        rc, bad, plan = _pack(orc, ex, policy)
        assert rc == 0
        np.testing.assert_array_equal(plan.place, np.array(want["place"]), err_msg=ex["name"])
        np.testing.assert_array_equal(plan.order, np.array(want["order"]), err_msg=ex["name"])
        np.testing.assert_array_equal(plan.canvas_begin, np.array(want["canvas_begin"]))
        assert plan.n_canvases == len(want["canvas_begin"]) - 1
        cw, ch = ex["canvas"]
        assert orc.check_plan(ex["rois"], cw, ch, POLICIES[policy], plan.place, plan.order,
                              plan.canvas_begin, plan.n_canvases) == 0
        if "free" in want:
            free = orc.guillotine_free(np.array(ex["rois"]), cw, ch)
            np.testing.assert_array_equal(free, np.array(want["free"]), err_msg=ex["name"])
        n_checked += 1
    assert n_checked >= 2


@pytest.mark.parametrize("policy", list(POLICIES))
@pytest.mark.parametrize("C,s,n", [(10, 3, 20), (64, 8, 130), (1280, 320, 33), (7, 7, 3),
                                   (100, 1, 20000)])
def test_pack_equal_squares_closed_form(orc, policy, C, s, n):
    """n equal s x s squares on a C x C canvas: floor(C/s)^2 per canvas, every square
    on the grid of multiples of s, J = ceil(n / floor(C/s)^2)."""
    rois = np.array([[0, 0, 0, s, s]] * n)
    rc, _, plan = orc.pack(rois, C, C, C, C, 1, POLICIES[policy])
    assert rc == 0
    per = (C // s) ** 2
    assert plan.n_canvases == -(-n // per)
    assert np.all(np.diff(plan.canvas_begin)[:-1] == per)
    assert np.all(plan.place[:, 1:] % s == 0)
    if policy != "guillotine_bssf":  # shelves fill row-major
        k = np.arange(n) % per
        np.testing.assert_array_equal(plan.place[plan.order, 1], (k % (C // s)) * s)
        np.testing.assert_array_equal(plan.place[plan.order, 2], (k // (C // s)) * s)


def test_guillotine_grid_trace(orc):
    """Hand trace, C = 10, s = 3: every cut lies on a grid line."""
    rc, _, plan = orc.pack(np.array([[0, 0, 0, 3, 3]] * 9), 10, 10, 10, 10, 1, 2)
    want = [(0, 0), (3, 0), (6, 0), (0, 3), (0, 6), (3, 3), (6, 3), (3, 6), (6, 6)]
    assert [tuple(p) for p in plan.place[:, 1:]] == want


@pytest.mark.parametrize("policy", list(POLICIES))
def test_pack_single_and_full(orc, policy):
    rc, _, plan = orc.pack(np.array([[0, 5, 6, 7, 8]]), 16, 16, 32, 32, 1, POLICIES[policy])
    assert rc == 0 and plan.n_canvases == 1 and plan.place.tolist() == [[0, 0, 0]]
    rc, _, plan = orc.pack(np.array([[0, 0, 0, 16, 16]] * 3), 16, 16, 16, 16, 1, POLICIES[policy])
    assert plan.n_canvases == 3 and plan.place.tolist() == [[0, 0, 0], [1, 0, 0], [2, 0, 0]]
    rc, _, plan = orc.pack(np.zeros((0, 5)), 16, 16, 16, 16, 1, POLICIES[policy])
    assert rc == 0 and plan.n_canvases == 0 and plan.canvas_begin.tolist() == [0]


def test_pack_validation(orc):
    ok = [0, 0, 0, 4, 4]
    cases = [
        ([ok, [0, 0, 0, 0, 4]], orc.E_INVAL, 1),
        ([ok, ok, [0, 0, 0, 4, -1]], orc.E_INVAL, 2),
        ([[1, 0, 0, 4, 4]], orc.E_ROI_OOB, 0),      # frame id == n_frames
        ([ok, [-1, 0, 0, 4, 4]], orc.E_ROI_OOB, 1),
        ([ok, [0, 17, 0, 4, 4]], orc.E_ROI_OOB, 1),  # x + w > frame_w
        ([ok, [0, 0, -1, 4, 4]], orc.E_ROI_OOB, 1),
        ([ok, [0, 0, 0, 9, 4]], orc.E_ROI_TOO_LARGE, 1),
        ([[0, 0, 0, 4, 9], [0, 30, 0, 4, 4]], orc.E_ROI_TOO_LARGE, 0),  # first bad RoI wins
    ]
    for rois, code, bad in cases:
        for pol in range(3):
            rc, b, _ = orc.pack(np.array(rois), 8, 8, 20, 20, 1, pol)
            assert (rc, b) == (code, bad), (rois, pol)
    assert orc.pack(np.array([ok]), 8, 8, 20, 20, 1, 3)[0] == orc.E_INVAL
    assert orc.pack(np.array([ok]), 0, 8, 20, 20, 1, 0)[0] == orc.E_INVAL


def _random_case(rng):
    cw, ch = int(rng.integers(4, 90)), int(rng.integers(4, 90))
    fw, fh, nf = 100, 80, int(rng.integers(1, 4))
    n = int(rng.integers(0, 120))
    lo = 1
    rois = W.random_rois(rng, n, nf, fw, fh, lo, cw, ch)
    return rois, cw, ch, fw, fh, nf


@pytest.mark.parametrize("policy", list(POLICIES))
def test_pack_invariants_random(orc, policy):
    rng = np.random.default_rng(11 + POLICIES[policy])
    for _ in range(400):
        rois, cw, ch, fw, fh, nf = _random_case(rng)
        rc, _, plan = orc.pack(rois, cw, ch, fw, fh, nf, POLICIES[policy])
        assert rc == 0
        assert orc.check_plan(rois, cw, ch, POLICIES[policy], plan.place, plan.order,
                              plan.canvas_begin, plan.n_canvases) == 0


def test_guillotine_free_rects_tile_each_canvas(orc):
    """Placed rects and the final free rects cover every canvas exactly once."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        rois, cw, ch, fw, fh, nf = _random_case(rng)
        rc, _, plan = orc.pack(rois, cw, ch, fw, fh, nf, 2)
        free = orc.guillotine_free(rois, cw, ch)
        for j in range(plan.n_canvases):
            occ = np.zeros((ch, cw), dtype=np.int32)
            for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]:
                _, x, y = plan.place[i]
                occ[y:y + rois[i, 4], x:x + rois[i, 3]] += 1
            for c, x, y, w, h in free[free[:, 0] == j]:
                assert w > 0 and h > 0
                occ[y:y + h, x:x + w] += 1
            assert np.all(occ == 1)


def test_check_plan_catches_planted_mistakes(orc):
    """The invariant checker itself must reject broken plans."""
    ex = load_golden("pack_examples.json")["examples"][1]
    rois = np.array(ex["rois"])
    rc, _, plan = orc.pack(rois, 10, 8, 50, 50, 1, 0)

    def chk(place=None, order=None, cbeg=None, J=None, policy=0):
        return orc.check_plan(rois, 10, 8, policy,
                              plan.place if place is None else place,
                              plan.order if order is None else order,
                              plan.canvas_begin if cbeg is None else cbeg,
                              plan.n_canvases if J is None else J)

    assert chk() == 0
    o = plan.order.copy(); o[0] = o[1]
    assert chk(order=o) == 1
    assert chk(cbeg=np.array([0, 5, 8])) == 3
    assert chk(cbeg=np.array([0, 4, 7])) == 2
    p = plan.place.copy(); p[7, 1] = 10  # r7 pushed off the right edge
    assert chk(place=p) == 4
    p = plan.place.copy(); p[3, 1] = 5  # r3 slid onto r1
    assert chk(place=p) == 5
    o = plan.order.copy(); o[[0, 2]] = o[[2, 0]]  # breaks FFDH order (and shelves)
    assert chk(order=o) in (7, 8)
    # arrival policy demands input order
    assert chk(policy=1) == 8
    # next fit: move r2 back onto canvas 0's second shelf would overlap; instead claim
    # canvas 1's first RoI could not fit -- shrink it so it would have fitted
    rois_small = rois.copy(); rois_small[2, 3] = 1; rois_small[2, 4] = 2
    assert orc.check_plan(rois_small, 10, 8, 0, plan.place, plan.order,
                          plan.canvas_begin, plan.n_canvases) == 9


# --------------------------------------------------------------------------- stitch

def _tiny_stitch_case(rng, policy):
    fw, fh, nf = int(rng.integers(4, 17)), int(rng.integers(4, 17)), int(rng.integers(1, 3))
    cw, ch = int(rng.integers(4, 9)), int(rng.integers(4, 9))
    n = int(rng.integers(1, 7))
    rois = W.random_rois(rng, n, nf, fw, fh, 1, min(4, cw), min(4, ch))
    frames = W.random_frames_np(nf, fh, fw, int(rng.integers(1 << 30)))
    return frames, rois, cw, ch, fw, fh, nf


def test_stitch_matches_brute_force(orc):
    from oracle import brute

    rng = np.random.default_rng(21)
    mean, std, pad = W.MEAN, W.STD, W.PAD
    for _ in range(60):
        frames, rois, cw, ch, fw, fh, nf = _tiny_stitch_case(rng, 0)
        for policy in (0, 2):
            rc, _, plan = orc.pack(rois, cw, ch, fw, fh, nf, policy)
            assert rc == 0
            got = orc.stitch(frames, rois, plan, 0, plan.n_canvases, cw, ch, mean, std, pad)
            want = brute.stitch(frames, rois, plan.place, 0, plan.n_canvases, cw, ch,
                                mean, std, pad)
            np.testing.assert_array_equal(got, want)


def test_stitch_exhaustive_sizes(orc):
    """Every w, h in 1..4 for a single RoI on a 4x4 .. 6x6 canvas, two mean/std sets."""
    from oracle import brute

    frames = W.random_frames_np(1, 6, 7, 3)
    for (cw, ch), w, h in itertools.product([(4, 4), (6, 5)], range(1, 5), range(1, 5)):
        rois = np.array([[0, 7 - w, 6 - h, w, h], [0, 0, 0, 1, 1]])
        for mean, std in [(W.MEAN, W.STD), ((0, 0, 0), (255, 255, 255))]:
            rc, _, plan = orc.pack(rois, cw, ch, 7, 6, 1, 1)
            got = orc.stitch(frames, rois, plan, 0, plan.n_canvases, cw, ch, mean, std, (0, 128, 255))
            want = brute.stitch(frames, rois, plan.place, 0, plan.n_canvases, cw, ch,
                                mean, std, (0, 128, 255))
            np.testing.assert_array_equal(got, want)


def test_stitch_whole_frame_is_plain_normalise(orc):
    """One patch = the whole frame = the canvas: the result is the HWC -> CHW
    transpose of (x - mean) / std rounded to binary16 (numpy's rounding)."""
    frames = W.random_frames_np(2, 24, 40, 9)
    rois = np.array([[1, 0, 0, 40, 24]])
    rc, _, plan = orc.pack(rois, 40, 24, 40, 24, 2, 0)
    got = orc.stitch(frames, rois, plan, 0, 1, 40, 24, W.MEAN, W.STD, W.PAD)[0]
    m = np.asarray(W.MEAN, np.float32).astype(np.float64)
    s = np.asarray(W.STD, np.float32).astype(np.float64)
    ref = ((frames[1].astype(np.float64) - m) / s).astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(got, ref.transpose(2, 0, 1))


def test_stitch_invariants_random(orc):
    """Pad everywhere outside patches; each patch reads back as its normalised crop."""
    rng = np.random.default_rng(8)
    frames = W.random_frames_np(3, 60, 90, 10)
    table = orc.norm_table(W.MEAN, W.STD)
    for policy in (0, 1, 2):
        rois = W.random_rois(rng, 40, 3, 90, 60, 1, 30, 30)
        rc, _, plan = orc.pack(rois, 48, 40, 90, 60, 3, policy)
        out = orc.stitch(frames, rois, plan, 0, plan.n_canvases, 48, 40, W.MEAN, W.STD, W.PAD)
        covered = np.zeros((plan.n_canvases, 40, 48), dtype=bool)
        for i, (f, x, y, w, h) in enumerate(rois):
            c, dx, dy = plan.place[i]
            crop = frames[f, y:y + h, x:x + w]
            for k in range(3):
                np.testing.assert_array_equal(out[c, k, dy:dy + h, dx:dx + w], table[k][crop[..., k]])
            covered[c, dy:dy + h, dx:dx + w] = True
        for k in range(3):
            assert np.all(out[:, k][~covered] == table[k][W.PAD[k]])


def test_stitch_canvas_range(orc):
    frames = W.random_frames_np(1, 20, 20, 1)
    rois = np.array([[0, 0, 0, 10, 10]] * 5)
    rc, _, plan = orc.pack(rois, 10, 10, 20, 20, 1, 0)
    full = orc.stitch(frames, rois, plan, 0, 5, 10, 10, W.MEAN, W.STD, W.PAD)
    part = orc.stitch(frames, rois, plan, 2, 2, 10, 10, W.MEAN, W.STD, W.PAD)
    np.testing.assert_array_equal(part, full[2:4])
    with pytest.raises(ValueError):
        orc.stitch(frames, rois, plan, 4, 2, 10, 10, W.MEAN, W.STD, W.PAD)


def test_pixel_sources_agree_with_stitch(orc):
    rng = np.random.default_rng(4)
    frames = W.random_frames_np(2, 50, 70, 12)
    rois = W.random_rois(rng, 30, 2, 70, 50, 1, 25, 25)
    rc, _, plan = orc.pack(rois, 40, 40, 70, 50, 2, 0)
    out = orc.stitch(frames, rois, plan, 0, plan.n_canvases, 40, 40, W.MEAN, W.STD, W.PAD)
    pts = np.stack([rng.integers(0, plan.n_canvases, 3000), rng.integers(0, 40, 3000),
                    rng.integers(0, 40, 3000)], axis=1)
    src = orc.pixel_sources(rois, plan, 50 * 70 * 3, 70 * 3, pts)
    table = orc.norm_table(W.MEAN, W.STD)
    flat = frames.reshape(-1)
    for q, (c, X, Y) in enumerate(pts):
        for k in range(3):
            want = table[k][W.PAD[k]] if src[q] < 0 else table[k][flat[src[q] + k]]
            assert out[c, k, Y, X] == want


# --------------------------------------------------------------------------- unstitch

def test_unstitch_golden(orc):
    g = load_golden("unstitch_example.json")
    ex = load_golden("pack_examples.json")["examples"][0]
    rc, _, plan = _pack(orc, ex, "guillotine_bssf")
    boxes = np.array(g["boxes"], dtype=np.float32)
    boxes[g["box_nan_index"], 0] = np.nan
    for clip, key in ((1, "dets_clip"), (0, "dets_noclip")):
        rob, dets = orc.unstitch(boxes, g["box_canvas"], ex["rois"], plan, clip)
        assert rob.tolist() == g["roi_of_box"]
        got = [tuple(d) for d in dets.tolist()]
        want = [tuple(r[:3]) + tuple(np.float32(v) for v in r[3:]) for r in g[key]]
        assert got == want


def test_unstitch_matches_brute_force(orc):
    from oracle import brute

    rng = np.random.default_rng(31)
    for _ in range(30):
        rois = W.random_rois(rng, int(rng.integers(1, 40)), 3, 200, 100, 1, 40, 40)
        rc, _, plan = orc.pack(rois, 64, 48, 200, 100, 3, int(rng.integers(0, 3)))
        n = 300
        cx, cy = rng.uniform(-4, 68, n), rng.uniform(-4, 52, n)
        bw, bh = rng.uniform(0, 30, n), rng.uniform(0, 30, n)
        boxes = np.stack([cx - bw / 2, cy - bh / 2, cx + bw / 2, cy + bh / 2], 1).astype(np.float32)
        # integer and half-integer centres hit patch edges exactly
        boxes[:50] = np.round(boxes[:50] * 2) / 2
        boxes[50:55, 1] = np.nan
        canv = rng.integers(-1, plan.n_canvases + 1, n)
        for clip in (0, 1):
            rob, dets = orc.unstitch(boxes, canv, rois, plan, clip)
            rob_b, dets_b = brute.unstitch(boxes, canv, rois, plan.place, plan.n_canvases, clip)
            np.testing.assert_array_equal(rob, rob_b)
            assert [tuple(d) for d in dets.tolist()] == [tuple(d) for d in dets_b]


def test_unstitch_own_box_is_identity(orc):
    """Unstitching each patch's own placed rect returns its source rect on its frame."""
    rng = np.random.default_rng(2)
    rois = W.random_rois(rng, 300, 5, 3840, 2160, 8, 300, 300)
    rc, _, plan = orc.pack(rois, 640, 640, 3840, 2160, 5, 0)
    pl = plan.place
    boxes = np.stack([pl[:, 1], pl[:, 2], pl[:, 1] + rois[:, 3], pl[:, 2] + rois[:, 4]], 1)
    rob, dets = orc.unstitch(boxes.astype(np.float32), pl[:, 0], rois, plan, 1)
    assert rob.tolist() == list(range(300))
    assert dets["box"].tolist() == list(range(300))
    assert dets["frame"].tolist() == rois[:, 0].tolist()
    got = np.stack([dets["x1"], dets["y1"], dets["x2"], dets["y2"]], 1)
    want = np.stack([rois[:, 1], rois[:, 2], rois[:, 1] + rois[:, 3], rois[:, 2] + rois[:, 4]], 1)
    np.testing.assert_array_equal(got, want.astype(np.float32))


# --------------------------------------------------------------------------- workloads

@pytest.mark.parametrize("name", ["cam1_1080p", "cam5_4k", "cam20_4k", "small_roi_8cam"])
def test_workload_plans_are_valid(orc, name):
    wl = W.WORKLOADS[name]
    rois = W.make_rois(wl)
    assert rois.shape == (wl.n_rois, 5)
    rc, _, plan = orc.pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    assert rc == 0
    assert orc.check_plan(rois, wl.canvas, wl.canvas, 0, plan.place, plan.order,
                          plan.canvas_begin, plan.n_canvases) == 0


# ---------------------------------------------------------------- unstitch, overlap rule

def test_unstitch_overlap_rule_example(orc):
    """Hand-worked: RoI 0 at (0,0), RoI 1 at (10,0), RoI 2 at (0,10), all 10 x 10.
    A [4,2,16,8] overlaps RoI 0 and RoI 1 by 6x6 = 36 each: the tie goes to RoI 0 (its
    centre x = 10 belongs to RoI 1). B [8,0,13,5]: 2x5 = 10 against 3x5 = 15: RoI 1.
    C [-5,-5,2,2]: 2x2 = 4 with RoI 0 (its centre is on no patch). D overlaps nothing,
    E has a NaN. F [2,8,8,14]: 6x2 = 12 with RoI 0, 6x4 = 24 with RoI 2: RoI 2."""
    rois = np.array([[0, 100, 50, 10, 10], [1, 200, 0, 10, 10], [0, 0, 0, 10, 10]], np.int32)
    plan = orc.Plan(np.array([[0, 0, 0], [0, 10, 0], [0, 0, 10]], np.int32),
                    np.array([0, 1, 2], np.int32), np.array([0, 3], np.int32), 1)
    boxes = np.array([[4, 2, 16, 8], [8, 0, 13, 5], [-5, -5, 2, 2], [30, 30, 40, 40],
                      [np.nan, 0, 5, 5], [2, 8, 8, 14]], np.float32)
    canv = np.zeros(6, np.int32)
    rob, dets = orc.unstitch(boxes, canv, rois, plan, 1, rule=1)
    assert rob.tolist() == [0, 1, 0, -1, -1, 2]
    # A clipped to RoI 0 ([0,10] x [0,10]) and moved by (100, 50) on frame 0
    assert tuple(dets[0])[:3] == (0, 0, 0) and tuple(dets[0])[3:] == (104, 52, 110, 58)
    rob_c, _ = orc.unstitch(boxes, canv, rois, plan, 1, rule=0)
    assert rob_c.tolist() == [1, 1, -1, -1, -1, 2]


def test_unstitch_overlap_rule_matches_brute_force(orc):
    from oracle import brute

    rng = np.random.default_rng(41)
    for _ in range(30):
        rois = W.random_rois(rng, int(rng.integers(1, 40)), 3, 200, 100, 1, 40, 40)
        rc, _, plan = orc.pack(rois, 64, 48, 200, 100, 3, int(rng.integers(0, 3)))
        n = 300
        cx, cy = rng.uniform(-4, 68, n), rng.uniform(-4, 52, n)
        bw, bh = rng.uniform(0, 30, n), rng.uniform(0, 30, n)
        boxes = np.stack([cx - bw / 2, cy - bh / 2, cx + bw / 2, cy + bh / 2], 1).astype(np.float32)
        boxes[:80] = np.round(boxes[:80])  # integer corners: exact ties between patches
        boxes[80:85, 2] = np.nan
        boxes[85:90, 0] = -np.inf
        canv = rng.integers(-1, plan.n_canvases + 1, n)
        for clip in (0, 1):
            rob, dets = orc.unstitch(boxes, canv, rois, plan, clip, rule=1)
            rob_b, dets_b = brute.unstitch(boxes, canv, rois, plan.place, plan.n_canvases, clip,
                                           rule=1)
            np.testing.assert_array_equal(rob, rob_b)
            assert [tuple(d) for d in dets.tolist()] == [tuple(d) for d in dets_b]


def test_unstitch_rules_agree_inside_patches(orc):
    """A box inside one patch overlaps only that patch and has its centre there."""
    rng = np.random.default_rng(5)
    rois = W.random_rois(rng, 200, 4, 800, 600, 8, 120, 120)
    rc, _, plan = orc.pack(rois, 400, 400, 800, 600, 4, 0)
    pl = plan.place
    f = rng.uniform(0.1, 0.45, (200, 4))
    x0 = pl[:, 1] + f[:, 0] * rois[:, 3]
    y0 = pl[:, 2] + f[:, 1] * rois[:, 4]
    boxes = np.stack([x0, y0, x0 + f[:, 2] * rois[:, 3], y0 + f[:, 3] * rois[:, 4]], 1).astype(np.float32)
    r0, _ = orc.unstitch(boxes, pl[:, 0], rois, plan, 1, rule=0)
    r1, _ = orc.unstitch(boxes, pl[:, 0], rois, plan, 1, rule=1)
    assert r0.tolist() == r1.tolist() == list(range(200))
