"""tg_merge on the GPU against the oracle: keep flags, kept detections and counts,
bit-exact, through the C ABI, including the path fed directly by tg_unstitch."""
import numpy as np
import pytest

from gpu_helpers import say
from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W
from test_merge import golden_inputs, random_dets

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    tg.lib()
    return torch


def run_gpu(torch, dets, scores, n_frames, thr, cross_only, n_max=None):
    n = len(dets)
    n_max = n if n_max is None else n_max
    host = np.zeros((max(n_max, 1), tg.DET_WORDS), np.int32)
    host[:n] = dets.view(np.int32).reshape(n, tg.DET_WORDS)
    bufs = tg.MergeBuffers(n_max, n_frames)
    bufs.keep.fill_(-7)
    d = torch.from_numpy(host).cuda()
    if n_max == 0:
        d = d[:0]
    tg.merge(d, torch.tensor([n], dtype=torch.int32, device="cuda"),
             torch.from_numpy(np.ascontiguousarray(scores, np.float32)).cuda(), n_frames, thr,
             cross_only, bufs)
    torch.cuda.synchronize()
    return bufs.keep[:n].cpu().numpy(), bufs.kept_numpy(), int(bufs.n_kept.item())


def check(torch, dets, scores, n_frames, thr, cross_only, **kw):
    from oracle import merge

    say("merge", len(dets), n_frames, thr, cross_only)
    keep, kept, n_kept = run_gpu(torch, dets, scores, n_frames, thr, cross_only, **kw)
    want_keep, want_kept = merge.merge(dets, scores, n_frames, thr, cross_only)
    np.testing.assert_array_equal(keep, want_keep.astype(np.int32))
    assert n_kept == len(want_kept)
    np.testing.assert_array_equal(kept.view(np.int32), want_kept.view(np.int32))
    return keep


@pytest.mark.parametrize("cross_only,key", [(True, "keep_cross_only"), (False, "keep_all_pairs")])
def test_golden(torch, cross_only, key):
    g, dets, scores = golden_inputs()
    keep, _, _ = run_gpu(torch, dets, scores, g["n_frames"], g["threshold"], cross_only)
    assert keep.tolist() == g[key]


@pytest.mark.parametrize("cross_only,thr", [(True, 0.5), (False, 0.45), (True, 0.0), (False, 1.0)])
def test_random(torch, cross_only, thr):
    rng = np.random.default_rng(int(thr * 100) + cross_only)
    dets, scores = random_dets(rng, 5000, 40, 30)
    dets["frame"][rng.random(5000) < 0.02] = 40 + rng.integers(0, 5)  # outside [0, 40)
    check(torch, dets, scores, 40, thr, cross_only)


@pytest.mark.parametrize("name", ["cam20_4k", "small_roi_8cam"])
def test_after_unstitch_on_device(torch, name):
    """tg_unstitch's device outputs feed tg_merge directly (no host copy in between); on
    small_roi_8cam every frame holds several thousand detections (the workspace path)."""
    from oracle import merge

    say("unstitch -> merge", name)
    wl = W.WORKLOADS[name]
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    boxes, canv = W.make_boxes(wl, plan.n_canvases)
    dplan = tg.DevicePlan(rois, plan)
    ub = tg.UnstitchBuffers(len(boxes), len(rois))
    tg.unstitch(torch.from_numpy(boxes).cuda(), torch.from_numpy(canv).cuda(), dplan, 1, ub)
    scores = np.random.default_rng(2).uniform(0, 1, len(boxes)).astype(np.float32)
    mb = tg.MergeBuffers(len(boxes), wl.n_frames)
    tg.merge(ub.dets, ub.n_out, torch.from_numpy(scores).cuda(), wl.n_frames, 0.5, True, mb)
    torch.cuda.synchronize()
    dets = ub.dets_numpy()
    want_keep, want_kept = merge.merge(dets, scores, wl.n_frames, 0.5, True)
    np.testing.assert_array_equal(mb.keep[: len(dets)].cpu().numpy(), want_keep.astype(np.int32))
    np.testing.assert_array_equal(mb.kept_numpy().view(np.int32), want_kept.view(np.int32))
    assert 0 < len(want_kept) < len(dets)


def test_large_frames(torch):
    """Large frames: 1024, 1025, 2048, 2049, 5000 and 20000 detections in one frame next
    to a small frame, in crowded and sparse layouts, with and without cross_only."""
    rng = np.random.default_rng(9)
    for big, span, thr, cross in [(1024, 400.0, 0.5, True), (1025, 400.0, 0.5, True),
                                  (1025, 100.0, 0.3, False), (2048, 600.0, 0.5, True),
                                  (2049, 600.0, 0.5, True),
                                  (2049, 150.0, 0.3, False), (5000, 1500.0, 0.5, True),
                                  (5000, 300.0, 0.4, False), (20000, 3000.0, 0.5, True)]:
        dets, scores = random_dets(rng, big + 300, 2, 10, span=span)
        dets["frame"] = np.r_[np.zeros(big, np.int32), np.ones(300, np.int32)]
        check(torch, dets, scores, 2, thr, cross)


def test_large_frames_special_boxes(torch):
    """A 3000-detection frame with the cases the cell index treats apart: boxes with
    infinite corners, inverted boxes, boxes wider than the frame, duplicates of one box
    (up to 239 suppressors each: their whole lists go to the overflow area), and a
    negative threshold (every pair suppresses: the lists need about 4.5 M entries, far
    past the overflow area's 48,000, so most detections search their lists again in
    the rounds)."""
    rng = np.random.default_rng(19)
    dets, scores = random_dets(rng, 3000, 1, 12, span=800.0)
    k = rng.permutation(3000)
    dets["x2"][k[:40]] = np.inf
    dets["y1"][k[40:80]] = -np.inf
    dets["x1"][k[80:120]], dets["x2"][k[80:120]] = dets["x2"][k[80:120]], dets["x1"][k[80:120]]
    dets["x1"][k[120:160]], dets["x2"][k[120:160]] = -50.0, 2000.0
    for c in ("x1", "y1", "x2", "y2"):
        dets[c][k[160:400]] = dets[c][k[160]]
    check(torch, dets, scores, 1, 0.5, True)
    check(torch, dets, scores, 1, 0.5, False)
    check(torch, dets, scores, 1, -0.5, False)
    check(torch, dets, scores, 1, 0.0, True)


def test_frames_around_the_matrix_limit(torch):
    """Frames of 437, 439, 448, 512 and 513 detections side by side (through the spatial
    index: frames of up to 256 detections are decided in one workgroup's LDS)."""
    rng = np.random.default_rng(12)
    sizes = [437, 439, 448, 512, 513]
    dets, scores = random_dets(rng, sum(sizes), len(sizes), 8, span=400.0)
    dets["frame"] = np.repeat(np.arange(len(sizes)), sizes)
    check(torch, dets, scores, len(sizes), 0.4, True)
    check(torch, dets, scores, len(sizes), 0.6, False)


def test_frames_around_the_small_workgroup_limit(torch):
    """Frames averaging at most 256 detections take 256-thread workgroups: frames of 256
    are decided in LDS, of 257 through the spatial index, side by side."""
    rng = np.random.default_rng(14)
    sizes = [256, 257, 40, 1, 0, 120]
    dets, scores = random_dets(rng, sum(sizes), len(sizes), 6, span=250.0)
    dets["frame"] = np.repeat(np.arange(len(sizes)), sizes)
    check(torch, dets, scores, len(sizes), 0.45, True)
    check(torch, dets, scores, len(sizes), 0.5, False)


def test_small_frames_special_boxes(torch):
    """Frames of 1-256 detections (decided in LDS, each pair of boxes tested once) with
    NaN, infinite and signed-zero corners, inverted and empty boxes, duplicates of one box
    and equal scores, for thresholds of both signs, with and without cross_only."""
    rng = np.random.default_rng(23)
    sizes = [1, 2, 3, 4, 63, 64, 65, 128, 129, 200, 255, 256]
    dets, scores = random_dets(rng, sum(sizes), len(sizes), 4, span=120.0)
    dets["frame"] = np.repeat(np.arange(len(sizes)), sizes)
    k = rng.permutation(len(dets))
    special = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0], np.float32)
    for c in ("x1", "y1", "x2", "y2"):
        pick = k[rng.integers(0, 150, 20)]
        dets[c][pick] = rng.choice(special, 20)
    dets["x1"][k[150:170]], dets["x2"][k[150:170]] = dets["x2"][k[150:170]], dets["x1"][k[150:170]]
    dets["y2"][k[170:190]] = dets["y1"][k[170:190]]  # empty
    for c in ("x1", "y1", "x2", "y2"):
        dets[c][k[190:260]] = dets[c][k[190]]  # duplicates, spread over frames
    for thr, cross in [(0.5, True), (0.3, False), (0.0, False), (-0.5, True), (1.0, False)]:
        check(torch, dets, scores, len(sizes), thr, cross)


def test_many_frames(torch):
    """More frames than the LDS histograms hold (4096): direct global counters."""
    rng = np.random.default_rng(13)
    dets, scores = random_dets(rng, 20000, 5000, 6, span=100.0)
    check(torch, dets, scores, 5000, 0.5, True)


def test_many_frames_with_large_ones(torch):
    """3,000 frames of 25 detections with four of 257-600 among them, the large ones on
    both sides of frame 2048 (the rounds step through frames 2048 apart) and more than
    65,536 detections (the search steps through them 65,536 apart). Frames are merged
    independently, so the oracle checks the large frames and 200 others on their own; the
    compacted output is the kept detections in input order."""
    from oracle import merge

    rng = np.random.default_rng(15)
    sizes = np.full(3000, 25)
    big = [5, 2100, 2101, 2999]
    sizes[big] = [300, 400, 257, 600]
    dets, scores = random_dets(rng, int(sizes.sum()), 3000, 6, span=300.0)
    dets["frame"] = np.repeat(np.arange(3000), sizes)
    dets = dets[rng.permutation(len(dets))]
    say("merge, many frames with large ones", len(dets))
    keep, kept, n_kept = run_gpu(torch, dets, scores, 3000, 0.5, True)
    frames = np.r_[big, rng.choice(np.setdiff1d(np.arange(3000), big), 200, replace=False)]
    sub = np.nonzero(np.isin(dets["frame"], frames))[0]
    want_keep, _ = merge.merge(dets[sub], scores, 3000, 0.5, True)
    np.testing.assert_array_equal(keep[sub], want_keep.astype(np.int32))
    assert set(np.unique(keep)) <= {0, 1}
    assert n_kept == int(keep.sum())
    np.testing.assert_array_equal(kept.view(np.int32), dets[keep == 1].view(np.int32))


def test_partial_count_and_empty(torch):
    rng = np.random.default_rng(4)
    dets, scores = random_dets(rng, 800, 5, 4)
    # only the first 600 entries are valid (device count), capacity 800
    from oracle import merge

    keep, kept, n_kept = run_gpu(torch, dets[:600], scores, 5, 0.5, True, n_max=800)
    want_keep, want_kept = merge.merge(dets[:600], scores, 5, 0.5, True)
    np.testing.assert_array_equal(keep, want_keep.astype(np.int32))
    assert n_kept == len(want_kept)
    _, _, n_kept = run_gpu(torch, dets[:0], scores, 5, 0.5, True, n_max=64)
    assert n_kept == 0
    _, _, n_kept = run_gpu(torch, dets[:0], scores, 5, 0.5, True, n_max=0)
    assert n_kept == 0


def test_single_workgroup_path(torch):
    """Capacities up to 512 take the one-launch path (one workgroup, suppressor rows in
    LDS): against the oracle, and against the general path run on the same detections
    with a larger capacity, on frames sharing the 512 slots, NaN scores, frames out of
    range, special boxes, a negative threshold, and counts of 0, 1, 511 and 512."""
    from oracle import merge

    rng = np.random.default_rng(21)
    cases = [(1, 1, 0.5, True), (2, 1, 0.5, False), (41, 1, 0.5, True), (200, 3, 0.4, True),
             (511, 1, 0.3, False), (512, 1, 0.5, True), (512, 7, 0.5, False),
             (300, 2, -0.5, False), (300, 2, 0.0, True), (512, 600, 0.5, True)]
    for n, n_frames, thr, cross in cases:
        dets, scores = random_dets(rng, n, n_frames, 5, span=150.0)
        if n >= 300:
            k = rng.permutation(n)
            dets["frame"][k[:10]] = n_frames + 2                   # dropped
            dets["x2"][k[10:20]] = np.inf
            dets["x1"][k[20:30]], dets["x2"][k[20:30]] = dets["x2"][k[20:30]], dets["x1"][k[20:30]]
            for c in ("x1", "y1", "x2", "y2"):
                dets[c][k[30:60]] = dets[c][k[30]]                # duplicates of one box
        say("single workgroup", n, n_frames, thr, cross)
        want_keep, want_kept = merge.merge(dets, scores, n_frames, thr, cross)
        for n_max in (n, 513):
            keep, kept, n_kept = run_gpu(torch, dets, scores, n_frames, thr, cross, n_max=n_max)
            np.testing.assert_array_equal(keep, want_keep.astype(np.int32))
            assert n_kept == len(want_kept)
            np.testing.assert_array_equal(kept.view(np.int32), want_kept.view(np.int32))
    _, _, n_kept = run_gpu(torch, np.zeros(0, tg.DET_DTYPE), np.zeros(1, np.float32), 3, 0.5,
                           True, n_max=100)
    assert n_kept == 0
