"""tg_stitch on the GPU against the oracle (pixels within 1 fp16 ulp, pad bit-exact;
the library's table design makes it bit-exact everywhere, which is checked too)."""
import numpy as np
import pytest

import oracle
from gpu_helpers import (SENTINEL, assert_stitch_parity, coverage, oracle_plan, run_stitch,
                         say)
from stitch_geometry import records_per_unit, unit_pixels
from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    tg.lib()
    return torch


def _case(torch, rng, n_frames, fh, fw, cw, ch, n, lo, hi_w, hi_h, policy, mean=W.MEAN,
          std=W.STD, pad=W.PAD, with_rois=False):
    rois = W.random_rois(rng, n, n_frames, fw, fh, lo, min(hi_w, cw), min(hi_h, ch))
    frames = W.random_frames_np(n_frames, fh, fw, int(rng.integers(1 << 30)))
    plan = tg.plan_pack(rois, cw, ch, fw, fh, n_frames, policy)
    frames_d = torch.from_numpy(frames).cuda()
    got = run_stitch(frames_d, rois, plan, 0, plan.n_canvases, cw, ch, mean, std, pad)
    want = oracle.stitch(frames, rois, oracle_plan(plan), 0, plan.n_canvases, cw, ch,
                         mean, std, pad)
    cov = coverage(plan, rois, 0, plan.n_canvases, cw, ch)
    assert_stitch_parity(got, want, cov)
    np.testing.assert_array_equal(got, want)  # bit-exact by design
    return (plan, rois) if with_rois else plan


@pytest.mark.parametrize("cw,ch", [(64, 48), (256, 32), (264, 40), (8, 8), (300, 70),
                                   (37, 29), (1, 1), (513, 33), (5, 300)])
def test_small_random_plans(torch, cw, ch):
    rng = np.random.default_rng(cw * 1000 + ch)
    for policy in (0, 1, 2):
        say("small", cw, ch, "policy", policy)
        _case(torch, rng, 3, 70, 91, cw, ch, 60, 1, 40, 40, policy)


def test_odd_frame_widths_and_mean_std(torch):
    rng = np.random.default_rng(77)
    for fw in (1, 2, 3, 5, 37, 101):
        say("frame width", fw)
        _case(torch, rng, 2, 23, fw, 72, 40, 30, 1, 16, 16, 0, mean=(0, 0, 0),
              std=(255, 255, 255), pad=(0, 128, 255))
        _case(torch, rng, 2, 23, fw, 72, 40, 30, 1, 16, 16, 2, mean=(10.5, 300.0, -7.25),
              std=(0.01, 1000.0, 3.5), pad=(255, 0, 7))


def test_many_patches_per_run_take_further_lists(torch):
    """Runs met by more patches than one list holds (40; the rest take further lists): up
    to 8192 tiny RoIs on a small canvas, including 1 x 1, and exactly 40 and 41."""
    rng = np.random.default_rng(5)
    # expect: the exact maximum of patches per unit, or ">" (over 40), or "<=" (40 or fewer)
    for cw, ch, n, lo, hi, pol, expect in [
            (256, 3, 41, 1, 1, 1, 41), (256, 3, 40, 1, 1, 1, 40),
            (256, 3, 129, 1, 1, 1, 129), (256, 32, 8192, 1, 1, 1, ">"),
            (256, 32, 3000, 1, 4, 2, ">"), (64, 64, 30, 2, 6, 0, "<="),
            (300, 64, 600, 1, 2, 1, ">"), (1300, 6, 900, 1, 2, 0, ">"),
            (3000, 5, 700, 1, 3, 2, ">")]:
        say("dense", cw, ch, n, lo, hi, pol)
        plan, rois = _case(torch, rng, 2, 50, 60, cw, ch, n, lo, hi, hi, pol, with_rois=True)
        most = max(records_per_unit(rois, plan, 0, plan.n_canvases, cw, ch))
        if expect == ">":
            assert most > 40
        elif expect == "<=":
            assert most <= 40
        else:
            assert most == expect


def test_roi_at_end_of_frame_buffer(torch):
    """Patches that end on the frame buffer's last byte (no over-read past it)."""
    for fw, fh in [(40, 30), (41, 30), (42, 31), (43, 17)]:
        rois = np.array([[1, fw - 9, fh - 5, 9, 5], [1, fw - 17, fh - 1, 17, 1],
                         [0, 0, 0, 8, 8], [1, fw - 1, fh - 1, 1, 1]])
        frames = W.random_frames_np(2, fh, fw, fw)
        for policy in (0, 2):
            say("end of buffer", fw, fh, policy)
            plan = tg.plan_pack(rois, 24, 24, fw, fh, 2, policy)
            got = run_stitch(torch.from_numpy(frames).cuda(), rois, plan, 0, plan.n_canvases,
                             24, 24)
            want = oracle.stitch(frames, rois, oracle_plan(plan), 0, plan.n_canvases, 24, 24,
                                 W.MEAN, W.STD, W.PAD)
            np.testing.assert_array_equal(got, want)


def test_whole_frame_is_plain_normalise(torch):
    """One patch = whole frame = canvas: torch's own normalise, within 1 ulp."""
    from gpu_helpers import half_ord

    say("whole frame")
    frames = torch.randint(0, 256, (2, 96, 160, 3), dtype=torch.uint8, device="cuda",
                           generator=torch.Generator(device="cuda").manual_seed(9))
    rois = np.array([[1, 0, 0, 160, 96]])
    plan = tg.plan_pack(rois, 160, 96, 160, 96, 2, 0)
    got = run_stitch(frames, rois, plan, 0, 1, 160, 96)[0]
    mean = torch.tensor(W.MEAN, device="cuda").view(3, 1, 1)
    std = torch.tensor(W.STD, device="cuda").view(3, 1, 1)
    ref = ((frames[1].permute(2, 0, 1).float() - mean) / std).half()
    ref = ref.cpu().numpy().view(np.uint16)
    assert np.abs(half_ord(got) - half_ord(ref)).max() <= 1


def test_canvas_ranges_and_misaligned_output(torch):
    rng = np.random.default_rng(12)
    rois = W.random_rois(rng, 400, 2, 500, 400, 8, 120, 120)
    frames = W.random_frames_np(2, 400, 500, 3)
    frames_d = torch.from_numpy(frames).cuda()
    plan = tg.plan_pack(rois, 256, 256, 500, 400, 2, 0)
    assert plan.n_canvases >= 4
    want = oracle.stitch(frames, rois, oracle_plan(plan), 0, plan.n_canvases, 256, 256,
                         W.MEAN, W.STD, W.PAD)
    dplan = tg.DevicePlan(rois, plan)
    for first, count in [(0, 1), (1, 2), (plan.n_canvases - 1, 1), (0, plan.n_canvases)]:
        say("range", first, count)
        got = run_stitch(frames_d, rois, plan, first, count, 256, 256, dplan=dplan)
        np.testing.assert_array_equal(got, want[first:first + count])
    say("count 0")
    empty = torch.empty((0, 3, 256, 256), dtype=torch.int16, device="cuda")
    tg.stitch(frames_d, dplan, 0, 0, 256, 256, W.MEAN, W.STD, W.PAD, empty)
    with pytest.raises(tg.TgError):
        tg.stitch(frames_d, dplan, plan.n_canvases, 1, 256, 256, W.MEAN, W.STD, W.PAD,
                  torch.empty((1, 3, 256, 256), dtype=torch.int16, device="cuda"))
    say("misaligned out")  # element offset 1: 2-byte aligned only -> generic path
    buf = torch.full((2 * 3 * 256 * 256 + 1,), SENTINEL, dtype=torch.int16, device="cuda")
    out = buf[1:].view(2, 3, 256, 256)
    tg.stitch(frames_d, dplan, 1, 2, 256, 256, W.MEAN, W.STD, W.PAD, out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16), want[1:3])
    assert buf[0].item() == SENTINEL  # nothing written before the view


def test_corrupt_plan_entries_are_skipped(torch):
    """Out-of-range ids, wrong canvas, rects leaving canvas or frame: read as pad."""
    rng = np.random.default_rng(6)
    rois = W.random_rois(rng, 60, 2, 120, 90, 4, 30, 30)
    frames = W.random_frames_np(2, 90, 120, 4)
    plan = tg.plan_pack(rois, 128, 128, 120, 90, 2, 0)
    assert plan.canvas_begin[1] >= 5
    bad_rois, bad_place, bad_order = rois.copy(), plan.place.copy(), plan.order.copy()
    victims = plan.order[plan.canvas_begin[0]:plan.canvas_begin[1]][:5]
    bad_order[plan.canvas_begin[0]] = 10_000            # id out of range
    bad_place[victims[1], 0] = 99                        # names another canvas
    bad_place[victims[2], 1] = 128 - rois[victims[2], 3] + 1  # leaves the canvas
    bad_rois[victims[3], 0] = 5                          # frame id out of range
    bad_rois[victims[4], 1] = 120 - rois[victims[4], 3] + 1  # leaves the frame
    skipped = set(victims.tolist())
    keep = [i for i in plan.order if i not in skipped]
    # the oracle's answer for the plan without the corrupt entries
    cb = [0]
    for j in range(plan.n_canvases):
        seg = [i for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]
               if i not in skipped]
        cb.append(cb[-1] + len(seg))
    clean = oracle.Plan(plan.place, np.array(keep, np.int32), np.array(cb, np.int32),
                        plan.n_canvases)
    want = oracle.stitch(frames, rois, clean, 0, plan.n_canvases, 128, 128, W.MEAN, W.STD,
                         W.PAD)
    say("corrupt plan")
    corrupt = tg.Plan(bad_place, bad_order, plan.canvas_begin, plan.n_canvases)
    got = run_stitch(torch.from_numpy(frames).cuda(), bad_rois, corrupt, 0, plan.n_canvases,
                     128, 128)
    np.testing.assert_array_equal(got, want)


def test_empty_canvas_is_all_pad(torch):
    rois = np.array([[0, 0, 0, 4, 4], [0, 4, 4, 4, 4]])
    place = np.array([[0, 0, 0], [2, 3, 3]], np.int32)
    plan = tg.Plan(place, np.array([0, 1], np.int32), np.array([0, 1, 1, 2], np.int32), 3)
    frames = W.random_frames_np(1, 8, 8, 1)
    say("empty canvas")
    got = run_stitch(torch.from_numpy(frames).cuda(), rois, plan, 0, 3, 16, 16)
    want = oracle.stitch(frames, rois, oracle_plan(plan), 0, 3, 16, 16, W.MEAN, W.STD, W.PAD)
    np.testing.assert_array_equal(got, want)
    table = oracle.norm_table(W.MEAN, W.STD)
    for k in range(3):
        assert np.all(got[1, k] == table[k][W.PAD[k]])


def test_deterministic(torch):
    wl = W.WORKLOADS["cam5_4k"]
    rois = W.make_rois(wl)
    frames_d = W.make_frames(wl, "cuda")
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    say("determinism")
    a = run_stitch(frames_d, rois, plan, 0, plan.n_canvases, wl.canvas, wl.canvas)
    b = run_stitch(frames_d, rois, plan, 0, plan.n_canvases, wl.canvas, wl.canvas,
                   sentinel=False)
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name,policy,order", [("cam1_1080p", 0, None), ("cam5_4k", 0, None),
                                               ("cam20_4k", 0, None), ("cam20_4k", 0, "reverse"),
                                               ("cam20_4k", 2, None),
                                               ("small_roi_8cam", 0, None),
                                               ("small_roi_8cam", 1, "reverse")])
def test_workload_full_parity(torch, name, policy, order):
    """Whole workloads, batch by batch as the bench launches them (units in address
    order, or in reverse through the unit-order argument), against the oracle."""
    wl = W.WORKLOADS[name]
    say("workload", name, "policy", policy, "order", order)
    rois = W.make_rois(wl)
    frames_d = W.make_frames(wl, "cuda")
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, policy)
    dplan = tg.DevicePlan(rois, plan)
    frames = frames_d.cpu().numpy()
    for k in range(tg.batch_count(plan.n_canvases, wl.batch_cap)):
        first, count = tg.batch_range(plan.n_canvases, wl.batch_cap, k)
        say("  batch", k, first, count)
        unit_order = None
        if order == "reverse":
            n_units = tg.stitch_units(wl.canvas, wl.canvas, count)
            unit_order = torch.arange(n_units - 1, -1, -1, dtype=torch.int32, device="cuda")
        got = run_stitch(frames_d, rois, plan, first, count, wl.canvas, wl.canvas, dplan=dplan,
                         unit_order=unit_order)
        want = oracle.stitch(frames, rois, oracle_plan(plan), first, count, wl.canvas,
                             wl.canvas, W.MEAN, W.STD, W.PAD)
        cov = coverage(plan, rois, first, count, wl.canvas, wl.canvas)
        assert_stitch_parity(got, want, cov)
        np.testing.assert_array_equal(got, want)


def test_window_sampled_batches(torch):
    """The 64-camera x 30-frame window (about 48 GB of frames resident): first, middle
    and last batch. Every patch is read back against the oracle's normalisation of
    its crop, and every uncovered pixel must be the pad value."""
    wl = W.WORKLOADS["window_64x30"]
    say("window: plan + frames")
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    rc, _, oplan = oracle.pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h,
                               wl.n_frames, 0)
    np.testing.assert_array_equal(plan.place, oplan.place)
    frames_d = W.make_frames(wl, "cuda")
    dplan = tg.DevicePlan(rois, plan)
    table = oracle.norm_table(W.MEAN, W.STD)
    nb = tg.batch_count(plan.n_canvases, wl.batch_cap)
    for k in sorted({0, nb // 2, nb - 1}):
        first, count = tg.batch_range(plan.n_canvases, wl.batch_cap, k)
        say("window batch", k, first, count)
        got = run_stitch(frames_d, rois, plan, first, count, wl.canvas, wl.canvas, dplan=dplan)
        assert not np.any(got == SENTINEL)
        cov = np.zeros((count, wl.canvas, wl.canvas), dtype=bool)
        for j in range(first, first + count):
            for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]:
                f, sx, sy, w, h = rois[i]
                _, dx, dy = plan.place[i]
                crop = frames_d[f, sy:sy + h, sx:sx + w].cpu().numpy()
                for ch in range(3):
                    np.testing.assert_array_equal(got[j - first, ch, dy:dy + h, dx:dx + w],
                                                  table[ch][crop[..., ch]])
                cov[j - first, dy:dy + h, dx:dx + w] = True
        for ch in range(3):
            assert np.all(got[:, ch][~cov] == table[ch][W.PAD[ch]])
    del frames_d
    torch.cuda.empty_cache()


# mean/std for which tg_stitch normalises through its binary16 table (no fp32 fma
# constants reproduce every correctly rounded value); the CPU tests pin that choice
TABLE_MEAN = (174.00369262695312, 189.9988250732422, 150.99696350097656)
TABLE_STD = (0.031708136200904846, 1.5641870498657227, 1.5637657642364502)


def test_table_path_parity(torch):
    """The table path: small plans of every policy and a whole workload, bit-exact."""
    assert tg.stitch_norm_uses_table(TABLE_MEAN, TABLE_STD)
    rng = np.random.default_rng(31)
    for cw, ch in [(64, 48), (300, 70), (37, 29)]:
        for policy in (0, 1, 2):
            say("table path", cw, ch, policy)
            _case(torch, rng, 3, 70, 91, cw, ch, 60, 1, 40, 40, policy, mean=TABLE_MEAN,
                  std=TABLE_STD, pad=(3, 200, 90))
    wl = W.WORKLOADS["cam5_4k"]
    rois = W.make_rois(wl)
    frames_d = W.make_frames(wl, "cuda")
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    say("table path cam5_4k")
    got = run_stitch(frames_d, rois, plan, 0, plan.n_canvases, wl.canvas, wl.canvas,
                     TABLE_MEAN, TABLE_STD, (3, 200, 90))
    want = oracle.stitch(frames_d.cpu().numpy(), rois, oracle_plan(plan), 0, plan.n_canvases,
                         wl.canvas, wl.canvas, TABLE_MEAN, TABLE_STD, (3, 200, 90))
    np.testing.assert_array_equal(got, want)


def test_unit_order_that_is_not_a_permutation(torch):
    """Ids outside the unit range are ignored, a repeated id rewrites the same values, a
    missing id leaves its region unwritten -- and nothing outside `out` is touched."""
    rng = np.random.default_rng(8)
    cw = ch = 256
    rois = W.random_rois(rng, 80, 2, 400, 300, 8, 120, 120)
    frames = W.random_frames_np(2, 300, 400, 6)
    plan = tg.plan_pack(rois, cw, ch, 400, 300, 2, 0)
    count = min(plan.n_canvases, 2)
    n_units = tg.stitch_units(cw, ch, count)
    want = oracle.stitch(frames, rois, oracle_plan(plan), 0, count, cw, ch, W.MEAN, W.STD,
                         W.PAD)
    order = np.full(n_units, -1, np.int32)
    order[0] = order[1] = 0        # unit 0 twice
    order[2] = n_units             # out of range
    order[3] = n_units - 1         # the last unit
    order[4] = 2 ** 31 - 1
    say("unit order not a permutation", n_units)
    buf = torch.full((count * 3 * ch * cw + 64,), SENTINEL, dtype=torch.int16, device="cuda")
    out = buf[:count * 3 * ch * cw].view(count, 3, ch, cw)
    tg.stitch(torch.from_numpy(frames).cuda(), tg.DevicePlan(rois, plan), 0, count, cw, ch,
              W.MEAN, W.STD, W.PAD, out, unit_order=torch.from_numpy(order).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    assert np.all(buf[count * 3 * ch * cw:].cpu().numpy().view(np.uint16) == SENTINEL)
    written = np.zeros((count, ch * cw), bool)
    for u in (0, n_units - 1):
        c, p0, p1 = unit_pixels(cw, ch, count, u)
        written[c, p0:p1] = True
    flat = got.reshape(count, 3, ch * cw)
    want_flat = want.reshape(count, 3, ch * cw)
    for c in range(count):
        np.testing.assert_array_equal(flat[c][:, written[c]], want_flat[c][:, written[c]])
        assert np.all(flat[c][:, ~written[c]] == SENTINEL), c


def test_argument_struct_keeps_its_tensors(torch):
    """stitch_args returns a struct of raw device pointers; it holds the tensors they
    point into, so a launch order passed as a temporary lives as long as the struct."""
    import gc
    import weakref

    rng = np.random.default_rng(11)
    rois = W.random_rois(rng, 30, 2, 90, 70, 4, 40, 40)
    plan = tg.plan_pack(rois, 128, 96, 90, 70, 2, tg.SHELF_FFDH)
    frames = torch.from_numpy(W.random_frames_np(2, 70, 90, 3)).cuda()
    dplan = tg.DevicePlan(rois, plan)
    out = torch.empty((plan.n_canvases, 3, 96, 128), dtype=torch.float16, device="cuda")
    n_units = tg.stitch_units(128, 96, plan.n_canvases)
    order = torch.arange(n_units - 1, -1, -1, dtype=torch.int32, device="cuda")
    alive = weakref.ref(order)
    a = tg.stitch_args(frames, dplan, 0, plan.n_canvases, 128, 96, W.MEAN, W.STD, W.PAD, out,
                       unit_order=order)
    del order
    gc.collect()
    assert alive() is not None
    assert tg.lib().tg_stitch(tg.ctypes.byref(a), tg._stream_handle(None)) == tg.OK
    torch.cuda.synchronize()
    want = oracle.stitch(frames.cpu().numpy(), rois, oracle_plan(plan), 0, plan.n_canvases, 128,
                         96, W.MEAN, W.STD, W.PAD)
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16), want)
    del a
    gc.collect()
    assert alive() is None
