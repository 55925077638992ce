"""tg_unstitch on the GPU against the oracle: bit-exact roi_of_box, dets and n_out."""
import numpy as np
import pytest

import oracle
from conftest import load_golden
from gpu_helpers import oracle_plan, say
from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    tg.lib()
    return torch


def run_unstitch(torch, boxes, box_canvas, rois, plan, clip, dplan=None, rule=0):
    dplan = dplan or tg.DevicePlan(rois, plan)
    n = boxes.shape[0]
    b_d = torch.from_numpy(np.ascontiguousarray(boxes, np.float32).reshape(n, 4)).cuda()
    c_d = torch.from_numpy(np.ascontiguousarray(box_canvas, np.int32)).cuda()
    bufs = tg.UnstitchBuffers(n, dplan.n_rois)
    bufs.roi_of_box.fill_(-7)
    bufs.n_out.fill_(-7)
    tg.unstitch(b_d, c_d, dplan, clip, bufs, rule=rule)
    torch.cuda.synchronize()
    return bufs.roi_of_box.cpu().numpy(), bufs.dets_numpy(), int(bufs.n_out.item())


def check(torch, boxes, box_canvas, rois, plan, clip, dplan=None, rule=0):
    rob, dets, n_out = run_unstitch(torch, boxes, box_canvas, rois, plan, clip, dplan, rule)
    rob_o, dets_o = oracle.unstitch(boxes, box_canvas, rois, oracle_plan(plan), clip, rule)
    np.testing.assert_array_equal(rob, rob_o)
    assert n_out == len(dets_o)
    # compare bit patterns (NaN-free by construction: kept boxes have finite sums)
    np.testing.assert_array_equal(dets.view(np.int32).reshape(-1, 7),
                                  dets_o.view(np.int32).reshape(-1, 7))
    return rob, dets


def test_golden_example(torch):
    g = load_golden("unstitch_example.json")
    ex = load_golden("pack_examples.json")["examples"][0]
    cw, ch = ex["canvas"]
    fw, fh, nf = ex["frame"]
    rois = np.array(ex["rois"])
    plan = tg.plan_pack(rois, cw, ch, fw, fh, nf, tg.GUILLOTINE_BSSF)
    boxes = np.array(g["boxes"], dtype=np.float32)
    boxes[g["box_nan_index"], 0] = np.nan
    for clip, key in ((1, "dets_clip"), (0, "dets_noclip")):
        say("golden clip", clip)
        rob, dets, n_out = run_unstitch(torch, boxes, np.array(g["box_canvas"]), rois, plan, clip)
        assert rob.tolist() == g["roi_of_box"]
        assert n_out == len(g[key])
        got = [tuple(d) for d in dets.tolist()]
        assert got == [tuple(r[:3]) + tuple(np.float32(v) for v in r[3:]) for r in g[key]]


@pytest.mark.parametrize("per_canvas", [4, 24, 60, 300])
def test_random_plans(torch, per_canvas):
    """Patches per canvas around 16, 32 and 64+ select the three lane widths."""
    rng = np.random.default_rng(per_canvas)
    side = int(np.sqrt(200 * 200 / per_canvas))
    for policy in (0, 1, 2):
        rois = W.random_rois(rng, 30 * per_canvas, 4, 800, 600, max(1, side // 2), side, side)
        plan = tg.plan_pack(rois, 200, 200, 800, 600, 4, policy)
        n = 20000
        cx, cy = rng.uniform(-8, 208, n), rng.uniform(-8, 208, n)
        bw, bh = rng.uniform(0, 60, n), rng.uniform(0, 60, n)
        boxes = np.stack([cx - bw / 2, cy - bh / 2, cx + bw / 2, cy + bh / 2], 1).astype(np.float32)
        boxes[:3000] = np.round(boxes[:3000])          # centres on patch edges
        boxes[3000:3100, 0] = np.nan
        boxes[3100:3200, 3] = np.inf
        canv = rng.integers(-2, plan.n_canvases + 2, n).astype(np.int32)
        boxes[3200:3400] = np.round(boxes[3200:3400])  # integer corners: overlap ties
        for clip, rule in ((0, 0), (1, 0), (1, 1), (0, 1)):
            say("random", per_canvas, "policy", policy, "clip", clip, "rule", rule)
            check(torch, boxes, canv, rois, plan, clip, rule=rule)


@pytest.mark.parametrize("name", W.ORDERED)
def test_workload_boxes(torch, name):
    wl = W.WORKLOADS[name]
    say("workload", name)
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    boxes, canv = W.make_boxes(wl, plan.n_canvases)
    rob, dets = check(torch, boxes, canv, rois, plan, 1)
    assert (rob >= 0).sum() > 0.1 * len(rob)  # sanity: boxes do land on patches


def test_own_box_identity(torch):
    """Stitch then unstitch of each patch's own placed rect gives back its source rect."""
    wl = W.WORKLOADS["cam20_4k"]
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    pl = plan.place
    boxes = np.stack([pl[:, 1], pl[:, 2], pl[:, 1] + rois[:, 3], pl[:, 2] + rois[:, 4]],
                     1).astype(np.float32)
    say("identity")
    rob, dets, n_out = run_unstitch(torch, boxes, pl[:, 0], rois, plan, 1)
    assert rob.tolist() == list(range(len(rois))) and n_out == len(rois)
    got = np.stack([dets["x1"], dets["y1"], dets["x2"], dets["y2"]], 1)
    want = np.stack([rois[:, 1], rois[:, 2], rois[:, 1] + rois[:, 3], rois[:, 2] + rois[:, 4]], 1)
    np.testing.assert_array_equal(got, want.astype(np.float32))
    assert dets["frame"].tolist() == rois[:, 0].tolist()


def test_zero_boxes_and_no_canvases(torch):
    rois = np.array([[0, 0, 0, 4, 4]])
    plan = tg.plan_pack(rois, 8, 8, 8, 8, 1, 0)
    say("zero boxes")
    bufs = tg.UnstitchBuffers(0, 1)
    bufs.n_out.fill_(-5)
    dplan = tg.DevicePlan(rois, plan)
    tg.unstitch(torch.empty((0, 4), dtype=torch.float32, device="cuda"),
                torch.empty(0, dtype=torch.int32, device="cuda"), dplan, 1, bufs)
    torch.cuda.synchronize()
    assert bufs.n_out.item() == 0
    say("empty plan")
    empty = tg.plan_pack(np.zeros((0, 5)), 8, 8, 8, 8, 1, 0)
    boxes = np.array([[0, 0, 1, 1]], np.float32)
    rob, dets, n_out = run_unstitch(torch, boxes, np.array([0]), np.zeros((0, 5)), empty, 1)
    assert rob.tolist() == [-1] and n_out == 0


def test_deterministic(torch):
    wl = W.WORKLOADS["window_64x30"]
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    boxes, canv = W.make_boxes(wl, plan.n_canvases)
    dplan = tg.DevicePlan(rois, plan)
    say("determinism")
    a = run_unstitch(torch, boxes, canv, rois, plan, 1, dplan)
    b = run_unstitch(torch, boxes, canv, rois, plan, 1, dplan)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_overlap_rule_example(torch):
    """The hand-worked overlap example of the oracle tests, through the C ABI."""
    rois = np.array([[0, 100, 50, 10, 10], [1, 200, 0, 10, 10], [0, 0, 0, 10, 10]], np.int32)
    plan = tg.Plan(np.array([[0, 0, 0], [0, 10, 0], [0, 0, 10]], np.int32),
                   np.array([0, 1, 2], np.int32), np.array([0, 3], np.int32), 1)
    boxes = np.array([[4, 2, 16, 8], [8, 0, 13, 5], [-5, -5, 2, 2], [30, 30, 40, 40],
                      [np.nan, 0, 5, 5], [2, 8, 8, 14]], np.float32)
    rob, dets, n_out = run_unstitch(torch, boxes, np.zeros(6, np.int32), rois, plan, 1, rule=1)
    assert rob.tolist() == [0, 1, 0, -1, -1, 2]
    assert tuple(dets[0])[:3] == (0, 0, 0) and tuple(dets[0])[3:] == (104, 52, 110, 58)


@pytest.mark.parametrize("name", ["cam5_4k", "cam20_4k", "small_roi_8cam"])
def test_workload_boxes_overlap_rule(torch, name):
    wl = W.WORKLOADS[name]
    rois = W.make_rois(wl)
    plan = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, 0)
    boxes, canv = W.make_boxes(wl, plan.n_canvases)
    say("workload overlap rule", name)
    check(torch, boxes, canv, rois, plan, 1, rule=1)


def test_patch_records_switch(torch):
    """The calls on either side of the switch to patch records (at 2^21 box-patch tests,
    about n_boxes times the mean patches per canvas) agree with the oracle and with each
    other on their common boxes: the direct gathers and the records give one result."""
    rng = np.random.default_rng(91)
    rois = W.random_rois(rng, 9000, 4, 800, 600, 5, 11, 11)
    plan = tg.plan_pack(rois, 200, 200, 800, 600, 4, tg.SHELF_FFDH)
    per_canvas = -(-len(rois) // plan.n_canvases)
    n_switch = -(-(1 << 21) // per_canvas)
    n = n_switch + 100
    cx, cy = rng.uniform(-4, 204, n), rng.uniform(-4, 204, n)
    bw, bh = rng.uniform(0, 20, n), rng.uniform(0, 20, n)
    boxes = np.stack([cx - bw / 2, cy - bh / 2, cx + bw / 2, cy + bh / 2], 1).astype(np.float32)
    boxes[:500] = np.round(boxes[:500])
    canv = rng.integers(-1, plan.n_canvases + 1, n).astype(np.int32)
    dplan = tg.DevicePlan(rois, plan)
    for rule in (0, 1):
        say("records switch", per_canvas, n_switch, "rule", rule)
        lo = check(torch, boxes[:n_switch - 1], canv[:n_switch - 1], rois, plan, 1, dplan, rule)
        hi = check(torch, boxes, canv, rois, plan, 1, dplan, rule)
        np.testing.assert_array_equal(lo[0], hi[0][:n_switch - 1])


@pytest.mark.parametrize("rule", [0, 1])
def test_patch_records_with_small_canvases(torch, rule):
    """Patch records on canvases of about 24 patches (16 lanes per box, two rounds):
    120,000 boxes, centres on edges, NaN and infinite corners, bad canvases."""
    rng = np.random.default_rng(95 + rule)
    rois = W.random_rois(rng, 720, 4, 800, 600, 28, 48, 48)
    plan = tg.plan_pack(rois, 200, 200, 800, 600, 4, tg.SHELF_FFDH)
    n = 120_000
    cx, cy = rng.uniform(-8, 208, n), rng.uniform(-8, 208, n)
    bw, bh = rng.uniform(0, 60, n), rng.uniform(0, 60, n)
    boxes = np.stack([cx - bw / 2, cy - bh / 2, cx + bw / 2, cy + bh / 2], 1).astype(np.float32)
    boxes[:20000] = np.round(boxes[:20000])
    boxes[20000:20500, 1] = np.nan
    boxes[20500:21000, 2] = np.inf
    canv = rng.integers(-2, plan.n_canvases + 2, n).astype(np.int32)
    per_canvas = -(-len(rois) // plan.n_canvases)
    assert per_canvas <= 32 and n * per_canvas >= 1 << 21
    for clip in (0, 1):
        say("records, small canvases", per_canvas, "rule", rule, "clip", clip)
        check(torch, boxes, canv, rois, plan, clip, rule=rule)
