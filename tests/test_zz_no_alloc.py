"""tg_unstitch_noalloc (the allocation-free entry point) on the GPU through the C ABI,
against tg_unstitch on the same inputs: two calls in a row on the library's own device
scratch, the second with fewer boxes (its stale contents must not matter), with no
workspace passed. Collected last (`test_zz_...`) so that a failure here hides no other
test."""
import ctypes

import numpy as np
import pytest

from gpu_helpers import say
from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    tg.lib()
    return torch


def _case(torch, seed, n_boxes, rule):
    rng = np.random.default_rng(seed)
    rois = W.random_rois(rng, 300, 3, 700, 500, 4, 200, 200)
    plan = tg.plan_pack(rois, 320, 320, 700, 500, 3, tg.SHELF_FFDH)
    boxes, canv = W.make_boxes(W.WORKLOADS["cam1_1080p"], plan.n_canvases, seed=seed)
    reps = -(-n_boxes // len(boxes))
    boxes = np.tile(boxes, (reps, 1))[:n_boxes] * np.float32(320 / 1024)
    canv = np.tile(canv, reps)[:n_boxes]
    boxes[::97] = np.nan  # some boxes match nothing
    canv[::89] = plan.n_canvases + 3  # some name no canvas
    dplan = tg.DevicePlan(rois, plan)
    boxes_d = torch.from_numpy(np.ascontiguousarray(boxes, np.float32)).cuda()
    canv_d = torch.from_numpy(np.ascontiguousarray(canv, np.int32)).cuda()
    return dplan, boxes_d, canv_d


def _run(torch, dplan, boxes_d, canv_d, rule, noalloc):
    bufs = tg.UnstitchBuffers(boxes_d.shape[0], dplan.n_rois)
    bufs.roi_of_box.fill_(-7)
    bufs.dets.fill_(-7)
    bufs.n_out.fill_(-7)
    a = tg.unstitch_args(boxes_d, canv_d, dplan, 1, bufs, rule)
    if noalloc:
        a.workspace, a.workspace_bytes = None, 0  # ignored by the allocation-free entry
        rc = tg.unstitch_noalloc_raw(a)
    else:
        rc = tg.unstitch_raw(a)
    assert rc == tg.OK, tg.strerror(rc)
    torch.cuda.synchronize()
    return (bufs.roi_of_box.cpu().numpy(), bufs.dets_numpy(), int(bufs.n_out.item()))


@pytest.mark.parametrize("rule", [0, 1])
def test_noalloc_matches_unstitch_twice(torch, rule):
    for n_boxes, seed in [(300_000, 11), (4_000, 12)]:  # the second call is smaller
        say("noalloc", rule, n_boxes)
        dplan, boxes_d, canv_d = _case(torch, seed, n_boxes, rule)
        want = _run(torch, dplan, boxes_d, canv_d, rule, noalloc=False)
        got = _run(torch, dplan, boxes_d, canv_d, rule, noalloc=True)
        np.testing.assert_array_equal(got[0], want[0])
        assert got[2] == want[2] and got[2] > 0
        assert got[1].tobytes() == want[1].tobytes()


def test_noalloc_plan_beyond_record_area(torch):
    """A plan of more RoIs than the scratch array's patch records hold: the allocation-free
    entry reads it directly and still matches tg_unstitch (which uses records there)."""
    rng = np.random.default_rng(14)
    n_rois = tg.UNSTITCH_NOALLOC_MAX_ROIS + 5000
    rois = W.random_rois(rng, n_rois, 8, 3840, 2160, 4, 12, 12)
    plan = tg.plan_pack(rois, 640, 640, 3840, 2160, 8, tg.SHELF_FFDH)
    dplan = tg.DevicePlan(rois, plan)
    n = 4_000  # about 25 million box-patch tests: records in tg_unstitch
    cx, cy = rng.uniform(0, 640, n), rng.uniform(0, 640, n)
    boxes = np.stack([cx - 3, cy - 3, cx + 3, cy + 3], 1).astype(np.float32)
    canv = rng.integers(0, plan.n_canvases, n).astype(np.int32)
    boxes_d = torch.from_numpy(boxes).cuda()
    canv_d = torch.from_numpy(canv).cuda()
    for rule in (0, 1):
        say("noalloc large plan", n_rois, plan.n_canvases, rule)
        want = _run(torch, dplan, boxes_d, canv_d, rule, noalloc=False)
        got = _run(torch, dplan, boxes_d, canv_d, rule, noalloc=True)
        np.testing.assert_array_equal(got[0], want[0])
        assert got[2] == want[2] and got[2] > 0
        assert got[1].tobytes() == want[1].tobytes()


def test_noalloc_limits(torch):
    dplan, boxes_d, canv_d = _case(torch, 13, 10, 0)
    bufs = tg.UnstitchBuffers(10, dplan.n_rois)
    a = tg.unstitch_args(boxes_d, canv_d, dplan, 1, bufs, 0)
    a.n_boxes = tg.UNSTITCH_NOALLOC_MAX_BOXES + 1  # refused before anything is enqueued
    assert tg.unstitch_noalloc_raw(a) == tg.E_WORKSPACE
    a.n_boxes = 0  # only *n_out = 0 is written
    bufs.n_out.fill_(5)
    assert tg.unstitch_noalloc_raw(a) == tg.OK
    torch.cuda.synchronize()
    assert int(bufs.n_out.item()) == 0
