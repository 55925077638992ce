"""tg_partition on the GPU against the oracle (Alg. 1, Sec. III-A): zone of every RoI and
the patch list, bit-exact, through the C ABI."""
import numpy as np
import pytest

from conftest import load_golden
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


def run_gpu(torch, boxes, frame_begin, fw, fh, zx, zy):
    boxes = np.ascontiguousarray(boxes, dtype=np.int32).reshape(-1, 5)
    fb = np.ascontiguousarray(frame_begin, dtype=np.int32)
    bufs = tg.PartitionBuffers(len(boxes), len(fb) - 1)
    bufs.zone_of_box.fill_(-7)
    bufs.patches.fill_(-7)
    tg.partition(torch.from_numpy(boxes).cuda(), torch.from_numpy(fb).cuda(), fw, fh, zx, zy,
                 bufs)
    torch.cuda.synchronize()
    return bufs.zone_of_box[: len(boxes)].cpu().numpy(), bufs.patches_numpy()


def run_oracle(boxes, frame_begin, fw, fh, zx, zy):
    from oracle import partition

    z, p = partition.partition(np.asarray(boxes).tolist(), list(frame_begin), fw, fh, zx, zy)
    return np.array(z, dtype=np.int32), np.array(p, dtype=np.int32).reshape(-1, 5)


def check(torch, boxes, fb, fw, fh, zx, zy):
    say("partition", len(boxes), len(fb) - 1, fw, fh, zx, zy)
    gz, gp = run_gpu(torch, boxes, fb, fw, fh, zx, zy)
    oz, op = run_oracle(boxes, fb, fw, fh, zx, zy)
    np.testing.assert_array_equal(gz, oz)
    np.testing.assert_array_equal(gp, op)
    return gp


@pytest.mark.parametrize("case", load_golden("partition_examples.json")["cases"],
                         ids=lambda c: c["name"])
def test_golden(torch, case):
    boxes = np.array([[0] + b for b in case["boxes"]], dtype=np.int32)
    z, p = run_gpu(torch, boxes, [0, len(boxes)], *case["frame"], *case["zones"])
    assert z.tolist() == case["zone_of"]
    assert p[:, 1:].tolist() == case["patches"]


@pytest.mark.parametrize("fw,fh,zx,zy,frames,per", [
    (3840, 2160, 4, 4, 30, 60), (3840, 2160, 2, 2, 12, 40), (3840, 2160, 1, 1, 8, 30),
    (1001, 777, 7, 3, 20, 50), (3840, 2160, 32, 32, 6, 300), (640, 480, 5, 13, 40, 10)])
def test_parity(torch, fw, fh, zx, zy, frames, per):
    boxes, fb = W.make_gmm_boxes(frames, per, fw, fh, seed=fw + zx * 10 + zy + frames,
                                 hi=min(400, fw, fh))
    check(torch, boxes, fb, fw, fh, zx, zy)


def test_many_frames(torch):
    """A 64-camera x 30-frame window: 1,920 workgroups chained by the look-back."""
    boxes, fb = W.make_gmm_boxes(1920, 30, 3840, 2160, seed=77)
    assert (np.diff(fb) == 0).sum() > 10  # frames without RoIs occur
    p = check(torch, boxes, fb, 3840, 2160, 4, 4)
    assert len(p) > 1920


def test_skipped_rois_and_empty_inputs(torch):
    boxes, fb = W.make_gmm_boxes(10, 20, 300, 200, seed=8)
    bad = boxes.copy()
    k = np.arange(0, len(bad), 7)
    bad[k[0::4], 3] = 0                          # w = 0
    bad[k[1::4], 1] = 300 - bad[k[1::4], 3] + 1  # leaves the frame on the right
    bad[k[2::4], 0] = (bad[k[2::4], 0] + 1) % 10  # another frame's id
    bad[k[3::4], 2] = -1                          # above the frame
    gz, gp = run_gpu(torch, bad, fb, 300, 200, 3, 3)
    valid = np.ones(len(bad), bool)
    valid[k] = False
    keep_fb = np.concatenate([[0], np.cumsum([valid[fb[f]:fb[f + 1]].sum() for f in range(10)])])
    oz, op = run_oracle(bad[valid], keep_fb, 300, 200, 3, 3)
    assert (gz[~valid] == -1).all()
    np.testing.assert_array_equal(gz[valid], oz)
    np.testing.assert_array_equal(gp, op)
    # no RoIs at all, and no frames
    z, p = run_gpu(torch, np.zeros((0, 5), np.int32), [0, 0, 0], 64, 64, 2, 2)
    assert len(p) == 0
    z, p = run_gpu(torch, np.zeros((0, 5), np.int32), [0], 64, 64, 2, 2)
    assert len(p) == 0


def test_deterministic_and_ready_for_the_planner(torch):
    boxes, fb = W.make_gmm_boxes(20, 60, 3840, 2160, seed=21)
    a = run_gpu(torch, boxes, fb, 3840, 2160, 4, 4)[1]
    b = run_gpu(torch, boxes, fb, 3840, 2160, 4, 4)[1]
    np.testing.assert_array_equal(a, b)
    plan = tg.plan_pack(a, 1920, 1080, 3840, 2160, 20, tg.GUILLOTINE_BSSF)
    assert plan.n_canvases >= 1
