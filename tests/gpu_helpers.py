"""Shared helpers for the GPU parity tests (test infrastructure)."""
from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

SENTINEL = 0x7E00  # a binary16 NaN: any element the kernel fails to write keeps it


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def half_ord(bits: np.ndarray) -> np.ndarray:
    """Monotone integer order of binary16 bit patterns (+0 and -0 equal)."""
    b = bits.astype(np.int32)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def assert_stitch_parity(got: np.ndarray, want: np.ndarray, covered: np.ndarray | None = None):
    """Pixels within 1 binary16 ulp, pad bit-exact (when `covered` is given); this
    library is in fact bit-exact everywhere, which is asserted separately."""
    assert got.shape == want.shape
    assert not np.any(got == SENTINEL), "unwritten output elements"
    d = np.abs(half_ord(got) - half_ord(want))
    assert d.max(initial=0) <= 1, f"max ulp diff {d.max()}"
    if covered is not None:
        pad = ~covered[:, None, :, :].repeat(3, axis=1)
        np.testing.assert_array_equal(got[pad], want[pad])


def coverage(plan, rois, first, count, cw, ch) -> np.ndarray:
    cov = np.zeros((count, ch, cw), dtype=bool)
    for j in range(first, first + count):
        for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]:
            _, x, y = plan.place[i]
            cov[j - first, y:y + rois[i, 4], x:x + rois[i, 3]] = True
    return cov


def run_stitch(frames_d, rois, plan, first, count, cw, ch, mean=W.MEAN, std=W.STD, pad=W.PAD,
               dplan=None, sentinel=True, unit_order=None):
    import torch

    dplan = dplan or tg.DevicePlan(rois, plan)
    out = torch.empty((count, 3, ch, cw), dtype=torch.int16, device="cuda")
    if sentinel:
        out.fill_(SENTINEL)
    tg.stitch(frames_d, dplan, first, count, cw, ch, mean, std, pad, out, unit_order=unit_order)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint16)


def oracle_plan(plan: tg.Plan) -> oracle.Plan:
    return oracle.Plan(plan.place, plan.order, plan.canvas_begin, plan.n_canvases)
