#!/usr/bin/env python3
"""Throughput of the patch-stitching path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
  tg_plan_pack (host C++) -> plan uploaded to HBM (tg_plan_upload) -> tg_stitch once per batch of
  canvases -> tg_unstitch of every detector box.
Frames, the RoI table and the boxes are resident in HBM before timing starts. The
host plan of step s+1 overlaps the GPU work of step s (double-buffered pinned
staging), as a serving loop would run it.

Prints one JSON line. `value` is stitched canvas Mpixel/s over whole steps; the
roofline object covers the dominant kernel (tg_stitch) measured with HIP events on
the stream it runs on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
STITCH_RUN = 6144      # canvas pixels per tg_stitch work unit (include/tg.h, tg_stitch_units)
METRIC = "stitched canvas Mpixel/s and achieved HBM GB/s (% of peak), 20-cam 4K"
STITCH_SRC = os.path.join(ROOT, "paper_2404_09267_amd", "csrc", "stitch.hip")
def counters_path(workload: str) -> str:
    """Calibrated rocprofv3 traffic of tg_stitch on a workload, with the hash of the
    kernel source they were taken on (profiles/stitch_<workload>_counters.json)."""
    return os.path.join(ROOT, "profiles", f"stitch_{workload}_counters.json")


def source_hash(path=STITCH_SRC) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="cam20_4k")
    ap.add_argument("--policy", type=int, default=0, help="0 shelf FFDH, 1 shelf arrival, 2 guillotine")
    ap.add_argument("--unit-order", choices=["natural", "xcd"], default="natural",
                    help="tg_stitch launch order: units in address order (the default), or "
                         "each of the 8 XCDs sweeping its own contiguous eighth of the batch")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-aux", action="store_true",
                    help="only the path's own legs (stitch roofline, unstitch, merge, CPU "
                         "baseline): skip the streaming ceiling, invoker, partition and "
                         "background-model legs, which do not depend on --workload")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum wall time of the oracle's CPU sample")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="instead of the bench, run plain device copies of this size "
                         "(counter calibration for rocprofv3 --pmc)")
    return ap.parse_args()


def calib_copy(mb: int, steps: int):
    """Plain device copies of `mb` MiB, alternating between two source and two destination
    buffers so that no copy finds its bytes in the memory-side cache. Used to scale the
    rocprofv3 traffic counters (one copy moves a known byte count) and as the practical
    read + write streaming rate of the part."""
    import torch

    n = mb << 20
    src = [torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda") for _ in range(2)]
    dst = [torch.empty_like(src[0]) for _ in range(2)]
    stream = torch.cuda.current_stream()
    for i in range(2):
        dst[i].copy_(src[i])
    torch.cuda.synchronize()
    evs = [TimingEvent() for _ in range(steps + 1)]
    evs[0].record(stream)
    for i in range(steps):
        dst[i & 1].copy_(src[i & 1])
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    us = sum(evs[i].elapsed_time(evs[i + 1]) for i in range(steps)) * 1e3 / steps
    print(json.dumps({"calib_copy_bytes": n, "launches": steps + 2, "avg_copy_us": round(us, 2),
                      "read_plus_write_gbs": round(2 * n / us / 1e3, 1)}), flush=True)


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence: recording it
    performs no system-scope cache writeback and invalidation. An event torch creates does,
    and the GPU then idles about 5.7 us after it before the next kernel (kernel trace),
    which would charge each step for the measurement. Completion order is unchanged, so
    synchronize() still returns once the work recorded before the event has finished (all
    the host needs from it: the pinned staging read by the upload is free again); the
    timed region itself ends with a full device synchronisation. Made through the HIP
    runtime the process already uses (torch's), so that its streams are valid here."""
    _hip = None

    @classmethod
    def hip(cls):
        if cls._hip is None:
            import ctypes

            path = next((ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln),
                        None)
            if path is None:
                raise RuntimeError("the HIP runtime is not loaded")
            h = ctypes.CDLL(path)
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                              ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = h
        return cls._hip

    def __init__(self):
        import ctypes

        self.ev = ctypes.c_void_p()
        rc = self.hip().hipEventCreateWithFlags(ctypes.byref(self.ev), 0x20000000)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags: {rc}")

    def record(self, stream):
        import ctypes

        rc = self.hip().hipEventRecord(self.ev, ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord: {rc}")

    def synchronize(self):
        rc = self.hip().hipEventSynchronize(self.ev)
        if rc != 0:
            raise RuntimeError(f"hipEventSynchronize: {rc}")

    def elapsed_time(self, end) -> float:
        """Milliseconds from this event to `end`."""
        import ctypes

        ms = ctypes.c_float()
        rc = self.hip().hipEventElapsedTime(ctypes.byref(ms), self.ev, end.ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime: {rc}")
        return ms.value

    def __del__(self):
        if self._hip is not None and self.ev:
            self._hip.hipEventDestroy(self.ev)


def xcd_order(n: int) -> np.ndarray:
    """A launch order of n stitch units in which XCD x (the workgroups b with b % 8 == x,
    dealt round-robin by the dispatcher) runs one contiguous block of units in address
    order, instead of every eighth unit of the whole batch."""
    slots = [(n - x + 7) // 8 for x in range(8)]
    start = np.concatenate([[0], np.cumsum(slots)])
    b = np.arange(n)
    return (start[b % 8] + b // 8).astype(np.int32)


def stitch_bytes(rois, plan, first, count, canvas) -> int:
    """Algorithmic bytes of one tg_stitch launch: fp16 canvases written, source
    pixels read once, and 36 bytes of plan per patch (tg_roi, tg_place, order)."""
    lo, hi = int(plan.canvas_begin[first]), int(plan.canvas_begin[first + count])
    ids = plan.order[lo:hi]
    px = int((rois[ids, 3].astype(np.int64) * rois[ids, 4]).sum())
    return int(count) * canvas * canvas * 6 + 3 * px + 36 * (hi - lo)


def sample_frames(frames_d, rois, plan, sample_canvases):
    """The frames the first canvases read, copied to the host, and the RoI table with
    those RoIs' frame ids renumbered into that copy (other RoIs point at frame 0, which
    the sample's stitch does not read for them): the oracle's stitch of the sample needs
    no host copy of the whole window."""
    lo, hi = 0, int(plan.canvas_begin[sample_canvases])
    ids = plan.order[lo:hi]
    used = np.unique(rois[ids, 0])
    remap = np.zeros(int(rois[:, 0].max()) + 1, np.int32)
    remap[used] = np.arange(len(used), dtype=np.int32)
    r2 = rois.copy()
    r2[:, 0] = 0
    r2[ids, 0] = remap[rois[ids, 0]]
    idx = __import__("torch").from_numpy(used.astype(np.int64)).to(frames_d.device)
    return frames_d.index_select(0, idx).cpu().numpy(), r2


def cpu_baseline(wl, rois, frames_d, boxes, canv, plan, min_seconds: float):
    """The oracle, untuned, on a bounded sample of the same workload: the full plan,
    the first canvases' stitch and those canvases' boxes, repeated until at least
    `min_seconds` of wall time have passed."""
    import oracle

    sample_canvases = min(4, plan.n_canvases)
    frames_np, srois = sample_frames(frames_d, rois, plan, sample_canvases)
    t0 = time.perf_counter()
    reps = 0
    while True:
        rc, _, oplan = oracle.pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h,
                                   wl.n_frames, 0)
        oracle.stitch(frames_np, srois, oplan, 0, sample_canvases, wl.canvas, wl.canvas,
                      _W.MEAN, _W.STD, _W.PAD)
        sel = canv < sample_canvases
        oracle.unstitch(boxes[sel], canv[sel], rois, oplan, 1)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    px = reps * sample_canvases * wl.canvas * wl.canvas
    threads = oracle.threads()
    # the same sample on one thread, for at least a quarter of the time
    oracle.set_threads(1)
    t1, reps1 = time.perf_counter(), 0
    while True:
        rc, _, oplan = oracle.pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h,
                                   wl.n_frames, 0)
        oracle.stitch(frames_np, srois, oplan, 0, sample_canvases, wl.canvas, wl.canvas,
                      _W.MEAN, _W.STD, _W.PAD)
        oracle.unstitch(boxes[sel], canv[sel], rois, oplan, 1)
        reps1 += 1
        el1 = time.perf_counter() - t1
        if el1 >= min_seconds / 4:
            break
    oracle.set_threads(threads)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return {"value": round(px / el / 1e6, 3), "unit": "Mpixel/s", "cores": threads,
            "value_1_thread": round(reps1 * sample_canvases * wl.canvas * wl.canvas / el1 / 1e6, 3),
            "cpu_model": model, "nproc": os.cpu_count(),
            "kind": "oracle",
            "sample": f"{reps} x (plan of all {len(rois)} RoIs + stitch of canvases 0-"
                      f"{sample_canvases - 1} ({sample_canvases} x {wl.canvas}x{wl.canvas}) + "
                      f"unstitch of their {int((canv < sample_canvases).sum())} boxes), "
                      f"{el:.1f} s wall",
            "host_threads_available": len(os.sched_getaffinity(0))}


def invoker_cost(tg, W, with_oracle: bool):
    """Host cost of the SLO-aware batching invoker (tg_slo_replay, incremental packing)
    per patch arrival on a camera trace of cam20_4k's patches, next to the oracle's
    literal form (the whole queue re-packed on every arrival)."""
    wl = W.WORKLOADS["cam20_4k"]
    w, h, t, ddl, mean, std = W.camera_arrival_trace(wl)
    pt = tg.slo_patches(w, h, t, ddl)
    n = len(pt)
    reps, t0 = 0, time.perf_counter()
    while True:
        r = tg.slo_replay(pt, wl.canvas, wl.canvas, tg.GUILLOTINE_BSSF, len(mean), mean, std)
        reps += 1
        el = time.perf_counter() - t0
        if el >= 0.2:
            break
    reasons = np.bincount(r.invocations["reason"], minlength=3)
    out = {"trace": f"{n} patches of cam20_4k, 20 cameras at 30 fps, two rounds 0.3 s apart "
                    f"with SLO 0.5 s and 0.25 s, {wl.canvas}x{wl.canvas} canvases, "
                    f"guillotine, at most {len(mean)} canvases per invocation",
           "arrivals": n, "invocations": len(r.invocations),
           "fired_by": {"deadline": int(reasons[0]), "slo": int(reasons[1]),
                        "memory": int(reasons[2])},
           "us_per_arrival": round(el / reps / n * 1e6, 4)}
    if with_oracle:
        from oracle import slo

        t0 = time.perf_counter()
        slo.replay(w.tolist(), h.tolist(), t.tolist(), ddl.tolist(), wl.canvas, wl.canvas,
                   tg.GUILLOTINE_BSSF, len(mean), list(mean), list(std))
        out["oracle_us_per_arrival"] = round((time.perf_counter() - t0) / n * 1e6, 2)
    return out


def partition_cost(tg, W, torch, with_oracle: bool, launches: int = 50):
    """tg_partition (Alg. 1) over a 64-camera x 30-frame window of 3840x2160 frames with
    synthetic background-model RoIs and 4 x 4 zones, timed with HIP events on the stream
    it runs on; the oracle on a sample of the same frames."""
    import time as _t

    frames, fw, fh, zx, zy = 1920, 3840, 2160, 4, 4
    boxes, fb = W.make_gmm_boxes(frames, 30, fw, fh, seed=77)
    bufs = tg.PartitionBuffers(len(boxes), frames)
    boxes_d = torch.from_numpy(boxes).cuda()
    fb_d = torch.from_numpy(fb).cuda()
    a = tg.partition_args(boxes_d, fb_d, fw, fh, zx, zy, bufs, zone_of_box=False)
    stream = torch.cuda.current_stream()
    h = tg._vp(stream.cuda_stream)
    for _ in range(3):
        tg.lib().tg_partition(tg.ctypes.byref(a), h)
    torch.cuda.synchronize()
    evs = [TimingEvent() for _ in range(launches + 1)]
    evs[0].record(stream)
    for i in range(launches):
        rc = tg.lib().tg_partition(tg.ctypes.byref(a), h)
        if rc != tg.OK:
            raise tg.TgError("tg_partition", rc)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    us = sum(evs[i].elapsed_time(evs[i + 1]) for i in range(launches)) * 1e3 / launches
    n_patches = int(bufs.n_patches.item())
    out = {"workload": f"{frames} frames {fw}x{fh} (64 cameras x 30), {len(boxes)} RoIs, "
                       f"{zx}x{zy} zones", "patches": n_patches,
           "us_per_launch": round(us, 2), "mroi_per_s": round(len(boxes) / us, 1),
           "bound": "latency: 2 launches, one 256-thread workgroup per frame",
           "algorithmic_bytes": int(20 * len(boxes) + 4 * (frames + 1) + 20 * n_patches)}
    if with_oracle:
        from oracle import partition

        sample = frames  # the whole window: about a second
        t0 = _t.perf_counter()
        partition.partition(boxes[: fb[sample]].tolist(), fb[: sample + 1].tolist(), fw, fh, zx, zy)
        el = _t.perf_counter() - t0
        out["oracle_mroi_per_s"] = round(fb[sample] / el / 1e6, 4)
        out["oracle_sample"] = f"first {sample} frames ({int(fb[sample])} RoIs), {el:.2f} s"
    return out


def merge_cost(tg, W, torch, uargs, ubufs, name, n_frames, with_oracle: bool,
               launches: int = 50):
    """tg_merge on the bench's own tg_unstitch output (seeded detector scores, IoU 0.5
    across patches), timed with HIP events; the oracle beside."""
    stream = torch.cuda.current_stream()
    h = tg._vp(stream.cuda_stream)
    rc = tg.lib().tg_unstitch(tg.ctypes.byref(uargs), h)
    if rc != tg.OK:
        raise tg.TgError("tg_unstitch", rc)
    n_boxes = ubufs.n_boxes
    scores = torch.from_numpy(np.random.default_rng(2).uniform(0, 1, n_boxes)
                              .astype(np.float32)).cuda()
    mb = tg.MergeBuffers(n_boxes, n_frames)
    a = tg.merge_args(ubufs.dets, ubufs.n_out, scores, n_frames, 0.5, True, mb)
    for _ in range(3):
        tg.lib().tg_merge(tg.ctypes.byref(a), h)
    torch.cuda.synchronize()
    evs = [TimingEvent() for _ in range(launches + 1)]
    evs[0].record(stream)
    for i in range(launches):
        rc = tg.lib().tg_merge(tg.ctypes.byref(a), h)
        if rc != tg.OK:
            raise tg.TgError("tg_merge", rc)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    us = sum(evs[i].elapsed_time(evs[i + 1]) for i in range(launches)) * 1e3 / launches
    n_dets = int(ubufs.n_out.item())
    per_frame = np.bincount(ubufs.dets_numpy()["frame"], minlength=n_frames)
    out = {"input": f"tg_unstitch output of {name} ({n_dets} detections, {n_frames} frames, "
                    f"up to {int(per_frame.max())} per frame), IoU 0.5 across patches",
           "kept": int(mb.n_kept.item()), "us_per_call": round(us, 2),
           "bound": ("latency: one launch (capacities up to 512 detections)" if n_boxes <= 512 else
                     "latency: 8 launches (frame index and suppression rounds), about 0.3 KB "
                     "per detection")}
    if with_oracle:
        from oracle import merge

        dets = ubufs.dets_numpy()
        t0 = time.perf_counter()
        merge.merge(dets, scores.cpu().numpy(), n_frames, 0.5, True)
        out["oracle_us_per_call"] = round((time.perf_counter() - t0) * 1e6, 1)
    return out


def gmm_cost(tg, W, torch, with_oracle: bool, warm: int = 8, launches: int = 8):
    """tg_gmm_update on the 20-camera 3840x2160 background model (5 components) fed seeded
    synthetic video, then tg_mask_rois on its mask; HIP events on the stream they run on.
    Algorithmic bytes of an update: per pixel 3 sample bytes, the component count read and
    written, the mask byte, and 20 bytes per component in use before (read) and after
    (written) the frame."""
    cfg = W.GMM_BENCH
    cams, fw, fh, K = cfg["cameras"], cfg["width"], cfg["height"], cfg["n_mix"]
    video = W.SyntheticVideo(cams, fw, fh, objects=cfg["objects"], seed=cfg["seed"])
    n_video = warm + launches  # every update sees a new frame: objects keep moving
    frames = [torch.from_numpy(video.frame(t)).cuda() for t in range(n_video)]
    model = tg.GmmModel(cams, fw, fh, K)
    n = model.n_px
    stream = torch.cuda.current_stream()
    h = tg._vp(stream.cuda_stream)

    def update(t):
        a = tg.gmm_args(frames[t % n_video], model, tg.gmm_params(n_mix=K, alpha=W.gmm_alpha(t)))
        rc = tg.lib().tg_gmm_update(tg.ctypes.byref(a), h)
        if rc != tg.OK:
            raise tg.TgError("tg_gmm_update", rc)

    for t in range(warm):
        update(t)
    used = torch.zeros(launches + 1, dtype=torch.int64, device="cuda")
    used[0] = model.modes[:n].sum(dtype=torch.int64)
    evs = [(TimingEvent(), TimingEvent())
           for _ in range(launches)]
    for i in range(launches):
        evs[i][0].record(stream)
        update(warm + i)
        evs[i][1].record(stream)
        used[i + 1] = model.modes[:n].sum(dtype=torch.int64)
    torch.cuda.synchronize()
    us = [e0.elapsed_time(e1) * 1e3 for e0, e1 in evs]
    u = used.cpu().numpy()
    nbytes = [6 * n + 20 * int(u[i] + u[i + 1]) for i in range(launches)]
    gbs = float(np.mean(nbytes)) / float(np.mean(us)) / 1e3
    out = {"workload": f"{cams} cameras x {fw}x{fh}, {K} components, synthetic video "
                       f"({cfg['objects']} moving objects per camera), frames {warm}..{warm + launches - 1}",
           "us_per_update": round(float(np.mean(us)), 2),
           "gpx_per_s": round(n / float(np.mean(us)) / 1e3, 2),
           "components_per_pixel": round(float(u[1:].mean()) / n, 3),
           "foreground": round(float(model.mask[:n].float().mean()), 4),
           "algorithmic_bytes_per_update": int(np.mean(nbytes)),
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4)}}
    # tg_mask_rois on the last mask
    bufs = tg.MaskRoisBuffers(cams, fw, fh, 1 << 20, 1 << 22)
    ra = tg.mask_rois_args(model.mask, bufs, 16)
    for _ in range(2):
        tg.lib().tg_mask_rois(tg.ctypes.byref(ra), h)
    torch.cuda.synchronize()
    mevs = [TimingEvent() for _ in range(launches + 1)]
    mevs[0].record(stream)
    for i in range(launches):
        rc = tg.lib().tg_mask_rois(tg.ctypes.byref(ra), h)
        if rc != tg.OK:
            raise tg.TgError("tg_mask_rois", rc)
        mevs[i + 1].record(stream)
    torch.cuda.synchronize()
    mus = float(np.mean([mevs[i].elapsed_time(mevs[i + 1]) * 1e3 for i in range(launches)]))
    _, _, _, n_rois, n_comp = bufs.result()
    out["mask_rois"] = {"us_per_call": round(mus, 2), "rois": int(n_rois),
                        "components": int(n_comp), "min_area": 16,
                        "gpx_per_s": round(n / mus / 1e3, 2)}
    if with_oracle:
        import oracle

        px = fw * fh  # the oracle on camera 0 only, two frames
        st, md = oracle.gmm_state(px, K)
        host = [video.frame(t)[0].reshape(-1, 3) for t in range(2)]
        t0 = time.perf_counter()
        for t in range(2):
            oracle.gmm_update(host[t], st, md, oracle.gmm_params(n_mix=K, alpha=W.gmm_alpha(t)))
        el = time.perf_counter() - t0
        out["oracle_gpx_per_s"] = round(2 * px / el / 1e9, 4)
        out["oracle_sample"] = f"camera 0, frames 0-1 ({2 * px} pixel updates), {el:.2f} s, 1 thread"
    del frames, model
    return out


def replay_chunks(rois, plan, first, count, canvas, frame_stride, row_pitch):
    """The source byte ranges each stitch unit of a launch reads (canvases [first, first +
    count)): one range per patch row and STITCH_RUN-pixel run it meets, as (unit, byte
    offset into the frames, length), sorted by unit."""
    lo, hi = int(plan.canvas_begin[first]), int(plan.canvas_begin[first + count])
    ids = plan.order[lo:hi]
    pl = plan.place[ids].astype(np.int64)
    r = rois[ids].astype(np.int64)
    h = r[:, 4]
    row = np.repeat(np.arange(len(ids)), h)
    y = np.arange(int(h.sum())) - np.repeat(np.cumsum(h) - h, h)
    runs = -(-canvas * canvas // STITCH_RUN)
    assert int(r[:, 3].max(initial=0)) <= STITCH_RUN  # a patch row meets at most two runs
    s = (pl[row, 2] + y) * canvas + pl[row, 1]  # first canvas pixel of the row segment
    e = s + r[row, 3]
    src = r[row, 0] * frame_stride + (r[row, 2] + y) * row_pitch + 3 * r[row, 1]
    split = np.minimum(e, (s // STITCH_RUN + 1) * STITCH_RUN)
    unit0 = (pl[row, 0] - first) * runs + s // STITCH_RUN
    two = split < e
    unit = np.r_[unit0, unit0[two] + 1]
    off = np.r_[src, src[two] + 3 * (split[two] - s[two])]
    ln = np.r_[3 * (split - s), 3 * (e[two] - split[two])]
    o = np.argsort(unit, kind="stable")
    begin = np.searchsorted(unit[o], np.arange(count * runs + 1)).astype(np.int32)
    return off[o].astype(np.int64), ln[o].astype(np.int32), begin, runs


def replay_ceiling(torch, frames_d, rois, plan, batches, out, canvas, stitch_us,
                   launches: int = 40):
    """The stitch launches' own memory traffic replayed with no work of their own
    (libtg_probe.so tg_probe_replay): one workgroup per stitch unit reads the source byte
    ranges that unit reads and writes the unit's run of each fp16 plane, batches
    alternating as in the steps. The time is what the memory system needs for exactly this
    access pattern; stitch_frac = replay time / stitch time."""
    import ctypes

    L = ctypes.CDLL(os.path.join(ROOT, "paper_2404_09267_amd", "libtg_probe.so"))
    L.tg_probe_replay.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                  ctypes.c_int64, ctypes.c_void_p]
    F, H, Wd, _ = frames_d.shape
    src_bytes = frames_d.numel()
    import paper_2404_09267_amd.tg as tgm
    if tgm.stitch_units(canvas, canvas, 1) != -(-canvas * canvas // STITCH_RUN):
        raise RuntimeError("STITCH_RUN differs from the library's unit size")
    descs = []
    for first, count in batches:
        off, ln, begin, runs = replay_chunks(rois, plan, first, count, canvas, H * Wd * 3, Wd * 3)
        if len(off) and int(((off + ln + 15) // 16 * 16).max()) > (src_bytes + 15) // 16 * 16:
            raise RuntimeError("replay range outside the frames")
        descs.append((torch.from_numpy(off).cuda(), torch.from_numpy(ln).cuda(),
                      torch.from_numpy(begin).cuda(), count * runs, runs,
                      out[first:first + count]))
    stream = torch.cuda.current_stream()
    h = ctypes.c_void_p(stream.cuda_stream)

    def launch(i):
        off, ln, begin, n_units, runs, dst = descs[i % len(descs)]
        rc = L.tg_probe_replay(ctypes.c_void_p(frames_d.data_ptr()), src_bytes,
                               ctypes.c_void_p(off.data_ptr()), ctypes.c_void_p(ln.data_ptr()),
                               ctypes.c_void_p(begin.data_ptr()), n_units, runs,
                               ctypes.c_void_p(dst.data_ptr()), canvas * canvas * 2,
                               STITCH_RUN * 2, h)
        if rc != 0:
            raise RuntimeError(f"tg_probe_replay: {rc}")
    for i in range(4):
        launch(i)
    torch.cuda.synchronize()
    evs = [TimingEvent() for _ in range(launches + 1)]
    evs[0].record(stream)
    for i in range(launches):
        launch(i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    us = sum(evs[i].elapsed_time(evs[i + 1]) for i in range(launches)) * 1e3 / launches
    return {"kernel": "stitch traffic replayed, libtg_probe.so tg_probe_replay",
            "ranges_per_launch": int(np.mean([len(d[0]) for d in descs])),
            "us": round(us, 2), "stitch_frac": round(us / stitch_us, 4)}


def stream_ceiling(torch, read_bytes: int, write_bytes: int, launches: int = 40):
    """A plain streaming kernel (libtg_probe.so) moving the stitch launch's algorithmic
    reads and writes, writes alternating between two outputs and reads cycling through a
    pool of five read regions, as consecutive stitch batches do: what the memory system
    gives a kernel with no work of its own for this mix. Swept over the bytes each
    workgroup writes, once with each workgroup writing one contiguous run (`sweep`; the
    best rate is the ceiling) and once with its writes cut into three runs at the same
    offset of three planes, as a stitch unit writes its rows' fp16 planes (`planes3`)."""
    import ctypes

    L = ctypes.CDLL(os.path.join(ROOT, "paper_2404_09267_amd", "libtg_probe.so"))
    L.tg_probe_stream_planes.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                         ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_void_p]
    r = read_bytes // 4096 * 4096
    w = write_bytes // 4096 * 4096 // 48 * 48
    regions = 5
    pool = torch.empty(regions * r, dtype=torch.uint8, device="cuda").fill_(1)
    outs = [torch.empty(w, dtype=torch.uint8, device="cuda") for _ in range(2)]
    stream = torch.cuda.current_stream()
    h = ctypes.c_void_p(stream.cuda_stream)
    out = {"kernel": "plain stream, libtg_probe.so", "read_bytes": r, "write_bytes": w}

    def sweep(planes):
        res = {}
        for chunk in (8192, 16384, 32768, 49152, 131072):
            def launch(i):
                rc = L.tg_probe_stream_planes(
                    ctypes.c_void_p(pool.data_ptr() + (i % regions) * r), r,
                    ctypes.c_void_p(outs[i & 1].data_ptr()), w, chunk, planes, h)
                if rc != 0:
                    raise RuntimeError(f"tg_probe_stream_planes: {rc}")
            for i in range(4):
                launch(i)
            torch.cuda.synchronize()
            evs = [TimingEvent() for _ in range(launches + 1)]
            evs[0].record(stream)
            for i in range(launches):
                launch(i)
                evs[i + 1].record(stream)
            torch.cuda.synchronize()
            us = sum(evs[i].elapsed_time(evs[i + 1]) for i in range(launches)) * 1e3 / launches
            res[f"{chunk // 1024}k"] = {"us": round(us, 2), "gbs": round((r + w) / us / 1e3, 1)}
        return res

    out["sweep"] = sweep(1)
    best = max(out["sweep"], key=lambda k: out["sweep"][k]["gbs"])
    out["best_chunk"] = best
    out["gbs"] = out["sweep"][best]["gbs"]
    p3 = sweep(3)
    b3 = max(p3, key=lambda k: p3[k]["gbs"])
    out["planes3"] = {"sweep": p3, "best_chunk": b3, "gbs": p3[b3]["gbs"]}
    del pool, outs
    return out


def unstitch_cost(tg, torch, uargs, ubufs, launches: int = 50):
    """tg_unstitch alone (assign + emit), timed with HIP events after the timed steps."""
    stream = torch.cuda.current_stream()
    h = tg._vp(stream.cuda_stream)
    for _ in range(3):
        tg.lib().tg_unstitch(tg.ctypes.byref(uargs), h)
    torch.cuda.synchronize()
    evs = [TimingEvent() for _ in range(launches + 1)]
    evs[0].record(stream)
    for i in range(launches):
        rc = tg.lib().tg_unstitch(tg.ctypes.byref(uargs), h)
        if rc != tg.OK:
            raise tg.TgError("tg_unstitch", rc)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    t = sorted(evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(launches))
    us = sum(t) / launches
    # boxes and canvas ids in, a patch id per box and the detections out
    n_boxes = ubufs.n_boxes
    mb = (n_boxes * (16 + 4 + 4) + int(ubufs.n_out.item()) * 28) / 1e6
    return {"boxes": n_boxes, "us_per_call": round(us, 2), "median_us": round(t[launches // 2], 2),
            "mboxes_per_s": round(n_boxes / us, 1),
            "bound": f"latency: 2 or 3 launches, {mb:.2f} MB moved"}


_W = None


def main():
    global _W
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only; run with --gpus 1"}),
              file=sys.stderr, flush=True)
        sys.exit(2)

    import torch

    from paper_2404_09267_amd import tg
    from paper_2404_09267_amd import workload as W

    _W = W
    if args.calib_copy_mb:
        calib_copy(args.calib_copy_mb, args.steps)
        return
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    tg.lib()
    wl = W.WORKLOADS[args.workload]
    dev = torch.device("cuda")
    stream = torch.cuda.current_stream()

    # ---- resident inputs -------------------------------------------------------
    rois = W.make_rois(wl)
    frames_d = W.make_frames(wl, dev)
    plan0 = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames,
                         args.policy)
    J = plan0.n_canvases
    boxes, canv = W.make_boxes(wl, J)
    n_rois, n_boxes = len(rois), len(boxes)
    rois_d = torch.from_numpy(rois).to(dev)
    boxes_d = torch.from_numpy(boxes).to(dev)
    canv_d = torch.from_numpy(canv).to(dev)
    out = torch.empty((J, 3, wl.canvas, wl.canvas), dtype=torch.float16, device=dev)
    ubufs = tg.UnstitchBuffers(n_boxes, n_rois)
    batches = [tg.batch_range(J, wl.batch_cap, k) for k in range(tg.batch_count(J, wl.batch_cap))]

    # device plan arrays, refreshed every step from double-buffered pinned staging
    words = 5 * n_rois + 1
    staging = [torch.empty(words, dtype=torch.int32, pin_memory=True) for _ in range(2)]
    staging_np = [s.numpy() for s in staging]
    plan_d = torch.zeros(words, dtype=torch.int32, device=dev)
    dplan = tg.DevicePlan.from_tensors(rois_d, plan_d[: 3 * n_rois].view(n_rois, 3),
                                       plan_d[3 * n_rois: 4 * n_rois],
                                       plan_d[4 * n_rois: 4 * n_rois + J + 1], J)
    upload_done = [None, None]
    J_buf = np.zeros(1, np.int32)
    bad_buf = np.zeros(1, np.int32)
    params = tg.PackParams(wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, args.policy)
    unit_orders = [torch.from_numpy(xcd_order(tg.stitch_units(wl.canvas, wl.canvas, c))).to(dev)
                   if args.unit_order == "xcd" else None for _, c in batches]
    # argument blocks are built once: no pointer changes between steps
    stitch_args = [tg.stitch_args(frames_d, dplan, first, count, wl.canvas, wl.canvas,
                                  W.MEAN, W.STD, W.PAD, out[first:first + count],
                                  unit_order=unit_orders[k])
                   for k, (first, count) in enumerate(batches)]
    uargs = tg.unstitch_args(boxes_d, canv_d, dplan, 1, ubufs)
    stitch_events = []
    plan_s = []
    timing = {"on": False}

    def step(s: int):
        buf = s & 1
        if upload_done[buf] is not None:
            upload_done[buf].synchronize()  # staging of step s-2 has reached the GPU
        st = staging_np[buf]
        place = st[: 3 * n_rois].reshape(n_rois, 3)
        order = st[3 * n_rois: 4 * n_rois]
        cbeg = st[4 * n_rois: 5 * n_rois + 1]
        tp = time.perf_counter()
        rc = tg.lib().tg_plan_pack(rois.ctypes.data, n_rois, tg.ctypes.byref(params),
                                   place.ctypes.data, order.ctypes.data, cbeg.ctypes.data,
                                   J_buf.ctypes.data, bad_buf.ctypes.data)
        if timing["on"]:
            plan_s.append(time.perf_counter() - tp)
        if rc != tg.OK or J_buf[0] != J:
            raise tg.TgError("tg_plan_pack", rc)
        tg.plan_upload(staging[buf], plan_d, stream)  # one kernel reading the pinned buffer
        # Two timing events per step, one before the step's first tg_stitch launch (it also
        # marks the staging upload as done) and one after its last: every event recorded
        # between two kernels can leave the GPU idle for a few microseconds, so none is put
        # between the launches themselves (and they are made without a system fence).
        evs = [TimingEvent() for _ in range(2)]
        evs[0].record(stream)
        upload_done[buf] = evs[0]
        h = tg._vp(stream.cuda_stream)
        for a in stitch_args:
            rc = tg.lib().tg_stitch(tg.ctypes.byref(a), h)
            if rc != tg.OK:
                raise tg.TgError("tg_stitch", rc)
        evs[1].record(stream)
        if timing["on"]:
            stitch_events.append((evs[0], evs[1]))
        rc = tg.lib().tg_unstitch(tg.ctypes.byref(uargs), h)
        if rc != tg.OK:
            raise tg.TgError("tg_unstitch", rc)

    for s in range(args.warmup):
        step(s)
    torch.cuda.synchronize()
    # sanity: the plan the steps recompute equals the one the buffers were sized for
    chk = plan_d.cpu().numpy()
    assert np.array_equal(chk[: 3 * n_rois].reshape(n_rois, 3), plan0.place)
    timing["on"] = True
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.warmup, args.warmup + args.steps):
        step(s)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    timing["on"] = False

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    canvas_px = J * wl.canvas * wl.canvas
    value = canvas_px / (ms_per_step * 1e-3) / 1e6

    # ---- dominant kernel: tg_stitch ------------------------------------------------
    # each step's launches run back to back between its two events: the average launch
    # is the events' interval over all steps divided by the number of launches
    step_ms = [e0.elapsed_time(e1) for e0, e1 in stitch_events]
    n_launch = len(batches) * len(stitch_events)
    avg_ms = float(np.sum(step_ms)) / n_launch
    avg_bytes = sum(stitch_bytes(rois, plan0, f, c, wl.canvas) for f, c in batches) / len(batches)
    achieved = avg_bytes / (avg_ms * 1e-3) / 1e9
    traffic = None
    if os.path.exists(counters_path(wl.name)):
        with open(counters_path(wl.name)) as f:
            cnt = json.load(f)
        if cnt.get("stitch_source_sha256_16") == source_hash() and \
                cnt.get("workload") == wl.name:
            traffic = cnt.get("hbm_bytes_per_launch")
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "stitch_kernel<true, false>", "launches": n_launch,
                "avg_launch_us": round(avg_ms * 1e3, 2),
                "median_step_launch_us": round(float(np.median(step_ms)) * 1e3 / len(batches), 2),
                "algorithmic_bytes_per_launch": int(avg_bytes)}

    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "Mpixel/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.n_frames} x {wl.frame_w}x{wl.frame_h} u8 RGB "
                               f"frames, {n_rois} RoIs ({wl.roi_dist} {wl.roi_lo}..{wl.roi_hi} px),"
                               f" {wl.canvas}x{wl.canvas} canvases, batch cap {wl.batch_cap}, "
                               f"{n_boxes} boxes",
                   "canvases": J, "batches": len(batches), "policy": args.policy,
                   "unit_order": args.unit_order,
                   "canvas_efficiency": round(float((rois[:, 3].astype(np.int64) *
                                                     rois[:, 4]).sum()) / canvas_px, 4)},
        "roofline": roofline,
        "stitch_gbs": round(achieved, 1),
        "stitch_pct_hbm_peak": round(100 * achieved / HBM_PEAK_GBS, 2),
        # per step, over the timed steps: the host plan (overlapped with the previous
        # step's GPU work) and the GPU time of all of the step's stitch launches; then
        # tg_unstitch, timed alone after the steps (no event inside the steps separates it)
        "step_parts": {
            "plan_ms": round(1e3 * float(np.mean(plan_s)), 4),
            "stitch_ms": round(float(np.mean(step_ms)), 4),
            "unstitch_ms": None,
            "stitch_launches": len(batches)},
    }
    if not args.no_aux:
        write_bytes = int(np.mean([c * wl.canvas * wl.canvas * 6 for _, c in batches]))
        ceil = stream_ceiling(torch, int(avg_bytes) - write_bytes, write_bytes)
        ceil["stitch_frac"] = round(achieved / ceil["gbs"], 4)
        ceil["planes3"]["stitch_frac"] = round(achieved / ceil["planes3"]["gbs"], 4)
        ceil["replay"] = replay_ceiling(torch, frames_d, rois, plan0, batches, out, wl.canvas,
                                        avg_ms * 1e3)
        ceil["replay"]["gbs"] = round(avg_bytes / ceil["replay"]["us"] / 1e3, 1)
        result["ceiling"] = ceil
    result["unstitch"] = unstitch_cost(tg, torch, uargs, ubufs)
    result["step_parts"]["unstitch_ms"] = round(result["unstitch"]["us_per_call"] / 1e3, 4)
    if not args.no_aux:
        result["invoker"] = invoker_cost(tg, W, not args.no_cpu_baseline)
        result["partition"] = partition_cost(tg, W, torch, not args.no_cpu_baseline)
    result["merge"] = merge_cost(tg, W, torch, uargs, ubufs, wl.name, wl.n_frames,
                                 not args.no_cpu_baseline)
    if not args.no_aux:
        result["gmm"] = gmm_cost(tg, W, torch, not args.no_cpu_baseline)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, rois, frames_d, boxes, canv, plan0,
                                              args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
