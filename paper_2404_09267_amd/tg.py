"""Python binding of libtg.so (include/tg.h): argument marshalling only.

Every step of the path runs in the native library: packing in its host C++ code,
stitch and unstitch in its HIP kernels. PyTorch supplies device memory and the
stream. There is no fallback: if libtg.so is missing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

# TG_LIBTG names another build of the same library (the host-sanitizer build, say).
LIB_PATH = os.environ.get("TG_LIBTG") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                      "libtg.so")

SHELF_FFDH, SHELF_ARRIVAL, GUILLOTINE_BSSF = 0, 1, 2
OK = 0
E_INVAL, E_ROI_TOO_LARGE, E_ROI_OOB, E_RANGE, E_WORKSPACE, E_HIP, E_INTERNAL = range(-1, -8, -1)

ROI_DTYPE = np.dtype([("frame", "<i4"), ("x", "<i4"), ("y", "<i4"), ("w", "<i4"), ("h", "<i4")])
DET_DTYPE = np.dtype([("box", "<i4"), ("roi", "<i4"), ("frame", "<i4"),
                      ("x1", "<f4"), ("y1", "<f4"), ("x2", "<f4"), ("y2", "<f4")])
DET_WORDS = 7  # int32 words per tg_det
SLO_PATCH_DTYPE = np.dtype([("w", "<i4"), ("h", "<i4"), ("t_arrive", "<f8"), ("t_ddl", "<f8")])
INVOCATION_DTYPE = np.dtype([("t_fire", "<f8"), ("t_ddl", "<f8"), ("t_slack", "<f8"),
                             ("first", "<i4"), ("count", "<i4"), ("n_canvases", "<i4"),
                             ("reason", "<i4")])
FIRE_DEADLINE, FIRE_SLO, FIRE_MEMORY = 0, 1, 2

_i32, _i64, _f32, _u8, _vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_uint8,
                              ctypes.c_void_p)


class PackParams(ctypes.Structure):
    _fields_ = [("canvas_w", _i32), ("canvas_h", _i32), ("frame_w", _i32), ("frame_h", _i32),
                ("n_frames", _i32), ("policy", _i32)]


class StitchArgs(ctypes.Structure):
    _fields_ = [("frames", _vp), ("frame_stride", _i64), ("n_frames", _i32), ("frame_w", _i32),
                ("frame_h", _i32), ("row_pitch", _i32), ("rois", _vp), ("place", _vp),
                ("order", _vp), ("canvas_begin", _vp), ("n_rois", _i32), ("n_canvases", _i32),
                ("canvas_first", _i32), ("canvas_count", _i32), ("canvas_w", _i32),
                ("canvas_h", _i32), ("mean", _f32 * 3), ("std", _f32 * 3), ("pad", _u8 * 3),
                ("out", _vp), ("unit_order", _vp)]


class UnstitchArgs(ctypes.Structure):
    _fields_ = [("boxes", _vp), ("box_canvas", _vp), ("n_boxes", _i32), ("rois", _vp),
                ("place", _vp), ("order", _vp), ("canvas_begin", _vp), ("n_rois", _i32),
                ("n_canvases", _i32), ("clip", _i32), ("roi_of_box", _vp), ("dets", _vp),
                ("n_out", _vp), ("workspace", _vp), ("workspace_bytes", ctypes.c_size_t),
                ("rule", _i32)]


class PartitionArgs(ctypes.Structure):
    _fields_ = [("boxes", _vp), ("frame_begin", _vp), ("n_boxes", _i32), ("n_frames", _i32),
                ("frame_w", _i32), ("frame_h", _i32), ("zones_x", _i32), ("zones_y", _i32),
                ("patches", _vp), ("zone_of_box", _vp), ("n_patches", _vp), ("workspace", _vp),
                ("workspace_bytes", ctypes.c_size_t)]


class MergeArgs(ctypes.Structure):
    _fields_ = [("dets", _vp), ("n_dets", _vp), ("n_max", _i32), ("scores", _vp),
                ("n_scores", _i32), ("n_frames", _i32), ("iou_threshold", _f32),
                ("cross_only", _i32), ("keep", _vp), ("out", _vp), ("n_kept", _vp),
                ("workspace", _vp), ("workspace_bytes", ctypes.c_size_t)]


class SloParams(ctypes.Structure):
    _fields_ = [("canvas_w", _i32), ("canvas_h", _i32), ("policy", _i32), ("max_canvases", _i32),
                ("n_lat", _i32), ("lat_mean", _vp), ("lat_std", _vp)]


class GmmParams(ctypes.Structure):
    _fields_ = [("n_mix", _i32), ("alpha", _f32), ("var_threshold", _f32),
                ("var_threshold_gen", _f32), ("var_init", _f32), ("var_min", _f32),
                ("var_max", _f32), ("background_ratio", _f32), ("complexity_reduction", _f32)]


class GmmArgs(ctypes.Structure):
    _fields_ = [("frames", _vp), ("n_frames", _i32), ("width", _i32), ("height", _i32),
                ("state", _vp), ("modes", _vp), ("mask", _vp), ("params", GmmParams)]


class MaskRoisArgs(ctypes.Structure):
    _fields_ = [("mask", _vp), ("n_frames", _i32), ("width", _i32), ("height", _i32),
                ("min_area", _i32), ("rois", _vp), ("areas", _vp), ("max_rois", _i32),
                ("frame_begin", _vp), ("n_rois", _vp), ("n_components", _vp),
                ("max_components", _i32), ("workspace", _vp),
                ("workspace_bytes", ctypes.c_size_t)]


GMM_MAX_MIX = 5

EXPORTS = ["tg_gmm_plane_stride", "tg_gmm_state_bytes", "tg_gmm_update",
           "tg_mask_rois_workspace_bytes", "tg_mask_rois", "tg_partition_workspace_bytes", "tg_partition", "tg_plan_pack", "tg_batch_count",
           "tg_batch_range", "tg_plan_upload", "tg_slo_replay", "tg_stitch",
           "tg_stitch_units", "tg_stitch_norm_uses_table",
           "tg_unstitch_workspace_bytes", "tg_unstitch", "tg_unstitch_noalloc",
           "tg_merge_workspace_bytes", "tg_merge",
           "tg_strerror", "tg_abi_version"]

_lib = None


class TgError(RuntimeError):
    def __init__(self, call, code, bad_index=-1):
        msg = f"{call}: {strerror(code)} ({code})"
        if bad_index >= 0:
            msg += f", first bad RoI {bad_index}"
        super().__init__(msg)
        self.code = code
        self.bad_index = bad_index


def _device_count(call: str, value) -> int:
    """A count a kernel wrote: negative values are status codes (TG_E_INTERNAL when a
    device pass could not complete), raised as TgError."""
    n = int(value)
    if n < 0:
        raise TgError(call, n)
    return n


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2404_09267_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.tg_plan_pack.argtypes = [_vp, _i32, ctypes.POINTER(PackParams), _vp, _vp, _vp, _vp, _vp]
        L.tg_plan_pack.restype = ctypes.c_int
        L.tg_batch_count.argtypes = [_i32, _i32]
        L.tg_batch_count.restype = _i32
        L.tg_batch_range.argtypes = [_i32, _i32, _i32, _vp, _vp]
        L.tg_batch_range.restype = ctypes.c_int
        L.tg_plan_upload.argtypes = [_vp, _vp, ctypes.c_size_t, _vp]
        L.tg_plan_upload.restype = ctypes.c_int
        L.tg_partition_workspace_bytes.argtypes = [_i32]
        L.tg_partition_workspace_bytes.restype = ctypes.c_size_t
        L.tg_partition.argtypes = [ctypes.POINTER(PartitionArgs), _vp]
        L.tg_partition.restype = ctypes.c_int
        L.tg_slo_replay.argtypes = [_vp, _i32, ctypes.POINTER(SloParams), _vp, _vp, _vp, _vp,
                                    _vp]
        L.tg_slo_replay.restype = ctypes.c_int
        L.tg_stitch.argtypes = [ctypes.POINTER(StitchArgs), _vp]
        L.tg_stitch.restype = ctypes.c_int
        L.tg_stitch_norm_uses_table.argtypes = [ctypes.POINTER(_f32), ctypes.POINTER(_f32)]
        L.tg_stitch_norm_uses_table.restype = _i32
        L.tg_stitch_units.argtypes = [_i32, _i32, _i32]
        L.tg_stitch_units.restype = _i32
        L.tg_unstitch_workspace_bytes.argtypes = [_i32, _i32]
        L.tg_unstitch_workspace_bytes.restype = ctypes.c_size_t
        L.tg_unstitch.argtypes = [ctypes.POINTER(UnstitchArgs), _vp]
        L.tg_unstitch.restype = ctypes.c_int
        L.tg_unstitch_noalloc.argtypes = [ctypes.POINTER(UnstitchArgs), _vp]
        L.tg_unstitch_noalloc.restype = ctypes.c_int
        L.tg_merge_workspace_bytes.argtypes = [_i32, _i32]
        L.tg_merge_workspace_bytes.restype = ctypes.c_size_t
        L.tg_merge.argtypes = [ctypes.POINTER(MergeArgs), _vp]
        L.tg_merge.restype = ctypes.c_int
        L.tg_gmm_plane_stride.argtypes = [ctypes.c_int64]
        L.tg_gmm_plane_stride.restype = ctypes.c_int64
        L.tg_gmm_state_bytes.argtypes = [ctypes.c_int64, _i32]
        L.tg_gmm_state_bytes.restype = ctypes.c_size_t
        L.tg_gmm_update.argtypes = [ctypes.POINTER(GmmArgs), _vp]
        L.tg_gmm_update.restype = ctypes.c_int
        L.tg_mask_rois_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32]
        L.tg_mask_rois_workspace_bytes.restype = ctypes.c_size_t
        L.tg_mask_rois.argtypes = [ctypes.POINTER(MaskRoisArgs), _vp]
        L.tg_mask_rois.restype = ctypes.c_int
        L.tg_strerror.argtypes = [ctypes.c_int]
        L.tg_strerror.restype = ctypes.c_char_p
        L.tg_abi_version.argtypes = []
        L.tg_abi_version.restype = _i32
        _lib = L
    return _lib


def strerror(code: int) -> str:
    return lib().tg_strerror(int(code)).decode()


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(_vp)


# --------------------------------------------------------------------------- planning

@dataclass
class Plan:
    """Host outputs of tg_plan_pack."""
    place: np.ndarray         # int32 [n, 3] = {canvas, x, y}
    order: np.ndarray         # int32 [n]
    canvas_begin: np.ndarray  # int32 [J + 1]
    n_canvases: int


def plan_pack(rois: np.ndarray, canvas_w: int, canvas_h: int, frame_w: int, frame_h: int,
              n_frames: int, policy: int = SHELF_FFDH) -> Plan:
    r = np.ascontiguousarray(rois, dtype=np.int32).reshape(-1, 5)
    n = r.shape[0]
    place = np.empty((n, 3), dtype=np.int32)
    order = np.empty(n, dtype=np.int32)
    cbeg = np.empty(n + 1, dtype=np.int32)
    J = np.zeros(1, dtype=np.int32)
    bad = np.full(1, -1, dtype=np.int32)
    p = PackParams(canvas_w, canvas_h, frame_w, frame_h, n_frames, policy)
    rc = lib().tg_plan_pack(_np_ptr(r), n, ctypes.byref(p), _np_ptr(place), _np_ptr(order),
                            _np_ptr(cbeg), _np_ptr(J), _np_ptr(bad))
    if rc != OK:
        raise TgError("tg_plan_pack", rc, int(bad[0]))
    j = int(J[0])
    return Plan(place, order, cbeg[: j + 1].copy(), j)


def plan_pack_raw(rois: np.ndarray, params: PackParams, place, order, cbeg, J, bad) -> int:
    """Unchecked call on caller-provided numpy buffers (for tests of error codes)."""
    r = np.ascontiguousarray(rois, dtype=np.int32).reshape(-1, 5)
    return lib().tg_plan_pack(_np_ptr(r), r.shape[0], ctypes.byref(params), _np_ptr(place),
                              _np_ptr(order), _np_ptr(cbeg), _np_ptr(J), _np_ptr(bad))


def batch_count(n_canvases: int, batch_cap: int) -> int:
    return int(lib().tg_batch_count(n_canvases, batch_cap))


def batch_range(n_canvases: int, batch_cap: int, k: int):
    first = np.zeros(1, dtype=np.int32)
    count = np.zeros(1, dtype=np.int32)
    rc = lib().tg_batch_range(n_canvases, batch_cap, k, _np_ptr(first), _np_ptr(count))
    if rc != OK:
        raise TgError("tg_batch_range", rc)
    return int(first[0]), int(count[0])


def plan_upload(src, dst, stream=None) -> None:
    """Copies pinned host tensor `src` into device tensor `dst` (same byte size) with
    tg_plan_upload on `stream` (the current stream by default)."""
    import torch

    if not src.is_pinned():
        raise ValueError("plan_upload: the source must be pinned host memory")
    if not dst.is_cuda or not dst.is_contiguous() or not src.is_contiguous():
        raise ValueError("plan_upload: a contiguous pinned source and device destination")
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise ValueError("plan_upload: source and destination sizes differ")
    s = stream or torch.cuda.current_stream()
    rc = lib().tg_plan_upload(_vp(src.data_ptr()), _vp(dst.data_ptr()), n, _vp(s.cuda_stream))
    if rc != OK:
        raise TgError("tg_plan_upload", rc)


@dataclass
class SloReplay:
    """Host outputs of tg_slo_replay."""
    order: np.ndarray        # int32 [n]: patch ids grouped by invocation
    place: np.ndarray        # int32 [n, 3]: {canvas inside its invocation, x, y} per patch
    invocations: np.ndarray  # INVOCATION_DTYPE [n_inv]


def slo_patches(w, h, t_arrive, t_ddl) -> np.ndarray:
    """Packs per-patch arrays into tg_slo_patch records."""
    out = np.zeros(len(w), dtype=SLO_PATCH_DTYPE)
    out["w"], out["h"], out["t_arrive"], out["t_ddl"] = w, h, t_arrive, t_ddl
    return out


def slo_replay(patches: np.ndarray, canvas_w: int, canvas_h: int, policy: int, max_canvases: int,
               lat_mean, lat_std) -> SloReplay:
    pt = np.ascontiguousarray(patches, dtype=SLO_PATCH_DTYPE)
    n = pt.shape[0]
    mean = np.ascontiguousarray(lat_mean, dtype=np.float64)
    sd = np.ascontiguousarray(lat_std, dtype=np.float64)
    if mean.shape != sd.shape:
        raise ValueError("latency mean and std tables differ in length")
    p = SloParams(canvas_w, canvas_h, policy, max_canvases, mean.shape[0], _np_ptr(mean),
                  _np_ptr(sd))
    order = np.empty(n, dtype=np.int32)
    place = np.empty((n, 3), dtype=np.int32)
    inv = np.empty(max(n, 1), dtype=INVOCATION_DTYPE)
    n_inv = np.zeros(1, dtype=np.int32)
    bad = np.full(1, -1, dtype=np.int32)
    rc = lib().tg_slo_replay(_np_ptr(pt), n, ctypes.byref(p), _np_ptr(order), _np_ptr(place),
                             _np_ptr(inv), _np_ptr(n_inv), _np_ptr(bad))
    if rc != OK:
        raise TgError("tg_slo_replay", rc, int(bad[0]))
    return SloReplay(order, place, inv[: int(n_inv[0])].copy())


# --------------------------------------------------------------------------- device side

def _stream_handle(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return _vp(s.cuda_stream)


def _check(t, dtype, shape=None, name="tensor"):
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


class DevicePlan:
    """Device copies of a plan's arrays (int32, contiguous) for tg_stitch/tg_unstitch."""

    def __init__(self, rois: np.ndarray, plan: Plan, device="cuda"):
        import torch

        r = np.ascontiguousarray(rois, dtype=np.int32).reshape(-1, 5)
        self.n_rois = r.shape[0]
        self.n_canvases = plan.n_canvases
        self.rois = torch.from_numpy(r).to(device)
        self.place = torch.from_numpy(np.ascontiguousarray(plan.place, np.int32)).to(device)
        self.order = torch.from_numpy(np.ascontiguousarray(plan.order, np.int32)).to(device)
        self.canvas_begin = torch.from_numpy(
            np.ascontiguousarray(plan.canvas_begin, np.int32)).to(device)

    @classmethod
    def from_tensors(cls, rois, place, order, canvas_begin, n_canvases: int) -> "DevicePlan":
        """Wrap existing device tensors (e.g. views of one staging-backed buffer)."""
        self = cls.__new__(cls)
        self.n_rois = int(rois.shape[0])
        self.n_canvases = int(n_canvases)
        self.rois, self.place, self.order, self.canvas_begin = rois, place, order, canvas_begin
        self.check()
        return self

    def check(self):
        import torch

        _check(self.rois, torch.int32, (self.n_rois, 5), "rois")
        _check(self.place, torch.int32, (self.n_rois, 3), "place")
        _check(self.order, torch.int32, (self.n_rois,), "order")
        _check(self.canvas_begin, torch.int32, (self.n_canvases + 1,), "canvas_begin")


def stitch_norm_uses_table(mean, std) -> bool:
    """True when tg_stitch normalises through its binary16 table (no exact fp32 fma
    constants exist for this mean/std), False when it computes each value."""
    m = (_f32 * 3)(*[float(v) for v in mean])
    s = (_f32 * 3)(*[float(v) for v in std])
    rc = int(lib().tg_stitch_norm_uses_table(m, s))
    if rc < 0:
        raise TgError("tg_stitch_norm_uses_table", rc)
    return bool(rc)


def stitch_units(canvas_w: int, canvas_h: int, canvas_count: int) -> int:
    """Number of work units of one tg_stitch launch (the length of a unit order)."""
    n = int(lib().tg_stitch_units(canvas_w, canvas_h, canvas_count))
    if n < 0:
        raise TgError("tg_stitch_units", n)
    return n


def stitch_args(frames, dplan: DevicePlan, canvas_first, canvas_count, canvas_w, canvas_h,
                mean, std, pad, out, unit_order=None) -> StitchArgs:
    import torch

    dplan.check()
    if frames.dim() != 4 or frames.shape[3] != 3:
        raise ValueError("frames must be uint8 [F, H, W, 3]")
    _check(frames, torch.uint8, name="frames")
    if out.dtype not in (torch.float16, torch.int16):
        raise ValueError("out must be float16 (or int16 bit patterns)")
    _check(out, out.dtype, (canvas_count, 3, canvas_h, canvas_w), "out")
    F, H, W, _ = frames.shape
    a = StitchArgs()
    a.frames = frames.data_ptr()
    a.frame_stride = H * W * 3
    a.n_frames, a.frame_w, a.frame_h, a.row_pitch = F, W, H, W * 3
    a.rois, a.place = dplan.rois.data_ptr(), dplan.place.data_ptr()
    a.order, a.canvas_begin = dplan.order.data_ptr(), dplan.canvas_begin.data_ptr()
    a.n_rois, a.n_canvases = dplan.n_rois, dplan.n_canvases
    a.canvas_first, a.canvas_count = canvas_first, canvas_count
    a.canvas_w, a.canvas_h = canvas_w, canvas_h
    a.mean[:] = [float(v) for v in mean]
    a.std[:] = [float(v) for v in std]
    a.pad[:] = [int(v) for v in pad]
    a.out = out.data_ptr()
    a.unit_order = None
    if unit_order is not None:
        n_units = stitch_units(canvas_w, canvas_h, canvas_count) if canvas_count > 0 else 0
        _check(unit_order, torch.int32, name="unit_order")
        if unit_order.numel() < n_units:
            raise ValueError(f"unit_order must hold {n_units} unit ids")
        a.unit_order = unit_order.data_ptr()
    a._keep = (frames, dplan, out, unit_order)  # the struct holds raw pointers: keep their owners alive
    return a


def stitch(frames, dplan: DevicePlan, canvas_first, canvas_count, canvas_w, canvas_h,
           mean, std, pad, out, stream=None, unit_order=None) -> None:
    """Enqueue tg_stitch for canvases [canvas_first, +canvas_count) into `out`
    (`unit_order`: optional device int32 launch order of the units)."""
    a = stitch_args(frames, dplan, canvas_first, canvas_count, canvas_w, canvas_h,
                    mean, std, pad, out, unit_order)
    rc = lib().tg_stitch(ctypes.byref(a), _stream_handle(stream))
    if rc != OK:
        raise TgError("tg_stitch", rc)


def stitch_raw(args: StitchArgs, stream=None) -> int:
    return int(lib().tg_stitch(ctypes.byref(args), _stream_handle(stream)))


def unstitch_workspace_bytes(n_boxes: int, n_rois: int) -> int:
    return int(lib().tg_unstitch_workspace_bytes(n_boxes, n_rois))


class PartitionBuffers:
    """Caller-owned device outputs and scratch for tg_partition."""

    def __init__(self, n_boxes: int, n_frames: int, device="cuda"):
        import torch

        self.n_boxes, self.n_frames = n_boxes, n_frames
        self.patches = torch.empty((max(n_boxes, 1), 5), dtype=torch.int32, device=device)
        self.zone_of_box = torch.empty(max(n_boxes, 1), dtype=torch.int32, device=device)
        self.n_patches = torch.empty(1, dtype=torch.int32, device=device)
        ws = int(lib().tg_partition_workspace_bytes(n_frames))
        self.workspace = torch.empty(max(ws, 8), dtype=torch.uint8, device=device)
        self.workspace_bytes = ws

    def patches_numpy(self) -> np.ndarray:
        n = _device_count("tg_partition", self.n_patches.item())
        return self.patches[:n].cpu().numpy()


def partition_args(boxes, frame_begin, frame_w, frame_h, zones_x, zones_y,
                   bufs: PartitionBuffers, zone_of_box=True) -> PartitionArgs:
    import torch

    _check(boxes, torch.int32, (bufs.n_boxes, 5), "boxes")
    _check(frame_begin, torch.int32, (bufs.n_frames + 1,), "frame_begin")
    a = PartitionArgs()
    a.boxes, a.frame_begin = boxes.data_ptr(), frame_begin.data_ptr()
    a.n_boxes, a.n_frames, a.frame_w, a.frame_h = bufs.n_boxes, bufs.n_frames, frame_w, frame_h
    a.zones_x, a.zones_y = zones_x, zones_y
    a.patches = bufs.patches.data_ptr()
    a.zone_of_box = bufs.zone_of_box.data_ptr() if zone_of_box else None
    a.n_patches = bufs.n_patches.data_ptr()
    a.workspace, a.workspace_bytes = bufs.workspace.data_ptr(), bufs.workspace_bytes
    a._keep = (boxes, frame_begin, bufs)  # the struct holds raw pointers: keep their owners alive
    return a


def partition(boxes, frame_begin, frame_w, frame_h, zones_x, zones_y, bufs: PartitionBuffers,
              stream=None, zone_of_box=True) -> None:
    """Enqueue tg_partition; patches land in `bufs`."""
    a = partition_args(boxes, frame_begin, frame_w, frame_h, zones_x, zones_y, bufs, zone_of_box)
    rc = lib().tg_partition(ctypes.byref(a), _stream_handle(stream))
    if rc != OK:
        raise TgError("tg_partition", rc)


class UnstitchBuffers:
    """Caller-owned device outputs and scratch for tg_unstitch of n_boxes boxes over a plan
    of n_rois RoIs."""

    def __init__(self, n_boxes: int, n_rois: int, device="cuda"):
        import torch

        self.n_boxes, self.n_rois = n_boxes, n_rois
        self.roi_of_box = torch.empty(n_boxes, dtype=torch.int32, device=device)
        self.dets = torch.empty((n_boxes, DET_WORDS), dtype=torch.int32, device=device)
        self.n_out = torch.empty(1, dtype=torch.int32, device=device)
        ws = unstitch_workspace_bytes(n_boxes, n_rois)
        self.workspace = torch.empty(max(ws, 16), dtype=torch.uint8, device=device)
        self.workspace_bytes = ws

    def dets_numpy(self) -> np.ndarray:
        n = _device_count("tg_unstitch", self.n_out.item())
        return self.dets[:n].cpu().numpy().view(DET_DTYPE).reshape(-1)


def unstitch_args(boxes, box_canvas, dplan: DevicePlan, clip, bufs: UnstitchBuffers,
                  rule: int = 0) -> UnstitchArgs:
    import torch

    dplan.check()
    n = bufs.n_boxes
    _check(boxes, torch.float32, (n, 4), "boxes")
    _check(box_canvas, torch.int32, (n,), "box_canvas")
    if bufs.n_rois < dplan.n_rois:
        raise ValueError(f"UnstitchBuffers sized for {bufs.n_rois} RoIs, the plan has {dplan.n_rois}")
    a = UnstitchArgs()
    a.boxes, a.box_canvas, a.n_boxes = boxes.data_ptr(), box_canvas.data_ptr(), n
    a.rois, a.place = dplan.rois.data_ptr(), dplan.place.data_ptr()
    a.order, a.canvas_begin = dplan.order.data_ptr(), dplan.canvas_begin.data_ptr()
    a.n_rois, a.n_canvases, a.clip = dplan.n_rois, dplan.n_canvases, int(bool(clip))
    a.roi_of_box, a.dets, a.n_out = (bufs.roi_of_box.data_ptr(), bufs.dets.data_ptr(),
                                     bufs.n_out.data_ptr())
    a.workspace, a.workspace_bytes = bufs.workspace.data_ptr(), bufs.workspace_bytes
    a.rule = int(rule)
    a._keep = (boxes, box_canvas, dplan, bufs)  # the struct holds raw pointers: keep their owners alive
    return a


def unstitch(boxes, box_canvas, dplan: DevicePlan, clip, bufs: UnstitchBuffers,
             stream=None, rule: int = 0) -> None:
    """Enqueue tg_unstitch; results land in `bufs` (rule 0 centre, 1 largest overlap)."""
    a = unstitch_args(boxes, box_canvas, dplan, clip, bufs, rule)
    rc = lib().tg_unstitch(ctypes.byref(a), _stream_handle(stream))
    if rc != OK:
        raise TgError("tg_unstitch", rc)


def unstitch_raw(args: UnstitchArgs, stream=None) -> int:
    return int(lib().tg_unstitch(ctypes.byref(args), _stream_handle(stream)))


UNSTITCH_NOALLOC_MAX_BOXES = 1 << 24
UNSTITCH_NOALLOC_MAX_ROIS = 1 << 17


def unstitch_noalloc_raw(args: UnstitchArgs, stream=None) -> int:
    """tg_unstitch_noalloc: tg_unstitch on the library's own device scratch (the args'
    workspace fields are ignored); calls that may overlap on one GPU must be serialised."""
    return int(lib().tg_unstitch_noalloc(ctypes.byref(args), _stream_handle(stream)))


class MergeBuffers:
    """Caller-owned device outputs and scratch for tg_merge."""

    def __init__(self, n_max: int, n_frames: int, device="cuda"):
        import torch

        self.n_max, self.n_frames = n_max, n_frames
        self.keep = torch.empty(max(n_max, 1), dtype=torch.int32, device=device)
        self.out = torch.empty((max(n_max, 1), DET_WORDS), dtype=torch.int32, device=device)
        self.n_kept = torch.empty(1, dtype=torch.int32, device=device)
        ws = int(lib().tg_merge_workspace_bytes(n_max, n_frames))
        self.workspace = torch.empty(max(ws, 8), dtype=torch.uint8, device=device)
        self.workspace_bytes = ws

    def kept_numpy(self) -> np.ndarray:
        n = _device_count("tg_merge", self.n_kept.item())
        return self.out[:n].cpu().numpy().view(DET_DTYPE).reshape(-1)


def merge_args(dets, n_dets, scores, n_frames, iou_threshold, cross_only,
               bufs: MergeBuffers) -> MergeArgs:
    """dets: int32 [n_max, 7] device tensor of tg_det (e.g. UnstitchBuffers.dets); n_dets:
    device int32 [1] (e.g. UnstitchBuffers.n_out); scores: device float32 per box."""
    import torch

    _check(dets, torch.int32, (bufs.n_max, DET_WORDS), "dets")
    _check(n_dets, torch.int32, (1,), "n_dets")
    _check(scores, torch.float32, None, "scores")
    a = MergeArgs()
    a.dets, a.n_dets, a.n_max = dets.data_ptr(), n_dets.data_ptr(), bufs.n_max
    a.scores, a.n_scores = scores.data_ptr(), scores.numel()
    a.n_frames, a.iou_threshold, a.cross_only = n_frames, float(iou_threshold), int(bool(cross_only))
    a.keep, a.out = bufs.keep.data_ptr(), bufs.out.data_ptr()
    a.n_kept = bufs.n_kept.data_ptr()
    a.workspace, a.workspace_bytes = bufs.workspace.data_ptr(), bufs.workspace_bytes
    a._keep = (dets, n_dets, scores, bufs)  # the struct holds raw pointers: keep their owners alive
    return a


def merge(dets, n_dets, scores, n_frames, iou_threshold, cross_only, bufs: MergeBuffers,
          stream=None) -> None:
    """Enqueue tg_merge; results land in `bufs`."""
    a = merge_args(dets, n_dets, scores, n_frames, iou_threshold, cross_only, bufs)
    rc = lib().tg_merge(ctypes.byref(a), _stream_handle(stream))
    if rc != OK:
        raise TgError("tg_merge", rc)


# ---- background model and mask -> RoIs --------------------------------------------

def gmm_params(n_mix=5, alpha=0.002, var_threshold=16.0, var_threshold_gen=9.0, var_init=15.0,
               var_min=4.0, var_max=75.0, background_ratio=0.9,
               complexity_reduction=0.05) -> GmmParams:
    return GmmParams(n_mix, alpha, var_threshold, var_threshold_gen, var_init, var_min, var_max,
                     background_ratio, complexity_reduction)


class GmmModel:
    """Device state of the per-pixel background model of n_frames cameras (tg_gmm_update):
    5 n_mix planes of `stride` floats, the component counts and the last mask."""

    def __init__(self, n_frames: int, width: int, height: int, n_mix: int, device="cuda"):
        import torch

        self.n_frames, self.width, self.height, self.n_mix = n_frames, width, height, n_mix
        self.n_px = n_frames * width * height
        self.stride = int(lib().tg_gmm_plane_stride(self.n_px))
        nbytes = int(lib().tg_gmm_state_bytes(self.n_px, n_mix))
        if nbytes == 0:
            raise ValueError("bad model size")
        self.state = torch.zeros(nbytes // 4, dtype=torch.float32, device=device)
        self.modes = torch.zeros(max(self.n_px, 4), dtype=torch.uint8, device=device)
        self.mask = torch.zeros(max(self.n_px, 4), dtype=torch.uint8, device=device)

    def planes(self):
        """State as [n_mix, 5, n_px] (a view): weight, mean r, g, b, variance."""
        return self.state.view(self.n_mix, 5, self.stride)[:, :, : self.n_px]

    def reset(self):
        self.modes.zero_()


def gmm_args(frames, model: GmmModel, params: GmmParams) -> GmmArgs:
    import torch

    _check(frames, torch.uint8, (model.n_frames, model.height, model.width, 3), "frames")
    if params.n_mix != model.n_mix:
        raise ValueError("params.n_mix differs from the model's")
    a = GmmArgs()
    a.frames = frames.data_ptr()
    a.n_frames, a.width, a.height = model.n_frames, model.width, model.height
    a.state, a.modes, a.mask = model.state.data_ptr(), model.modes.data_ptr(), model.mask.data_ptr()
    a.params = params
    a._keep = (frames, model)  # the struct holds raw pointers: keep their owners alive
    return a


def gmm_update(frames, model: GmmModel, params: GmmParams, stream=None) -> None:
    """Enqueue tg_gmm_update: one frame per camera; the mask lands in model.mask."""
    a = gmm_args(frames, model, params)
    rc = lib().tg_gmm_update(ctypes.byref(a), _stream_handle(stream))
    if rc != OK:
        raise TgError("tg_gmm_update", rc)


class MaskRoisBuffers:
    """Caller-owned device outputs and scratch for tg_mask_rois."""

    def __init__(self, n_frames: int, width: int, height: int, max_rois: int,
                 max_components: int, device="cuda"):
        import torch

        self.n_frames, self.width, self.height = n_frames, width, height
        self.max_rois, self.max_components = max_rois, max_components
        self.rois = torch.empty((max(max_rois, 1), 5), dtype=torch.int32, device=device)
        self.areas = torch.empty(max(max_rois, 1), dtype=torch.int32, device=device)
        self.frame_begin = torch.empty(n_frames + 1, dtype=torch.int32, device=device)
        self.counts = torch.empty(2, dtype=torch.int32, device=device)  # n_rois, n_components
        ws = int(lib().tg_mask_rois_workspace_bytes(n_frames, width, height, max_components))
        if ws == 0:
            raise ValueError("bad mask size or max_components")
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)
        self.workspace_bytes = ws

    def result(self):
        """(rois int32 [n][5], areas int32 [n], frame_begin, n_rois, n_components)."""
        n_rois, n_comp = (int(v) for v in self.counts.cpu().tolist())
        _device_count("tg_mask_rois", n_rois)
        n = min(n_rois, self.max_rois)
        return (self.rois[:n].cpu().numpy(), self.areas[:n].cpu().numpy(),
                self.frame_begin.cpu().numpy(), n_rois, n_comp)


def mask_rois_args(mask, bufs: MaskRoisBuffers, min_area: int) -> MaskRoisArgs:
    import torch

    _check(mask, torch.uint8, None, "mask")
    if mask.numel() < bufs.n_frames * bufs.width * bufs.height:
        raise ValueError("mask smaller than n_frames * height * width")
    a = MaskRoisArgs()
    a.mask = mask.data_ptr()
    a.n_frames, a.width, a.height, a.min_area = bufs.n_frames, bufs.width, bufs.height, min_area
    a.rois, a.areas, a.max_rois = bufs.rois.data_ptr(), bufs.areas.data_ptr(), bufs.max_rois
    a.frame_begin = bufs.frame_begin.data_ptr()
    a.n_rois = bufs.counts.data_ptr()
    a.n_components = bufs.counts.data_ptr() + 4
    a.max_components = bufs.max_components
    a.workspace, a.workspace_bytes = bufs.workspace.data_ptr(), bufs.workspace_bytes
    a._keep = (mask, bufs)  # the struct holds raw pointers: keep their owners alive
    return a


def mask_rois(mask, bufs: MaskRoisBuffers, min_area: int = 1, stream=None) -> None:
    """Enqueue tg_mask_rois; RoIs land in `bufs`."""
    a = mask_rois_args(mask, bufs, min_area)
    rc = lib().tg_mask_rois(ctypes.byref(a), _stream_handle(stream))
    if rc != OK:
        raise TgError("tg_mask_rois", rc)
