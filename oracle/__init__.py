"""Test infrastructure only: ctypes wrapper around the plain C oracle.

Only tests/, ``__graft_entry__.smoke()`` and the bench's CPU-baseline leg may import
this package. The product path (``paper_2404_09267_amd``) never does, and the two
share no code: the only common module is the seeded input generator, which holds
none of the method's arithmetic.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# TG_LIBORACLE names another build of the oracle (the host-sanitizer build, say).
LIB_PATH = os.environ.get("TG_LIBORACLE") or os.path.join(HERE, "liboracle.so")
SOURCES = [os.path.join(HERE, "tg_oracle.c"), os.path.join(HERE, "gmm_oracle.c")]

SHELF_FFDH, SHELF_ARRIVAL, GUILLOTINE_BSSF = 0, 1, 2
OK, E_INVAL, E_ROI_OOB, E_ROI_TOO_LARGE, E_RANGE = 0, 1, 2, 3, 4
ERROR_NAMES = {OK: "ok", E_INVAL: "inval", E_ROI_OOB: "roi_oob",
               E_ROI_TOO_LARGE: "roi_too_large", E_RANGE: "range"}

DET_DTYPE = np.dtype([("box", "<i4"), ("roi", "<i4"), ("frame", "<i4"),
                      ("x1", "<f4"), ("y1", "<f4"), ("x2", "<f4"), ("y2", "<f4")])


def build(force: bool = True, path: str | None = None, sanitize: bool = False) -> str:
    """Compile liboracle.so with gcc (always, when ``force``); with ``sanitize`` under
    ASan + UBSan (every undefined-behaviour report fatal) into ``path``."""
    path = path or LIB_PATH
    if force or not os.path.exists(path):
        san = (["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                "-fno-omit-frame-pointer", "-g"] if sanitize else [])
        cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", *san,
               "-shared", "-Wall", "-Wextra", "-o", path + ".tmp", *SOURCES, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(path + ".tmp", path)
    return path


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        _lib = ctypes.CDLL(LIB_PATH)
        _declare(_lib)
    return _lib


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64


def _declare(L):
    L.oracle_half_from_double.argtypes = [ctypes.c_double]
    L.oracle_half_from_double.restype = ctypes.c_uint16
    L.oracle_norm_table.argtypes = [_P, _P, _P]
    L.oracle_norm_table.restype = None
    L.oracle_pack.argtypes = [_P, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P]
    L.oracle_pack.restype = ctypes.c_int
    L.oracle_guillotine_free.argtypes = [_P, _I32, _I32, _I32, _P, _I32]
    L.oracle_guillotine_free.restype = _I32
    L.oracle_check_plan.argtypes = [_P, _I32, _I32, _I32, _I32, _P, _P, _P, _I32]
    L.oracle_check_plan.restype = ctypes.c_int
    L.oracle_stitch.argtypes = [_P, _I64, _I32, _P, _P, _P, _P, _I32, _I32, _I32, _I32, _I32,
                                _P, _P, _P, _P]
    L.oracle_stitch.restype = ctypes.c_int
    L.oracle_pixel_sources.argtypes = [_P, _P, _P, _P, _I32, _I64, _I32, _P, _I32, _P]
    L.oracle_pixel_sources.restype = None
    L.oracle_unstitch.argtypes = [_P, _P, _I32, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P]
    L.oracle_unstitch.restype = ctypes.c_int
    L.oracle_threads.argtypes = []
    L.oracle_threads.restype = _I32
    L.oracle_set_threads.argtypes = [_I32]
    L.oracle_set_threads.restype = None
    L.oracle_gmm_pixel.argtypes = [_P, _P, _P, _P]
    L.oracle_gmm_pixel.restype = ctypes.c_int
    L.oracle_gmm_update.argtypes = [_P, _I64, _P, _P, _P, _P]
    L.oracle_gmm_update.restype = ctypes.c_int
    L.oracle_mask_rois.argtypes = [_P, _I32, _I32, _I32, _I32, _P, _P, _I64, _P]
    L.oracle_mask_rois.restype = _I64


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def half_from_double(v: float) -> int:
    return int(lib().oracle_half_from_double(float(v)))


def norm_table(mean, std) -> np.ndarray:
    """uint16 [3, 256]: binary16 bits of (x - mean_k) / std_k."""
    m = np.ascontiguousarray(mean, dtype=np.float32)
    s = np.ascontiguousarray(std, dtype=np.float32)
    t = np.zeros((3, 256), dtype=np.uint16)
    lib().oracle_norm_table(_ptr(m), _ptr(s), _ptr(t))
    return t


class Plan:
    def __init__(self, place, order, canvas_begin, n_canvases):
        self.place = place
        self.order = order
        self.canvas_begin = canvas_begin
        self.n_canvases = n_canvases


def pack(rois, canvas_w, canvas_h, frame_w, frame_h, n_frames, policy=SHELF_FFDH):
    """Returns (code, bad_index, Plan or None)."""
    r = _i32(rois).reshape(-1, 5)
    n = r.shape[0]
    place = np.zeros((n, 3), dtype=np.int32)
    order = np.zeros(n, dtype=np.int32)
    cbeg = np.zeros(n + 1, dtype=np.int32)
    J = np.zeros(1, dtype=np.int32)
    bad = np.full(1, -1, dtype=np.int32)
    rc = lib().oracle_pack(_ptr(r), n, canvas_w, canvas_h, frame_w, frame_h, n_frames, policy,
                           _ptr(place), _ptr(order), _ptr(cbeg), _ptr(J), _ptr(bad))
    if rc != OK:
        return rc, int(bad[0]), None
    j = int(J[0])
    return rc, -1, Plan(place, order, cbeg[: j + 1].copy(), j)


def guillotine_free(rois, canvas_w, canvas_h) -> np.ndarray:
    r = _i32(rois).reshape(-1, 5)
    cap = 2 * r.shape[0] + 2
    out = np.zeros((cap, 5), dtype=np.int32)
    m = lib().oracle_guillotine_free(_ptr(r), r.shape[0], canvas_w, canvas_h, _ptr(out), cap)
    if m < 0:
        raise ValueError("invalid input to guillotine_free")
    return out[:m].copy()


def check_plan(rois, canvas_w, canvas_h, policy, place, order, canvas_begin, n_canvases) -> int:
    r = _i32(rois).reshape(-1, 5)
    pl, od, cb = _i32(place).reshape(-1, 3), _i32(order), _i32(canvas_begin)
    return int(lib().oracle_check_plan(_ptr(r), r.shape[0], canvas_w, canvas_h, policy,
                                       _ptr(pl), _ptr(od), _ptr(cb), int(n_canvases)))


def stitch(frames: np.ndarray, rois, plan: Plan, first, count, canvas_w, canvas_h,
           mean, std, pad, frame_stride=None, row_pitch=None) -> np.ndarray:
    """frames: uint8 [F, H, W, 3] (or a flat buffer with explicit strides)."""
    fr = np.ascontiguousarray(frames)
    if frame_stride is None:
        frame_stride = fr.shape[1] * fr.shape[2] * 3
        row_pitch = fr.shape[2] * 3
    r = _i32(rois).reshape(-1, 5)
    out = np.empty((count, 3, canvas_h, canvas_w), dtype=np.uint16)
    m = np.ascontiguousarray(mean, dtype=np.float32)
    s = np.ascontiguousarray(std, dtype=np.float32)
    p = np.ascontiguousarray(pad, dtype=np.uint8)
    rc = lib().oracle_stitch(_ptr(fr), frame_stride, row_pitch, _ptr(r), _ptr(_i32(plan.place)),
                             _ptr(_i32(plan.order)), _ptr(_i32(plan.canvas_begin)),
                             plan.n_canvases, first, count, canvas_w, canvas_h,
                             _ptr(m), _ptr(s), _ptr(p), _ptr(out))
    if rc != OK:
        raise ValueError(f"oracle_stitch: {ERROR_NAMES.get(rc, rc)}")
    return out


def pixel_sources(rois, plan: Plan, frame_stride, row_pitch, pts) -> np.ndarray:
    """int64 byte offsets of channel 0 for sample points {canvas, X, Y}; -1 = pad."""
    q = _i32(pts).reshape(-1, 3)
    src = np.empty(q.shape[0], dtype=np.int64)
    lib().oracle_pixel_sources(_ptr(_i32(rois).reshape(-1, 5)), _ptr(_i32(plan.place)),
                               _ptr(_i32(plan.order)), _ptr(_i32(plan.canvas_begin)),
                               plan.n_canvases, frame_stride, row_pitch, _ptr(q), q.shape[0],
                               _ptr(src))
    return src


def unstitch(boxes, box_canvas, rois, plan: Plan, clip=1, rule=0):
    """Returns (roi_of_box int32 [n], dets DET_DTYPE [n_out]); rule 0 centre, 1 overlap."""
    bx = np.ascontiguousarray(boxes, dtype=np.float32).reshape(-1, 4)
    bc = _i32(box_canvas)
    n = bx.shape[0]
    rob = np.empty(n, dtype=np.int32)
    dets = np.zeros(n, dtype=DET_DTYPE)
    n_out = np.zeros(1, dtype=np.int32)
    lib().oracle_unstitch(_ptr(bx), _ptr(bc), n, _ptr(_i32(rois).reshape(-1, 5)),
                          _ptr(_i32(plan.place)), _ptr(_i32(plan.order)),
                          _ptr(_i32(plan.canvas_begin)), plan.n_canvases, int(clip), int(rule),
                          _ptr(rob), _ptr(dets), _ptr(n_out))
    return rob, dets[: int(n_out[0])].copy()


def threads() -> int:
    return int(lib().oracle_threads())


def set_threads(n: int) -> None:
    lib().oracle_set_threads(int(n))


class GmmParams(ctypes.Structure):
    """orc_gmm_params (gmm_oracle.h)."""
    _fields_ = [("n_mix", ctypes.c_int32), ("alpha", ctypes.c_float),
                ("var_threshold", ctypes.c_float), ("var_threshold_gen", ctypes.c_float),
                ("var_init", ctypes.c_float), ("var_min", ctypes.c_float),
                ("var_max", ctypes.c_float), ("background_ratio", ctypes.c_float),
                ("complexity_reduction", ctypes.c_float)]


def gmm_params(n_mix=5, alpha=0.002, var_threshold=16.0, var_threshold_gen=9.0, var_init=15.0,
               var_min=4.0, var_max=75.0, background_ratio=0.9, complexity_reduction=0.05):
    return GmmParams(n_mix, alpha, var_threshold, var_threshold_gen, var_init, var_min,
                     var_max, background_ratio, complexity_reduction)


def gmm_state(n_px: int, n_mix: int):
    """A fresh model: (state float32 [n_px][n_mix][5], modes uint8 [n_px])."""
    return (np.zeros((n_px, n_mix, 5), dtype=np.float32), np.zeros(n_px, dtype=np.uint8))


def gmm_update(frames, state, modes, params: GmmParams) -> np.ndarray:
    """One sample per pixel (frames uint8 [..., 3], pixel-major); updates state and modes
    in place and returns the foreground mask (uint8, frames' shape without the channel)."""
    fr = np.ascontiguousarray(frames, dtype=np.uint8)
    n = fr.size // 3
    assert state.dtype == np.float32 and state.flags.c_contiguous
    if 1 <= params.n_mix <= 8:  # other counts are refused by the C side before any access
        assert state.shape == (n, params.n_mix, 5)
    assert modes.dtype == np.uint8 and modes.flags.c_contiguous and modes.size == n
    mask = np.empty(fr.shape[:-1], dtype=np.uint8)
    rc = lib().oracle_gmm_update(_ptr(fr), n, _ptr(state), _ptr(modes), _ptr(mask),
                                 ctypes.byref(params))
    if rc != 0:
        raise ValueError("oracle_gmm_update: bad parameters")
    return mask


def gmm_pixel(sample, state_px, modes_px, params: GmmParams) -> int:
    """One sample of one pixel: state_px float32 [n_mix][5], modes_px uint8 [1]."""
    x = np.ascontiguousarray(sample, dtype=np.uint8).reshape(3)
    return int(lib().oracle_gmm_pixel(_ptr(x), _ptr(state_px), _ptr(modes_px),
                                      ctypes.byref(params)))


def mask_rois(mask, min_area=1):
    """mask uint8 [F, H, W]. Returns (rows int32 [n][5] = frame, x, y, w, h; areas int64
    [n]; frame_begin int32 [F + 1])."""
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    F, H, W = m.shape
    fb = np.zeros(F + 1, dtype=np.int32)
    cap = 1024
    while True:
        rows = np.zeros((cap, 5), dtype=np.int32)
        areas = np.zeros(cap, dtype=np.int64)
        n = lib().oracle_mask_rois(_ptr(m), F, W, H, int(min_area), _ptr(rows), _ptr(areas),
                                   cap, _ptr(fb))
        if n < 0:
            raise ValueError("oracle_mask_rois: bad arguments")
        if n <= cap:
            return rows[:n].copy(), areas[:n].copy(), fb
        cap = int(n)
