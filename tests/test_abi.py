"""The C ABI: the library loads, exports every function tg.h declares, the ctypes
structs match the header's layout, and argument validation rejects bad calls before
any HIP work (so these run without a GPU)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2404_09267_amd import tg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tg.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tg_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(tg.EXPORTS)
    L = tg.lib()
    for n in names:
        assert hasattr(L, n), n


def test_abi_version():
    assert tg.lib().tg_abi_version() == 8


def test_strerror():
    for code in range(0, -8, -1):
        assert tg.strerror(code) not in ("", "unknown status")
    assert tg.strerror(-99) == "unknown status"


def _c_layout(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(r"""
#include <stdio.h>
#include <stddef.h>
#include "tg.h"
#define F(T, m) printf(#T "." #m " %zu\n", offsetof(T, m))
int main(void) {
  printf("tg_roi %zu\ntg_place %zu\ntg_box %zu\ntg_det %zu\ntg_pack_params %zu\n",
         sizeof(tg_roi), sizeof(tg_place), sizeof(tg_box), sizeof(tg_det), sizeof(tg_pack_params));
  printf("tg_stitch_args %zu\ntg_unstitch_args %zu\n", sizeof(tg_stitch_args), sizeof(tg_unstitch_args));
  printf("tg_slo_patch %zu\ntg_slo_params %zu\ntg_invocation %zu\n", sizeof(tg_slo_patch),
         sizeof(tg_slo_params), sizeof(tg_invocation));
  F(tg_slo_patch, w); F(tg_slo_patch, h); F(tg_slo_patch, t_arrive); F(tg_slo_patch, t_ddl);
  F(tg_slo_params, canvas_w); F(tg_slo_params, policy); F(tg_slo_params, max_canvases);
  F(tg_slo_params, n_lat); F(tg_slo_params, lat_mean); F(tg_slo_params, lat_std);
  F(tg_invocation, t_fire); F(tg_invocation, t_ddl); F(tg_invocation, t_slack);
  F(tg_invocation, first); F(tg_invocation, count); F(tg_invocation, n_canvases);
  F(tg_invocation, reason);
  F(tg_stitch_args, frames); F(tg_stitch_args, frame_stride); F(tg_stitch_args, n_frames);
  F(tg_stitch_args, row_pitch); F(tg_stitch_args, rois); F(tg_stitch_args, canvas_begin);
  F(tg_stitch_args, n_rois); F(tg_stitch_args, canvas_first); F(tg_stitch_args, canvas_h);
  F(tg_stitch_args, mean); F(tg_stitch_args, std); F(tg_stitch_args, pad); F(tg_stitch_args, out);
  F(tg_stitch_args, unit_order);
  F(tg_unstitch_args, boxes); F(tg_unstitch_args, n_boxes); F(tg_unstitch_args, rois);
  F(tg_unstitch_args, n_rois); F(tg_unstitch_args, clip); F(tg_unstitch_args, roi_of_box);
  F(tg_unstitch_args, n_out); F(tg_unstitch_args, workspace); F(tg_unstitch_args, workspace_bytes);
  F(tg_unstitch_args, rule);
  printf("noalloc_max_boxes %d\nnoalloc_max_rois %d\n", TG_UNSTITCH_NOALLOC_MAX_BOXES,
         TG_UNSTITCH_NOALLOC_MAX_ROIS);
  printf("tg_gmm_params %zu\ntg_gmm_args %zu\ntg_mask_rois_args %zu\n", sizeof(tg_gmm_params),
         sizeof(tg_gmm_args), sizeof(tg_mask_rois_args));
  F(tg_gmm_params, alpha); F(tg_gmm_params, var_threshold_gen); F(tg_gmm_params, var_max);
  F(tg_gmm_params, complexity_reduction);
  F(tg_gmm_args, frames); F(tg_gmm_args, n_frames); F(tg_gmm_args, height); F(tg_gmm_args, state);
  F(tg_gmm_args, modes); F(tg_gmm_args, mask); F(tg_gmm_args, params);
  F(tg_mask_rois_args, mask); F(tg_mask_rois_args, min_area); F(tg_mask_rois_args, rois);
  F(tg_mask_rois_args, areas); F(tg_mask_rois_args, max_rois); F(tg_mask_rois_args, frame_begin);
  F(tg_mask_rois_args, n_rois); F(tg_mask_rois_args, n_components);
  F(tg_mask_rois_args, max_components); F(tg_mask_rois_args, workspace);
  F(tg_mask_rois_args, workspace_bytes);
  return 0;
}
""")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    return dict(line.rsplit(" ", 1) for line in out.strip().splitlines())


def test_struct_layout_matches_header(tmp_path):
    c = {k: int(v) for k, v in _c_layout(tmp_path).items()}
    assert c["tg_roi"] == 20 and c["tg_place"] == 12 and c["tg_box"] == 16 and c["tg_det"] == 28
    assert c["tg_roi"] == tg.ROI_DTYPE.itemsize and c["tg_det"] == tg.DET_DTYPE.itemsize
    assert c["tg_pack_params"] == ctypes.sizeof(tg.PackParams)
    assert c["tg_stitch_args"] == ctypes.sizeof(tg.StitchArgs)
    assert c["tg_unstitch_args"] == ctypes.sizeof(tg.UnstitchArgs)
    assert c["noalloc_max_boxes"] == tg.UNSTITCH_NOALLOC_MAX_BOXES
    assert c["noalloc_max_rois"] == tg.UNSTITCH_NOALLOC_MAX_ROIS
    assert c["tg_slo_patch"] == tg.SLO_PATCH_DTYPE.itemsize == 24
    assert c["tg_slo_params"] == ctypes.sizeof(tg.SloParams)
    assert c["tg_invocation"] == tg.INVOCATION_DTYPE.itemsize == 40
    assert c["tg_gmm_params"] == ctypes.sizeof(tg.GmmParams) == 36
    assert c["tg_gmm_args"] == ctypes.sizeof(tg.GmmArgs)
    assert c["tg_mask_rois_args"] == ctypes.sizeof(tg.MaskRoisArgs)
    structs = {"tg_stitch_args": tg.StitchArgs, "tg_unstitch_args": tg.UnstitchArgs,
               "tg_slo_params": tg.SloParams, "tg_gmm_params": tg.GmmParams,
               "tg_gmm_args": tg.GmmArgs, "tg_mask_rois_args": tg.MaskRoisArgs}
    dtypes = {"tg_slo_patch": tg.SLO_PATCH_DTYPE, "tg_invocation": tg.INVOCATION_DTYPE}
    for key, off in c.items():
        if "." not in key:
            continue
        struct, field = key.split(".")
        if struct in dtypes:
            assert dtypes[struct].fields[field][1] == off, key
        else:
            assert getattr(structs[struct], field).offset == off, key


def _valid_stitch_args():
    a = tg.StitchArgs()
    a.frames = 0x1000
    a.frame_stride = 64 * 64 * 3
    a.n_frames, a.frame_w, a.frame_h, a.row_pitch = 1, 64, 64, 192
    a.rois = a.place = a.order = a.canvas_begin = 0x2000
    a.n_rois, a.n_canvases, a.canvas_first, a.canvas_count = 4, 2, 0, 0
    a.canvas_w = a.canvas_h = 32
    a.mean[:] = [0.0, 0.0, 0.0]
    a.std[:] = [1.0, 1.0, 1.0]
    a.out = 0x3000
    return a


def _raw_stitch(a):
    return int(tg.lib().tg_stitch(ctypes.byref(a), None))


def test_stitch_validation_without_gpu():
    """Every rejection happens before any HIP call; canvas_count == 0 is a no-op."""
    a = _valid_stitch_args()
    assert _raw_stitch(a) == tg.OK  # nothing to do
    assert int(tg.lib().tg_stitch(None, None)) == tg.E_INVAL
    cases = [("canvas_w", 0, tg.E_INVAL), ("frame_h", 0, tg.E_INVAL),
             ("row_pitch", 191, tg.E_INVAL), ("frame_stride", 100, tg.E_INVAL),
             ("canvas_count", -1, tg.E_INVAL), ("canvas_first", -1, tg.E_INVAL),
             ("n_rois", -1, tg.E_INVAL)]
    for field, val, code in cases:
        b = _valid_stitch_args()
        setattr(b, field, val)
        assert _raw_stitch(b) == code, field
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        b = _valid_stitch_args()
        b.std[1] = bad
        assert _raw_stitch(b) == tg.E_INVAL
    b = _valid_stitch_args()
    b.mean[2] = float("nan")
    assert _raw_stitch(b) == tg.E_INVAL
    b = _valid_stitch_args()
    b.canvas_first, b.canvas_count = 1, 2
    assert _raw_stitch(b) == tg.E_RANGE
    b = _valid_stitch_args()
    b.canvas_count = 1
    b.out = None
    assert _raw_stitch(b) == tg.E_INVAL


def test_unstitch_validation_without_gpu():
    a = tg.UnstitchArgs()
    a.n_boxes = -1
    a.n_out = 0x1000
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_INVAL
    a.n_boxes = 10
    a.n_out = None
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_INVAL
    a.n_out = 0x1000
    a.boxes = a.box_canvas = a.roi_of_box = a.dets = 0x2000
    a.rois = a.place = a.order = a.canvas_begin = 0x3000
    a.n_rois, a.n_canvases = 3, 1
    a.workspace, a.workspace_bytes = 0x4000, tg.unstitch_workspace_bytes(10, 3) - 1
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_WORKSPACE
    a.n_rois, a.workspace_bytes = 4, tg.unstitch_workspace_bytes(10, 3)  # records for 3 only
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_WORKSPACE
    a.n_rois = 3
    a.workspace = None
    a.workspace_bytes = 1 << 20
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_WORKSPACE
    a.workspace = 0x4004  # misaligned
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_WORKSPACE
    a.workspace = 0x4008  # 8-byte but not 16-byte aligned (the patch records are float4)
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_WORKSPACE
    a.workspace = 0x4000
    a.rois = None
    assert int(tg.lib().tg_unstitch(ctypes.byref(a), None)) == tg.E_INVAL


def test_plan_upload_validation_without_gpu():
    L = tg.lib()
    assert int(L.tg_plan_upload(None, None, 0, None)) == tg.OK         # nothing to move
    assert int(L.tg_plan_upload(None, ctypes.c_void_p(0x1000), 8, None)) == tg.E_INVAL
    assert int(L.tg_plan_upload(ctypes.c_void_p(0x1000), None, 8, None)) == tg.E_INVAL


def test_workspace_sizes():
    assert tg.unstitch_workspace_bytes(0, 100) == 0
    assert tg.unstitch_workspace_bytes(-5, 100) == 0
    # one ticket word and one look-back word per 1024 boxes, rounded up to 16 bytes, then
    # 24 bytes of patch record per RoI
    assert tg.unstitch_workspace_bytes(1, 0) == 16
    assert tg.unstitch_workspace_bytes(1024, 0) == 16
    assert tg.unstitch_workspace_bytes(1025, 0) == 32
    assert tg.unstitch_workspace_bytes(200000, 0) == 1584  # 8 * (1 + 196), rounded up
    assert tg.unstitch_workspace_bytes(1, 3) == 16 + 72
    assert tg.unstitch_workspace_bytes(200000, 115200) == 1584 + 24 * 115200
    assert tg.unstitch_workspace_bytes(10, -1) == 16


def test_gmm_and_mask_rois_validation_without_gpu():
    L = tg.lib()
    assert L.tg_gmm_plane_stride(1) == 64 and L.tg_gmm_plane_stride(64) == 64
    assert L.tg_gmm_plane_stride(65) == 128 and L.tg_gmm_plane_stride(0) == 0
    assert L.tg_gmm_state_bytes(100, 3) == 4 * 5 * 3 * 128
    assert L.tg_gmm_state_bytes(100, 0) == 0 and L.tg_gmm_state_bytes(100, 6) == 0
    a = tg.GmmArgs()
    a.frames = a.state = a.modes = a.mask = 0x1000
    a.n_frames, a.width, a.height = 1, 8, 8
    a.params = tg.gmm_params(n_mix=3)
    for field, bad in (("n_mix", 0), ("n_mix", 6), ("alpha", 0.0), ("alpha", 2.0),
                       ("var_min", 0.0), ("complexity_reduction", 1.0),
                       ("background_ratio", float("nan"))):
        b = tg.GmmArgs.from_buffer_copy(a)
        setattr(b.params, field, bad)
        assert L.tg_gmm_update(ctypes.byref(b), None) == tg.E_INVAL, field
    b = tg.GmmArgs.from_buffer_copy(a)
    b.state = 0x1004  # not 16-byte aligned
    assert L.tg_gmm_update(ctypes.byref(b), None) == tg.E_INVAL
    b = tg.GmmArgs.from_buffer_copy(a)
    b.n_frames = 0
    assert L.tg_gmm_update(ctypes.byref(b), None) == tg.OK  # nothing to do, no launch
    assert L.tg_gmm_update(None, None) == tg.E_INVAL

    assert L.tg_mask_rois_workspace_bytes(1, 8, 8, 0) == 0
    assert L.tg_mask_rois_workspace_bytes(70000, 8, 8, 4) == 0
    assert L.tg_mask_rois_workspace_bytes(1, 1 << 16, 1 << 15, 4) == 0
    assert L.tg_mask_rois_workspace_bytes(1, 1 << 15, 1 << 15, 4) == 0  # 2^30 pixels: no flag bit
    assert L.tg_mask_rois_workspace_bytes(1, 1 << 15, (1 << 15) - 1, 4) > 0
    # tile slots are 28-bit: 65535 frames of 64 x 64 tiles fit (268,431,360 < 2^28), of
    # 64 x 65 tiles do not
    assert L.tg_mask_rois_workspace_bytes(65535, 2048, 2048, 4) > 0
    assert L.tg_mask_rois_workspace_bytes(65535, 2048, 2080, 4) == 0
    ws = L.tg_mask_rois_workspace_bytes(2, 100, 50, 1000)
    # labels, component records, and per 32 x 32 tile (2 frames x 4 x 2
    # tiles) its list entry, records (row masks, root masks, border roots), entry slots
    # and entry count
    tiles = 2 * 4 * 2
    assert ws >= 4 * 2 * 100 * 50 + 32 * 1000 + tiles * (4 + 128 + 128 + 512 + 2048 + 4)
    assert ws % 256 == 0
    m = tg.MaskRoisArgs()
    m.mask = m.rois = m.areas = m.frame_begin = m.n_rois = m.n_components = 0x1000
    m.n_frames, m.width, m.height, m.min_area, m.max_rois, m.max_components = 2, 100, 50, 1, 10, 1000
    m.workspace, m.workspace_bytes = 0x2000, ws - 1
    assert L.tg_mask_rois(ctypes.byref(m), None) == tg.E_WORKSPACE
    m.workspace = 0x2008
    m.workspace_bytes = ws
    assert L.tg_mask_rois(ctypes.byref(m), None) == tg.E_WORKSPACE  # misaligned
    for field, bad in (("max_components", 0), ("max_rois", -1), ("width", 0), ("n_frames", -1)):
        b = tg.MaskRoisArgs.from_buffer_copy(m)
        setattr(b, field, bad)
        assert L.tg_mask_rois(ctypes.byref(b), None) == tg.E_INVAL, field
    b = tg.MaskRoisArgs.from_buffer_copy(m)
    b.n_rois = None
    assert L.tg_mask_rois(ctypes.byref(b), None) == tg.E_INVAL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(tg, "LIB_PATH", str(tmp_path / "nope.so"))
    monkeypatch.setattr(tg, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        tg.lib()


def test_probe_library_exports_its_header():
    """libtg_probe.so (the benchmark's streaming probe) exports what tg_probe.h declares
    and rejects bad arguments before any HIP call."""
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "tg_probe.h")).read(),
                  flags=re.S)
    names = sorted(set(re.findall(r"\b(tg_\w+)\s*\(", text)))
    assert names == ["tg_probe_replay", "tg_probe_stream", "tg_probe_stream_planes"]
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2404_09267_amd", "libtg_probe.so"))
    f = L.tg_probe_stream
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_int32, ctypes.c_void_p]
    ok = ctypes.c_void_p(4096)
    assert f(None, 4096, ok, 4096, 4096, None) == -1          # null source
    assert f(ok, 4096, ok, 0, 4096, None) == -1               # nothing to write
    assert f(ok, 4100, ok, 4096, 4096, None) == -1            # size not a multiple of 16
    assert f(ok, 4096, ok, 4096, 1000, None) == -1            # chunk not whole pages
    assert f(ctypes.c_void_p(4104), 4096, ok, 4096, 4096, None) == -1  # misaligned
    g = L.tg_probe_stream_planes
    g.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
    assert g(ok, 4096, ok, 4800, 4096, 0, None) == -1        # no planes
    assert g(ok, 4096, ok, 4800, 4096, 5, None) == -1        # too many planes
    assert g(ok, 4096, ok, 4816, 4096, 3, None) == -1        # planes of whole 16-byte words
    r = L.tg_probe_replay
    r.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                  ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
    assert r(None, 4096, ok, ok, ok, 4, 2, ok, 4096, 4096, None) == -1  # null source
    assert r(ok, 4096, ok, ok, ok, 0, 1, ok, 4096, 4096, None) == -1    # no units
    assert r(ok, 4096, ok, ok, ok, 5, 2, ok, 4096, 4096, None) == -1    # not whole canvases
    assert r(ok, 4096, ok, ok, ok, 4, 2, ok, 4100, 4096, None) == -1    # plane not whole words
    assert r(ok, 4096, ok, ok, ok, 4, 2, ok, 4096, 4100, None) == -1    # run not whole words
    assert r(ok, 4096, ok, ok, ok, 4, 2, ctypes.c_void_p(4104), 4096, 4096, None) == -1


def test_unstitch_noalloc_validation_without_gpu():
    """The allocation-free entry point checks its arguments like tg_unstitch and refuses
    more boxes than its device scratch holds, before anything is enqueued."""
    L = tg.lib()
    a = tg.UnstitchArgs()
    a.n_boxes = -1
    a.n_out = 0x1000
    assert int(L.tg_unstitch_noalloc(ctypes.byref(a), None)) == tg.E_INVAL
    a.n_boxes = 10
    a.n_out = 0x1000
    a.boxes = a.box_canvas = a.roi_of_box = a.dets = 0x2000
    a.rois = a.place = a.order = a.canvas_begin = 0x3000
    a.n_rois, a.n_canvases = 3, 1
    a.rule = 2
    assert int(L.tg_unstitch_noalloc(ctypes.byref(a), None)) == tg.E_INVAL
    a.rule = 0
    a.n_boxes = tg.UNSTITCH_NOALLOC_MAX_BOXES + 1
    assert int(L.tg_unstitch_noalloc(ctypes.byref(a), None)) == tg.E_WORKSPACE
    a.n_boxes = 10
    a.dets = None
    assert int(L.tg_unstitch_noalloc(ctypes.byref(a), None)) == tg.E_INVAL
