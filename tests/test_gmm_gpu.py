"""tg_gmm_update and tg_mask_rois on the GPU against the oracle, through the C ABI: the
foreground mask bit for bit every frame, the model state (weights, means, variances and
component counts) bit for bit, and the RoIs (boxes, pixel counts, frame_begin, counts)
exactly."""
import numpy as np
import pytest

import oracle
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


def _gpu_state(model):
    """Device planes [n_mix, 5, n_px] -> host [n_px, n_mix, 5] like the oracle's."""
    return model.planes().permute(2, 0, 1).contiguous().cpu().numpy()


def _compare_state(got, got_modes, want, want_modes, where=None):
    np.testing.assert_array_equal(got_modes, want_modes)
    K = want.shape[1]
    used = np.arange(K)[None, :] < want_modes[:, None]
    if where is not None:
        used &= where[:, None]
    np.testing.assert_array_equal(got[used].view(np.uint32), want[used].view(np.uint32))


def _params(K, t, ct=0.05, history=500):
    kw = dict(n_mix=K, alpha=W.gmm_alpha(t, history), complexity_reduction=ct)
    return tg.gmm_params(**kw), oracle.gmm_params(**kw)


@pytest.mark.parametrize("K,cams,w,h,frames,ct", [(1, 2, 131, 97, 30, 0.05),
                                                  (3, 2, 131, 97, 40, 0.05),
                                                  (5, 2, 131, 97, 40, 0.05),
                                                  (5, 1, 64, 48, 60, 0.4),
                                                  (2, 3, 33, 7, 25, 0.0),
                                                  (4, 1, 5, 1, 12, 0.1)])
def test_gmm_matches_oracle_frame_by_frame(torch, K, cams, w, h, frames, ct):
    say("gmm", K, cams, w, h, frames, ct)
    video = W.SyntheticVideo(cams, w, h, objects=6, lo=3, hi=max(4, min(w, h) // 2),
                             max_speed=3.0, seed=K * 100 + w)
    model = tg.GmmModel(cams, w, h, K)
    n = cams * w * h
    st, md = oracle.gmm_state(n, K)
    for t in range(frames):
        # a short history so that objects leave and re-enter the background in the test
        gp, op = _params(K, t, ct, history=12)
        f = video.frame(t)
        tg.gmm_update(torch.from_numpy(f).cuda(), model, gp)
        want = oracle.gmm_update(f.reshape(-1, 3), st, md, op)
        got = model.mask[:n].cpu().numpy()
        np.testing.assert_array_equal(got, want, err_msg=f"mask, frame {t}")
    assert 0 < want.mean() < 1
    _compare_state(_gpu_state(model), model.modes[:n].cpu().numpy(), st, md)


def test_gmm_first_frame_and_reset(torch):
    """A fresh model marks every pixel foreground and holds one component of weight 1;
    zeroing the counts restarts it."""
    video = W.SyntheticVideo(1, 40, 30, seed=3)
    model = tg.GmmModel(1, 40, 30, 3)
    gp, _ = _params(3, 0)
    f = torch.from_numpy(video.frame(0)).cuda()
    for _ in range(2):
        model.state.fill_(float("nan"))  # contents past the counts are never read
        model.reset()
        tg.gmm_update(f, model, gp)
        assert model.mask[:1200].cpu().numpy().all()
        assert (model.modes[:1200].cpu().numpy() == 1).all()
        pl = model.planes()
        assert (pl[0, 0] == 1).all()
        np.testing.assert_array_equal(pl[0, 1:4].T.cpu().numpy(),
                                      video.frame(0).reshape(-1, 3).astype(np.float32))


def test_gmm_full_size_bench_configuration(torch):
    """The bench's model: 20 cameras of 3840x2160, 5 components, two frames after a fresh
    start; every pixel's mask and component count, and the state of sampled pixels."""
    cfg = W.GMM_BENCH
    cams, w, h, K = cfg["cameras"], cfg["width"], cfg["height"], cfg["n_mix"]
    say("gmm full size", cams, w, h, K)
    video = W.SyntheticVideo(cams, w, h, objects=cfg["objects"], seed=cfg["seed"])
    model = tg.GmmModel(cams, w, h, K)
    n = cams * w * h
    st, md = oracle.gmm_state(n, K)
    for t in range(3):
        gp, op = _params(K, t)
        f = video.frame(t)
        tg.gmm_update(torch.from_numpy(f).cuda(), model, gp)
        want = oracle.gmm_update(f.reshape(-1, 3), st, md, op)
        np.testing.assert_array_equal(model.mask[:n].cpu().numpy(), want, err_msg=f"frame {t}")
        say("frame", t, "foreground", float(want.mean()))
    rng = np.random.default_rng(0)
    pick = np.unique(rng.integers(0, n, 2_000_000))
    got = model.planes()[:, :, torch.from_numpy(pick).cuda()].permute(2, 0, 1).cpu().numpy()
    _compare_state(got, model.modes[:n].cpu().numpy()[pick], st[pick], md[pick])
    np.testing.assert_array_equal(model.modes[:n].cpu().numpy(), md)


# ---- mask -> RoIs ----------------------------------------------------------------

def _run_rois(torch, mask, min_area=1, max_rois=None, max_components=None):
    F, H, Wd = mask.shape
    max_rois = max_rois if max_rois is not None else F * H * Wd // 2 + 1
    max_components = max_components if max_components is not None else F * H * Wd // 2 + 1
    bufs = tg.MaskRoisBuffers(F, Wd, H, max_rois, max_components)
    bufs.rois.fill_(-7)
    bufs.frame_begin.fill_(-7)
    tg.mask_rois(torch.from_numpy(np.ascontiguousarray(mask)).cuda(), bufs, min_area)
    torch.cuda.synchronize()
    return bufs.result()


def _assert_rois(torch, mask, min_area=1):
    rows, areas, fb, n_rois, n_comp = _run_rois(torch, mask, min_area)
    want_rows, want_areas, want_fb = oracle.mask_rois(mask, min_area)
    all_rows, _, _ = oracle.mask_rois(mask, 1)
    np.testing.assert_array_equal(rows, want_rows)
    np.testing.assert_array_equal(areas, want_areas)
    np.testing.assert_array_equal(fb, want_fb)
    assert n_rois == len(want_rows) and n_comp == len(all_rows)


@pytest.mark.parametrize("shape,density,min_area", [((3, 97, 131), 0.1, 1), ((2, 64, 64), 0.35, 1),
                                                    ((2, 70, 41), 0.5, 3), ((1, 33, 90), 0.6, 1),
                                                    ((4, 16, 16), 0.8, 5), ((2, 1, 200), 0.5, 1),
                                                    ((2, 200, 1), 0.5, 2), ((1, 1, 1), 1.0, 1),
                                                    ((5, 3, 3), 0.5, 1), ((1, 257, 511), 0.45, 2)])
def test_mask_rois_random_masks(torch, shape, density, min_area):
    say("mask_rois", shape, density, min_area)
    rng = np.random.default_rng(shape[1] * 1000 + shape[2])
    mask = (rng.random(shape) < density).astype(np.uint8) * rng.integers(1, 256, shape).astype(np.uint8)
    _assert_rois(torch, mask, min_area)


def test_mask_rois_structured(torch):
    """Shapes that cross many tiles: serpentine, spiral-like rings, a full frame, a
    checkerboard of isolated pixels (the most components 8-connectivity allows), empty
    frames, diagonal chains across tile corners."""
    F, H, Wd = 6, 130, 161
    m = np.zeros((F, H, Wd), np.uint8)
    for y in range(0, H, 4):
        m[0, y, 1:Wd - 1] = 1
    for y in range(0, H - 4, 8):
        m[0, y:y + 5, Wd - 2] = 1
    for y in range(4, H - 4, 8):
        m[0, y:y + 5, 1] = 1
    for r in range(2, 60, 6):
        m[1, 65 - r:65 + r, 80 - r] = m[1, 65 - r:65 + r, 80 + r] = 1
        m[1, 65 - r, 80 - r:80 + r + 1] = m[1, 65 + r, 80 - r:80 + r + 1] = 1
    m[2] = 1
    m[3, ::2, ::2] = 1
    for k in range(-H, Wd):  # anti-diagonals touching only at corners
        ys = np.arange(H)
        xs = ys + k
        ok = (xs >= 0) & (xs < Wd) & (k % 7 == 0)
        m[5, ys[ok], xs[ok]] = 1
    _assert_rois(torch, m, 1)
    _assert_rois(torch, m, 10)


def _labels_after(torch, bufs, n_px):
    """The label array and the status word that a tg_mask_rois call left in its
    workspace. The labels are the workspace's last region, 256-byte aligned and padded to
    256 bytes, so they start round_up(4 n_px, 256) bytes before its end; the status word
    is the workspace's third 8-byte word."""
    ws = bufs.workspace.cpu().numpy()
    lab_bytes = (4 * n_px + 255) // 256 * 256
    start = bufs.workspace_bytes - lab_bytes
    labels = ws[start:start + 4 * n_px].view(np.int32)
    status = int(ws[16:20].view(np.uint32)[0])
    return labels, status


def test_mask_rois_empty_frames(torch):
    """frame_begin over leading, inner and trailing frames without components, a frame
    whose components are all below min_area, and a mask with no foreground at all."""
    F, H, Wd = 7, 40, 70
    m = np.zeros((F, H, Wd), np.uint8)
    m[1, 3:9, 5:60] = 1
    m[1, 30, 2] = 1
    m[3, 10, 10] = 1          # one pixel: below min_area 2
    m[4, 0:40, 33] = 1
    m[4, 39, 0:70] = 1
    say("mask_rois empty frames", m.shape)
    _assert_rois(torch, m, 1)
    _assert_rois(torch, m, 2)
    _assert_rois(torch, np.zeros((3, 33, 65), np.uint8), 1)


def test_mask_rois_wide_frames(torch):
    """Frames more than 256 tiles (8192 pixels) wide, numbered by the per-chunk walk of
    the band instead of the listed tiles, with a long component across most of a band
    and noise; and a frame exactly 256 tiles wide, the widest the listed walk takes."""
    rng = np.random.default_rng(31)
    for shape in ((2, 40, 8300), (1, 45, 8192)):
        m = (rng.random(shape) < 0.12).astype(np.uint8)
        m[0, 5:30, 100:8100] = 1
        m[-1, 0:shape[1], 4000:4100] = 1
        say("mask_rois wide", shape)
        _assert_rois(torch, m, 2)


def test_mask_rois_many_bands(torch):
    """More than 4096 bands of 32 rows (150 frames of 29 tile rows): the numbering takes
    each band's first number from a scan over the bands' counts instead of summing them
    in each band's workgroup."""
    rng = np.random.default_rng(41)
    m = (rng.random((150, 900, 20)) < 0.2).astype(np.uint8)
    m[3, 100:800, 5:15] = 1
    m[149, 0:900:3, :] = 1
    say("mask_rois many bands", m.shape)
    _assert_rois(torch, m, 1)


def _tile_local_roots(mask2d):
    """Frame indices of the tile-local roots of one frame: per 32x32 tile, the first pixel
    (raster order) of each of the tile's own 8-connected components."""
    from scipy import ndimage

    H, Wd = mask2d.shape
    out = []
    for y0 in range(0, H, 32):
        for x0 in range(0, Wd, 32):
            sub = mask2d[y0:y0 + 32, x0:x0 + 32]
            lab, n = ndimage.label(sub, structure=np.ones((3, 3), np.int32))
            for k in range(1, n + 1):
                ys, xs = np.nonzero(lab == k)
                out.append((y0 + ys[0]) * Wd + x0 + xs[0])
    return np.sort(np.array(out, np.int64))


def test_mask_rois_labels_keep_the_union_find_invariant(torch):
    """After a call, the label words of the tile-local roots (per 32x32 tile, the first
    pixel of each of the tile's own 8-connected components; no other label word is read
    by the labelling), read back from the workspace, satisfy, checked on the CPU against
    scipy's 8-connected labelling: each holds a flagged link to a smaller tile-local root
    of the same component, or the negated component number; each component is numbered
    once, at its first pixel in raster order, in raster order over the frames; following
    the links from any tile-local root ends at its component's number. The status word is
    clear."""
    from scipy import ndimage

    rng = np.random.default_rng(21)
    F, H, Wd = 3, 197, 261
    mask = (rng.random((F, H, Wd)) < 0.5).astype(np.uint8)
    mask[1, 40:120, 30:200] = 1                     # one blob over many tiles
    mask[2, ::2, ::2] = 1                           # isolated pixels next to noise
    say("mask_rois labels", mask.shape)
    n_px = F * H * Wd
    bufs = tg.MaskRoisBuffers(F, Wd, H, n_px // 2 + 1, n_px // 2 + 1)
    tg.mask_rois(torch.from_numpy(mask).cuda(), bufs, 1)
    torch.cuda.synchronize()
    _, _, _, n_rois, n_comp = bufs.result()
    labels, status = _labels_after(torch, bufs, n_px)
    assert status == 0
    labels = labels.reshape(F, H * Wd).astype(np.int64)
    flag, index = 1 << 30, (1 << 30) - 1
    offset = 0
    for f in range(F):
        lab = labels[f]
        comp, n = ndimage.label(mask[f], structure=np.ones((3, 3), np.int32))
        comp = comp.reshape(-1)
        idx = _tile_local_roots(mask[f])
        is_local_root = np.zeros(H * Wd, bool)
        is_local_root[idx] = True
        v = lab[idx]
        numbered = v < 0
        flagged = (v >= 0) & ((v & flag) != 0)
        assert np.all(numbered | flagged)

        p, i = v[flagged] & index, idx[flagged]  # link to a smaller tile-local root
        assert np.all(p < i)
        assert np.all(is_local_root[p]) and np.array_equal(comp[p], comp[i])

        first = np.full(n + 1, np.iinfo(np.int64).max)
        np.minimum.at(first, comp[idx], idx)
        roots = idx[numbered]
        assert np.array_equal(roots, np.sort(first[1:]))
        ids = -v[numbered] - 1
        assert np.array_equal(ids, np.arange(offset, offset + len(roots)))
        id_of_comp = np.empty(n + 1, np.int64)
        id_of_comp[comp[roots]] = ids

        cur = v.copy()
        for _ in range(len(idx) + 2):  # each link strictly lowers the index: bounded
            live = cur >= 0
            if not live.any():
                break
            cur[live] = lab[cur[live] & index]
        assert np.all(cur < 0)
        assert np.array_equal(-cur - 1, id_of_comp[comp[idx]])
        offset += len(roots)
    assert offset == n_comp and n_rois == n_comp


def test_mask_rois_caps(torch):
    rng = np.random.default_rng(5)
    mask = (rng.random((2, 50, 70)) < 0.3).astype(np.uint8)
    all_rows, all_areas, all_fb = oracle.mask_rois(mask, 1)
    n = len(all_rows)
    # fewer row slots than kept components: the first max_rois are written, all counted,
    # and frame_begin indexes the full list of kept components
    rows, areas, fb, n_rois, n_comp = _run_rois(torch, mask, 1, max_rois=n // 3)
    assert n_rois == n_comp == n
    np.testing.assert_array_equal(rows, all_rows[: n // 3])
    np.testing.assert_array_equal(fb, all_fb)
    # fewer component records than components: those past the cap (raster order) are not
    # measured, and the count says so; frame_begin covers the measured ones
    cap = n // 2
    rows, areas, fb, n_rois, n_comp = _run_rois(torch, mask, 1, max_components=cap)
    assert n_comp == n and n_rois == cap
    np.testing.assert_array_equal(rows, all_rows[:cap])
    np.testing.assert_array_equal(areas, all_areas[:cap])
    frames = np.asarray(all_rows[:cap])[:, 0]
    np.testing.assert_array_equal(fb, np.searchsorted(frames, np.arange(mask.shape[0] + 1)))
    # no row slots at all
    rows, areas, fb, n_rois, n_comp = _run_rois(torch, mask, 1, max_rois=0)
    assert n_rois == n and len(rows) == 0
    np.testing.assert_array_equal(fb, all_fb)


def test_mask_rois_twice_reuses_workspace(torch):
    rng = np.random.default_rng(9)
    bufs = tg.MaskRoisBuffers(2, 90, 60, 4000, 4000)
    for d in (0.4, 0.05):
        mask = (rng.random((2, 60, 90)) < d).astype(np.uint8)
        tg.mask_rois(torch.from_numpy(mask).cuda(), bufs, 2)
        rows, areas, fb, n_rois, _ = bufs.result()
        want_rows, want_areas, want_fb = oracle.mask_rois(mask, 2)
        np.testing.assert_array_equal(rows, want_rows)
        np.testing.assert_array_equal(fb, want_fb)


def test_roi_source_end_to_end_full_size(torch):
    """Background model then mask -> RoIs then adaptive partitioning, all on the GPU, at
    the bench's size, against the oracle's model, labelling and partitioning."""
    from oracle import partition as opart

    cfg = W.GMM_BENCH
    cams, w, h, K = 4, cfg["width"], cfg["height"], cfg["n_mix"]
    say("roi source end to end", cams, w, h, K)
    video = W.SyntheticVideo(cams, w, h, objects=cfg["objects"], seed=cfg["seed"])
    model = tg.GmmModel(cams, w, h, K)
    n = cams * w * h
    st, md = oracle.gmm_state(n, K)
    for t in range(8):
        gp, op = _params(K, t, history=4)
        f = video.frame(t)
        tg.gmm_update(torch.from_numpy(f).cuda(), model, gp)
        want_mask = oracle.gmm_update(f.reshape(-1, 3), st, md, op)
    bufs = tg.MaskRoisBuffers(cams, w, h, 1 << 20, 1 << 22)
    tg.mask_rois(model.mask, bufs, 16)
    rows, areas, fb, n_rois, n_comp = bufs.result()
    want_rows, want_areas, want_fb = oracle.mask_rois(want_mask.reshape(cams, h, w), 16)
    np.testing.assert_array_equal(rows, want_rows)
    np.testing.assert_array_equal(areas, want_areas)
    np.testing.assert_array_equal(fb, want_fb)
    say("rois", n_rois, "components", n_comp)
    assert n_rois > 0
    pb = tg.PartitionBuffers(n_rois, cams)
    tg.partition(bufs.rois[:n_rois], bufs.frame_begin, w, h, 4, 4, pb)
    torch.cuda.synchronize()
    _, want_patches = opart.partition(want_rows.tolist(), want_fb.tolist(), w, h, 4, 4)
    np.testing.assert_array_equal(pb.patches_numpy(), np.array(want_patches, np.int32).reshape(-1, 5))


def test_mask_rois_unaligned_mask_pointer(torch):
    """A mask that starts one byte into its buffer: every pass takes its byte-wise reads
    (the dword, 16-byte and span loads need aligned rows); several 65,536-pixel spans and
    rows whose width is a multiple of 16, so only the pointer differs from the fast paths."""
    rng = np.random.default_rng(21)
    F, H, Wd = 3, 200, 160
    mask = np.zeros((F, H, Wd), np.uint8)
    for f in range(F):
        for _ in range(25):
            h, w = (int(v) for v in rng.integers(2, 70, 2))
            y, x = int(rng.integers(0, H - h)), int(rng.integers(0, Wd - w))
            mask[f, y:y + h, x:x + w] = 1
    mask |= (rng.random(mask.shape) < 0.02).astype(np.uint8)
    buf = torch.zeros(mask.size + 16, dtype=torch.uint8, device="cuda")
    buf[1:1 + mask.size] = torch.from_numpy(mask.reshape(-1)).cuda()
    view = buf[1:1 + mask.size]
    assert view.data_ptr() % 4 == 1
    say("mask_rois unaligned", mask.shape)
    bufs = tg.MaskRoisBuffers(F, Wd, H, 1 << 16, 1 << 16)
    tg.mask_rois(view, bufs, 2)
    rows, areas, fb, n_rois, n_comp = bufs.result()
    want_rows, want_areas, want_fb = oracle.mask_rois(mask, 2)
    np.testing.assert_array_equal(rows, want_rows)
    np.testing.assert_array_equal(areas, want_areas)
    np.testing.assert_array_equal(fb, want_fb)
    assert n_rois == len(want_rows) and n_comp == len(oracle.mask_rois(mask, 1)[0])
