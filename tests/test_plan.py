"""tg_plan_pack (host, no GPU) against the oracle: bit-exact plans and error codes."""
import numpy as np
import pytest

import oracle
from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

POLICIES = [tg.SHELF_FFDH, tg.SHELF_ARRIVAL, tg.GUILLOTINE_BSSF]
CODE_MAP = {oracle.E_INVAL: tg.E_INVAL, oracle.E_ROI_OOB: tg.E_ROI_OOB,
            oracle.E_ROI_TOO_LARGE: tg.E_ROI_TOO_LARGE}


def _same_plan(p, q):
    np.testing.assert_array_equal(p.place, q.place)
    np.testing.assert_array_equal(p.order, q.order)
    np.testing.assert_array_equal(p.canvas_begin, q.canvas_begin)
    assert p.n_canvases == q.n_canvases


@pytest.mark.parametrize("policy", POLICIES)
def test_random_plans_match_oracle(policy):
    rng = np.random.default_rng(100 + policy)
    for trial in range(1500):
        cw, ch = int(rng.integers(1, 120)), int(rng.integers(1, 120))
        fw, fh, nf = int(rng.integers(1, 300)), int(rng.integers(1, 200)), int(rng.integers(1, 5))
        n = int(rng.integers(0, 150))
        rois = W.random_rois(rng, n, nf, fw, fh, 1, min(cw, fw), min(ch, fh))
        if trial % 3 == 0 and n > 0:  # many equal heights / widths exercise tie-breaks
            rois[:, 4] = np.minimum(rng.integers(1, 4, size=n) * max(1, min(ch, fh) // 4),
                                    min(ch, fh))
            rois[:, 2] = 0
        got = tg.plan_pack(rois, cw, ch, fw, fh, nf, policy)
        rc, _, want = oracle.pack(rois, cw, ch, fw, fh, nf, policy)
        assert rc == 0
        _same_plan(got, want)


@pytest.mark.parametrize("name", W.ORDERED)
@pytest.mark.parametrize("policy", POLICIES)
def test_workload_plans_match_oracle(name, policy):
    wl = W.WORKLOADS[name]
    rois = W.make_rois(wl)
    got = tg.plan_pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h, wl.n_frames, policy)
    rc, _, want = oracle.pack(rois, wl.canvas, wl.canvas, wl.frame_w, wl.frame_h,
                              wl.n_frames, policy)
    assert rc == 0
    _same_plan(got, want)
    if name != "window_64x30":  # the invariant checker's occupancy maps are slow at 4,000 canvases
        assert oracle.check_plan(rois, wl.canvas, wl.canvas, policy, got.place, got.order,
                                 got.canvas_begin, got.n_canvases) == 0


def test_golden_examples():
    from conftest import load_golden

    names = {"shelf_ffdh": 0, "shelf_arrival": 1, "guillotine_bssf": 2}
    for ex in load_golden("pack_examples.json")["examples"]:
        cw, ch = ex["canvas"]
        fw, fh, nf = ex["frame"]
        for key, pol in names.items():
            if key not in ex:
                continue
            p = tg.plan_pack(np.array(ex["rois"]), cw, ch, fw, fh, nf, pol)
            np.testing.assert_array_equal(p.place, np.array(ex[key]["place"]))
            np.testing.assert_array_equal(p.order, np.array(ex[key]["order"]))
            np.testing.assert_array_equal(p.canvas_begin, np.array(ex[key]["canvas_begin"]))


def test_error_codes_match_oracle():
    rng = np.random.default_rng(3)
    for _ in range(600):
        n = int(rng.integers(1, 12))
        rois = rng.integers(-3, 25, size=(n, 5)).astype(np.int32)
        rois[:, 0] = rng.integers(-1, 3, size=n)
        cw, ch, fw, fh, nf = 12, 10, 20, 18, 2
        rc, bad, _ = oracle.pack(rois, cw, ch, fw, fh, nf, 0)
        for pol in POLICIES:
            if rc == oracle.OK:
                got = tg.plan_pack(rois, cw, ch, fw, fh, nf, pol)
                _, _, want = oracle.pack(rois, cw, ch, fw, fh, nf, pol)
                _same_plan(got, want)
            else:
                with pytest.raises(tg.TgError) as ei:
                    tg.plan_pack(rois, cw, ch, fw, fh, nf, pol)
                assert ei.value.code == CODE_MAP[rc]
                assert ei.value.bad_index == bad


def test_bad_arguments():
    place = np.zeros((1, 3), np.int32)
    order = np.zeros(1, np.int32)
    cbeg = np.zeros(2, np.int32)
    J = np.zeros(1, np.int32)
    bad = np.zeros(1, np.int32)
    rois = np.array([[0, 0, 0, 2, 2]])
    for params in [tg.PackParams(0, 4, 8, 8, 1, 0), tg.PackParams(4, 4, 8, 0, 1, 0),
                   tg.PackParams(4, 4, 8, 8, -1, 0), tg.PackParams(4, 4, 8, 8, 1, 7)]:
        assert tg.plan_pack_raw(rois, params, place, order, cbeg, J, bad) == tg.E_INVAL
    ok = tg.PackParams(4, 4, 8, 8, 1, 0)
    assert tg.plan_pack_raw(rois, ok, place, order, cbeg, J, bad) == tg.OK
    assert J[0] == 1 and cbeg.tolist() == [0, 1]


def test_empty_plan():
    p = tg.plan_pack(np.zeros((0, 5)), 8, 8, 8, 8, 1, 0)
    assert p.n_canvases == 0 and p.canvas_begin.tolist() == [0]


def test_batch_split():
    assert tg.batch_count(0, 32) == 0
    assert tg.batch_count(63, 32) == 2
    assert tg.batch_count(64, 32) == 2
    assert tg.batch_count(65, 32) == 3
    assert tg.batch_count(7, 0) == 1
    assert tg.batch_range(63, 32, 0) == (0, 32)
    assert tg.batch_range(63, 32, 1) == (32, 31)
    assert tg.batch_range(7, 0, 0) == (0, 7)
    with pytest.raises(tg.TgError):
        tg.batch_range(63, 32, 2)
    with pytest.raises(tg.TgError):
        tg.batch_range(63, 32, -1)
    J, cap = 4010, 64
    ranges = [tg.batch_range(J, cap, k) for k in range(tg.batch_count(J, cap))]
    assert sum(c for _, c in ranges) == J
    assert all(f == k * cap for k, (f, _) in enumerate(ranges))
