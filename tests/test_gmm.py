"""The oracle's Gaussian-mixture background model and mask-to-RoI step, pinned to
hand-worked samples, closed forms, a library filter and a library labeller."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.ndimage as ndi
from scipy.signal import lfilter

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _params(d):
    return oracle.gmm_params(**d)


def _run(samples, params, n_mix=None):
    st = np.zeros((params.n_mix, 5), np.float32)
    md = np.zeros(1, np.uint8)
    out = []
    for x in samples:
        fg = oracle.gmm_pixel(x, st, md, params)
        out.append((fg, st[: md[0]].copy()))
    return out


def _close(got: float, want: Fraction) -> bool:
    w = float(want)
    return abs(got - w) <= 4 * np.spacing(np.float32(max(abs(w), 1e-30)))


@pytest.mark.parametrize("k", range(8))
def test_hand_worked_samples(k):
    sc = json.load(open(os.path.join(GOLDEN, "gmm_example.json")))["scenarios"][k]
    res = _run(sc["samples"], _params(sc["params"]))
    for t, ((fg, st), want_fg, want) in enumerate(zip(res, sc["foreground"], sc["states"])):
        assert fg == want_fg, (sc["name"], t)
        assert len(st) == len(want), (sc["name"], t)
        for c, (w, mu, v) in zip(st, want):
            assert _close(c[0], Fraction(w)), (sc["name"], t, c, w)
            for ch in range(3):
                assert _close(c[1 + ch], Fraction(mu[ch])), (sc["name"], t, c, mu)
            assert _close(c[4], Fraction(v)), (sc["name"], t, c, v)


@pytest.mark.parametrize("ct", [0.0, 0.05, 0.4])
def test_constant_pixel_variance_decays_geometrically(ct):
    """A constant sample keeps one component of weight 1, is background from the second
    frame on, and its variance follows var_init (1 - r)^t down to var_min, where
    r = alpha / (1 - alpha c_T) is the owner's rate at its pre-normalisation weight."""
    alpha, vinit, vmin = 0.05, 15.0, 4.0
    p = oracle.gmm_params(n_mix=5, alpha=alpha, var_init=vinit, var_min=vmin,
                          complexity_reduction=ct)
    r = alpha / (1 - alpha * ct)
    res = _run([[77, 140, 12]] * 60, p)
    for t, (fg, st) in enumerate(res):
        assert fg == (t == 0)
        assert len(st) == 1 and st[0][0] == 1.0
        assert tuple(st[0][1:4]) == (77.0, 140.0, 12.0)
        want = max(vinit * (1 - r) ** t, vmin)
        assert st[0][4] == pytest.approx(want, rel=1e-5), t


@pytest.mark.parametrize("alpha,ratio", [(0.05, 0.9), (0.02, 0.7), (0.1, 0.75), (0.01, 0.9),
                                         (0.2, 0.6)])
def test_step_change_switches_at_closed_form_frame(alpha, ratio):
    """Background a, then b from frame T0 on. The new component's weight after j frames is
    1 - (1 - alpha)^j, so b is first background at the smallest j >= 1 with
    (1 - alpha)^j <= ratio (ratio >= 1/2: b is in the background set once the old
    component alone no longer covers the ratio)."""
    j_star = math.ceil(math.log(ratio) / math.log(1 - alpha))
    frac = math.log(ratio) / math.log(1 - alpha)
    assert abs(frac - round(frac)) > 0.01  # not a tie the rounding could flip
    p = oracle.gmm_params(n_mix=3, alpha=alpha, background_ratio=ratio, complexity_reduction=0)
    t0 = 40
    samples = [[30, 30, 30]] * t0 + [[220, 220, 220]] * (j_star + 5)
    fg = [r[0] for r in _run(samples, p)]
    assert fg[0] == 1 and not any(fg[1:t0])
    after = fg[t0:]
    assert after[: j_star] == [1] * j_star
    assert not any(after[j_star:])


def test_owner_mean_and_variance_are_exponential_filters():
    """With one component of weight 1 (every sample owned, c_T = 0) rho = alpha, so the
    mean is the exponentially weighted average of the samples and the variance that of
    the squared innovations |x_t - mu_(t-1)|^2: checked against scipy's IIR filter."""
    rng = np.random.default_rng(3)
    T, alpha, vinit = 400, 0.05, 15.0
    x = (128 + rng.integers(-1, 2, size=(T, 3))).astype(np.float64)
    p = oracle.gmm_params(n_mix=4, alpha=alpha, var_init=vinit, var_min=1e-6, var_max=1e6,
                          var_threshold_gen=1e4, complexity_reduction=0)
    res = _run(x.astype(np.uint8), p)
    assert all(len(st) == 1 for _, st in res)
    mu = np.empty((T, 3))
    mu[0] = x[0]
    for ch in range(3):
        mu[1:, ch], _ = lfilter([alpha], [1, alpha - 1], x[1:, ch], zi=[(1 - alpha) * x[0, ch]])
    d2 = ((x[1:] - mu[:-1]) ** 2).sum(axis=1)
    v = np.empty(T)
    v[0] = vinit
    v[1:], _ = lfilter([alpha], [1, alpha - 1], d2, zi=[(1 - alpha) * vinit])
    got_mu = np.array([st[0][1:4] for _, st in res], dtype=np.float64)
    got_v = np.array([st[0][4] for _, st in res], dtype=np.float64)
    np.testing.assert_allclose(got_mu, mu, atol=2e-3)
    np.testing.assert_allclose(got_v, v, rtol=2e-3, atol=1e-4)


def test_invariants_on_random_sequences():
    rng = np.random.default_rng(11)
    n_px, T = 3000, 60
    for K, alpha, ct in [(5, 0.05, 0.05), (3, 0.2, 0.0), (1, 0.1, 0.0), (8, 0.5, 0.3)]:
        p = oracle.gmm_params(n_mix=K, alpha=alpha, complexity_reduction=ct)
        st, md = oracle.gmm_state(n_px, K)
        modes_of_pixel = rng.integers(0, 256, size=(n_px, 4, 3))
        for t in range(T):
            pick = rng.integers(0, 4, size=n_px)
            frame = np.clip(modes_of_pixel[np.arange(n_px), pick] + rng.normal(0, 3, (n_px, 3)),
                            0, 255).astype(np.uint8)
            mask = oracle.gmm_update(frame, st, md, p)
            assert set(np.unique(mask)) <= {0, 1}
            assert md.min() >= 1 and md.max() <= K
            for i in range(0, n_px, 97):
                c = st[i, : md[i]]
                w = c[:, 0]
                assert (w >= 0).all()
                assert abs(float(w.astype(np.float64).sum()) - 1) < 1e-5 * K
                assert (np.diff(w) <= 0).all()
                assert ((c[:, 4] >= p.var_min) & (c[:, 4] <= p.var_max)).all()
                if ct == 0:  # then rho = alpha / w <= 1: the mean is a convex combination
                    assert ((c[:, 1:4] >= 0) & (c[:, 1:4] <= 255)).all()
        if t == 0:
            assert mask.all()


def test_bad_parameters_are_rejected():
    st, md = oracle.gmm_state(4, 2)
    fr = np.zeros((4, 3), np.uint8)
    for bad in (dict(n_mix=0), dict(n_mix=9), dict(alpha=0.0), dict(alpha=1.5),
                dict(var_min=0.0), dict(var_init=100.0, var_max=75.0),
                dict(complexity_reduction=1.0)):
        kw = dict(n_mix=2)
        kw.update(bad)
        p = oracle.gmm_params(**kw)
        with pytest.raises(ValueError):
            oracle.gmm_update(fr, np.zeros((4, p.n_mix, 5), np.float32) if 0 < p.n_mix <= 8
                              else st, md, p)


# ---- mask -> RoIs ----------------------------------------------------------------

def _scipy_rois(mask, min_area):
    rows, areas = [], []
    eight = np.ones((3, 3), dtype=int)
    for f in range(mask.shape[0]):
        lab, n = ndi.label(mask[f] != 0, structure=eight)
        if n == 0:
            continue
        flat = lab.ravel()
        idx = np.nonzero(flat)[0]
        first = np.full(n + 1, flat.size)
        np.minimum.at(first, flat[idx], idx)
        sizes = np.bincount(flat, minlength=n + 1)
        objs = ndi.find_objects(lab)
        for k in sorted(range(1, n + 1), key=lambda k: first[k]):
            if sizes[k] < min_area:
                continue
            sy, sx = objs[k - 1]
            rows.append((f, sx.start, sy.start, sx.stop - sx.start, sy.stop - sy.start))
            areas.append(sizes[k])
    return np.array(rows, dtype=np.int64).reshape(-1, 5), np.array(areas, dtype=np.int64)


@pytest.mark.parametrize("shape,density,min_area", [((3, 37, 53), 0.1, 1), ((2, 64, 64), 0.3, 1),
                                                    ((2, 41, 70), 0.5, 3), ((1, 90, 33), 0.62, 1),
                                                    ((4, 16, 16), 0.8, 5), ((2, 1, 40), 0.5, 1),
                                                    ((2, 40, 1), 0.5, 2)])
def test_mask_rois_match_scipy_labelling(shape, density, min_area):
    rng = np.random.default_rng(hash((shape, density)) % 2**32)
    mask = (rng.random(shape) < density).astype(np.uint8) * rng.integers(1, 256, shape).astype(np.uint8)
    rows, areas, fb = oracle.mask_rois(mask, min_area)
    want_rows, want_areas = _scipy_rois(mask, min_area)
    np.testing.assert_array_equal(rows, want_rows)
    np.testing.assert_array_equal(areas, want_areas)
    counts = np.bincount(want_rows[:, 0], minlength=shape[0]) if len(want_rows) else np.zeros(shape[0], int)
    np.testing.assert_array_equal(fb, np.concatenate([[0], np.cumsum(counts)]))


def test_mask_rois_hand_drawn():
    """Diagonal contact joins (8-connectivity), a U joins through its base, an island in a
    ring's hole is its own component, and the area threshold drops single pixels."""
    art = [
        "#........#####",
        ".#.......#...#",
        "..#..#.#.#.#.#",
        ".....#.#.#...#",
        ".....###.#####",
        "#.............",
    ]
    mask = np.array([[c == "#" for c in r] for r in art], dtype=np.uint8)[None]
    rows, areas, fb = oracle.mask_rois(mask, 1)
    assert rows.tolist() == [[0, 0, 0, 3, 3], [0, 9, 0, 5, 5], [0, 5, 2, 3, 3], [0, 11, 2, 1, 1],
                             [0, 0, 5, 1, 1]]
    assert areas.tolist() == [3, 16, 7, 1, 1]
    rows, areas, fb = oracle.mask_rois(mask, 2)
    assert rows.tolist() == [[0, 0, 0, 3, 3], [0, 9, 0, 5, 5], [0, 5, 2, 3, 3]]
    assert fb.tolist() == [0, 3]


def test_mask_rois_empty_frames():
    mask = np.zeros((3, 5, 7), np.uint8)
    mask[1, 2, 3] = 1
    rows, areas, fb = oracle.mask_rois(mask, 1)
    assert rows.tolist() == [[1, 3, 2, 1, 1]] and fb.tolist() == [0, 0, 1, 1]
