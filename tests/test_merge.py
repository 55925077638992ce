"""Per-frame merge after unstitch: the oracle pinned by a hand-worked example, exact
rational overlap tests, an independently formulated greedy, and closed forms; argument
checks of tg_merge that fail before any GPU work. GPU parity is in test_merge_gpu.py."""
from fractions import Fraction

import numpy as np
import pytest

from conftest import load_golden
from paper_2404_09267_amd import tg


def golden_inputs():
    g = load_golden("merge_example.json")
    dets = np.zeros(len(g["dets"]), dtype=tg.DET_DTYPE)
    for k, row in enumerate(g["dets"]):
        dets[k] = tuple(row)
    scores = np.array([float(s) for s in g["scores"]], dtype=np.float32)
    return g, dets, scores


@pytest.mark.parametrize("cross_only,key", [(True, "keep_cross_only"), (False, "keep_all_pairs")])
def test_oracle_golden(cross_only, key):
    from oracle import merge

    g, dets, scores = golden_inputs()
    keep, kept = merge.merge(dets, scores, g["n_frames"], g["threshold"], cross_only)
    assert keep.astype(int).tolist() == g[key]
    assert kept["box"].tolist() == [d[0] for d, k in zip(g["dets"], g[key]) if k]


def test_overlap_test_is_exact_on_small_integers():
    """With integer corners below 2^10 and dyadic thresholds every binary32 operation is
    exact, so the decision must equal the rational one."""
    from oracle import merge

    rng = np.random.default_rng(11)
    for _ in range(3000):
        a = np.sort(rng.integers(0, 1000, (2, 2)), axis=0).T.reshape(-1)[[0, 2, 1, 3]]
        b = np.sort(rng.integers(0, 1000, (2, 2)), axis=0).T.reshape(-1)[[0, 2, 1, 3]]
        if rng.random() < 0.3:  # force overlaps
            b = a + rng.integers(-30, 30, 4)
        thr = Fraction(int(rng.integers(1, 16)), 16)
        w = max(0, min(a[2], b[2]) - max(a[0], b[0]))
        h = max(0, min(a[3], b[3]) - max(a[1], b[1]))
        area = lambda r: max(0, r[2] - r[0]) * max(0, r[3] - r[1])
        inter = w * h
        union = area(a) + area(b) - inter
        want = Fraction(inter) > thr * union
        got = merge.suppresses(tuple(np.float32(v) for v in a), tuple(np.float32(v) for v in b),
                               float(thr))
        assert got == want, (a, b, thr)


def test_vectorised_overlap_equals_scalar():
    """suppressed_by_any (the merge's test against a whole kept list) equals any() of the
    scalar suppresses over the same rows, on boxes mixing ordinary corners with NaN,
    infinities, signed zeros, empty and inverted boxes and huge values, for thresholds of
    both signs and with and without the patch mask."""
    from oracle import merge

    rng = np.random.default_rng(21)
    special = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, 1e38, -1e38, 3.0, 3.0000002],
                       np.float32)

    def boxes(k):
        x = rng.uniform(-50, 150, (k, 4)).astype(np.float32)
        x[:, 2:] = x[:, :2] + rng.uniform(-5, 60, (k, 2)).astype(np.float32)
        odd = rng.random((k, 4)) < 0.08
        x[odd] = rng.choice(special, odd.sum())
        return x

    for trial in range(400):
        K = int(rng.integers(0, 12))
        kept = boxes(K)
        b = boxes(1)[0]
        thr = float(rng.choice([0.5, 0.0, -0.0, -0.5, 1.0, 0.1, 2.0]))
        roi = rng.integers(0, 3, K)
        rb = int(rng.integers(0, 3))
        bt = tuple(np.float32(v) for v in b)
        rows = [tuple(np.float32(v) for v in r) for r in kept]
        want_all = any(merge.suppresses(r, bt, thr) for r in rows)
        want_cross = any(merge.suppresses(r, bt, thr) for r, q in zip(rows, roi) if q != rb)
        assert merge.suppressed_by_any(kept, b, thr) == want_all, (kept, b, thr)
        assert merge.suppressed_by_any(kept, b, thr, roi, rb) == want_cross, (kept, b, thr)


def other_greedy(dets, scores, n_frames, thr, cross_only):
    """The same greedy, written as 'take the best remaining, drop what it overlaps'."""
    from oracle.merge import suppresses

    keep = np.zeros(len(dets), bool)
    for f in range(n_frames):
        left = [k for k in range(len(dets)) if dets[k]["frame"] == f]
        score = lambda k: (-np.inf if np.isnan(scores[dets[k]["box"]]) else scores[dets[k]["box"]])
        while left:
            best = max(left, key=lambda k: (score(k), -int(dets[k]["box"])))
            keep[best] = True
            bb = tuple(np.float32(dets[best][c]) for c in ("x1", "y1", "x2", "y2"))
            left = [k for k in left if k != best and not (
                (not cross_only or dets[k]["roi"] != dets[best]["roi"]) and
                suppresses(bb, tuple(np.float32(dets[k][c]) for c in ("x1", "y1", "x2", "y2")), thr))]
    return keep


def random_dets(rng, n, n_frames, n_rois, span=200.0):
    dets = np.zeros(n, dtype=tg.DET_DTYPE)
    dets["box"] = rng.permutation(n)
    dets["roi"] = rng.integers(0, n_rois, n)
    dets["frame"] = rng.integers(0, n_frames, n)
    x1 = rng.uniform(0, span, n).astype(np.float32)
    y1 = rng.uniform(0, span, n).astype(np.float32)
    dets["x1"], dets["y1"] = x1, y1
    dets["x2"] = x1 + rng.uniform(5, 60, n).astype(np.float32)
    dets["y2"] = y1 + rng.uniform(5, 60, n).astype(np.float32)
    scores = np.round(rng.uniform(0, 1, n), 1).astype(np.float32)  # many ties
    scores[rng.random(n) < 0.05] = np.nan
    return dets, scores


@pytest.mark.parametrize("cross_only,thr", [(True, 0.5), (False, 0.3), (True, 0.0)])
def test_oracle_against_other_greedy(cross_only, thr):
    from oracle import merge

    rng = np.random.default_rng(int(thr * 10) + cross_only)
    for _ in range(5):
        dets, scores = random_dets(rng, 150, 3, 6)
        keep, _ = merge.merge(dets, scores, 3, thr, cross_only)
        assert (keep == other_greedy(dets, scores, 3, thr, cross_only)).all()


def test_oracle_closed_forms():
    from oracle import merge

    rng = np.random.default_rng(3)
    dets, scores = random_dets(rng, 200, 4, 5)
    keep, _ = merge.merge(dets, scores, 4, 1.0, True)
    assert keep.all()  # inter > union never holds
    keep, _ = merge.merge(dets, scores, 4, -1.0, False)
    for f in range(4):  # every pair suppresses: one detection per frame, the top-ranked
        idx = np.nonzero(dets["frame"] == f)[0]
        s = np.where(np.isnan(scores[dets["box"][idx]]), -np.inf, scores[dets["box"][idx]])
        top = idx[np.lexsort((dets["box"][idx], -s))[0]]
        assert keep[idx].sum() == 1 and keep[top]
    keep, _ = merge.merge(dets, scores, 2, 0.5, True)
    assert not keep[dets["frame"] >= 2].any()  # frames outside [0, n_frames)


def test_cyclic_pair_schedule_covers_each_pair_once():
    """The LDS path of frames up to 256 detections tests each unordered pair once: thread i
    takes the detections 1 .. last(i) places after it, cyclically, where last(i) is n/2 for
    even n and i < n/2, else (n - 1)/2. Every pair of distinct detections must come up
    exactly once, for every frame size."""
    for n in range(1, 258):
        seen = {}
        for i in range(n):
            last = n // 2 if (n % 2 == 0 and i < n // 2) else (n - 1) // 2
            for d in range(1, last + 1):
                j = i + d
                j = j - n if j >= n else j
                assert j != i and 0 <= j < n
                key = (min(i, j), max(i, j))
                seen[key] = seen.get(key, 0) + 1
        assert len(seen) == n * (n - 1) // 2 and set(seen.values()) <= {1}, n


def test_merge_argument_checks():
    L = tg.lib()
    a = tg.MergeArgs()
    a.dets, a.n_dets, a.scores, a.keep, a.out = 0x1000, 0x2000, 0x3000, 0x4000, 0x5000
    a.n_kept, a.workspace = 0x6000, 0x8000
    a.n_max, a.n_scores, a.n_frames, a.iou_threshold, a.cross_only = 100, 100, 4, 0.5, 1
    a.workspace_bytes = L.tg_merge_workspace_bytes(100, 4)

    def call(**kw):
        b = tg.MergeArgs.from_buffer_copy(a)
        for k, v in kw.items():
            setattr(b, k, v)
        return L.tg_merge(tg.ctypes.byref(b), None)

    assert L.tg_merge(None, None) == tg.E_INVAL
    assert call(n_max=-1) == tg.E_INVAL
    assert call(n_frames=-1) == tg.E_INVAL
    assert call(iou_threshold=float("nan")) == tg.E_INVAL
    assert call(n_kept=None) == tg.E_INVAL
    assert call(dets=None) == tg.E_INVAL
    assert call(n_dets=None) == tg.E_INVAL
    assert call(scores=None) == tg.E_INVAL
    assert call(workspace=None) == tg.E_WORKSPACE
    assert call(workspace_bytes=a.workspace_bytes - 1) == tg.E_WORKSPACE
    assert call(workspace=0x8008) == tg.E_WORKSPACE  # not 16-byte aligned
    assert L.tg_merge_workspace_bytes(0, 4) == 0
    # ticket and status, the overflow cursor, the large-frame flag, one look-back word
    # (32), counts and cursors one 256-byte slot apart (3 + 3 slots of 64 int32), starts
    # (4 int32), grouped ids (4 n); then, 16-byte aligned, per detection its box (16),
    # ranking key (8), patch id, cell range and state (4 each), its lists to
    # search (5 starts and 5 sizes: 40), 16 suppressors in place, their count and the
    # start of a longer list (72), and 16 entries of the overflow area (64); then, 16-byte
    # aligned, the cell lists (4 n entries of a box and an int4: 32 bytes)
    n = 1024
    small = 8 * 4 + 4 * (64 * (3 + 3) + 4) + 4 * n
    per_det = 16 + 8 + 4 + 4 + 4 + 40 + 72 + 64
    assert L.tg_merge_workspace_bytes(n, 3) == \
        ((small + 15) // 16 * 16 + per_det * n + 15) // 16 * 16 + 4 * 32 * n
    # past 16,384 frames the counters are packed, one int32 each
    packed = 8 * 4 + 4 * (2 * 20000 + 20001) + 4 * n
    assert L.tg_merge_workspace_bytes(n, 20000) == \
        ((packed + 15) // 16 * 16 + per_det * n + 15) // 16 * 16 + 4 * 32 * n
    padded = 8 * 4 + 4 * (64 * 2 * 16384 + 16385) + 4 * n
    assert L.tg_merge_workspace_bytes(n, 16384) == \
        ((padded + 15) // 16 * 16 + per_det * n + 15) // 16 * 16 + 4 * 32 * n
