"""SLO-aware batching invoker (Alg. 2, Sec. III-C): the oracle pinned by hand-worked
traces and closed forms, then the library (incremental packing, tg_slo_replay) against
the oracle (full re-solve on every arrival) on random traces. Host only."""
import math

import numpy as np
import pytest

from conftest import load_golden
from paper_2404_09267_amd import tg

GUILLOTINE, ARRIVAL = 2, 1


def lib_invocations(r: tg.SloReplay):
    out = []
    for v in r.invocations:
        ids = r.order[v["first"]: v["first"] + v["count"]].tolist()
        out.append({"t_fire": float(v["t_fire"]), "t_ddl": float(v["t_ddl"]),
                    "t_slack": float(v["t_slack"]), "patches": ids,
                    "n_canvases": int(v["n_canvases"]), "reason": int(v["reason"]),
                    "place": {p: tuple(int(x) for x in r.place[p]) for p in ids}})
    return out


def run_lib(pt, cw, ch, policy, cap, mean, std):
    return lib_invocations(tg.slo_replay(pt, cw, ch, policy, cap, mean, std))


def run_oracle(pt, cw, ch, policy, cap, mean, std):
    from oracle import slo

    return slo.replay(pt["w"].tolist(), pt["h"].tolist(), pt["t_arrive"].tolist(),
                      pt["t_ddl"].tolist(), cw, ch, policy, cap, list(mean), list(std))


def assert_matches_golden(got, case):
    want = case["invocations"]
    assert len(got) == len(want)
    for g, w in zip(got, want):
        assert g["patches"] == w["patches"]
        assert g["reason"] == w["reason"] and g["n_canvases"] == w["n_canvases"]
        for k in ("t_fire", "t_ddl", "t_slack"):
            assert math.isclose(g[k], w[k], rel_tol=1e-12, abs_tol=1e-12), (k, g[k], w[k])
        for p in g["patches"]:
            assert list(g["place"][p]) == case["place"][p]


def golden_patches(case):
    a = np.array(case["patches"], dtype=np.float64)
    return tg.slo_patches(a[:, 0].astype(int), a[:, 1].astype(int), a[:, 2], a[:, 3])


@pytest.mark.parametrize("case", load_golden("slo_examples.json")["traces"],
                         ids=lambda c: c["name"])
def test_oracle_golden(orc, case):
    got = run_oracle(golden_patches(case), *case["canvas"], case["policy"],
                     case["max_canvases"], case["lat_mean"], case["lat_std"])
    assert_matches_golden(got, case)


@pytest.mark.parametrize("case", load_golden("slo_examples.json")["traces"],
                         ids=lambda c: c["name"])
def test_library_golden(case):
    got = run_lib(golden_patches(case), *case["canvas"], case["policy"], case["max_canvases"],
                  case["lat_mean"], case["lat_std"])
    assert_matches_golden(got, case)


def random_trace(rng, n, cw, ch, lo, hi, slo, spread=1.0, ties=False):
    w = rng.integers(lo, min(hi, cw) + 1, n)
    h = rng.integers(lo, min(hi, ch) + 1, n)
    t = np.sort(rng.uniform(0, spread * n, n))
    if ties:
        t = np.floor(t)  # many equal arrival times
    ddl = t + rng.uniform(0.2, 1.0, n) * slo
    return tg.slo_patches(w, h, t, ddl)


@pytest.mark.parametrize("policy", [GUILLOTINE, ARRIVAL])
def test_oracle_closed_form_far_deadlines(orc, policy):
    """With deadlines out of reach only the memory cap splits the queue, so invocation k
    holds canvases [k*cap, (k+1)*cap) of one packing of the whole trace in arrival order,
    with the same positions."""
    rng = np.random.default_rng(3 + policy)
    n, cw, cap = 300, 128, 3
    pt = random_trace(rng, n, cw, cw, 8, 80, slo=1.0)
    pt["t_ddl"] = 1e9
    got = run_oracle(pt, cw, cw, policy, cap, [1.0] * cap, [0.1] * cap)
    rois = np.stack([np.zeros(n), np.zeros(n), np.zeros(n), pt["w"], pt["h"]], 1).astype(np.int32)
    rc, _, plan = orc.pack(rois, cw, cw, cw, cw, 1, policy)
    assert rc == 0
    J = plan.n_canvases
    assert len(got) == -(-J // cap)
    for k, v in enumerate(got):
        first, count = k * cap, min(cap, J - k * cap)
        want_ids = plan.order[plan.canvas_begin[first]:plan.canvas_begin[first + count]].tolist()
        assert v["patches"] == want_ids
        assert v["n_canvases"] == count
        assert v["reason"] == (2 if k < len(got) - 1 else 0)
        for p in want_ids:
            c, x, y = plan.place[p]
            assert v["place"][p] == (c - first, x, y)


def test_oracle_closed_form_no_slack(orc):
    """Zero latency and deadlines equal to arrival times: every patch is due the moment it
    arrives, so each is invoked alone at its arrival time."""
    rng = np.random.default_rng(9)
    pt = random_trace(rng, 50, 64, 64, 4, 30, slo=1.0)
    pt["t_ddl"] = pt["t_arrive"]
    got = run_oracle(pt, 64, 64, GUILLOTINE, 2, [0.0, 0.0], [0.0, 0.0])
    assert [v["patches"] for v in got] == [[i] for i in range(50)]
    assert [v["t_fire"] for v in got] == pt["t_arrive"].tolist()


def check_invariants(orc, got, pt, cw, ch, policy, cap, mean, std):
    ids = [p for v in got for p in v["patches"]]
    assert ids == list(range(len(pt))), "every patch once, in arrival order"
    for k, v in enumerate(got):
        last = v["patches"][-1]
        assert v["t_fire"] >= pt["t_arrive"][last]
        if k + 1 < len(got):
            assert v["t_fire"] <= pt["t_arrive"][got[k + 1]["patches"][0]]
        assert v["t_ddl"] == min(pt["t_ddl"][p] for p in v["patches"])
        assert v["t_slack"] == mean[v["n_canvases"] - 1] + 3 * std[v["n_canvases"] - 1]
        assert 1 <= v["n_canvases"] <= cap
        if v["reason"] == 0:
            assert v["t_fire"] == max(v["t_ddl"] - v["t_slack"], pt["t_arrive"][last])
        else:  # fired when the next patch arrived
            assert v["t_fire"] == pt["t_arrive"][got[k + 1]["patches"][0]]
        # the invocation's placement is a valid plan of its patches
        pp = v["patches"]
        rois = np.stack([np.zeros(len(pp)), np.zeros(len(pp)), np.zeros(len(pp)),
                         pt["w"][pp], pt["h"][pp]], 1).astype(np.int32)
        place = np.array([v["place"][p] for p in pp], dtype=np.int32)
        order = np.arange(len(pp), dtype=np.int32)
        cbeg = np.searchsorted(place[:, 0], np.arange(v["n_canvases"] + 1)).astype(np.int32)
        assert orc.check_plan(rois, cw, ch, policy, place, order, cbeg, v["n_canvases"]) == 0


@pytest.mark.parametrize("seed,policy,cap,ties", [(0, GUILLOTINE, 4, False),
                                                  (1, ARRIVAL, 2, False),
                                                  (2, GUILLOTINE, 1, True),
                                                  (3, ARRIVAL, 6, True)])
def test_oracle_invariants_and_library_parity(orc, seed, policy, cap, ties):
    rng = np.random.default_rng(100 + seed)
    cw = ch = 96
    mean = np.linspace(0.5, 2.0, cap)
    std = np.linspace(0.05, 0.3, cap)
    pt = random_trace(rng, 400, cw, ch, 4, 60, slo=8.0, spread=0.05, ties=ties)
    want = run_oracle(pt, cw, ch, policy, cap, mean, std)
    check_invariants(orc, want, pt, cw, ch, policy, cap, mean, std)
    assert {v["reason"] for v in want} >= {0}
    got = run_lib(pt, cw, ch, policy, cap, mean, std)
    assert got == want  # same invocations, times, placements (exact)


def camera_trace():
    """cam20_4k's patches from 20 cameras at 30 fps, sent twice 0.3 s apart: the first
    round with a 0.5 s SLO (the memory cap splits it), the second with 0.25 s (SLO
    violations split it)."""
    from paper_2404_09267_amd import workload as W

    wl = W.WORKLOADS["cam20_4k"]
    w, h, t, ddl, mean, std = W.camera_arrival_trace(wl)
    return tg.slo_patches(w, h, t, ddl), wl.canvas, len(mean), mean, std


def test_library_parity_on_a_camera_trace(orc):
    pt, canvas, cap, mean, std = camera_trace()
    got = run_lib(pt, canvas, canvas, GUILLOTINE, cap, mean, std)
    want = run_oracle(pt, canvas, canvas, GUILLOTINE, cap, mean, std)
    assert got == want
    assert {v["reason"] for v in want} == {0, 1, 2}
    check_invariants(orc, want, pt, canvas, canvas, GUILLOTINE, cap, mean, std)


def test_replay_errors():
    pt = tg.slo_patches([4, 4], [4, 4], [0.0, 1.0], [5.0, 5.0])
    ok = dict(canvas_w=8, canvas_h=8, policy=GUILLOTINE, max_canvases=2, lat_mean=[1, 1],
              lat_std=[0, 0])
    assert len(tg.slo_replay(pt, **ok).invocations) == 1
    assert len(tg.slo_replay(pt[:0], **ok).invocations) == 0

    def code(patches, **kw):
        args = dict(ok)
        args.update(kw)
        with pytest.raises(tg.TgError) as e:
            tg.slo_replay(patches, **args)
        return e.value.code, e.value.bad_index

    assert code(pt, policy=0) == (tg.E_INVAL, -1)          # FFDH reorders the queue
    assert code(pt, max_canvases=3) == (tg.E_INVAL, -1)    # table shorter than the cap
    assert code(pt, max_canvases=0) == (tg.E_INVAL, -1)
    assert code(pt, lat_mean=[1, float("nan")]) == (tg.E_INVAL, -1)
    late = pt.copy()
    late["t_arrive"] = [1.0, 0.5]
    assert code(late) == (tg.E_INVAL, 1)                   # arrivals out of order
    big = pt.copy()
    big["w"][1] = 9
    assert code(big) == (tg.E_ROI_TOO_LARGE, 1)
    bad = pt.copy()
    bad["t_ddl"][0] = float("inf")
    assert code(bad) == (tg.E_INVAL, 0)
    zero = pt.copy()
    zero["h"][0] = 0
    assert code(zero) == (tg.E_INVAL, 0)
    L = tg.lib()
    n_inv = np.zeros(1, np.int32)
    badi = np.zeros(1, np.int32)
    p = tg.SloParams(8, 8, GUILLOTINE, 2, 2, None, None)
    assert L.tg_slo_replay(None, 0, tg.ctypes.byref(p), None, None, None, n_inv.ctypes.data,
                           badi.ctypes.data) == tg.E_INVAL  # null table
