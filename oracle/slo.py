"""Test infrastructure only: the SLO-aware batching invoker, written out step by step.

Follows Alg. 2 and the text of Sec. III-C (Online SLO-aware Batching Invoker, Latency
Estimator, Patch-stitching Solver): every arrival joins the queue, the deadline of the
queue is its earliest patch deadline, the whole queue is packed afresh (as the algorithm
states), the estimator prices the resulting canvases at mean + 3 standard deviations, and
t_remain = t_DDL - T_slack. Readings where the paper is garbled or silent:
  - a patch violates the SLO when t_remain < t (the text; the pseudo-code's test is
    inverted), and then the previous queue is invoked at t and the patch starts anew;
  - the memory test memory(C) > m_G - tau becomes "more than max_canvases canvases";
  - the queue fires when t >= t_remain: at t_remain between arrivals, at once if already
    due; a firing that falls exactly on an arrival time comes before that arrival;
  - after the last arrival the queue fires at its t_remain;
  - t_DDL is recomputed over the new queue after a violation.
Packing goes through the oracle's own packer; nothing here imports the library.
"""
from __future__ import annotations

import numpy as np

from . import pack as _pack

DEADLINE, SLO, MEMORY = 0, 1, 2


def latency_estimator(n_canvases, lat_mean, lat_std):
    """T_slack = mu + 3 sigma of a batch of n_canvases canvases (Sec. III-C)."""
    return lat_mean[n_canvases - 1] + 3 * lat_std[n_canvases - 1]


def stitching_solver(queue, w, h, canvas_w, canvas_h, policy):
    """Packs the queued patches in queue order (Alg. 2's Patch-stitching Solver); the
    patches need no frame, so each is given as a rectangle of a canvas-sized frame."""
    rois = np.array([[0, 0, 0, w[i], h[i]] for i in queue], dtype=np.int32).reshape(-1, 5)
    rc, bad, plan = _pack(rois, canvas_w, canvas_h, canvas_w, canvas_h, 1, policy)
    if rc != 0:
        raise ValueError(f"patch {queue[bad]} cannot be packed (code {rc})")
    return plan


def replay(w, h, t_arrive, t_ddl, canvas_w, canvas_h, policy, max_canvases, lat_mean, lat_std):
    """Returns the invocations in firing order; each is a dict with t_fire, t_ddl, t_slack,
    patches (ids in queue order), n_canvases, reason and place ({id: (canvas, x, y)})."""
    invocations = []

    def invoke(queue, plan, t_fire, t_ddl_q, reason):
        invocations.append({
            "t_fire": t_fire, "t_ddl": t_ddl_q,
            "t_slack": latency_estimator(plan.n_canvases, lat_mean, lat_std),
            "patches": list(queue), "n_canvases": plan.n_canvases, "reason": reason,
            "place": {p: tuple(int(v) for v in plan.place[k]) for k, p in enumerate(queue)}})

    queue, plan, t_DDL, t_remain = [], None, None, None
    for i in range(len(w)):
        t = t_arrive[i]
        if queue and t >= t_remain:  # the clock reached t_remain before this arrival
            invoke(queue, plan, t_remain, t_DDL, DEADLINE)
            queue, plan = [], None
        old_queue, old_plan, old_DDL = queue, plan, t_DDL
        queue = queue + [i]
        t_DDL = min(t_ddl[j] for j in queue)
        plan = stitching_solver(queue, w, h, canvas_w, canvas_h, policy)
        too_big = plan.n_canvases > max_canvases
        if not too_big:
            t_rem = t_DDL - latency_estimator(plan.n_canvases, lat_mean, lat_std)
        if old_queue and (too_big or t_rem < t):
            invoke(old_queue, old_plan, t, old_DDL, MEMORY if too_big else SLO)
            queue = [i]
            t_DDL = t_ddl[i]
            plan = stitching_solver(queue, w, h, canvas_w, canvas_h, policy)
            t_rem = t_DDL - latency_estimator(plan.n_canvases, lat_mean, lat_std)
        t_remain = t_rem
        if t >= t_remain:  # already due
            invoke(queue, plan, t, t_DDL, DEADLINE)
            queue, plan = [], None
    if queue:
        invoke(queue, plan, t_remain, t_DDL, DEADLINE)
    return invocations
