"""tg_stitch's unit geometry restated from its definition (test infrastructure): each
canvas plane cut in raster order into runs of 6144 pixels, one unit per run."""
import math

RUN = 6144


def geometry(cw, ch, count):
    """(runs per canvas, units) of a launch over `count` canvases of cw x ch."""
    runs = math.ceil(cw * ch / RUN)
    return runs, runs * count


def unit_pixels(cw, ch, count, u):
    """Canvas (local index) and the raster pixel range [p0, p1) of unit u."""
    runs, _ = geometry(cw, ch, count)
    c, r = divmod(u, runs)
    return c, r * RUN, min((r + 1) * RUN, cw * ch)


def records_per_unit(rois, plan, first, count, cw, ch):
    """Patches of each unit of a launch: those with at least one pixel in the unit's run."""
    runs, n_units = geometry(cw, ch, count)
    rec = [0] * n_units
    for c in range(count):
        j = first + c
        for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]:
            _, x, y = (int(v) for v in plan.place[i])
            w, h = int(rois[i, 3]), int(rois[i, 4])
            hit = set()
            for yy in range(y, y + h):
                a, b = yy * cw + x, yy * cw + x + w - 1
                hit.update(range(a // RUN, b // RUN + 1))
            for r in hit:
                rec[c * runs + r] += 1
    return rec
