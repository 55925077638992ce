"""tg_stitch's unit geometry restated from its definition (test infrastructure): tiles of
at most 1280 columns, bands of whole 3-row steps, about 6144 units per launch, at most
1024 steps per band."""
import math

TILE_W, STEP_ROWS, UNIT_TARGET, MAX_STEPS = 1280, 3, 6144, 1024


def geometry(cw, ch, count):
    """(tiles across, rows per band, bands down, units) of a launch over `count`
    canvases of cw x ch."""
    tiles = math.ceil(cw / TILE_W)
    steps = math.ceil(ch / STEP_ROWS)
    band_steps = min(max(math.ceil(steps * tiles * count / UNIT_TARGET), 1), MAX_STEPS)
    bands = math.ceil(steps / band_steps)
    return tiles, band_steps * STEP_ROWS, bands, bands * tiles * count


def records_per_unit(rois, plan, first, count, cw, ch):
    """Patches of each unit of a launch: those whose placed rectangle meets the unit's
    band of rows and tile of columns."""
    tiles, band_rows, bands, n_units = geometry(cw, ch, count)
    rec = [0] * n_units
    for c in range(count):
        j = first + c
        for i in plan.order[plan.canvas_begin[j]:plan.canvas_begin[j + 1]]:
            _, x, y = (int(v) for v in plan.place[i])
            w, h = int(rois[i, 3]), int(rois[i, 4])
            for b in range(y // band_rows, (y + h - 1) // band_rows + 1):
                for t in range(x // TILE_W, (x + w - 1) // TILE_W + 1):
                    rec[(c * bands + b) * tiles + t] += 1
    return rec
