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
