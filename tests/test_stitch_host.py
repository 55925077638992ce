"""Host side of tg_stitch's launch: unit geometry (tg_stitch_units) and which exact
normalisation path a mean/std takes (tg_stitch_norm_uses_table). No GPU needed."""
import ctypes
import math

import numpy as np
import pytest

from paper_2404_09267_amd import tg
from paper_2404_09267_amd import workload as W

from stitch_geometry import geometry


@pytest.mark.parametrize("cw,ch,count", [(1280, 1280, 32), (1280, 1280, 31), (1024, 1024, 9),
                                         (640, 640, 53), (1024, 1024, 1), (1920, 1080, 5),
                                         (1, 1, 1), (2561, 7, 3), (64, 50000, 1), (45, 91, 7)])
def test_unit_count_matches_geometry(cw, ch, count):
    assert tg.stitch_units(cw, ch, count) == geometry(cw, ch, count)[1]


def test_unit_count_edges():
    assert tg.stitch_units(1280, 1280, 0) == 0
    for bad in [(0, 10, 1), (10, 0, 1), (10, 10, -1), (65536, 65536, 4096)]:  # last: > 2^31 - 1 units
        assert tg.lib().tg_stitch_units(*bad) == tg.E_INVAL
    # the largest launch: 2^31 - 1 units at most
    assert tg.stitch_units(2048, 1, 2 ** 31 - 1) == 2 ** 31 - 1


# Triples for which no fp32 (a, c) reproduces every correctly rounded byte exactly
# (found by a search over random mean/std); ImageNet's statistics have such pairs.
TABLE_CASES = [((174.00369262695312, 189.9988250732422, 150.99696350097656),
                (0.031708136200904846, 1.5641870498657227, 1.5637657642364502))]


def test_norm_path_selection():
    assert tg.stitch_norm_uses_table(W.MEAN, W.STD) is False
    assert tg.stitch_norm_uses_table((0, 0, 0), (255, 255, 255)) is False
    assert tg.stitch_norm_uses_table((10.5, 300.0, -7.25), (0.01, 1000.0, 3.5)) is False
    for mean, std in TABLE_CASES:
        assert tg.stitch_norm_uses_table(mean, std) is True
    for mean, std in [((0, 0, 0), (1, 0, 1)), ((0, float("nan"), 0), (1, 1, 1)),
                      ((0, 0, 0), (1, 1, float("inf")))]:
        with pytest.raises(tg.TgError):
            tg.stitch_norm_uses_table(mean, std)
    f3 = ctypes.c_float * 3
    assert tg.lib().tg_stitch_norm_uses_table(None, f3(1, 1, 1)) == tg.E_INVAL
