"""Pins against the numbers the paper prints (tests/golden/paper_printed_values.txt): the Sec. 3 work
example through the work model, and the Sec. 3.1 pyramid facts through the oracle's plan of the
25-scale, 10-per-octave pyramid of a 768 x 1024 image stitched onto 1200 x 1200 planes."""
import os

import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import workmodel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_printed_values.txt")


def load():
    vals = {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = (x.strip() for x in line.split("=", 1))
            vals[k] = [int(x) for x in v.split(",")] if "," in v else int(v)
    return vals


G = load()


def test_sec3_example():
    N, M, s = G["sec3_N"], G["sec3_M"], G["sec3_stride"]
    assert workmodel.region_count(N, M, s) == G["sec3_regions"]
    assert workmodel.dense_speedup(N, M, s) == G["sec3_dense_ops_ratio"]


@pytest.fixture(scope="module")
def plan25():
    w = C.XGA_25SCALE
    return w, oracle.plan(w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side,
                          w.pad, w.plane_h, w.plane_w)


def test_sec31_pyramid_shape(plan25):
    w, p = plan25
    assert w.steps_per_octave in G["sec31_scales_per_octave"]
    lo, hi = G["sec31_levels"]
    assert lo <= w.n_scales <= hi
    assert w.pad == G["sec31_border_px"]
    assert w.plane_h in G["sec31_plane_sides"] and w.plane_w in G["sec31_plane_sides"]
    ratio = float(np.sum(p.field("h").astype(np.int64) * p.field("w"))) / (w.H * w.W)
    lo, hi = G["sec31_pixel_ratio"]
    assert lo <= ratio <= hi, ratio


def test_sec31_gap_between_stitched_images(plan25):
    """Real pixels of two different scales on one plane are at least 32 px apart along some axis."""
    w, p = plan25
    pad = w.pad
    real = []
    for k in range(w.n_scales):
        y, x, h, wd = (int(p.field(f)[k]) for f in ("y", "x", "h", "w"))
        real.append((int(p.field("plane")[k]), y + pad, x + pad, y + pad + h, x + pad + wd))
    for i in range(len(real)):
        for j in range(i + 1, len(real)):
            a, b = real[i], real[j]
            if a[0] != b[0]:
                continue
            gap_y = max(b[1] - a[3], a[1] - b[3])
            gap_x = max(b[2] - a[4], a[2] - b[4])
            assert max(gap_y, gap_x) >= G["sec31_min_gap_px"], (i, j, gap_y, gap_x)
