"""Pins of the oracle's aspect-ratio pyramids (Sec. 3.3: warp the image to each aspect ratio and build a
whole pyramid per ratio, all stitched together): ratio 1 is the plain pyramid, exact warped sizes,
area preservation, stitching invariants over all entries, per-entry planes equal the plain resize,
and region windows read each box where it is closest to a T x T square."""
import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import synth

MEAN = synth.IMAGENET_MEAN


def test_ratio_one_is_the_plain_pyramid():
    a = oracle.plan(768, 1024, 25, 10, 1.0, 0, 16, 1200, 1200)
    b = oracle.plan(768, 1024, 25, 10, 1.0, 0, 16, 1200, 1200, aspects=[1.0])
    np.testing.assert_array_equal(a.gi, b.gi)
    np.testing.assert_array_equal(a.gd, b.gd)
    assert a.plane_sizes == b.plane_sizes


def test_exact_warped_sizes_and_aspect_field():
    p = oracle.plan(64, 64, 2, 1, 1.0, 0, 0, 0, 0, aspects=[4.0, 0.25, 1.0])
    h, w, asp = p.field("h"), p.field("w"), p.field("aspect")
    # entry a*K + k: ratio 4 halves the height and doubles the width (area kept), ratio 1/4 the reverse
    np.testing.assert_array_equal(h, [32, 16, 128, 64, 64, 32])
    np.testing.assert_array_equal(w, [128, 64, 32, 16, 64, 32])
    np.testing.assert_array_equal(asp, [0, 0, 1, 1, 2, 2])
    np.testing.assert_array_equal(p.field("k"), np.arange(6))


def test_area_is_kept_across_ratios():
    H, W, K = 480, 640, 8
    r = [1 / 3, 0.5, 1.0, 2.0, 3.0]
    p = oracle.plan(H, W, K, 4, 1.0, 0, 16, 1200, 1200, aspects=r)
    h, w = p.field("h").astype(np.float64), p.field("w").astype(np.float64)
    for a in range(len(r)):
        for k in range(K):
            s = p.gd[a * K + k, 0]
            e = a * K + k
            assert abs(h[e] * w[e] - H * W * s * s) <= (h[e] + w[e] + 1) * 0.5 + 1e-9
            assert abs(np.log((w[e] / h[e]) / (W / H * r[a]))) < 0.02


def test_stitching_invariants_over_all_entries():
    K, r = 12, [0.5, 1.0, 2.0]
    p = oracle.plan(480, 640, K, 4, 1.0, 0, 16, 1200, 1200, aspects=r)
    E = K * len(r)
    assert p.gi.shape[0] == E
    y, x, rh, rw, pl = (p.field(f) for f in ("y", "x", "rh", "rw", "plane"))
    assert (y % 16 == 0).all() and (x % 16 == 0).all() and (rh % 16 == 0).all() and (rw % 16 == 0).all()
    assert (y + rh <= 1200).all() and (x + rw <= 1200).all()
    for i in range(E):
        for j in range(i + 1, E):
            if pl[i] == pl[j]:
                assert y[i] + rh[i] <= y[j] or y[j] + rh[j] <= y[i] or x[i] + rw[i] <= x[j] or \
                    x[j] + rw[j] <= x[i]
    assert p.n_planes >= int(np.ceil((rh.astype(np.int64) * rw).sum() / 1200 ** 2))


def test_entry_planes_equal_the_plain_resize():
    H, W, pad = 90, 120, 16
    img = synth.image(41, H, W)
    p = oracle.plan(H, W, 3, 2, 1.0, 0, pad, 400, 400, aspects=[0.5, 2.0])
    planes = oracle.build_planes(img, p, 1, MEAN)
    for e in range(p.gi.shape[0]):
        h, w, pl, y, x = (int(p.field(f)[e]) for f in ("h", "w", "plane", "y", "x"))
        got = planes[pl][:, y + pad:y + pad + h, x + pad:x + pad + w]
        np.testing.assert_array_equal(got, oracle.resize_center(img, h, w, MEAN))


def test_regions_pick_the_aspect_that_squares_the_box():
    H, W, K = 600, 800, 10
    r = [0.5, 1.0, 2.0]
    p = oracle.plan(H, W, K, 4, 1.0, 0, 16, 1200, 1200, aspects=r)
    maps = [np.zeros((256, oracle.conv5_side(h), oracle.conv5_side(w)), np.float32)
            for h, w in p.plane_sizes]
    boxes = np.array([[50, 100, 650, 400],     # wide 2:1 -> ratio 1/2 squares it
                      [200, 30, 470, 570],     # tall 1:2 -> ratio 2
                      [100, 100, 400, 400]],   # square -> ratio 1
                     np.float32)
    _, scale, _, _ = oracle.region_windows(maps, p, boxes)
    asp = p.field("aspect")[scale]
    np.testing.assert_array_equal(asp, [0, 2, 1])
    # and the chosen entry brings the box area within half a scale step (2^-1/4 per step) of T^2
    for b, e in zip(boxes, scale):
        a = (p.gd[e, 1] * (b[3] - b[1])) * (p.gd[e, 2] * (b[2] - b[0]))
        assert abs(np.log2(a / 227.0 ** 2)) <= 2 * 0.5 / 4 + 0.05


def test_single_warped_pyramid_uses_the_area_rule():
    """One ratio other than 1: the region rule stays the area rule (no aspect factor)."""
    H, W, K = 600, 800, 10
    p = oracle.plan(H, W, K, 4, 1.0, 0, 16, 1200, 1200, aspects=[2.0])
    maps = [np.zeros((256, oracle.conv5_side(h), oracle.conv5_side(w)), np.float32)
            for h, w in p.plane_sizes]
    boxes = synth.boxes(3, 50, H, W)
    _, scale, _, _ = oracle.region_windows(maps, p, boxes)
    bw, bh = boxes[:, 2] - boxes[:, 0], boxes[:, 3] - boxes[:, 1]
    cost = np.maximum.reduce([(p.gd[None, :, 1] * bh[:, None]) * (p.gd[None, :, 2] * bw[:, None]) / 227.0 ** 2,
                              227.0 ** 2 / ((p.gd[None, :, 1] * bh[:, None]) * (p.gd[None, :, 2] * bw[:, None]))])
    np.testing.assert_array_equal(scale, np.argmin(cost, axis=1))
