"""Pins for region windows ("crop after", Sec. 4): constant maps give constant descriptors, bin centres
on cell centres give exact gathers, torch grid_sample (align_corners, border) in fp64 reproduces the
bilinear sampling, the chosen scale is monotone in box area, degenerate boxes give scale -1 and zeros.
The scale rule itself (closest area to 227^2) is a reading of the paper: parity unpinned."""
import numpy as np
import torch

import oracle
from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import synth

w = C.XGA_25SCALE


def _plan():
    return oracle.plan(w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side,
                       w.pad, w.plane_h, w.plane_w)


def _maps(p, seed=3):
    rng = np.random.default_rng(seed)
    return [rng.normal(size=(256, 74, 74)).astype(np.float32) for _ in range(p.n_planes)]


def test_constant_map_gives_constant_descriptor():
    p = _plan()
    vals = np.random.default_rng(1).normal(size=256).astype(np.float32)
    maps = [np.ascontiguousarray(np.broadcast_to(vals[:, None, None], (256, 74, 74))) for _ in
            range(p.n_planes)]
    boxes = synth.boxes(9, 50, w.H, w.W)
    desc, scale, _, _ = oracle.region_windows(maps, p, boxes)
    assert (scale >= 0).all()
    np.testing.assert_array_equal(desc.reshape(50, 256, 36), np.broadcast_to(vals[None, :, None],
                                                                             (50, 256, 36)))


def test_bin_centres_on_cell_centres_are_exact_gathers():
    p = _plan()
    maps = _maps(p)
    k = 10                     # scale 0.5, exact factors sy = sx = 0.5
    h, wd, pl, y, x = (int(v) for v in p.gi[k, 1:6])
    assert p.gd[k, 1] == 0.5 and p.gd[k, 2] == 0.5
    # a box whose 6 bin centres fall on conv5 cell centres 16 i + 17.5 of the plane:
    # plane X = x_orig * 0.5 + x + 16; bins 16 cells apart need a box 6*16*... = 96 plane px wide
    i0, j0 = int(p.gi[k, 8]) + 2, int(p.gi[k, 10]) + 2
    X1 = 16 * j0 + 17.5 - 8.0           # bin b centre = X1 + (b + 0.5) * 16
    Y1 = 16 * i0 + 17.5 - 8.0
    x1 = (X1 - x - 16) / 0.5
    y1 = (Y1 - y - 16) / 0.5
    box = np.array([[x1, y1, x1 + 192.0, y1 + 192.0]], np.float32)   # 96 plane px, 6 bins of 16
    desc, scale, idx, lam = oracle.region_windows(maps, p, box, T=96.0)
    assert scale[0] == k
    assert (lam == 0).all()
    ref = maps[pl][:, i0:i0 + 6, j0:j0 + 6].reshape(-1)
    np.testing.assert_array_equal(desc[0], ref)


def test_sampling_matches_grid_sample():
    p = _plan()
    maps = _maps(p, 4)
    boxes = synth.boxes(105, 200, w.H, w.W)
    desc, scale, idx, lam = oracle.region_windows(maps, p, boxes)
    for r in range(0, 200, 7):
        k = scale[r]
        g = p.gi[k]
        pl, r0, r1, c0, c1 = int(g[3]), int(g[8]), int(g[9]), int(g[10]), int(g[11])
        win = torch.from_numpy(maps[pl][:, r0:r1 + 1, c0:c1 + 1]).double()[None]
        # sample positions in window cells, rebuilt from the oracle's own (index, fraction) output
        gy = idx[r, :, :, 0] + lam[r, :, :, 0] - r0
        gx = idx[r, :, :, 1] + lam[r, :, :, 1] - c0
        grid = torch.stack([torch.from_numpy(2 * gx / max(c1 - c0, 1) - 1),
                            torch.from_numpy(2 * gy / max(r1 - r0, 1) - 1)], -1)[None]
        ref = torch.nn.functional.grid_sample(win, grid, mode="bilinear", padding_mode="border",
                                              align_corners=True)[0]
        np.testing.assert_allclose(desc[r].reshape(256, 6, 6), ref.numpy(), rtol=1e-6, atol=1e-6)


def test_bin_positions_follow_box_linearly():
    # unclamped bin positions are an affine image of the box: equal steps between bins
    p = _plan()
    maps = _maps(p)
    boxes = np.array([[300, 200, 500, 330]], np.float32)
    _, scale, idx, lam = oracle.region_windows(maps, p, boxes)
    k = scale[0]
    g = p.gi[k]
    gx = idx[0, 0, :, 1] + lam[0, 0, :, 1]
    gy = idx[0, :, 0, 0] + lam[0, :, 0, 0]
    sx, sy = p.gd[k, 2], p.gd[k, 1]
    np.testing.assert_allclose(np.diff(gx), 200 * sx / 6 / 16, rtol=1e-12)
    np.testing.assert_allclose(np.diff(gy), 130 * sy / 6 / 16, rtol=1e-12)
    # first bin centre: (x1 sx + x + 16 + (1/12)(200 sx) - 17.5) / 16
    np.testing.assert_allclose(gx[0], (300 * sx + g[5] + 16 + 200 * sx / 12 - 17.5) / 16, rtol=1e-12)


def test_scale_choice_monotone_and_degenerate_boxes():
    p = _plan()
    maps = _maps(p)
    sizes = np.geomspace(20, 760, 60)
    boxes = np.stack([np.full(60, 2.0), np.full(60, 2.0), 2 + sizes, 2 + sizes], 1).astype(np.float32)
    _, scale, _, _ = oracle.region_windows(maps, p, boxes)
    assert (np.diff(scale) >= 0).all()           # larger boxes never pick a finer scale
    assert scale[0] == 0 and scale[-1] > 0
    # inside the pyramid's range the chosen scale brings the box within half a step (2^0.05) of 227
    for sz, k in zip(sizes, scale):
        side = sz * np.sqrt(p.gd[k, 1] * p.gd[k, 2])
        if 227 / p.gd[0, 1] < sz < 227 / p.gd[-1, 1]:
            assert abs(np.log2(side / 227)) <= 0.05 + 2e-3
    bad = np.array([[10, 10, 10, 50], [10, 10, 5, 50], [np.nan, 0, 5, 5], [0, 0, np.inf, 5]],
                   np.float32)
    desc, scale, _, _ = oracle.region_windows(maps, p, bad)
    assert (scale == -1).all() and not desc.any()
