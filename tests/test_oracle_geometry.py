"""Pins for the oracle's pyramid geometry (Sec. 3.1): closed-form scale sizes, the conv5 receptive
field measured through the oracle's own layers on delta inputs, and the stitching invariants.  The
Bottom-Left-Fill variant itself is a reading of the paper (parity unpinned): only its invariants are
checked here."""
import math

import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import configs as C


def P(w):
    return oracle.plan(w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side,
                       w.pad, w.plane_h, w.plane_w)


def test_scale_sizes_at_exact_octaves():
    p = P(C.XGA_25SCALE)
    hw = {int(k): (int(h), int(w)) for k, h, w in p.gi[:, :3]}
    assert hw[0] == (768, 1024)
    assert hw[10] == (384, 512)      # 2^-1 exactly
    assert hw[20] == (192, 256)      # 2^-2 exactly
    assert hw[5] == (543, 724)       # 768/sqrt 2 = 543.06, 1024/sqrt 2 = 724.08
    assert len(hw) == 25
    # 25 scales span (25 - 1)/10 octaves; the pyramid holds 3-8x the source pixels (Sec. 3.1)
    area = sum(h * w for h, w in hw.values()) / (768 * 1024)
    assert 3 <= area <= 8
    p2 = P(C.VGA_8SCALE)
    assert tuple(p2.gi[0, 1:3]) == (768, 1024)   # longest side 1024 from 640: 1.6 x (480, 640)
    assert tuple(p2.gi[4, 1:3]) == (384, 512)    # one octave down
    p1 = P(C.ALEXNET_227)
    assert tuple(p1.gi[1, 1:3]) == (161, 161)    # 227 / sqrt 2 = 160.5
    assert p1.n_planes == 2 and p1.plane_sizes == [(227, 227), (161, 161)]


def _support_rows(n_rows, width=40):
    """For every input row y of a 1-channel plane, the conv5 rows reached by a delta at (y, x0),
    through the oracle's conv and pool layers with positive filters."""
    ones = lambda R: np.ones((1, 1, R, R), np.float32)
    z = np.zeros(1, np.float32)
    masks = []
    for y in range(n_rows):
        x = np.zeros((1, n_rows, width), np.float32)
        x[0, y, width // 2] = 1
        a = oracle.maxpool(oracle.conv2d(x, ones(11), z, 4, 0))
        a = oracle.maxpool(oracle.conv2d(a, ones(5), z, 1, 2))
        for _ in range(3):
            a = oracle.conv2d(a, ones(3), z, 1, 1)
        masks.append(a[0].max(axis=1) > 0)
    return np.array(masks)  # [y][i]


def test_conv5_receptive_field_and_centre():
    n = 320
    m = _support_rows(n)
    Hc = m.shape[1]
    assert Hc == oracle.conv5_side(n)
    for i in range(Hc):
        ys = np.nonzero(m[:, i])[0]
        lo, hi = ys.min(), ys.max()
        assert hi - lo + 1 == min(163, hi + 1 - max(lo, 0)) or lo == 0 or hi == n - 1
        if 16 * i - 64 >= 0 and 16 * i + 98 < n:
            assert (lo, hi) == (16 * i - 64, 16 * i + 98)       # 163-px field at stride 16
            assert (lo + hi + 1) / 2 == 16 * i + 17.5           # continuous centre


def test_windows_follow_receptive_field_centres():
    # Cells kept for a scale are exactly those whose receptive-field centre lies on its real pixels.
    for w in (C.VGA_8SCALE, C.XGA_25SCALE, C.ALEXNET_227):
        p = P(w)
        for g in p.gi:
            k, h, wd, pl, y, x, rh, rw, r0, r1, c0, c1, PH, PW = (int(v) for v in g[:14])
            Hc, Wc = oracle.conv5_side(PH), oracle.conv5_side(PW)
            rows = [i for i in range(Hc) if y + w.pad <= 16 * i + 17.5 < y + w.pad + h]
            cols = [j for j in range(Wc) if x + w.pad <= 16 * j + 17.5 < x + w.pad + wd]
            assert (r0, r1) == (rows[0], rows[-1]) and (c0, c1) == (cols[0], cols[-1])


@pytest.mark.parametrize("w", [C.XGA_25SCALE, C.VGA_8SCALE, C.ALEXNET_227])
def test_stitching_invariants(w):
    p = P(w)
    K = w.n_scales
    assert sorted(p.gi[:, 0]) == list(range(K))
    rects = {}
    for g in p.gi:
        k, h, wd, pl, y, x, rh, rw = (int(v) for v in g[:8])
        PH, PW = p.plane_sizes[pl]
        assert 0 <= y and y + rh <= PH and 0 <= x and x + rw <= PW
        assert rh >= h + 2 * w.pad and rw >= wd + 2 * w.pad
        if w.plane_h:
            assert y % 16 == 0 and x % 16 == 0 and rh % 16 == 0 and rw % 16 == 0
            assert rh - (h + 2 * w.pad) < 16 and rw - (wd + 2 * w.pad) < 16
        rects.setdefault(pl, []).append((y, x, rh, rw))
    for pl, rs in rects.items():
        for a in range(len(rs)):
            for b in range(a + 1, len(rs)):
                ya, xa, ha, wa = rs[a]
                yb, xb, hb, wb = rs[b]
                assert ya + ha <= yb or yb + hb <= ya or xa + wa <= xb or xb + wb <= xa
    if w.plane_h:
        area = sum(int(g[6]) * int(g[7]) for g in p.gi)
        assert p.n_planes >= math.ceil(area / (w.plane_h * w.plane_w))
        # at least 2p px between real pixels of neighbouring scales (Sec. 3.1)
        assert w.pad == 16


def test_cfg3_plane_count_and_first_fit():
    p = P(C.XGA_25SCALE)
    assert p.n_planes == 6                     # area lower bound is 5
    assert all(s == (1200, 1200) for s in p.plane_sizes)
    # the five largest scales each open a plane at the origin
    assert [tuple(int(v) for v in p.gi[k, 3:6]) for k in range(5)] == [(k, 0, 0) for k in range(5)]


def test_plan_errors_and_tiny_scale():
    with pytest.raises(ValueError):
        oracle.plan(768, 1024, 3, 10, 1.0, 0, 16, 700, 700)   # scale 0 does not fit a 700 plane
    p = oracle.plan(1, 1, 1, 1, 1.0, 0, 16, 0, 0)               # a 1x1 image at scale 1
    assert tuple(p.gi[0, 1:3]) == (1, 1) and p.plane_sizes == [(33, 33)]
