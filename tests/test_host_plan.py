"""The library's host geometry (written independently of the oracle) equals the oracle's plan bit for
bit: sizes, factors, planes, rectangles, offsets and conv5 windows (Sec. 3.1)."""
import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import densenet as D

CASES = list(C.ALL) + [
    C.Workload("odd_small", 37, 53, (1,), 6, 3, pad=16, pad_mode=1, plane_h=400, plane_w=480),
    C.Workload("upsampled", 300, 200, (1,), 12, 5, base_scale=2.0, pad=16, pad_mode=1, plane_h=2000,
               plane_w=2000),
    C.Workload("tiny", 1, 1, (1,), 1, 1, pad=16),
    C.Workload("wide", 64, 1000, (1,), 9, 3, pad=8, plane_h=600, plane_w=1200),
    C.Workload("many_small", 120, 160, (1,), 40, 10, pad=16, pad_mode=1, plane_h=480, plane_w=480),
    C.Workload("aspects3", 480, 640, (1,), 12, 4, pad=16, pad_mode=1, plane_h=1200, plane_w=1200,
               aspects=(0.5, 1.0, 2.0)),
    C.Workload("aspects_per_scale_planes", 97, 131, (1,), 5, 2, pad=16, aspects=(1 / 3, 3.0)),
    C.Workload("aspect_single", 300, 200, (1,), 6, 3, pad=8, plane_h=800, plane_w=800, aspects=(1.7,)),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_plan_bit_exact_vs_oracle(w):
    lib = D.densenet_plan_pyramid(w.H, w.W, D.params_for(w))
    ref = oracle.plan(w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side,
                      w.pad, w.plane_h, w.plane_w, aspects=list(w.aspects) or None)
    assert len(lib.planes) == ref.n_planes
    np.testing.assert_array_equal(lib.geom_array(), ref.gi[:, [*range(12), 14]])
    np.testing.assert_array_equal(lib.scale_array(), ref.gd)   # bitwise equal fp64
    assert [(p.h, p.w) for p in lib.planes] == ref.plane_sizes
    # rows padded to a multiple of 64 elements
    pitch = [(w_ + 63) // 64 * 64 for _, w_ in ref.plane_sizes]
    assert [p.pitch for p in lib.planes] == pitch
    off = np.cumsum([0] + [3 * h * p for (h, _), p in zip(ref.plane_sizes, pitch)])
    assert [p.offset for p in lib.planes] == list(off[:-1])
    assert lib.image_elems == off[-1]


def test_plan_is_deterministic():
    w = C.XGA_25SCALE
    a = D.densenet_plan_pyramid(w.H, w.W, D.params_for(w)).geom_array()
    b = D.densenet_plan_pyramid(w.H, w.W, D.params_for(w)).geom_array()
    np.testing.assert_array_equal(a, b)


BATCH_CASES = [
    (16, C.XGA_25SCALE_B16),
    (5, C.Workload("vga_batch", 480, 640, (1,), 8, 4, pad=16, pad_mode=1, plane_h=1200, plane_w=1200)),
    (7, C.Workload("small_batch", 300, 200, (1,), 6, 3, pad=16, pad_mode=1, plane_h=400, plane_w=400)),
    (4, C.Workload("aspect_batch", 240, 320, (1,), 6, 3, pad=16, pad_mode=1, plane_h=800, plane_w=800,
                   aspects=(0.5, 2.0))),
    (3, C.Workload("wide_batch", 64, 1000, (1,), 9, 3, pad=8, plane_h=600, plane_w=1200)),
    (1, C.XGA_25SCALE),
]


@pytest.mark.parametrize("n_img,w", BATCH_CASES, ids=lambda v: getattr(v, "name", str(v)))
def test_batch_plan_bit_exact_vs_oracle(n_img, w):
    lib = D.BatchPlan(n_img, w.H, w.W, D.params_for(w), device=None)
    ref = oracle.plan_batch(n_img, w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale,
                            w.base_longest_side, w.pad, w.plane_h, w.plane_w,
                            aspects=list(w.aspects) or None)
    assert lib.n_planes == ref.n_planes
    np.testing.assert_array_equal(lib.geom_array(), ref.gi[:, [*range(12), 14, 15]])
    np.testing.assert_array_equal(np.array([[g.s, g.sy, g.sx] for g in lib.geom]), ref.gd)
    pitch = (w.plane_w + 63) // 64 * 64
    pe = 3 * w.plane_h * pitch
    assert [(p.h, p.w, p.pitch, p.offset) for p in lib.planes] == [(w.plane_h, w.plane_w, pitch, j * pe)
                                                                   for j in range(ref.n_planes)]
    assert lib.total_elems == ref.n_planes * pe


def test_batch_of_one_is_the_image_plan():
    w = C.XGA_25SCALE
    a = D.densenet_plan_pyramid(w.H, w.W, D.params_for(w))
    b = D.BatchPlan(1, w.H, w.W, D.params_for(w), device=None)
    np.testing.assert_array_equal(a.geom_array(), b.geom_array()[:, :13])
    assert b.n_planes == len(a.planes)
