"""GPU parity on edge cases of the path, through the C ABI, against the oracle: ragged image sizes on
small stitched planes, the smallest plane that still has a conv5 cell, the pool-then-LRN order,
a 2000 x 2000 plane (the paper's larger plane size), region windows with no boxes, 1 x 1 and 8 x 8
bins and out-of-range image indices, and planes too small for conv5 rejected before any launch."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import synth
from tests.parity import plane_tol, assert_layer_close, chw, round_to, ulp

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DTS = {"f32": 0, "f16": 1, "bf16": 2}
W7 = synth.weights(7)


@pytest.fixture(scope="module")
def D():
    from paper_1404_1869_amd import densenet
    assert torch.cuda.is_available()
    densenet.lib()
    return densenet


_packed = {}


def packed(D, dt):
    if dt not in _packed:
        ws = [(torch.from_numpy(w).cuda(), torch.from_numpy(b).cuda()) for w, b in W7]
        _packed[dt] = D.densenet_pack_weights(ws, DTS[dt])
    return _packed[dt]


def run(D, img, p, dt, net=None):
    pyra = D.convnet_featpyramid(torch.from_numpy(img).cuda()[None], p, packed(D, dt), DTS[dt], net)
    torch.cuda.synchronize()
    return pyra


@pytest.mark.parametrize("dt", ["f16", "bf16", "f32"])
def test_ragged_image_small_stitched_planes(D, dt):
    H, W = 97, 131
    img = synth.image(77, H, W)
    p = D.pyramid_params(4, 3, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=208, plane_w=240,
                         mean=synth.IMAGENET_MEAN)
    pyra = run(D, img, p, dt)
    op = oracle.plan(H, W, 4, 3, 1.0, 0, 16, 208, 240)
    planes = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)
    maps = pyra.conv.conv5_maps()
    assert len(maps) == op.n_planes
    for j, pl in enumerate(planes):
        ref = oracle.net(pl.astype(np.float32), W7)
        assert_layer_close(chw(maps[j].float().cpu().numpy()), ref, dt, f"ragged plane {j}")


@pytest.mark.parametrize("W", [4000, 3999])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_planes_strongly_reduced_wide_image(D, W, dt):
    """Scales 0.3 .. 0.106 of a 4000-px-wide image: a wave's 256 plane columns span up to 2400
    source columns; rows of 4000 px start on 4-byte boundaries, rows of 3999 px do not."""
    H = 40
    img = synth.image(91, H, W)
    p = D.pyramid_params(4, 2, base_scale=0.3, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=64,
                         plane_w=1248, mean=synth.IMAGENET_MEAN)
    planes, plan = D.densenet_build_pyramid(torch.from_numpy(img).cuda()[None], p, DTS[dt])
    op = oracle.plan(H, W, 4, 2, 0.3, 0, 16, 64, 1248)
    ref = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)
    assert len(plan.planes) == op.n_planes
    for j, d in enumerate(plan.planes):
        got = D.plane_view(planes, d).float().cpu().numpy()
        assert np.all(np.abs(got - ref[j]) <= plane_tol(ref[j], dt)), f"plane {j}"


@pytest.mark.parametrize("W,base", [(32767, 1.0), (16384, 2.0), (17000, 2.0)])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_planes_widest_scales(D, W, base, dt):
    """Scaled widths up to 32767 px take exact integer horizontal taps (weights 2 w - rx and rx as
    16-bit integers: 32767 and 32768 px wide scales sit on either side of that limit); a pyramid with
    a wider scale (34000 px) blends its columns in fp32 instead.  Per-scale planes, ramp border."""
    H = 3
    img = synth.image(95, H, W)
    p = D.pyramid_params(2, 2, base_scale=base, pad=16, pad_mode=D.DN_PAD_RAMP,
                         mean=synth.IMAGENET_MEAN)
    planes, plan = D.densenet_build_pyramid(torch.from_numpy(img).cuda()[None], p, DTS[dt])
    op = oracle.plan(H, W, 2, 2, base, 0, 16, 0, 0)
    ref = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)
    assert len(plan.planes) == op.n_planes
    for j, d in enumerate(plan.planes):
        got = D.plane_view(planes, d).float().cpu().numpy()
        assert np.all(np.abs(got - ref[j]) <= plane_tol(ref[j], dt)), f"plane {j}"


@pytest.mark.parametrize("W", [1, 2, 3])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_planes_narrow_images(D, W, dt):
    """Images 1-3 px wide, upscaled up to 40x: every plane column samples the last source column
    (the clamped tap), with the two taps of a row loaded separately (W = 1) or as one pair."""
    H = 5
    img = synth.image(93 + W, H, W)
    p = D.pyramid_params(3, 2, base_scale=40.0, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=256,
                         plane_w=192, mean=synth.IMAGENET_MEAN)
    planes, plan = D.densenet_build_pyramid(torch.from_numpy(img).cuda()[None], p, DTS[dt])
    op = oracle.plan(H, W, 3, 2, 40.0, 0, 16, 256, 192)
    ref = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)
    assert len(plan.planes) == op.n_planes
    for j, d in enumerate(plan.planes):
        got = D.plane_view(planes, d).float().cpu().numpy()
        assert np.all(np.abs(got - ref[j]) <= plane_tol(ref[j], dt)), f"plane {j}"


def test_smallest_plane_with_a_conv5_cell(D):
    # a 1 x 1 image with 13 px of zero padding is a 27 x 27 plane: conv5 is 1 x 1
    img = synth.image(5, 1, 1)
    p = D.pyramid_params(1, 1, pad=13, pad_mode=D.DN_PAD_ZERO, mean=synth.IMAGENET_MEAN)
    pyra = run(D, img, p, "f32")
    op = oracle.plan(1, 1, 1, 1, 1.0, 0, 13, 0, 0)
    pl = oracle.build_planes(img, op, 0, synth.IMAGENET_MEAN)[0]
    assert pl.shape == (3, 27, 27)
    ref = oracle.net(pl.astype(np.float32), W7)
    got = pyra.conv.conv5_maps()[0]
    assert tuple(got.shape) == (1, 1, 256)
    assert_layer_close(chw(got.cpu().numpy()), ref, "f32", "27x27 plane")


def test_plane_too_small_is_rejected_before_launch(D):
    img = torch.from_numpy(synth.image(5, 1, 1)).cuda()[None]
    p = D.pyramid_params(1, 1, pad=8, pad_mode=D.DN_PAD_ZERO)   # 17 x 17 plane: conv5 empty
    planes, plan = D.densenet_build_pyramid(img, p, DTS["f16"])
    with pytest.raises(D.DenseNetError) as e:
        D.ConvFeatures(plan.planes, DTS["f16"], D.net_params())
    assert e.value.status == D.DN_E_INVALID_ARG and "too small" in D.last_error()


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_pool_then_lrn_order_end_to_end(D, dt):
    img = synth.image(101, 227, 227)
    p = D.pyramid_params(2, 2, mean=synth.IMAGENET_MEAN)
    pyra = run(D, img, p, dt, D.net_params(lrn_before_pool=False, pool5=True))
    op = oracle.plan(227, 227, 2, 2)
    planes = oracle.build_planes(img, op, 0, synth.IMAGENET_MEAN)
    for j, pl in enumerate(planes):
        c5, p5 = oracle.net(pl.astype(np.float32), W7, lrn_before_pool=False, pool5=True)
        assert_layer_close(chw(pyra.conv.conv5_maps()[j].float().cpu().numpy()), c5, dt, f"conv5 {j}")
        assert_layer_close(chw(pyra.conv.pool5_maps()[j].float().cpu().numpy()), p5, dt, f"pool5 {j}")


def test_2000_plane_f16(D):
    # one 1536 x 2000 image at scale 1 with ramp padding, stitched onto a 2000 x 2000 plane
    H, W = 1536, 1900
    img = synth.image(2000, H, W)
    p = D.pyramid_params(1, 1, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=2000, plane_w=2000,
                         mean=synth.IMAGENET_MEAN)
    pyra = run(D, img, p, "f16")
    op = oracle.plan(H, W, 1, 1, 1.0, 0, 16, 2000, 2000)
    pl = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)[0]
    ref = oracle.net(pl.astype(np.float32), W7)
    got = pyra.conv.conv5_maps()[0]
    assert tuple(got.shape) == (124, 124, 256)
    assert_layer_close(chw(got.float().cpu().numpy()), ref, "f16", "2000 plane")


def _shared_maps(p, seed):
    rng = np.random.default_rng(seed)
    return [rng.normal(0, 1, (256, oracle.conv5_side(h), oracle.conv5_side(w))).astype(np.float32)
            for h, w in p.plane_sizes]


def _descs(D, maps, n_img=1):
    descs, off = [], 0
    for _ in range(n_img):
        for m in maps:
            d = D.dn_plane_desc()
            d.h, d.w, d.offset = m.shape[1], m.shape[2], off
            off += m.size
            descs.append(d)
    return descs


@pytest.mark.parametrize("S", [1, 8])
def test_region_windows_bins_and_edges(D, S):
    H, W = 480, 640
    p = oracle.plan(H, W, 8, 4, 1.0, 0, 16, 800, 800)
    plan = D.densenet_plan_pyramid(H, W, D.pyramid_params(8, 4, pad=16, pad_mode=D.DN_PAD_RAMP,
                                                          plane_h=800, plane_w=800))
    maps = _shared_maps(p, 3)
    flat = np.concatenate([np.moveaxis(m, 0, -1).ravel() for m in maps] * 2)
    c5 = torch.from_numpy(flat).cuda()
    boxes = synth.boxes(11, 300, H, W)
    box_img = np.zeros(300, np.int32)
    box_img[::3] = 1
    box_img[5] = 2          # out of range: scale -1, zero row
    box_img[7] = -1
    out, sc, ix = D.densenet_region_windows(c5, _descs(D, maps, 2), DTS["f32"], plan, 16, p.n_planes,
                                            torch.from_numpy(boxes).cuda(),
                                            torch.from_numpy(box_img).cuda(), target=227.0, S=S,
                                            want_idx=True)
    torch.cuda.synchronize()
    # image 1's maps are a copy of image 0's: the oracle sees image 0 for all valid boxes
    desc, scale, idx, _ = oracle.region_windows(maps, p, boxes, S=S)
    sc = sc.cpu().numpy()
    valid = (box_img >= 0) & (box_img < 2)
    np.testing.assert_array_equal(sc[valid], scale[valid])
    np.testing.assert_array_equal(ix.cpu().numpy()[valid], idx[valid])
    np.testing.assert_allclose(out.cpu().numpy()[valid], desc[valid], rtol=2e-6, atol=2e-6)
    assert (sc[~valid] == -1).all() and not out.cpu().numpy()[~valid].any()


def test_region_windows_no_boxes(D):
    p = oracle.plan(227, 227, 2, 2)
    plan = D.densenet_plan_pyramid(227, 227, D.pyramid_params(2, 2))
    maps = _shared_maps(p, 1)
    c5 = torch.from_numpy(np.concatenate([np.moveaxis(m, 0, -1).ravel() for m in maps])).cuda()
    out, sc, _ = D.densenet_region_windows(c5, _descs(D, maps), DTS["f32"], plan, 0, 2,
                                           torch.zeros((0, 4), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    assert out.shape == (0, 9216) and sc.shape == (0,)


@pytest.mark.parametrize("spo,base,plane,dt", [(5, 2.0, 2000, "bf16"), (3, 1.0, 1200, "f16")])
def test_scale_and_plane_variants_end_to_end(D, spo, base, plane, dt):
    """Sec. 3.1's other pyramid recipes: a maximum scale of 2 (upsampling) with 5 scales per octave on
    2000 x 2000 planes, and 3 scales per octave on 1200 x 1200 planes; planes, conv5 of the fullest
    plane, and region windows of the whole pyramid against the oracle."""
    H, W, K = 240, 320, 2 * spo
    img = synth.image(300 + spo, H, W)
    p = D.pyramid_params(K, spo, base_scale=base, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=plane,
                         plane_w=plane, mean=synth.IMAGENET_MEAN)
    pyra = run(D, img, p, dt)
    op = oracle.plan(H, W, K, spo, base, 0, 16, plane, plane)
    assert len(pyra.plan.planes) == op.n_planes
    ref_planes = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)
    for j, d in enumerate(pyra.plan.planes):
        got = D.plane_view(pyra.planes, d).float().cpu().numpy()
        assert np.all(np.abs(got - ref_planes[j]) <= plane_tol(ref_planes[j], dt)), f"plane {j}"
    maps = pyra.conv.conv5_maps()
    c5 = {}
    for j in range(op.n_planes):
        c5[j] = oracle.net(ref_planes[j].astype(np.float32), W7)
        assert_layer_close(chw(maps[j].float().cpu().numpy()), c5[j], dt, f"conv5 plane {j}")
    boxes = synth.boxes(12, 200, H, W, smin=16, smax=240)
    desc, scale, _ = D.densenet_region_windows(pyra.conv.conv5, list(pyra.conv.c5d), DTS[dt], pyra.plan,
                                               16, op.n_planes, torch.from_numpy(boxes).cuda())
    rd, rs, _, _ = oracle.region_windows([c5[j] for j in range(op.n_planes)], op, boxes)
    np.testing.assert_array_equal(scale.cpu().numpy(), rs)
    assert_layer_close(desc.cpu().numpy(), rd, dt, "region windows")


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_aspect_ratio_pyramids_end_to_end(D, dt):
    """Sec. 3.3: one area-keeping warped pyramid per aspect ratio (1/2, 1, 2), all stitched onto shared
    1200 x 1200 planes; planes, conv5 of every plane, and region windows (entry choice bit for bit,
    including boxes whose aspect picks the warped pyramids) against the oracle."""
    H, W, K, r = 480, 640, 6, (0.5, 1.0, 2.0)
    img = synth.image(333, H, W)
    p = D.pyramid_params(K, 4, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=1200, plane_w=1200,
                         mean=synth.IMAGENET_MEAN, aspects=r)
    pyra = run(D, img, p, dt)
    op = oracle.plan(H, W, K, 4, 1.0, 0, 16, 1200, 1200, aspects=list(r))
    assert len(pyra.plan.geom) == K * len(r) and len(pyra.plan.planes) == op.n_planes
    ref_planes = oracle.build_planes(img, op, 1, synth.IMAGENET_MEAN)
    for j, d in enumerate(pyra.plan.planes):
        got = D.plane_view(pyra.planes, d).float().cpu().numpy()
        assert np.all(np.abs(got - ref_planes[j]) <= plane_tol(ref_planes[j], dt)), f"plane {j}"
    maps = pyra.conv.conv5_maps()
    c5 = []
    for j in range(op.n_planes):
        c5.append(oracle.net(ref_planes[j].astype(np.float32), W7))
        assert_layer_close(chw(maps[j].float().cpu().numpy()), c5[j], dt, f"conv5 plane {j}")
    boxes = np.concatenate([synth.boxes(14, 300, H, W), np.array(
        [[20, 100, 620, 400], [250, 10, 400, 470], [100, 100, 350, 350]], np.float32)])
    desc, scale, _ = D.densenet_region_windows(pyra.conv.conv5, list(pyra.conv.c5d), DTS[dt], pyra.plan,
                                               16, op.n_planes, torch.from_numpy(boxes).cuda())
    rd, rs, _, _ = oracle.region_windows(c5, op, boxes)
    sc = scale.cpu().numpy()
    np.testing.assert_array_equal(sc, rs)
    np.testing.assert_array_equal(op.field("aspect")[sc[-3:]], [0, 2, 1])
    assert len(set(op.field("aspect")[sc])) == 3
    assert_layer_close(desc.cpu().numpy(), rd, dt, "region windows")


@pytest.mark.parametrize("dt,S", [("f32", 6), ("bf16", 6), ("f16", 1), ("bf16", 8)])
def test_region_pool_bit_exact(D, dt, S):
    """Max-pooled region bins on shared conv5 maps (two images, stored in the path's dtype): chosen
    entries, bin cell ranges and every descriptor value bit for bit against the oracle, including
    degenerate boxes and image indices out of range (scale -1, zero row)."""
    H, W = 480, 640
    p = oracle.plan(H, W, 8, 4, 1.0, 0, 16, 800, 800)
    plan = D.densenet_plan_pyramid(H, W, D.pyramid_params(8, 4, pad=16, pad_mode=D.DN_PAD_RAMP,
                                                          plane_h=800, plane_w=800))
    maps = [round_to(m, dt) for m in _shared_maps(p, 9)]
    flat = np.concatenate([np.moveaxis(m, 0, -1).ravel() for m in maps] * 2)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]
    c5 = torch.from_numpy(flat).to("cuda", tdt)
    boxes = np.concatenate([synth.boxes(31, 400, H, W, smin=8, smax=480),
                            np.array([[5, 5, 5, 40], [10, 10, 12.5, 11], [np.nan, 0, 4, 4]], np.float32)])
    box_img = (np.arange(len(boxes)) % 2).astype(np.int32)
    box_img[3] = 2
    out, sc, ix = D.densenet_region_pool(c5, _descs(D, maps, 2), DTS[dt], plan, 16, p.n_planes,
                                         torch.from_numpy(boxes).cuda(), torch.from_numpy(box_img).cuda(),
                                         S=S, want_idx=True)
    torch.cuda.synchronize()
    desc, scale, idx = oracle.region_pool(maps, p, boxes, S=S)
    sc, ix, out = sc.cpu().numpy(), ix.cpu().numpy(), out.cpu().numpy()
    valid = box_img < 2
    np.testing.assert_array_equal(sc[valid], scale[valid])
    np.testing.assert_array_equal(ix[valid], idx[valid])
    np.testing.assert_array_equal(out[valid], desc[valid])
    assert (sc[~valid] == -1).all() and not out[~valid].any()
    assert (sc[-3] == scale[-3]) and (sc[-1] == -1)
