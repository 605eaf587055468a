"""GPU parity of cross-image packing (the rectangles of a whole batch stitched together, Sec. 3.1)
through the C ABI: packed planes against the oracle's, every packed rectangle at full batch size equal
bit for bit to the same rectangle built per image, the conv stack on sampled packed planes, and region
windows / max-pooled bins read through the packed layout (entries and indices bit for bit)."""
import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import synth
from tests.parity import plane_tol, assert_layer_close, chw, round_to, ulp

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DTS = {"f32": 0, "f16": 1, "bf16": 2}
TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
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


def oplan_batch(n_img, w):
    return oracle.plan_batch(n_img, w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale,
                             w.base_longest_side, w.pad, w.plane_h, w.plane_w,
                             aspects=list(w.aspects) or None)


def views(D, planes, plan):
    return [D.plane_view(planes, plan.planes[j]) for j in range(plan.n_planes)]


def check_planes(got, ref, dt):
    got = got.float().cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= plane_tol(ref, dt))


SMALL = [
    (5, C.Workload("b5_120x90", 120, 90, tuple(range(200, 205)), 5, 2, pad=16, pad_mode=1, plane_h=224,
                   plane_w=224)),
    (3, C.Workload("b3_300x240", 300, 240, (210, 211, 212), 6, 2, pad=16, pad_mode=1, plane_h=480,
                   plane_w=480)),
    (6, C.Workload("b6_97x131_zero", 97, 131, tuple(range(220, 226)), 4, 3, pad=16, pad_mode=0,
                   plane_h=200, plane_w=232)),
    (4, C.Workload("b4_aspects", 120, 160, tuple(range(230, 234)), 4, 2, pad=16, pad_mode=1, plane_h=320,
                   plane_w=320, aspects=(0.5, 2.0))),
]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n_img,w", SMALL, ids=lambda v: getattr(v, "name", str(v)))
def test_packed_planes(D, n_img, w, dt):
    imgs = synth.images(w.seeds, w.H, w.W)
    plan = D.BatchPlan(n_img, w.H, w.W, D.params_for(w))
    ref_plan = oplan_batch(n_img, w)
    assert plan.n_planes == ref_plan.n_planes
    assert plan.n_planes < n_img * len(D.densenet_plan_pyramid(w.H, w.W, D.params_for(w)).planes)
    planes = D.densenet_build_batch(torch.from_numpy(imgs).cuda(), plan, DTS[dt])
    torch.cuda.synchronize()
    ref = oracle.build_planes(imgs, ref_plan, w.pad_mode, w.mean)
    for j, v in enumerate(views(D, planes, plan)):
        check_planes(v, ref[j], dt)


def test_packed_rectangles_equal_per_image_rectangles_full_batch(D):
    """16 images of 768 x 1024 (25 scales, 1200 x 1200 planes): the 88 packed planes hold, rectangle
    for rectangle, exactly the values the per-image builder writes, and zeros elsewhere."""
    w = C.XGA_25SCALE_B16
    imgs = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).cuda()
    plan = D.BatchPlan(16, w.H, w.W, D.params_for(w))
    assert plan.n_planes == 88
    pk = views(D, D.densenet_build_batch(imgs, plan, DTS["bf16"]), plan)
    own, own_plan = D.densenet_build_pyramid(imgs, D.params_for(w), DTS["bf16"])
    torch.cuda.synchronize()
    covered = torch.zeros((88, 1200, 1200), dtype=torch.bool, device="cuda")
    for b in range(16):
        for e in range(plan.E):
            g1, gb = own_plan.geom[e], plan.entry(b, e)
            d = own_plan.planes[g1.plane]
            src = D.plane_view(own, d, b * own_plan.image_elems)[:, g1.y:g1.y + g1.rh, g1.x:g1.x + g1.rw]
            dst = pk[gb.plane][:, gb.y:gb.y + gb.rh, gb.x:gb.x + gb.rw]
            assert torch.equal(src, dst), (b, e)
            covered[gb.plane, gb.y:gb.y + gb.rh, gb.x:gb.x + gb.rw] = True
    for j in range(88):
        assert not pk[j][:, ~covered[j]].any()


def _sub_plan(pb, j):
    """The rows of a packed plan that sit on plane j, as a one-plane oracle plan."""
    rows = pb.gi[:, 3] == j
    gi = pb.gi[rows].copy()
    gi[:, 3] = 0
    return oracle.Plan(gi, pb.gd[rows].copy(), 1, pb.pad, [pb.plane_sizes[j]], pb.n_aspects, pb.n_img, True)


def test_packed_batch16_conv5_sampled_planes(D):
    """The benchmark's batch packed: conv1..conv5 over all 88 planes in one call, the first, a middle
    and the last (least full) plane checked against the oracle."""
    w = C.XGA_25SCALE_B16
    imgs_np = synth.images(w.seeds, w.H, w.W)
    pyra = D.convnet_featpyramid_batch(torch.from_numpy(imgs_np).cuda(), D.params_for(w),
                                       packed(D, "bf16"), DTS["bf16"])
    torch.cuda.synchronize()
    pb = oplan_batch(16, w)
    maps = pyra.conv.conv5_maps()
    assert len(maps) == 88
    for j in (0, 47, 87):
        plane = oracle.build_planes(imgs_np, _sub_plan(pb, j), w.pad_mode, w.mean)[0]
        c5 = oracle.net(plane.astype(np.float32), W7)
        assert_layer_close(chw(maps[j].float().cpu().numpy()), c5, "bf16", f"packed plane {j}")
    # per-(image, entry) feature maps are the conv5 windows of the batch plan
    for row, f in enumerate(pyra.feat):
        g = pb.gi[row]
        assert tuple(f.shape) == (g[9] - g[8] + 1, g[11] - g[10] + 1, 256)


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("pooled", [False, True])
def test_packed_region_reads_on_shared_maps(D, dt, pooled):
    """Same seeded conv5 maps on both sides: entries and indices bit for bit; bilinear values to fp32
    rounding, pooled values exact."""
    n_img, w = 16, C.XGA_25SCALE_B16
    pb = oplan_batch(n_img, w)
    plan = D.BatchPlan(n_img, w.H, w.W, D.params_for(w))
    Hc = oracle.conv5_side(1200)
    rng = np.random.default_rng(23)
    maps = [round_to(rng.normal(0, 1, (256, Hc, Hc)), dt) for _ in range(pb.n_planes)]
    boxes = synth.boxes(77, 3000, w.H, w.W)
    extra = np.array([[5, 5, 5, 40], [np.nan, 1, 2, 3], [0, 0, w.W, w.H], [10, 10, 11, 11]], np.float32)
    boxes = np.concatenate([boxes, extra])
    box_img = (np.arange(len(boxes)) * 7 % n_img).astype(np.int32)
    fn = oracle.region_pool if pooled else oracle.region_windows
    ref = fn(maps, pb, boxes, box_img=box_img)
    flat = np.concatenate([np.moveaxis(m, 0, -1).ravel() for m in maps])
    c5 = torch.from_numpy(flat).to("cuda", TORCH_DT[dt])
    descs = []
    for j in range(pb.n_planes):
        d = D.dn_plane_desc()
        d.h, d.w, d.offset = Hc, Hc, j * Hc * Hc * 256
        descs.append(d)
    out, sc, ix = D.densenet_region_windows_batch(c5, descs, DTS[dt], plan, torch.from_numpy(boxes).cuda(),
                                                  torch.from_numpy(box_img).cuda(), pooled=pooled,
                                                  want_idx=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sc.cpu().numpy(), ref[1])
    np.testing.assert_array_equal(ix.cpu().numpy(), ref[2])
    got = out.cpu().numpy()
    if pooled:
        np.testing.assert_array_equal(got, ref[0])
    else:
        np.testing.assert_allclose(got, ref[0], rtol=2e-6, atol=2e-6)
    assert ref[1][-3] == -1 and ref[1][-4] == -1 and not got[-3].any()


def test_packed_end_to_end_small(D):
    """Images -> packed planes -> conv stack -> region windows, all on the GPU, against the oracle's
    same steps (f16)."""
    n_img, w = SMALL[1]
    imgs = synth.images(w.seeds, w.H, w.W)
    pyra = D.convnet_featpyramid_batch(torch.from_numpy(imgs).cuda(), D.params_for(w), packed(D, "f16"),
                                       DTS["f16"])
    boxes = synth.boxes(31, 500, w.H, w.W)
    box_img = (np.arange(500) % n_img).astype(np.int32)
    out, sc, ix = D.densenet_region_windows_batch(pyra.conv.conv5, list(pyra.conv.c5d), DTS["f16"], pyra.plan,
                                                  torch.from_numpy(boxes).cuda(),
                                                  torch.from_numpy(box_img).cuda(), want_idx=True)
    torch.cuda.synchronize()
    pb = oplan_batch(n_img, w)
    planes = oracle.build_planes(imgs, pb, w.pad_mode, w.mean)
    c5 = [oracle.net(p.astype(np.float32), W7) for p in planes]
    maps = pyra.conv.conv5_maps()
    for j in range(pb.n_planes):
        assert_layer_close(chw(maps[j].float().cpu().numpy()), c5[j], "f16", f"plane {j}")
    desc, scale, idx, _ = oracle.region_windows(c5, pb, boxes, box_img=box_img)
    np.testing.assert_array_equal(sc.cpu().numpy(), scale)
    np.testing.assert_array_equal(ix.cpu().numpy(), idx)
    assert_layer_close(out.cpu().numpy(), desc, "f16", "packed region descriptors")
