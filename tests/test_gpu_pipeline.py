"""GPU parity of the whole path through the C ABI, against the oracle on the same seeded inputs:
planes (fused resize/centre/pad/stitch), the conv stack end to end on every workload (full size; the
batch of 16 checked on every plane of its first and last image, in the launch configuration the
benchmark times), and region windows (scales and sample indices bit for bit)."""
import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import configs as C
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


def oplan(w):
    return oracle.plan(w.H, w.W, w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side,
                       w.pad, w.plane_h, w.plane_w)


_oracle_cache = {}


def oracle_pyramid(w, img_index=0, planes=None):
    """Oracle planes (fp64) and conv5 maps (fp32, [256][Hc][Wc]) of one image of a workload."""
    key = (w.name, img_index, tuple(planes) if planes else None)
    if key not in _oracle_cache:
        img = synth.image(w.seeds[img_index], w.H, w.W)
        p = oplan(w)
        pl = oracle.build_planes(img, p, w.pad_mode, w.mean)
        idx = planes if planes is not None else range(p.n_planes)
        c5 = {}
        p5 = {}
        for j in idx:
            r = oracle.net(pl[j].astype(np.float32), W7, pool5=w.pool5)
            if w.pool5:
                c5[j], p5[j] = r
            else:
                c5[j] = r
        _oracle_cache[key] = (p, pl, c5, p5)
    return _oracle_cache[key]


def gpu_planes(D, w, dt, imgs):
    x = torch.from_numpy(imgs).cuda()
    planes, plan = D.densenet_build_pyramid(x, D.params_for(w), DTS[dt])
    return planes, plan


def plane_views(D, planes, plan, b):
    out = []
    for d in plan.planes:
        out.append(D.plane_view(planes, d, b * plan.image_elems))
    return out


def check_planes(got, ref, dt):
    got = got.float().cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= plane_tol(ref, dt))


@pytest.mark.parametrize("w,dt", [(C.ALEXNET_227, "f32"), (C.VGA_8SCALE, "f32"), (C.VGA_8SCALE, "f16"),
                                  (C.XGA_25SCALE, "f16"), (C.XGA_25SCALE, "bf16")],
                         ids=lambda v: getattr(v, "name", v))
def test_planes(D, w, dt):
    img = synth.image(w.seeds[0], w.H, w.W)
    planes, plan = gpu_planes(D, w, dt, img[None])
    p = oplan(w)
    ref = oracle.build_planes(img, p, w.pad_mode, w.mean)
    assert len(plan.planes) == p.n_planes
    for j, v in enumerate(plane_views(D, planes, plan, 0)):
        check_planes(v, ref[j], dt)


def test_planes_batch_first_and_last(D):
    w = C.XGA_25SCALE_B16
    imgs = synth.images(w.seeds, w.H, w.W)
    planes, plan = gpu_planes(D, w, "bf16", imgs)
    p = oplan(w)
    for b in (0, 15):
        ref = oracle.build_planes(imgs[b], p, w.pad_mode, w.mean)
        for j, v in enumerate(plane_views(D, planes, plan, b)):
            check_planes(v, ref[j], "bf16")


def run_gpu(D, w, dt, imgs, pool5=False):
    x = torch.from_numpy(imgs).cuda()
    pyra = D.convnet_featpyramid(x, D.params_for(w), packed(D, dt), DTS[dt],
                                 D.net_params(pool5=pool5))
    return pyra


@pytest.mark.parametrize("w,dt", [(C.ALEXNET_227, "f32"), (C.VGA_8SCALE, "f32"), (C.VGA_8SCALE, "f16")],
                         ids=lambda v: getattr(v, "name", v))
def test_end_to_end_per_scale_planes(D, w, dt):
    img = synth.image(w.seeds[0], w.H, w.W)
    pyra = run_gpu(D, w, dt, img[None], pool5=w.pool5)
    torch.cuda.synchronize()
    p, _, c5, p5 = oracle_pyramid(w)
    maps = pyra.conv.conv5_maps()
    for j in range(p.n_planes):
        assert_layer_close(chw(maps[j].float().cpu().numpy()), c5[j], dt, f"{w.name} plane {j} conv5")
    if w.pool5:
        pm = pyra.conv.pool5_maps()
        for j in range(p.n_planes):
            assert_layer_close(chw(pm[j].float().cpu().numpy()), p5[j], dt, f"{w.name} plane {j} pool5")
        assert pm[0].shape == (6, 6, 256)          # the classic 9216-d pool5 of a 227 input
    # per-scale feature maps are the conv5 windows of the plan
    for k, f in enumerate(pyra.feat):
        g = p.gi[k]
        assert tuple(f.shape) == (g[9] - g[8] + 1, g[11] - g[10] + 1, 256)


def test_end_to_end_stitched_f16(D):
    w = C.XGA_25SCALE
    img = synth.image(w.seeds[0], w.H, w.W)
    pyra = run_gpu(D, w, "f16", img[None])
    torch.cuda.synchronize()
    p, _, c5, _ = oracle_pyramid(w)
    maps = pyra.conv.conv5_maps()
    assert len(maps) == 6
    for j in range(6):
        assert_layer_close(chw(maps[j].float().cpu().numpy()), c5[j], "f16", f"xga plane {j}")


def test_end_to_end_batch16_bf16_first_and_last_image(D):
    """The benchmark's launch configuration (96 planes in one launch per layer): every plane of the
    batch's first and last image against the oracle."""
    w = C.XGA_25SCALE_B16
    imgs = synth.images(w.seeds, w.H, w.W)
    pyra = run_gpu(D, w, "bf16", imgs)
    torch.cuda.synchronize()
    maps = pyra.conv.conv5_maps()
    assert len(maps) == 96
    for b in (0, 15):
        p, _, c5, _ = oracle_pyramid(w, b)
        for j in range(6):
            assert_layer_close(chw(maps[b * 6 + j].float().cpu().numpy()), c5[j], "bf16",
                               f"batch image {b} plane {j}")
    # run-to-run determinism of the whole batch
    first = pyra.conv.conv5.clone()
    pyra.conv(pyra.planes, packed(D, "bf16"))
    torch.cuda.synchronize()
    assert torch.equal(first, pyra.conv.conv5)


def _maps_for_regions(p, seed):
    rng = np.random.default_rng(seed)
    return [rng.normal(0, 1, (256, oracle.conv5_side(h), oracle.conv5_side(wd))).astype(np.float32)
            for h, wd in p.plane_sizes]


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_region_windows_on_shared_maps(D, dt):
    """Same seeded conv5 maps into both sides: scales and indices bit-exact, values to fp32 rounding."""
    w = C.XGA_25SCALE_REGIONS
    p = oplan(w)
    maps = [round_to(m, dt) for m in _maps_for_regions(p, 17)]
    boxes = synth.boxes(w.box_seed, w.n_boxes, w.H, w.W)
    extra = np.array([[5, 5, 5, 40], [np.nan, 1, 2, 3], [0, 0, w.W, w.H], [10, 10, 11, 11]], np.float32)
    boxes = np.concatenate([boxes, extra])
    desc, scale, idx, _ = oracle.region_windows(maps, p, boxes)
    plan = D.densenet_plan_pyramid(w.H, w.W, D.params_for(w))
    flat = np.concatenate([np.moveaxis(m, 0, -1).ravel() for m in maps])
    tdt = {"f32": torch.float32, "f16": torch.float16}[dt]
    c5 = torch.from_numpy(flat).to("cuda", tdt)
    descs = []
    off = 0
    for m in maps:
        d = D.dn_plane_desc()
        d.h, d.w, d.offset = m.shape[1], m.shape[2], off
        off += m.size
        descs.append(d)
    bx = torch.from_numpy(boxes).cuda()
    out, sc, ix = D.densenet_region_windows(c5, descs, DTS[dt], plan, w.pad, p.n_planes, bx,
                                            want_idx=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sc.cpu().numpy(), scale)
    np.testing.assert_array_equal(ix.cpu().numpy(), idx)
    got = out.cpu().numpy()
    np.testing.assert_allclose(got, desc, rtol=2e-6, atol=2e-6)
    assert scale[-4] == -1 and scale[-3] == -1 and not got[-3].any()


def test_region_windows_end_to_end(D):
    w = C.XGA_25SCALE_REGIONS
    img = synth.image(w.seeds[0], w.H, w.W)
    pyra = run_gpu(D, w, "f16", img[None])
    boxes = synth.boxes(w.box_seed, w.n_boxes, w.H, w.W)
    bx = torch.from_numpy(boxes).cuda()
    out, sc, ix = D.densenet_region_windows(pyra.conv.conv5, list(pyra.conv.c5d), DTS["f16"], pyra.plan,
                                            w.pad, len(pyra.plan.planes), bx, want_idx=True)
    torch.cuda.synchronize()
    p, _, c5, _ = oracle_pyramid(C.XGA_25SCALE)
    desc, scale, idx, _ = oracle.region_windows([c5[j] for j in range(p.n_planes)], p, boxes)
    np.testing.assert_array_equal(sc.cpu().numpy(), scale)
    np.testing.assert_array_equal(ix.cpu().numpy(), idx)
    assert out.shape == (2000, 9216)
    assert_layer_close(out.cpu().numpy(), desc, "f16", "region descriptors")


def test_graph_replay_equals_eager(D):
    """The pyramid build and conv stack captured once into a graph (the library allocates nothing and
    issues no memset, so its launches are capturable) and replayed several times, with eager work and
    synchronisations in between: every replay's planes and conv5 maps equal the eager run's bit for
    bit."""
    w = C.XGA_25SCALE
    dt = "f16"
    img = torch.from_numpy(synth.image(w.seeds[0], w.H, w.W)).cuda()[None]
    params = D.params_for(w)
    planes, plan = D.densenet_build_pyramid(img, params, DTS[dt])
    cf = D.ConvFeatures(list(plan.planes), DTS[dt], D.net_params())

    def pyramid():
        D.densenet_build_pyramid(img, params, DTS[dt], out=planes)
        cf(planes, packed(D, dt))

    pyramid()
    torch.cuda.synchronize()
    ref_planes = planes[:plan.image_elems].clone()
    ref_c5 = cf.conv5.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pyramid()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pyramid()
    other = D.densenet_build_pyramid(torch.from_numpy(synth.image(7, w.H, w.W)).cuda()[None], params,
                                     DTS[dt])[0]
    for rep in range(4):
        planes.zero_()
        cf.conv5.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(planes[:plan.image_elems], ref_planes), f"replay {rep}: planes"
        assert torch.equal(cf.conv5, ref_c5), f"replay {rep}: conv5"
        other.add_(1)                      # eager work between replays
        torch.cuda.synchronize()
