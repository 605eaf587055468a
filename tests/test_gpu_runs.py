"""GPU: one launch per layer over planes of several sizes (Sec. 3.1 per-scale planes, several images).
The planes of three images' 8-scale pyramids, image-major, form 24 runs of one plane each, so every
layer takes two launches of a run table (16 + 8 runs); each plane's conv5 and pool5 maps must equal,
bit for bit (fp32: to 1e-5, as fp32 launches too small to fill the GPU split their sums, in an order
that depends on the launch), the maps of that plane run through the stack on its own.  All storage
types and both LRN orders; the workspace the call asks for is checked against the sum of the runs'
layer maps."""
import numpy as np
import pytest

from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import synth

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


def pyramid(D, dt, n_img, H, W):
    """n_img images, 8 scales at 2^-0.25 from longest side 512, each scale its own plane."""
    w = C.Workload("runs", H, W, tuple(300 + i for i in range(n_img)), 8, 4, base_longest_side=512,
                   pad=16, pad_mode=0)
    imgs = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).cuda()
    planes, plan = D.densenet_build_pyramid(imgs, D.params_for(w), DTS[dt])
    return planes, plan.image_descs(n_img)


@pytest.mark.parametrize("dt,lrn_first", [("f32", True), ("f16", True), ("bf16", True), ("f16", False)])
def test_mixed_sizes_one_launch_per_layer(D, dt, lrn_first):
    planes, descs = pyramid(D, dt, 3, 240, 320)
    assert len(descs) == 24 and len({(d.h, d.w) for d in descs}) == 8
    net = D.net_params(pool5=True, lrn_before_pool=lrn_first)
    cf = D.ConvFeatures(descs, DTS[dt], net, device="cuda")
    cf(planes, packed(D, dt))
    torch.cuda.synchronize()
    # workspace: two ping-pong buffers each holding a layer's maps of all runs back to back (fp32:
    # plus the partial sums of launches that split their input channels)
    es = 4 if dt == "f32" else 2
    hw = [D.layer_sizes(d.h, d.w) for d in descs]
    a = max(sum(c * h[i][0] * h[i][1] for h in hw) for c, i in ((96, 0), (256, 2), (384, 4)))
    b = max(sum(c * h[i][0] * h[i][1] for h in hw) for c, i in ((96, 1), (256, 3), (384, 5)))
    ab = (a * es + 255) // 256 * 256 + (b * es + 255) // 256 * 256
    if dt == "f32":
        assert cf.workspace.numel() >= ab
    else:
        assert cf.workspace.numel() == ab
    c5, p5 = cf.conv5_maps(), cf.pool5_maps()
    for i, d in enumerate(descs):
        one = D.ConvFeatures([d], DTS[dt], net, device="cuda")
        one(planes, packed(D, dt))
        torch.cuda.synchronize()
        if dt == "f32":
            # fp32 launches too small to fill the GPU split their input channels, and how many
            # splits a plane gets depends on the launch it is in: sums in another order
            for g, r, what in ((one.conv5_maps()[0], c5[i], "conv5"), (one.pool5_maps()[0], p5[i], "pool5")):
                assert torch.allclose(g, r, rtol=1e-5, atol=1e-5 * float(r.abs().max())), \
                    f"plane {i} ({d.h}x{d.w}) {what}"
        else:
            assert torch.equal(one.conv5_maps()[0], c5[i]), f"plane {i} ({d.h}x{d.w}) conv5"
            assert torch.equal(one.pool5_maps()[0], p5[i]), f"plane {i} ({d.h}x{d.w}) pool5"
        assert torch.isfinite(c5[i].float()).all() and c5[i].float().abs().max() > 0


def test_fp32_split_launches_match_layer_by_layer(D):
    """The 227 x 227 pyramid in fp32 (Sec. 3.1, one plane per scale): densenet_conv_features splits
    its small conv2-5 launches over input-channel copies (the workspace holds their partial sums);
    the same planes through densenet_conv_layer / densenet_lrn_pool / densenet_maxpool, which never
    split, must agree to 1e-5."""
    w = C.ALEXNET_227
    f32 = DTS["f32"]
    img = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).cuda()
    planes, plan = D.densenet_build_pyramid(img, D.params_for(w), f32)
    net = D.net_params(pool5=True)
    pk = packed(D, "f32")
    for d in plan.planes:
        cf = D.ConvFeatures([d], f32, net, device="cuda")
        hw = D.layer_sizes(d.h, d.w)
        ab = sum((max(c * hw[i][0] * hw[i][1] for c, i in pairs) * 4 + 255) // 256 * 256
                 for pairs in (((96, 0), (256, 2), (384, 4)), ((96, 1), (256, 3), (384, 5))))
        assert cf.workspace.numel() > ab, "the small fp32 launches should take partial-sum space"
        cf(planes, pk)
        x = D.plane_view(planes, d).contiguous().unsqueeze(0)
        a = D.densenet_conv_layer(1, x, 1, d.h, d.w, f32, pk)
        a = D.densenet_lrn_pool(a, f32, net)
        for layer in (2, 3, 4, 5):
            a = D.densenet_conv_layer(layer, a, 1, a.shape[1], a.shape[2], f32, pk)
            if layer == 2:
                a = D.densenet_lrn_pool(a, f32, net)
        p5 = D.densenet_maxpool(a, f32)
        torch.cuda.synchronize()
        for got, ref, what in ((cf.conv5_maps()[0], a[0], "conv5"), (cf.pool5_maps()[0], p5[0], "pool5")):
            assert got.shape == ref.shape
            assert torch.allclose(got, ref, rtol=1e-5, atol=1e-5 * float(ref.abs().max())), (d.h, what)
            assert float(ref.abs().max()) > 0


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_large_runs_share_batch_kernels(D, dt):
    """Two runs large enough for the batch configurations (16 planes of 1200 x 1200, 8 of 1000 x 1000,
    each run at its own pitch): one call launches conv1-5 and the lrn_pool2 strip kernel with a
    two-entry run table; each run through the stack alone (single-run kernels, and for the smaller run
    the per-pixel LRN kernel, which computes the same values) must give the same maps bit for bit."""
    runs = [(16, 1200, 1216), (8, 1000, 1024)]
    descs, off = [], 0
    for n, side, pitch in runs:
        for _ in range(n):
            q = D.dn_plane_desc()
            q.h, q.w, q.pitch, q.offset = side, side, pitch, off
            descs.append(q)
            off += 3 * side * pitch
    g = torch.Generator(device="cuda").manual_seed(11)
    planes = (torch.rand(off, generator=g, device="cuda") * 200 - 100).to(
        {"bf16": torch.bfloat16, "f16": torch.float16}[dt])
    net = D.net_params()
    both = D.ConvFeatures(descs, DTS[dt], net, device="cuda")
    both(planes, packed(D, dt))
    first, i0 = [], 0
    for n, _, _ in runs:
        one = D.ConvFeatures(descs[i0:i0 + n], DTS[dt], net, device="cuda")
        one(planes, packed(D, dt))
        first += [m.clone() for m in one.conv5_maps()]
        i0 += n
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(both.conv5_maps(), first)):
        assert torch.equal(a, b), f"plane {i}"
    assert float(first[0].float().abs().max()) > 0


@pytest.mark.parametrize("wname,dt", [("ALEXNET_227", "f32"), ("VGA_8SCALE", "f16")])
def test_graph_replay_per_scale_planes(D, wname, dt):
    """Per-scale planes (Sec. 3.1 without stitching) captured once into a graph and replayed several
    times with eager work in between: the multi-run launches, and for the 227 x 227 fp32 pyramid the
    split launches with their partial sums and reductions, reproduce the eager conv5 (and pool5) maps
    bit for bit on every replay (the workspace's partial sums are rewritten in full each time)."""
    w = getattr(C, wname)
    img = torch.from_numpy(synth.images(w.seeds, w.H, w.W)).cuda()
    params = D.params_for(w)
    planes, plan = D.densenet_build_pyramid(img, params, DTS[dt])
    cf = D.ConvFeatures(list(plan.planes), DTS[dt], D.net_params(pool5=w.pool5), device="cuda")

    def pyramid():
        D.densenet_build_pyramid(img, params, DTS[dt], out=planes)
        cf(planes, packed(D, dt))

    pyramid()
    torch.cuda.synchronize()
    ref_c5 = cf.conv5.clone()
    ref_p5 = cf.pool5.clone() if cf.pool5 is not None else None
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pyramid()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pyramid()
    other = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        cf.conv5.zero_()
        cf.workspace.fill_(0xFF)           # stale partial sums and maps would show
        if ref_p5 is not None:
            cf.pool5.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(cf.conv5, ref_c5), f"replay {rep}: conv5"
        if ref_p5 is not None:
            assert torch.equal(cf.pool5, ref_p5), f"replay {rep}: pool5"
        other.add_(1)                       # eager work between replays
        torch.cuda.synchronize()
