"""Guard bands around every output buffer of the path: each buffer the library writes (planes and the
builder's scratch, the conv workspace, conv5, pool5, region descriptors, scales and sample indices,
crop-before windows, single-layer outputs) is placed between two 4 KB bands filled with a sentinel
byte, and the bands are checked after the stream has finished.  A kernel that writes past the end or
before the start of its buffer changes a band.  The guarded run must also equal an unguarded run of
the same call bit for bit (deterministic kernels), so the bands do not hide a short write."""
import ctypes

import numpy as np
import pytest

from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DTS = {"f32": 0, "f16": 1, "bf16": 2}
TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
GUARD_BYTES = 4096      # a multiple of 256, so the guarded buffer keeps the allocator's alignment
SENTINEL = 0xA5
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


class Guarded:
    """A flat device buffer of `numel` elements between two sentinel bands."""

    def __init__(self, numel, dtype):
        es = torch.empty(0, dtype=dtype).element_size()
        self.g = GUARD_BYTES // es
        self.numel, self.es = numel, es
        self.full = torch.empty(numel + 2 * self.g, dtype=dtype, device="cuda")
        self.full.view(torch.uint8).fill_(SENTINEL)
        self.view = self.full[self.g:self.g + numel]

    def check(self, what):
        torch.cuda.synchronize()
        b = self.full.view(torch.uint8)
        head = b[:GUARD_BYTES]
        tail = b[(self.g + self.numel) * self.es:]
        assert bool(torch.all(head == SENTINEL)), f"{what}: bytes before the buffer were written"
        assert bool(torch.all(tail == SENTINEL)), f"{what}: bytes after the buffer were written"


def guard_like(t):
    g = Guarded(t.numel(), t.dtype)
    return g, g.view.view(t.shape)


def guard_conv(cf):
    """Swap a ConvFeatures' workspace, conv5 and pool5 for guarded buffers of the same sizes."""
    guards = {}
    for name in ("workspace", "conv5", "pool5"):
        t = getattr(cf, name)
        if t is None:
            continue
        g, v = guard_like(t)
        setattr(cf, name, v)
        guards[name] = g
    return guards


@pytest.mark.parametrize("w,dt,n_img", [(C.XGA_25SCALE, "f16", 2), (C.VGA_8SCALE, "f32", 1),
                                        (C.VGA_8SCALE, "f16", 1), (C.ALEXNET_227, "f32", 1)],
                         ids=lambda v: getattr(v, "name", v))
def test_guarded_pyramid_conv_and_regions(D, w, dt, n_img):
    imgs = torch.from_numpy(synth.images(tuple(w.seeds[0] + i for i in range(n_img)), w.H, w.W)).cuda()
    params = D.params_for(w)
    ref_planes, plan = D.densenet_build_pyramid(imgs, params, DTS[dt])
    gp, planes = guard_like(ref_planes)
    D.densenet_build_pyramid(imgs, params, DTS[dt], out=planes)
    gp.check("planes + builder scratch")
    pix = n_img * plan.image_elems
    assert torch.equal(planes[:pix], ref_planes[:pix])

    desc = plan.image_descs(n_img)
    net = D.net_params(pool5=True)
    ref_cf = D.ConvFeatures(desc, DTS[dt], net)
    ref_cf(ref_planes, packed(D, dt))
    cf = D.ConvFeatures(desc, DTS[dt], net)
    guards = guard_conv(cf)
    cf(planes, packed(D, dt))
    for name, g in guards.items():
        g.check(name)
    assert torch.equal(cf.conv5, ref_cf.conv5) and torch.equal(cf.pool5, ref_cf.pool5)

    n_boxes = 300
    boxes = np.concatenate([synth.boxes(105 + b, n_boxes, w.H, w.W) for b in range(n_img)])
    bx = torch.from_numpy(boxes).cuda()
    box_img = torch.arange(n_img, dtype=torch.int32, device="cuda").repeat_interleave(n_boxes)
    ppi = len(plan.planes)
    for fn, width in ((D.densenet_region_windows, 2), (D.densenet_region_pool, 4)):
        ro, rs, ri = fn(cf.conv5, list(cf.c5d), DTS[dt], plan, w.pad, ppi, bx, box_img, want_idx=True)
        go, out = guard_like(ro)
        gs, scale = guard_like(rs)
        n = boxes.shape[0]
        gi = Guarded(n * 36 * width, torch.int32)
        idx = gi.view.view(n, 6, 6, width)
        # the binding allocates idx itself; call the library directly with the guarded one
        geom = (D.dn_scale_geom * len(plan.geom))(*plan.geom)
        cd = (D.dn_plane_desc * len(cf.c5d))(*cf.c5d)
        lib_fn = D.lib().densenet_region_windows if width == 2 else D.lib().densenet_region_pool
        D.check(lib_fn(D._ptr(cf.conv5), cd, len(cd), DTS[dt], geom, len(geom), w.pad, ppi, D._ptr(bx),
                       D._ptr(box_img), n, 227.0, 6, D._ptr(out), D._ptr(scale), D._ptr(idx),
                       D._stream()))
        go.check("region descriptors")
        gs.check("region scales")
        gi.check("region indices")
        assert torch.equal(out, ro) and torch.equal(scale, rs) and torch.equal(idx, ri)


def test_guarded_packed_batch(D):
    w = C.XGA_25SCALE_B16
    n_img = 4
    imgs = torch.from_numpy(synth.images(w.seeds[:n_img], w.H, w.W)).cuda()
    plan = D.BatchPlan(n_img, w.H, w.W, D.params_for(w))
    ref = D.densenet_build_batch(imgs, plan, DTS["bf16"])
    g, planes = guard_like(ref)
    D.densenet_build_batch(imgs, plan, DTS["bf16"], out=planes)
    g.check("packed planes + scratch")
    pix = plan.total_elems
    assert torch.equal(planes[:pix], ref[:pix])
    cf = D.ConvFeatures(plan.planes, DTS["bf16"], D.net_params())
    guards = guard_conv(cf)
    cf(planes, packed(D, "bf16"))
    for name, gg in guards.items():
        gg.check(name)
    boxes = np.concatenate([synth.boxes(105 + b, 200, w.H, w.W) for b in range(n_img)])
    bx = torch.from_numpy(boxes).cuda()
    box_img = torch.arange(n_img, dtype=torch.int32, device="cuda").repeat_interleave(200)
    for pooled in (False, True):
        ro, rs, _ = D.densenet_region_windows_batch(cf.conv5, list(cf.c5d), DTS["bf16"], plan, bx,
                                                    box_img, pooled=pooled)
        go, out = guard_like(ro)
        gs, scale = guard_like(rs)
        D.densenet_region_windows_batch(cf.conv5, list(cf.c5d), DTS["bf16"], plan, bx, box_img,
                                        pooled=pooled, out=out, scale=scale)
        go.check("packed region descriptors")
        gs.check("packed region scales")
        assert torch.equal(out, ro) and torch.equal(scale, rs)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_guarded_per_window(D, dt):
    w = C.XGA_25SCALE
    img = torch.from_numpy(synth.image(w.seeds[0], w.H, w.W)).cuda()
    boxes = torch.from_numpy(synth.boxes(105, 64, w.H, w.W)).cuda()
    pw = D.PerWindow(64, DTS[dt], 227)
    ref = pw(img, boxes, packed(D, dt), w.mean).clone()
    gw, win = guard_like(pw.windows)
    D.densenet_warp_regions(img, boxes, DTS[dt], 227, w.mean, out=win, pitch=pw.pitch)
    gw.check("crop-before windows")
    assert torch.equal(win, pw.windows)
    guards = guard_conv(pw.conv)
    got = pw(img, boxes, packed(D, dt), w.mean)
    for name, g in guards.items():
        g.check(f"per-window {name}")
    assert torch.equal(got, ref)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_guarded_single_layers(D, dt):
    rng = np.random.default_rng(3)
    n, H, W = 2, 83, 120
    x = torch.from_numpy(rng.normal(0, 50, (n, 3, H, W)).astype(np.float32)).to("cuda", TORCH_DT[dt])
    c1 = D.densenet_conv_layer(1, x, n, H, W, DTS[dt], packed(D, dt))
    Ho, Wo = c1.shape[1:3]
    sizes = {2: (96, 256), 3: (256, 384), 4: (384, 384), 5: (384, 256)}
    for layer in (1, 2, 3, 4, 5):
        if layer == 1:
            inp, h, wd, M = x, H, W, 96
            oh, ow = Ho, Wo
        else:
            Cin, M = sizes[layer]
            inp = torch.relu(torch.from_numpy(rng.normal(0, 3, (n, 19, 23, Cin)).astype(np.float32))).to(
                "cuda", TORCH_DT[dt])
            h, wd, oh, ow = 19, 23, 19, 23
        ref = D.densenet_conv_layer(layer, inp, n, h, wd, DTS[dt], packed(D, dt))
        g = Guarded(n * oh * ow * M, TORCH_DT[dt])
        D.check(D.lib().densenet_conv_layer(layer, D._ptr(inp), n, h, wd, DTS[dt], D._ptr(packed(D, dt)),
                                            D._ptr(g.view), D._stream()))
        g.check(f"conv{layer}")
        assert torch.equal(g.view.view(ref.shape), ref)
    for C_ in (96, 256):
        inp = torch.relu(torch.from_numpy(rng.normal(0, 30, (n, 27, 26, C_)).astype(np.float32))).to(
            "cuda", TORCH_DT[dt])
        for lrn_first in (True, False):
            ref = D.densenet_lrn_pool(inp, DTS[dt], D.net_params(lrn_before_pool=lrn_first))
            g = Guarded(ref.numel(), TORCH_DT[dt])
            D.check(D.lib().densenet_lrn_pool(D._ptr(inp), n, 27, 26, C_, DTS[dt],
                                              ctypes.byref(D.net_params(lrn_before_pool=lrn_first)),
                                              D._ptr(g.view), D._stream()))
            g.check(f"lrn_pool C={C_}")
            assert torch.equal(g.view.view(ref.shape), ref)
        ref = D.densenet_maxpool(inp, DTS[dt])
        g = Guarded(ref.numel(), TORCH_DT[dt])
        D.check(D.lib().densenet_maxpool(D._ptr(inp), n, 27, 26, C_, DTS[dt], D._ptr(g.view), D._stream()))
        g.check(f"maxpool C={C_}")
        assert torch.equal(g.view.view(ref.shape), ref)
