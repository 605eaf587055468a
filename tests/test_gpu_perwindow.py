"""GPU parity of the per-window baseline (Sec. 3.4: every proposal run through the network on its own;
Sec. 4: crop before), through the C ABI against the oracle on the same seeded inputs: the crop-before
warp of every box (taps bit for bit, values to the plane bars), and per-window pool5 descriptors end to
end, including the 2000-box launch configuration the benchmark times (sampled windows)."""
import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import synth
from tests.parity import BARS, plane_tol, assert_layer_close, hwc, ulp

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DTS = {"f32": 0, "f16": 1, "bf16": 2}
W7 = synth.weights(7)
WL = C.XGA_25SCALE
MEAN = synth.IMAGENET_MEAN


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


def special_boxes(H, W):
    """Degenerate, partly outside, sub-pixel, whole-image and non-finite boxes."""
    return np.array([[10, 10, 10, 50], [40, 30, 20, 60], [np.inf, 0, 5, 5], [0, 0, W, H],
                     [-30.5, -12.25, 100.75, 90.5], [W - 40, H - 25, W + 60, H + 35],
                     [100.3, 200.7, 100.9, 201.1], [3.5, 700.25, 1020.75, 767.5]], np.float32)


def check_windows(got, ref, dt):
    got = got.float().cpu().numpy().astype(np.float64)
    ref = ref.astype(np.float64)
    assert np.all(np.abs(got - ref) <= plane_tol(ref, dt))


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("S", [227, 13, 1])
def test_warp_regions(D, dt, S):
    imgs = synth.images((103, 104), WL.H, WL.W)
    boxes = np.concatenate([synth.boxes(105, 300, WL.H, WL.W), special_boxes(WL.H, WL.W)])
    bimg = (np.arange(len(boxes)) % 2).astype(np.int32)
    bimg[-1] = 5  # image index out of range: zero window
    got = D.densenet_warp_regions(torch.from_numpy(imgs).cuda(), torch.from_numpy(boxes).cuda(), DTS[dt],
                                  S, MEAN, torch.from_numpy(bimg).cuda())
    ref = oracle.warp_regions(imgs, boxes, S, MEAN, box_img=np.where(bimg < 2, bimg, 99))
    check_windows(got, ref, dt)
    assert not got[-1].any() and not got[len(boxes) - 8].any() and not got[len(boxes) - 6].any()


def test_warp_regions_no_box_img_and_odd_image(D):
    img = synth.image(7, 97, 131)
    boxes = np.concatenate([synth.boxes(8, 50, 97, 131, smin=4, smax=90), special_boxes(97, 131)])
    got = D.densenet_warp_regions(torch.from_numpy(img).cuda(), torch.from_numpy(boxes).cuda(), DTS["f32"],
                                  33, MEAN)
    check_windows(got, oracle.warp_regions(img, boxes, 33, MEAN), "f32")


_oracle_desc = {}


def oracle_pool5(imgs, boxes, bimg, i):
    key = (id(imgs), tuple(float(v) for v in boxes[i]), int(bimg[i]))
    if key not in _oracle_desc:
        win = oracle.warp_regions(imgs, boxes[i:i + 1], 227, MEAN, box_img=bimg[i:i + 1])[0]
        _oracle_desc[key] = oracle.net(win, W7, pool5=True)[1]
    return _oracle_desc[key]


IMGS = synth.images((103,), WL.H, WL.W)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_per_window_descriptors(D, dt):
    boxes = np.concatenate([synth.boxes(105, 5, WL.H, WL.W), special_boxes(WL.H, WL.W)[[0, 4]]])
    bimg = np.zeros(len(boxes), np.int32)
    pw = D.PerWindow(len(boxes), DTS[dt])
    p5 = pw(torch.from_numpy(IMGS).cuda(), torch.from_numpy(boxes).cuda(), packed(D, dt), MEAN)
    assert tuple(p5.shape) == (len(boxes), 6, 6, 256)
    got = p5.float().cpu().numpy()
    for i in range(len(boxes)):
        ref = oracle_pool5(IMGS, boxes, bimg, i)
        assert_layer_close(np.moveaxis(got[i], -1, 0), ref, dt, f"per-window pool5 box {i}")


def test_per_window_2000_boxes_sampled(D):
    """The benchmark's launch configuration: 2000 boxes of one 768 x 1024 image, bf16, one launch per
    layer over all windows; sampled windows against the oracle, and run-to-run determinism."""
    boxes = synth.boxes(105, 2000, WL.H, WL.W)
    boxes[1234] = (50, 50, 50, 90)  # a degenerate box inside the batch: the window is all zeros
    bimg = np.zeros(len(boxes), np.int32)
    pw = D.PerWindow(len(boxes), DTS["bf16"])
    x, b = torch.from_numpy(IMGS).cuda(), torch.from_numpy(boxes).cuda()
    p5 = pw(x, b, packed(D, "bf16"), MEAN).clone()
    p5b = pw(x, b, packed(D, "bf16"), MEAN)
    assert torch.equal(p5, p5b)
    got = p5.float().cpu().numpy()
    for i in (0, 999, 1234, 1999):
        ref = oracle_pool5(IMGS, boxes, bimg, i)
        assert_layer_close(np.moveaxis(got[i], -1, 0), ref, "bf16", f"per-window pool5 box {i}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_warp_regions_row_pitch(D, dt):
    boxes = np.concatenate([synth.boxes(106, 40, WL.H, WL.W), special_boxes(WL.H, WL.W)])
    x, b = torch.from_numpy(IMGS).cuda(), torch.from_numpy(boxes).cuda()
    got = D.densenet_warp_regions(x, b, DTS[dt], 227, MEAN, pitch=232)
    assert tuple(got.shape) == (len(boxes), 3, 227, 232)
    check_windows(got[..., :227], oracle.warp_regions(IMGS, boxes, 227, MEAN), dt)
    assert not got[..., 227:].any()


def test_conv_features_row_pitch_matches_packed_rows(D):
    """The same windows as pitch-232 planes (conv1 loads rows straight into LDS) and as packed 227-wide
    planes (register-staged conv1) give the same pool5 descriptors, up to the order of conv1's fp32
    accumulation (the two kernels group the 363 taps into MFMA k-steps differently): a wrong row pitch
    or padding read would differ by far more."""
    boxes = synth.boxes(107, 24, WL.H, WL.W)
    x, b = torch.from_numpy(IMGS).cuda(), torch.from_numpy(boxes).cuda()
    pk = packed(D, "bf16")
    a = D.PerWindow(len(boxes), DTS["bf16"])(x, b, pk, MEAN).float()
    win = D.densenet_warp_regions(x, b, DTS["bf16"], 227, MEAN)
    desc = []
    for i in range(len(boxes)):
        q = D.dn_plane_desc()
        q.h, q.w, q.offset = 227, 227, i * 3 * 227 * 227
        desc.append(q)
    cf = D.densenet_conv_features(win, desc, DTS["bf16"], pk, D.net_params(pool5=True))
    c = torch.stack([m.float() for m in cf.pool5_maps()])
    d = (a - c).abs()
    rms = c.pow(2).mean().sqrt()
    # the bf16 layer bar (a one-ulp difference at the largest values is ~0.05 rms), and most equal
    assert torch.isfinite(a).all() and d.max() <= BARS["bf16"] * rms, (d.max().item(), rms.item())
    assert (d > 0).float().mean() < 0.1
