"""GPU parity, layer by layer and teacher-forced: each HIP layer kernel, called through the C ABI, is
compared with the oracle on the same (storage-rounded) input, element by element, at sizes that span
several tiles with ragged tails."""
import numpy as np
import pytest

import oracle
from paper_1404_1869_amd import synth
from tests.parity import assert_layer_close, chw, hwc, round_to

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DTS = {"f32": 0, "f16": 1, "bf16": 2}
TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
W7 = synth.weights(7)
LAYERS = [(96, 3, 11, 4, 0, 1), (256, 96, 5, 1, 2, 2), (384, 256, 3, 1, 1, 1), (384, 384, 3, 1, 1, 2),
          (256, 384, 3, 1, 1, 2)]


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


def oracle_weights(dt):
    """Weights as the GPU path holds them: rounded to the storage type."""
    return [(round_to(w, dt), b) for w, b in W7]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
# Widths that are not multiples of 8 take the register-staged kernel, the others the direct-load one
# (16-bit types); 1200 x 1200 is a full stitched plane, and four of them (1444 tiles) give every
# worker of the direct-load kernel several tiles in a row.
@pytest.mark.parametrize("shape", [(2, 227, 227), (1, 300, 263), (1, 83, 51), (2, 232, 240),
                                   (3, 48, 64), (1, 11, 16), (1, 1200, 1200), (4, 1200, 1200)])
def test_conv1(D, dt, shape):
    n, H, W = shape
    rng = np.random.default_rng(H * 7 + W)
    x = round_to(rng.normal(0, 50, (n, 3, H, W)), dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_conv_layer(1, xg, n, H, W, DTS[dt], packed(D, dt)).float().cpu().numpy()
    w, b = oracle_weights(dt)[0]
    for i in range(n):
        ref = oracle.conv2d(x[i], w, b, 4, 0, 1, True)
        assert out[i].shape == hwc(ref).shape
        assert_layer_close(chw(out[i]), ref, dt, f"conv1 {shape}[{i}]")


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("layer,shape", [(2, (2, 37, 45)), (2, (1, 16, 16)), (3, (2, 21, 35)),
                                         (4, (1, 33, 17)), (5, (2, 19, 40)), (3, (1, 74, 74))])
def test_conv_s1(D, dt, layer, shape):
    n, H, W = shape
    M, C, R, s, p, G = LAYERS[layer - 1]
    rng = np.random.default_rng(layer * 1000 + H)
    x = round_to(np.abs(rng.normal(0, 3, (n, H, W, C))), dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_conv_layer(layer, xg, n, H, W, DTS[dt], packed(D, dt)).float().cpu().numpy()
    w, b = oracle_weights(dt)[layer - 1]
    for i in range(n):
        ref = oracle.conv2d(chw(x[i]), w, b, s, p, G, True)
        assert_layer_close(chw(out[i]), ref, dt, f"conv{layer} {shape}[{i}]")


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layer", [3, 4, 5])
def test_conv_s1_many_planes(D, dt, layer):
    """128 planes: enough workgroups for the per-layer configuration of large launches (the small
    launches above take 64-channel sub-blocks); first, middle and last planes against the oracle."""
    n, H, W = 128, 19, 40
    M, C, R, s, p, G = LAYERS[layer - 1]
    rng = np.random.default_rng(layer * 77)
    x = round_to(np.abs(rng.normal(0, 3, (n, H, W, C))), dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_conv_layer(layer, xg, n, H, W, DTS[dt], packed(D, dt)).float().cpu().numpy()
    w, b = oracle_weights(dt)[layer - 1]
    for i in (0, 63, 127):
        ref = oracle.conv2d(chw(x[i]), w, b, s, p, G, True)
        assert_layer_close(chw(out[i]), ref, dt, f"conv{layer} {n} planes [{i}]")


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("C,shape", [(96, (2, 55, 55)), (256, (1, 27, 26)), (96, (1, 298, 31)),
                                     (256, (2, 4, 3))])
@pytest.mark.parametrize("lrn_first", [True, False])
def test_lrn_pool(D, dt, C, shape, lrn_first):
    n, H, W = shape
    rng = np.random.default_rng(C + H + W)
    x = round_to(np.abs(rng.normal(0, 30, (n, H, W, C))), dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_lrn_pool(xg, DTS[dt], D.net_params(lrn_before_pool=lrn_first)).float().cpu().numpy()
    for i in range(n):
        if lrn_first:
            ref = oracle.maxpool(oracle.lrn(chw(x[i])))
        else:
            ref = oracle.lrn(oracle.maxpool(chw(x[i])))
        assert_layer_close(chw(out[i]), ref, dt, f"lrn_pool {C} {shape}[{i}]")
        if dt == "f32":
            # fp32 output of an fp32 computation: well inside the bar
            assert np.max(np.abs(chw(out[i]) - ref) / np.maximum(np.abs(ref), 1e-3)) < 2e-5


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("C", [96, 256])
@pytest.mark.parametrize("beta,k", [(0.75, 1.0), (0.5, 1.0), (0.75, 2.0), (0.75, 0.5)])
def test_lrn_pool_power_paths(D, dt, C, beta, k):
    """(k + alpha/n s)^-beta for other beta and k than AlexNet's, and activations from 0 to ~500 (every
    third row 8x larger, sums of squares far past the usual range), against the oracle."""
    n, H, W = 1, 29, 33
    rng = np.random.default_rng(C + 11)
    x = np.abs(rng.normal(0, 30, (n, H, W, C)))
    x[:, ::3] *= 8.0                   # every third row large: sums of squares far past 12 500
    x = round_to(x, dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_lrn_pool(xg, DTS[dt], D.net_params(beta=beta, k=k)).float().cpu().numpy()
    ref = oracle.maxpool(oracle.lrn(chw(x[0]), beta=beta, k=k))
    assert_layer_close(chw(out[0]), ref, dt, f"lrn_pool C={C} beta={beta} k={k}")
    if dt == "f32":
        assert np.max(np.abs(chw(out[0]) - ref) / np.maximum(np.abs(ref), 1e-3)) < 2e-5


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_lrn_pool2_strips_many_planes(D, dt):
    """20 planes of conv2's 149 x 149 x 256 maps: a launch large enough for the column-strip kernel
    (one image's planes take the tile kernel).  Sampled planes against the oracle, and every plane
    bit-identical to the same plane pooled alone (the tile kernel: the same arithmetic per element)."""
    n, H, W, C = 20, 149, 149, 256
    g = torch.Generator().manual_seed(256 + H)
    x = (torch.randn((n, H, W, C), generator=g) * 30).abs()
    x[7] = -x[7]                       # one plane of negative values pools in fp32
    xg = x.to("cuda", TORCH_DT[dt]).contiguous()
    del x
    out = D.densenet_lrn_pool(xg, DTS[dt], D.net_params())
    for i in (0, 7, 19):
        xi = xg[i].float().cpu().numpy()
        ref = oracle.maxpool(oracle.lrn(chw(xi)))
        assert_layer_close(chw(out[i].float().cpu().numpy()), ref, dt, f"lrn_pool2 strips [{i}]")
    for i in (0, 7, 13, 19):
        one = D.densenet_lrn_pool(xg[i:i + 1].contiguous(), DTS[dt], D.net_params())
        assert torch.equal(one[0].view(torch.int16), out[i].view(torch.int16)), f"plane {i}"


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("C", [96, 256])
def test_lrn_pool_signed_and_zero_inputs(D, dt, C):
    """Inputs of both signs (tiles holding negative LRN values pool in fp32), all-zero and negative-zero
    regions (tiles of values >= +0 pool on the raw 16-bit patterns)."""
    n, H, W = 1, 41, 38
    rng = np.random.default_rng(C + 3)
    x = rng.normal(0, 30, (n, H, W, C))
    x[:, :20] = np.abs(x[:, :20])      # upper rows non-negative
    x[:, :6, :9] = 0.0                 # zeros
    x[:, 6:10, :9] = -0.0              # negative zeros
    x = round_to(x, dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_lrn_pool(xg, DTS[dt], D.net_params()).float().cpu().numpy()
    ref = oracle.maxpool(oracle.lrn(chw(x[0])))
    assert_layer_close(chw(out[0]), ref, dt, f"signed lrn_pool {C}")
    assert np.array_equal(chw(out[0])[:, :2, :4], ref[:, :2, :4])   # pooled zeros are exact


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_maxpool_exact(D, dt):
    rng = np.random.default_rng(5)
    x = round_to(rng.normal(0, 1, (3, 13, 14, 256)), dt)
    xg = torch.from_numpy(x).to("cuda", TORCH_DT[dt]).contiguous()
    out = D.densenet_maxpool(xg, DTS[dt]).float().cpu().numpy()
    for i in range(3):
        np.testing.assert_array_equal(chw(out[i]), oracle.maxpool(chw(x[i])))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("W,pitch", [(227, 232), (235, 240), (229, 240)])
def test_conv1_ignores_row_padding(D, dt, W, pitch):
    """Planes whose rows are padded (pitch > width, width not a multiple of 8) take the direct-load
    conv1; the padding columns hold NaN here and must not reach any output (for widths with
    (W - 11) % 4 == 0 the last output column's zero-weight tap sits on column W).  The result equals
    the same planes stored unpadded (which take the register-staged conv1) and the oracle."""
    n, H = 3, 227
    rng = np.random.default_rng(W + pitch)
    x = round_to(rng.normal(0, 50, (n, 3, H, W)), dt)
    padded = np.full((n, 3, H, pitch), np.nan, np.float32)
    padded[..., :W] = x
    outs = []
    for arr, p in ((padded, pitch), (x, W)):
        xg = torch.from_numpy(np.ascontiguousarray(arr)).to("cuda", TORCH_DT[dt]).reshape(-1)
        desc = []
        for i in range(n):
            q = D.dn_plane_desc()
            q.h, q.w, q.offset, q.pitch = H, W, i * 3 * H * p, p
            desc.append(q)
        cf = D.ConvFeatures(desc, DTS[dt], D.net_params(pool5=True), device="cuda")
        cf(xg, packed(D, dt))
        torch.cuda.synchronize()
        outs.append([m.float().cpu().numpy() for m in cf.pool5_maps()])
    w = oracle_weights(dt)
    for i in range(n):
        assert np.all(np.isfinite(outs[0][i])), f"NaN from the row padding reached plane {i}"
        assert_layer_close(chw(outs[0][i]), chw(outs[1][i]), dt, f"padded vs unpadded [{i}]")
        _, ref = oracle.net(x[i], w, pool5=True)
        assert_layer_close(chw(outs[0][i]), ref, dt, f"padded pool5 [{i}]")
