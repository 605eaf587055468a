"""Pins of the oracle's crop-before windows (Sec. 3.4 per-window baseline, Sec. 4 crop before): exact
crops, exact 2x reductions, identity, agreement with torch's bilinear resize of the crop in fp64, and
with the oracle's own pyramid resize for a whole-image box."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

MEAN = (123.68, 116.779, 103.939)


def img(seed, H, W, n=None):
    shape = (3, H, W) if n is None else (n, 3, H, W)
    return np.random.default_rng(seed).integers(0, 256, shape, dtype=np.uint8)


def test_identity_box_is_centred_image():
    S = 24
    I = img(1, S, S)
    out = oracle.warp_regions(I, np.array([[0, 0, S, S]], np.float32), S=S, mean=MEAN)[0]
    ref = I.astype(np.float64) - np.array(MEAN)[:, None, None]
    np.testing.assert_array_equal(out, ref.astype(np.float32))


def test_integer_box_of_side_S_is_exact_crop():
    S = 16
    I = img(2, 60, 70)
    x, y = 23, 9
    out = oracle.warp_regions(I, np.array([[x, y, x + S, y + S]], np.float32), S=S)[0]
    np.testing.assert_array_equal(out, I[:, y:y + S, x:x + S].astype(np.float32))


def test_exact_2x_reduction_is_2x2_mean():
    S = 12
    I = img(3, 50, 50)
    x, y = 5, 11
    out = oracle.warp_regions(I, np.array([[x, y, x + 2 * S, y + 2 * S]], np.float32), S=S)[0]
    c = I[:, y:y + 2 * S, x:x + 2 * S].astype(np.float64)
    ref = 0.25 * (c[:, 0::2, 0::2] + c[:, 1::2, 0::2] + c[:, 0::2, 1::2] + c[:, 1::2, 1::2])
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-5)


@pytest.mark.parametrize("box,S", [((13, 7, 313, 177), 64), ((40, 31, 227, 290), 51)])
def test_downsampling_matches_torch_bilinear_of_crop(box, S):
    I = img(4, 320, 330)
    x1, y1, x2, y2 = box
    out = oracle.warp_regions(I, np.array([box], np.float32), S=S)[0]
    crop = torch.from_numpy(I[:, y1:y2, x1:x2].astype(np.float64))[None]
    ref = F.interpolate(crop, size=(S, S), mode="bilinear", align_corners=False)[0].numpy()
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-4)


def test_whole_image_upsampling_matches_torch_and_pyramid_resize():
    H, W, S = 37, 53, 90
    I = img(5, H, W)
    out = oracle.warp_regions(I, np.array([[0, 0, W, H]], np.float32), S=S, mean=MEAN)[0]
    ref = F.interpolate(torch.from_numpy(I.astype(np.float64))[None], size=(S, S), mode="bilinear",
                        align_corners=False)[0].numpy() - np.array(MEAN)[:, None, None]
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-4)
    np.testing.assert_allclose(out, oracle.resize_center(I, S, S, MEAN), rtol=0, atol=2e-5)  # fp32 rounding


def test_box_outside_image_repeats_edge_pixels():
    """Clamping the coordinate to the image: a box entirely right of / below the image gives the
    bottom-right pixel everywhere; one straddling the left edge repeats the first column."""
    I = img(7, 20, 30)
    out = oracle.warp_regions(I, np.array([[40, 25, 70, 50], [-20, 0, 10, 20]], np.float32), S=10)
    np.testing.assert_array_equal(out[0], np.broadcast_to(I[:, -1:, -1:], (3, 10, 10)).astype(np.float32))
    # left box: output columns whose coordinate falls below 0 equal column 0 of the image rows
    sx = -20 + (np.arange(10) + 0.5) * 3 - 0.5
    cols = np.where(sx <= 0)[0]
    sy = (np.arange(10) + 0.5) * 2 - 0.5
    for i in range(10):
        y = min(max(sy[i], 0), 19)
        y0 = int(np.floor(y)); y1 = min(y0 + 1, 19); ly = y - y0
        ref = (1 - ly) * I[:, y0, 0].astype(np.float64) + ly * I[:, y1, 0]
        for j in cols:
            np.testing.assert_allclose(out[1][:, i, j], ref, rtol=0, atol=1e-4)


def test_degenerate_boxes_give_zero_windows_and_box_img_selects_image():
    I = img(6, 30, 40, n=2)
    boxes = np.array([[5, 5, 5, 20], [10, 10, 3, 20], [np.nan, 0, 10, 10], [0, 0, 40, 30]], np.float32)
    out = oracle.warp_regions(I, boxes, S=8, box_img=np.array([0, 0, 0, 1], np.int32))
    assert not out[:3].any()
    np.testing.assert_array_equal(out[3], oracle.warp_regions(I[1], boxes[3:], S=8)[0])
    assert not np.array_equal(out[3], oracle.warp_regions(I[0], boxes[3:], S=8)[0])
