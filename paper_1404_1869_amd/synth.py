"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module holds random draws only, none of the pyramid or network arithmetic.  The paper measures on
natural images with a trained AlexNet (ImageNet / PASCAL); neither is available, so uniform uint8 images,
N(0, 0.01) weights with 0.1 biases and log-uniform boxes of the same shapes and sizes stand in for them.
All draws use numpy's PCG64 ``default_rng``.
"""
from __future__ import annotations

import numpy as np

# Widely published ImageNet RGB mean pixel, paired with input channels 0, 1, 2 (Sec. 3.2 centres on one
# mean pixel value; its exact value does not affect parity, it is a caller parameter).
IMAGENET_MEAN = (123.68, 116.78, 103.94)

# Weight shapes of the five conv layers of the AlexNet topology, OIHW: (M, C/G, R, R).
WEIGHT_SHAPES = ((96, 3, 11, 11), (256, 48, 5, 5), (384, 256, 3, 3), (384, 192, 3, 3),
                 (256, 192, 3, 3))


def image(seed: int, H: int, W: int) -> np.ndarray:
    """uint8 [3][H][W], uniform 0..255."""
    return np.random.default_rng(seed).integers(0, 256, (3, H, W), dtype=np.uint8)


def images(seeds, H: int, W: int) -> np.ndarray:
    return np.stack([image(s, H, W) for s in seeds])


def weights(seed: int = 7, std: float = 0.01, bias: float = 0.1):
    """[(w, b)] for conv1..conv5, w ~ N(0, std) drawn in layer order, b = bias."""
    rng = np.random.default_rng(seed)
    out = []
    for shape in WEIGHT_SHAPES:
        w = rng.normal(0.0, std, shape).astype(np.float32)
        out.append((w, np.full(shape[0], bias, np.float32)))
    return out


def boxes(seed: int, n: int, H: int, W: int, smin=32.0, smax=512.0, armax=3.0) -> np.ndarray:
    """[n][4] fp32 (x1, y1, x2, y2) in original pixel-edge coordinates.

    size = sqrt(w h) log-uniform in [smin, smax], aspect w/h log-uniform in [1/armax, armax], drawn in
    the order sizes, aspects, u_x, u_y; sides clamped to the image; top-left uniform so the box lies
    inside the image.
    """
    rng = np.random.default_rng(seed)
    size = np.exp(rng.uniform(np.log(smin), np.log(smax), n))
    ar = np.exp(rng.uniform(-np.log(armax), np.log(armax), n))
    ux = rng.random(n)
    uy = rng.random(n)
    bw = np.minimum(size * np.sqrt(ar), W)
    bh = np.minimum(size / np.sqrt(ar), H)
    x1 = ux * (W - bw)
    y1 = uy * (H - bh)
    return np.stack([x1, y1, x1 + bw, y1 + bh], axis=1).astype(np.float32)
