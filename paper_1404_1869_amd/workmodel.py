"""Algorithmic work of the path, for throughput and roofline reporting (not part of the computation).

FLOPs count 2 per multiply-add over whole planes (the method computes whole stitched planes, Sec. 3.1);
MFMA K-padding is not counted.  Bytes are compulsory traffic: every input read once, every output
written once.
"""
from __future__ import annotations

# (M, C, R, stride, pad, groups) of conv1..conv5 of the AlexNet topology
CONV_LAYERS = ((96, 3, 11, 4, 0, 1), (256, 96, 5, 1, 2, 2), (384, 256, 3, 1, 1, 1),
               (384, 384, 3, 1, 1, 2), (256, 384, 3, 1, 1, 2))


def _conv(n, R, s, p):
    return (n + 2 * p - R) // s + 1


def _pool(n):
    o = -((3 - n) // 2) + 1          # ceil((n - 3) / 2) + 1
    while (o - 1) * 2 >= n:
        o -= 1
    return o


def sides(n: int):
    """Output side after conv1, pool1, conv2, pool2, conv3, conv4, conv5, pool5 for an n-px side."""
    c1 = _conv(n, 11, 4, 0)
    p1 = _pool(c1)
    c2 = _conv(p1, 5, 1, 2)
    p2 = _pool(c2)
    return c1, p1, c2, p2, p2, p2, p2, _pool(p2)


def conv_flops(PH: int, PW: int):
    """Per-layer conv FLOPs on one PH x PW plane."""
    sh, sw = sides(PH), sides(PW)
    outs = [(sh[0], sw[0]), (sh[2], sw[2]), (sh[4], sw[4]), (sh[5], sw[5]), (sh[6], sw[6])]
    return [2 * M * (C // G) * R * R * ho * wo for (M, C, R, s, p, G), (ho, wo) in zip(CONV_LAYERS, outs)]


def region_count(N: int, M: int, stride: int = 16) -> float:
    """Number of M x M regions at the given stride in an N x N image (Sec. 3 example)."""
    return ((N - M) / stride) ** 2


def dense_speedup(N: int, M: int, stride: int = 16) -> float:
    """Per-region work R M^2 over dense work N^2 (Sec. 3 example)."""
    return region_count(N, M, stride) * M * M / (N * N)
