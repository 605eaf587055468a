"""Pins for the oracle's convolution (the conv layers of Sec. 3), independent of the oracle itself:
brute force in pure Python, torch.conv2d in fp64, delta filters, all-ones filters against a
summed-area table, grouped = concatenated per-group convs, closed-form output sizes."""
import numpy as np
import pytest
import torch

import oracle


def brute_conv(x, w, b, s, p, G, relu):
    C, H, W = x.shape
    M, Cg, R, _ = w.shape
    Ho, Wo = (H + 2 * p - R) // s + 1, (W + 2 * p - R) // s + 1
    out = np.zeros((M, Ho, Wo))
    Mg = M // G
    for m in range(M):
        g = m // Mg
        for i in range(Ho):
            for j in range(Wo):
                acc = float(b[m])
                for cl in range(Cg):
                    for ky in range(R):
                        for kx in range(R):
                            yy, xx = s * i + ky - p, s * j + kx - p
                            if 0 <= yy < H and 0 <= xx < W:
                                acc += float(w[m, cl, ky, kx]) * float(x[g * Cg + cl, yy, xx])
                out[m, i, j] = max(acc, 0.0) if relu else acc
    return out


@pytest.mark.parametrize("C,M,R,s,p,G", [(2, 3, 3, 1, 1, 1), (4, 4, 5, 1, 2, 2), (3, 2, 3, 2, 0, 1),
                                         (6, 6, 3, 1, 1, 3), (3, 5, 4, 3, 1, 1)])
def test_conv_brute_force_8x8(C, M, R, s, p, G):
    rng = np.random.default_rng(C * 100 + M * 10 + R)
    x = rng.normal(size=(C, 8, 8)).astype(np.float32)
    w = rng.normal(size=(M, C // G, R, R)).astype(np.float32)
    b = rng.normal(size=M).astype(np.float32)
    for relu in (False, True):
        got = oracle.conv2d(x, w, b, s, p, G, relu)
        ref = brute_conv(x, w, b, s, p, G, relu)
        np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("C,M,R,s,p,G,H", [(3, 96, 11, 4, 0, 1, 35), (96, 256, 5, 1, 2, 2, 13),
                                           (256, 384, 3, 1, 1, 1, 9), (384, 384, 3, 1, 1, 2, 7),
                                           (384, 256, 3, 1, 1, 2, 6)])
def test_conv_vs_torch_fp64(C, M, R, s, p, G, H):
    rng = np.random.default_rng(H)
    x = rng.normal(size=(C, H, H + 3)).astype(np.float32)
    w = (0.05 * rng.normal(size=(M, C // G, R, R))).astype(np.float32)
    b = rng.normal(size=M).astype(np.float32)
    got = oracle.conv2d(x, w, b, s, p, G, relu=False)
    ref = torch.nn.functional.conv2d(torch.from_numpy(x).double()[None], torch.from_numpy(w).double(),
                                     torch.from_numpy(b).double(), stride=s, padding=p, groups=G)[0]
    np.testing.assert_allclose(got, ref.numpy(), rtol=2e-6, atol=2e-6)


def test_delta_filters():
    rng = np.random.default_rng(5)
    x = rng.normal(size=(4, 10, 12)).astype(np.float32)
    # 3x3 pad 1: a 1 at the centre tap of the matching input channel gives the identity.
    w = np.zeros((4, 4, 3, 3), np.float32)
    for m in range(4):
        w[m, m, 1, 1] = 1
    b = np.zeros(4, np.float32)
    np.testing.assert_array_equal(oracle.conv2d(x, w, b, 1, 1, 1, relu=False), x)
    # conv1 geometry: a 1 at (5,5) of an 11x11 stride-4 filter picks in(4i+5, 4j+5).
    x1 = rng.normal(size=(3, 47, 51)).astype(np.float32)
    w1 = np.zeros((3, 3, 11, 11), np.float32)
    for m in range(3):
        w1[m, m, 5, 5] = 1
    got = oracle.conv2d(x1, w1, np.zeros(3, np.float32), 4, 0, 1, relu=False)
    assert got.shape == (3, 10, 11)
    np.testing.assert_array_equal(got, x1[:, 5:5 + 4 * 10:4, 5:5 + 4 * 11:4])


def test_all_ones_is_box_sum():
    rng = np.random.default_rng(6)
    x = rng.integers(0, 4, size=(2, 20, 23)).astype(np.float32)
    R, p = 5, 2
    w = np.ones((1, 2, R, R), np.float32)
    got = oracle.conv2d(x, w, np.zeros(1, np.float32), 1, p, 1, relu=False)[0]
    s = x.sum(0)
    sp = np.pad(s, p)
    sat = np.zeros((sp.shape[0] + 1, sp.shape[1] + 1))
    sat[1:, 1:] = sp.cumsum(0).cumsum(1)
    H, W = s.shape
    ref = sat[R:R + H, R:R + W] - sat[0:H, R:R + W] - sat[R:R + H, 0:W] + sat[0:H, 0:W]
    np.testing.assert_array_equal(got, ref)


def test_grouped_is_concatenation():
    rng = np.random.default_rng(8)
    x = rng.normal(size=(8, 9, 9)).astype(np.float32)
    w = rng.normal(size=(6, 4, 3, 3)).astype(np.float32)
    b = rng.normal(size=6).astype(np.float32)
    got = oracle.conv2d(x, w, b, 1, 1, 2, relu=True)
    a = oracle.conv2d(x[:4], w[:3], b[:3], 1, 1, 1, relu=True)
    c = oracle.conv2d(x[4:], w[3:], b[3:], 1, 1, 1, relu=True)
    np.testing.assert_array_equal(got, np.concatenate([a, c]))


def test_layer_sizes_closed_form():
    # AlexNet at 227: 55 / 27 / 27 / 13 / 13 / 6; a 1200 plane: 298 / 149 / 149 / 74 / 74 / 37.
    for n, expect in ((227, (55, 27, 27, 13, 13, 6)), (1200, (298, 149, 149, 74, 74, 37))):
        c1 = oracle.conv_side(n, 11, 4, 0)
        p1 = oracle.pool_side(c1)
        c2 = oracle.conv_side(p1, 5, 1, 2)
        p2 = oracle.pool_side(c2)
        c5 = oracle.conv_side(oracle.conv_side(oracle.conv_side(p2, 3, 1, 1), 3, 1, 1), 3, 1, 1)
        p5 = oracle.pool_side(c5)
        assert (c1, p1, c2, p2, c5, p5) == expect
        assert oracle.conv5_side(n) == expect[4]
