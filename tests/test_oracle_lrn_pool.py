"""Pins for LRN and max-pool: closed forms for constant inputs, torch routines in fp64, monotone ramps."""
import numpy as np
import pytest
import torch

import oracle


@pytest.mark.parametrize("a", [0.5, 3.0, 10.0])
def test_lrn_constant_closed_form(a):
    C, n, alpha, beta, k = 9, 5, 1e-4, 0.75, 1.0
    x = np.full((C, 3, 4), a, np.float32)
    got = oracle.lrn(x, n, alpha, beta, k)
    # the clipped window holds 3, 4, 5 channels at the edge, next to the edge and inside
    cnt = np.array([3, 4, 5, 5, 5, 5, 5, 4, 3])
    ref = a * (k + alpha / n * cnt * a * a) ** (-beta)
    np.testing.assert_allclose(got[:, 0, 0], ref, rtol=1e-7)


def test_lrn_stress_vs_torch():
    rng = np.random.default_rng(1)
    x = (10 * rng.normal(size=(17, 5, 6))).astype(np.float32)
    for alpha, beta, k, n in ((1.0, 0.75, 1.0, 5), (1e-4, 0.75, 1.0, 5), (0.3, 0.5, 2.0, 3)):
        got = oracle.lrn(x, n, alpha, beta, k)
        ref = torch.nn.functional.local_response_norm(torch.from_numpy(x).double()[None], n, alpha, beta,
                                                      k)[0].numpy()
        np.testing.assert_allclose(got, ref, rtol=2e-6, atol=1e-30)


def test_lrn_is_not_a_noop_at_config_scale():
    x = np.full((96, 1, 1), 30.0, np.float32)
    assert abs(oracle.lrn(x)[50, 0, 0] / 30.0 - 1) > 0.01


@pytest.mark.parametrize("H,W", [(7, 9), (8, 8), (298, 5), (13, 13), (2, 4)])
def test_pool_ceil_vs_torch(H, W):
    rng = np.random.default_rng(H * W)
    x = rng.normal(size=(3, H, W)).astype(np.float32)
    got = oracle.maxpool(x)
    ref = torch.nn.functional.max_pool2d(torch.from_numpy(x).double()[None], 3, 2, ceil_mode=True)[0]
    np.testing.assert_array_equal(got, ref.numpy().astype(np.float32))


def test_pool_monotone_ramp_takes_bottom_right():
    H, W = 298, 12
    x = (np.arange(H)[:, None] * 1000 + np.arange(W)[None, :]).astype(np.float32)[None]
    got = oracle.maxpool(x)[0]
    assert got.shape == (149, 6)
    for i in range(149):
        for j in range(6):
            assert got[i, j] == x[0, min(2 * i + 2, H - 1), min(2 * j + 2, W - 1)]
