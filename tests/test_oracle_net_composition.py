"""Pin of the oracle's whole conv stack as a composition (Sec. 3: the first five conv layers of the
AlexNet topology, read as conv1 -> ReLU -> LRN -> pool, conv2 (2 groups) -> ReLU -> LRN -> pool,
conv3 -> ReLU, conv4 (2 groups) -> ReLU, conv5 (2 groups) -> ReLU, optional pool5).

The reference chain here is built from torch's own fp64 layers (``conv2d`` with groups, ``relu``,
``local_response_norm``, ``max_pool2d`` in ceil mode), so a dropped, swapped or misplaced layer in the
oracle (a missing LRN, LRN and pool in the wrong order, a missing ReLU, floor-mode pooling) fails here
on the CPU, independently of the GPU path.  The oracle stores fp32 between layers; the chain keeps
fp64 throughout, so the bar allows for fp32 storage only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_1404_1869_amd import synth

W7 = synth.weights(7)
GROUPS = (1, 2, 1, 2, 2)
STRIDES = (4, 1, 1, 1, 1)
PADS = (0, 2, 1, 1, 1)
# fp32 storage between the layers (rounding 2^-24 relative, five conv layers deep, with cancellation
# in the sums) stays far below this; every composition mistake tried moves the result by > 1e-3.
BAR = 1e-5


def torch_chain(plane, weights, lrn_params, lrn_before_pool, pool5):
    a, be, k, n = lrn_params
    x = torch.from_numpy(np.asarray(plane, np.float64))[None]
    for l in range(5):
        w = torch.from_numpy(weights[l][0].astype(np.float64))
        b = torch.from_numpy(weights[l][1].astype(np.float64))
        x = F.relu(F.conv2d(x, w, b, stride=STRIDES[l], padding=PADS[l], groups=GROUPS[l]))
        if l < 2:
            if lrn_before_pool:
                x = F.max_pool2d(F.local_response_norm(x, n, alpha=a, beta=be, k=k), 3, 2,
                                 ceil_mode=True)
            else:
                x = F.local_response_norm(F.max_pool2d(x, 3, 2, ceil_mode=True), n, alpha=a, beta=be,
                                          k=k)
    c5 = x[0].numpy()
    p5 = F.max_pool2d(x, 3, 2, ceil_mode=True)[0].numpy() if pool5 else None
    return c5, p5


def rel(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return float(np.max(np.abs(g - o)) / np.sqrt(np.mean(o * o)))


@pytest.mark.parametrize("shape", [(227, 227), (131, 97), (163, 210)])
@pytest.mark.parametrize("lrn_before_pool", [True, False])
@pytest.mark.parametrize("lrn_params", [(1e-4, 0.75, 1.0, 5), (1.0, 0.75, 2.0, 5)],
                         ids=["alexnet_lrn", "strong_lrn"])
def test_oracle_net_equals_torch_fp64_chain(shape, lrn_before_pool, lrn_params):
    H, W = shape
    rng = np.random.default_rng(H * 1000 + W)
    plane = rng.uniform(-128.0, 128.0, (3, H, W)).astype(np.float32)
    c5, p5 = oracle.net(plane, W7, lrn_params=lrn_params, lrn_before_pool=lrn_before_pool, pool5=True)
    t5, tp5 = torch_chain(plane, W7, lrn_params, lrn_before_pool, pool5=True)
    assert c5.shape == t5.shape and p5.shape == tp5.shape
    assert rel(c5, t5) <= BAR, rel(c5, t5)
    assert rel(p5, tp5) <= BAR, rel(p5, tp5)


def test_alexnet_227_output_shapes():
    """227 x 227 in -> conv5 256 x 13 x 13 -> pool5 256 x 6 x 6 (9216 values, AlexNet's pool5)."""
    plane = np.zeros((3, 227, 227), np.float32)
    c5, p5 = oracle.net(plane, W7, pool5=True)
    assert c5.shape == (256, 13, 13) and p5.shape == (256, 6, 6)


@pytest.mark.parametrize("lrn_params", [(1e-4, 0.75, 1.0, 5), (1.0, 0.75, 2.0, 5)],
                         ids=["alexnet_lrn", "strong_lrn"])
def test_chain_distinguishes_plausible_mistakes(lrn_params):
    """The bar above separates the right composition from each plausible wrong one: the wrong chains,
    built from the same torch layers, all differ from the oracle by far more than BAR."""
    rng = np.random.default_rng(5)
    plane = rng.uniform(-128.0, 128.0, (3, 131, 97)).astype(np.float32)
    c5 = oracle.net(plane, W7, lrn_params=lrn_params)
    a, be, k, n = lrn_params

    def chain(order=True, lrn_layers=(0, 1), relu_last=True, ceil=True):
        x = torch.from_numpy(plane.astype(np.float64))[None]
        for l in range(5):
            w = torch.from_numpy(W7[l][0].astype(np.float64))
            b = torch.from_numpy(W7[l][1].astype(np.float64))
            x = F.conv2d(x, w, b, stride=STRIDES[l], padding=PADS[l], groups=GROUPS[l])
            if l < 4 or relu_last:
                x = F.relu(x)
            if l < 2:
                lrn = (lambda t: F.local_response_norm(t, n, alpha=a, beta=be, k=k)) \
                    if l in lrn_layers else (lambda t: t)
                pool = lambda t: F.max_pool2d(t, 3, 2, ceil_mode=ceil)
                x = pool(lrn(x)) if order else lrn(pool(x))
        return x[0].numpy()

    assert rel(c5, chain()) <= BAR
    assert rel(c5, chain(order=False)) > 100 * BAR
    assert rel(c5, chain(lrn_layers=(1,))) > 100 * BAR
    assert rel(c5, chain(lrn_layers=(0,))) > 100 * BAR
    assert rel(c5, chain(relu_last=False)) > 100 * BAR
    wrong = chain(ceil=False)
    assert wrong.shape != c5.shape or rel(c5, wrong) > 100 * BAR
