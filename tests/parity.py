"""Shared helpers of the GPU parity tests: tolerance metrics and layout conversions (no method
arithmetic)."""
import numpy as np

# Bars per storage type.  fp32: max relative error with an RMS guard; fp16: max abs error over the
# layer's output RMS; bf16: the same metric with the bar its 8-bit mantissa forces, plus an RMS bar.
BARS = {"f32": 1e-4, "f16": 2e-2, "bf16": 6e-2}
BF16_RMS_BAR = 1e-2


def rel_err_guarded(g, o):
    """max_i |g_i - o_i| / max(|o_i|, RMS(o))."""
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    rms = np.sqrt(np.mean(o * o))
    return float(np.max(np.abs(g - o) / np.maximum(np.abs(o), rms)))


def norm_max_abs(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return float(np.max(np.abs(g - o)) / np.sqrt(np.mean(o * o)))


def norm_rms(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return float(np.sqrt(np.mean((g - o) ** 2)) / np.sqrt(np.mean(o * o)))


def assert_layer_close(g, o, dt, what=""):
    if dt == "f32":
        e = rel_err_guarded(g, o)
    else:
        e = norm_max_abs(g, o)
    assert e <= BARS[dt], f"{what} {dt}: error {e:.3e} > {BARS[dt]:.1e}"
    if dt == "bf16":
        r = norm_rms(g, o)
        assert r <= BF16_RMS_BAR, f"{what} bf16: rms error {r:.3e} > {BF16_RMS_BAR:.1e}"
    return e


def round_to(x, dt):
    """Round an fp32/fp64 array to the storage type and back to fp32 (for teacher forcing)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    if dt == "f16":
        t = t.half().float()
    elif dt == "bf16":
        t = t.bfloat16().float()
    return t.numpy()


def ulp(x, dt):
    """Spacing of the storage type at |x| (normal range)."""
    ax = np.maximum(np.abs(np.asarray(x, np.float64)), 1e-30)
    mant = {"f16": 10, "bf16": 7, "f32": 23}[dt]
    e = np.floor(np.log2(ax))
    if dt == "f16":
        e = np.maximum(e, -14)
    return 2.0 ** (e - mant)


# fp32 error of a plane value before its final rounding to the storage type.  The builder (and the
# crop-before warp) blends four uint8 taps in fp32: lerp-x twice, lerp-y, minus the mean pixel, times the
# border weight.  Every intermediate is below 256 in magnitude, so each rounding costs at most
# h = 2^-17 (half an fp32 ulp at 128..256); the fractions and weights are fp32 roundings of exact
# rationals (relative error 2^-24, times values below 256: at most h each).  Counting terms:
# lerp-x 3h per row, the lerp-y of the two rows 7h, the mean 8h, the border weight 15h < 2^-13.
PLANE_FP32_ERR = 2.0 ** -13


def plane_tol(ref, dt):
    """Bound on |GPU plane value - fp64 oracle value|: the fp32 error above, plus half an ulp of the
    storage type at the largest magnitude the fp32 value can have."""
    ref = np.abs(np.asarray(ref, np.float64))
    return 0.5 * ulp(ref + PLANE_FP32_ERR, dt) + PLANE_FP32_ERR


def chw(nhwc):
    return np.ascontiguousarray(np.moveaxis(np.asarray(nhwc), -1, 0))


def hwc(chw_):
    return np.ascontiguousarray(np.moveaxis(np.asarray(chw_), 0, -1))
