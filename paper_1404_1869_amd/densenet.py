"""ctypes binding of libdensenet.so: the C ABI of include/densenet.h, same names, argument marshalling
only.  Device memory comes from torch tensors and the stream from torch.cuda.current_stream(); every
step of the computation runs in the library's HIP kernels.  There is no fallback: if the library or a
GPU is missing the calls raise.

On top of the raw entry points, ``convnet_featpyramid`` mirrors the paper's interface
(``pyra = convnet_featpyramid(image)``, Sec. 3.5): image(s) in, per-scale conv5 maps plus geometry out.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdensenet.so")

DN_OK, DN_E_INVALID_ARG, DN_E_TOO_LARGE, DN_E_BUFFER_TOO_SMALL = 0, -1, -2, -3
DN_E_UNSUPPORTED, DN_E_HIP, DN_E_INTERNAL = -4, -5, -6
DN_F32, DN_F16, DN_BF16 = 0, 1, 2
DN_PAD_ZERO, DN_PAD_RAMP = 0, 1
DN_MAX_SCALES, DN_MAX_PLANES_PER_IMAGE, DN_MAX_WARP_SIDE, DN_MAX_ASPECTS = 64, 64, 1024, 8
DN_MAX_BATCH_ITEMS = 65536
DN_STATIC_SCRATCH_BYTES = 64 << 20
DTYPES = {"f32": DN_F32, "f16": DN_F16, "bf16": DN_BF16}

EXPORTS = ("densenet_plan_pyramid", "densenet_build_pyramid", "densenet_pack_weights",
           "densenet_conv_features", "densenet_region_windows", "densenet_conv_layer",
           "densenet_lrn_pool", "densenet_maxpool", "densenet_layer_sizes", "densenet_warp_regions",
           "densenet_region_pool", "densenet_plan_batch", "densenet_build_batch",
           "densenet_region_windows_batch", "densenet_build_pyramid_noalloc", "densenet_profile_start",
           "densenet_profile_stop", "densenet_last_error")


class dn_pyramid_params(ctypes.Structure):
    _fields_ = [("n_scales", ctypes.c_int32), ("steps_per_octave", ctypes.c_int32),
                ("base_scale", ctypes.c_double), ("base_longest_side", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("pad_mode", ctypes.c_int32), ("plane_h", ctypes.c_int32),
                ("plane_w", ctypes.c_int32), ("mean", ctypes.c_float * 3), ("n_aspects", ctypes.c_int32),
                ("aspects", ctypes.c_double * DN_MAX_ASPECTS)]


class dn_scale_geom(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("k", "h", "w", "plane", "y", "x", "rh", "rw", "r0",
                                              "r1", "c0", "c1", "aspect", "image")] + \
               [(n, ctypes.c_double) for n in ("s", "sy", "sx")]


class dn_plane_desc(ctypes.Structure):
    _fields_ = [("h", ctypes.c_int32), ("w", ctypes.c_int32), ("offset", ctypes.c_int64),
                ("pitch", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class dn_net_params(ctypes.Structure):
    _fields_ = [("lrn_alpha", ctypes.c_float), ("lrn_beta", ctypes.c_float),
                ("lrn_k", ctypes.c_float), ("lrn_n", ctypes.c_int32),
                ("lrn_before_pool", ctypes.c_int32), ("pool5", ctypes.c_int32)]


class dn_profile_entry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


class DenseNetError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"densenet error {status}: {msg}")
        self.status = status


_lib = None


def lib():
    """Load libdensenet.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, sz, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
        pp, pg, pd = ctypes.POINTER(dn_pyramid_params), ctypes.POINTER(dn_scale_geom), ctypes.POINTER(dn_plane_desc)
        pn = ctypes.POINTER(dn_net_params)
        psz, pi32, pi64 = ctypes.POINTER(sz), ctypes.POINTER(i32), ctypes.POINTER(i64)
        sig = {
            "densenet_plan_pyramid": [i32, i32, pp, pg, pd, i32, pi32, pi64],
            "densenet_build_pyramid": [P, i32, i32, i32, pp, i32, P, sz, psz, pg, pd, i32, pi32, pi64, P],
            "densenet_build_pyramid_noalloc": [P, i32, i32, i32, pp, i32, P, sz, psz, pg, pd, i32, pi32, pi64,
                                               P],
            "densenet_pack_weights": [P, P, i32, P, sz, psz, P],
            "densenet_conv_features": [P, pd, i32, i32, P, pn, P, sz, psz, P, sz, psz, pd, P, sz, psz,
                                       pd, P],
            "densenet_region_windows": [P, pd, i32, i32, pg, i32, i32, i32, P, P, i32, f32, i32, P, P,
                                        P, P],
            "densenet_region_pool": [P, pd, i32, i32, pg, i32, i32, i32, P, P, i32, f32, i32, P, P, P,
                                     P],
            "densenet_conv_layer": [i32, P, i32, i32, i32, i32, P, P, P],
            "densenet_lrn_pool": [P, i32, i32, i32, i32, i32, pn, P, P],
            "densenet_maxpool": [P, i32, i32, i32, i32, i32, P, P],
            "densenet_layer_sizes": [i32, i32, pi32],
            "densenet_warp_regions": [P, i32, i32, i32, P, P, i32, i32, i32, ctypes.POINTER(f32), i32, P,
                                      sz, psz, P],
            "densenet_plan_batch": [i32, i32, i32, pp, pg, pd, i32, pi32, pi64],
            "densenet_build_batch": [P, i32, i32, i32, pp, i32, pg, P, i32, P, sz, psz, P],
            "densenet_region_windows_batch": [P, pd, i32, i32, pg, P, i32, i32, i32, i32, P, P, i32, f32,
                                              i32, P, P, P, P],
            "densenet_profile_start": [ctypes.c_char_p],
            "densenet_profile_stop": [ctypes.POINTER(dn_profile_entry), i32, pi32],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.densenet_last_error.argtypes = []
        L.densenet_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def last_error() -> str:
    return lib().densenet_last_error().decode()


def check(status: int):
    if status != DN_OK:
        raise DenseNetError(status, last_error())
    return status


# ------------------------------------------------------------------------------------------------
# torch plumbing: device memory and streams only
# ------------------------------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _ptr(t):
    if t is None:
        return None
    assert t.is_cuda and t.is_contiguous(), "device tensors must be contiguous CUDA/HIP tensors"
    return ctypes.c_void_p(t.data_ptr())


def _tdtype(dt: int):
    torch = _torch()
    return {DN_F32: torch.float32, DN_F16: torch.float16, DN_BF16: torch.bfloat16}[dt]


def pyramid_params(n_scales, steps_per_octave, base_scale=1.0, base_longest_side=0, pad=0,
                   pad_mode=DN_PAD_ZERO, plane_h=0, plane_w=0, mean=(0.0, 0.0, 0.0), aspects=()):
    p = dn_pyramid_params()
    p.n_scales, p.steps_per_octave, p.base_scale = n_scales, steps_per_octave, base_scale
    p.base_longest_side, p.pad, p.pad_mode = base_longest_side, pad, pad_mode
    p.plane_h, p.plane_w = plane_h, plane_w
    p.mean = (ctypes.c_float * 3)(*mean)
    p.n_aspects = len(aspects)
    for i, r in enumerate(aspects):
        p.aspects[i] = float(r)
    return p


def n_entries(p: dn_pyramid_params) -> int:
    """Pyramid entries (scales x aspect ratios) of a recipe: the length of its geometry arrays."""
    return p.n_scales * max(1, p.n_aspects)


def params_for(w):
    """dn_pyramid_params of a configs.Workload."""
    return pyramid_params(w.n_scales, w.steps_per_octave, w.base_scale, w.base_longest_side, w.pad,
                          w.pad_mode, w.plane_h, w.plane_w, w.mean, w.aspects)


def net_params(alpha=1e-4, beta=0.75, k=1.0, n=5, lrn_before_pool=True, pool5=False):
    q = dn_net_params()
    q.lrn_alpha, q.lrn_beta, q.lrn_k, q.lrn_n = alpha, beta, k, n
    q.lrn_before_pool, q.pool5 = int(lrn_before_pool), int(pool5)
    return q


# ------------------------------------------------------------------------------------------------
# Entry points
# ------------------------------------------------------------------------------------------------
@dataclass
class PlanResult:
    geom: list            # dn_scale_geom per scale
    planes: list          # dn_plane_desc per plane of one image
    image_elems: int

    def geom_array(self) -> np.ndarray:
        """[K][13] int32: k, h, w, plane, y, x, rh, rw, r0, r1, c0, c1, aspect."""
        return np.array([[getattr(g, f) for f in ("k", "h", "w", "plane", "y", "x", "rh", "rw", "r0",
                                                   "r1", "c0", "c1", "aspect")] for g in self.geom],
                        np.int32)

    def scale_array(self) -> np.ndarray:
        return np.array([[g.s, g.sy, g.sx] for g in self.geom], np.float64)

    def image_descs(self, n_img: int) -> list:
        """Descriptors of the planes of n_img images built with this plan (image b's planes at
        b * image_elems), image-major, for densenet_conv_features."""
        out = []
        for b in range(n_img):
            for d in self.planes:
                q = dn_plane_desc()
                q.h, q.w, q.pitch, q.offset = d.h, d.w, d.pitch, b * self.image_elems + d.offset
                out.append(q)
        return out


def plane_view(planes, d: dn_plane_desc, base: int = 0):
    """[3][h][w] view of the plane that descriptor d places in the flat planes tensor (rows d.pitch
    elements apart), shifted by base elements."""
    pitch = d.pitch or d.w
    o = base + d.offset
    return planes[o:o + 3 * d.h * pitch].view(3, d.h, pitch)[:, :, :d.w]


def densenet_plan_pyramid(H: int, W: int, p: dn_pyramid_params) -> PlanResult:
    geom = (dn_scale_geom * n_entries(p))()
    planes = (dn_plane_desc * DN_MAX_PLANES_PER_IMAGE)()
    n = ctypes.c_int32()
    e = ctypes.c_int64()
    check(lib().densenet_plan_pyramid(H, W, ctypes.byref(p), geom, planes, DN_MAX_PLANES_PER_IMAGE,
                                      ctypes.byref(n), ctypes.byref(e)))
    return PlanResult(list(geom), list(planes[:n.value]), e.value)


def densenet_build_pyramid(images, p: dn_pyramid_params, dtype: int, out=None):
    """images: uint8 device tensor [n][3][H][W] (or [3][H][W]).  Returns (planes tensor, PlanResult)."""
    torch = _torch()
    if images.dim() == 3:
        images = images[None]
    n_img, _, H, W = images.shape
    geom = (dn_scale_geom * n_entries(p))()
    planes = (dn_plane_desc * DN_MAX_PLANES_PER_IMAGE)()
    n = ctypes.c_int32()
    e = ctypes.c_int64()
    need = ctypes.c_size_t()
    L = lib()
    check(L.densenet_build_pyramid(None, n_img, H, W, ctypes.byref(p), dtype, None, 0,
                                   ctypes.byref(need), geom, planes, DN_MAX_PLANES_PER_IMAGE,
                                   ctypes.byref(n), ctypes.byref(e), None))
    es = 4 if dtype == DN_F32 else 2
    if out is None:
        out = torch.empty(need.value // es, dtype=_tdtype(dtype), device=images.device)
    check(L.densenet_build_pyramid(_ptr(images), n_img, H, W, ctypes.byref(p), dtype, _ptr(out),
                                   out.numel() * out.element_size(), ctypes.byref(need), geom, planes,
                                   DN_MAX_PLANES_PER_IMAGE, ctypes.byref(n), ctypes.byref(e),
                                   _stream()))
    return out, PlanResult(list(geom), list(planes[:n.value]), e.value)


def densenet_build_pyramid_noalloc(images, p: dn_pyramid_params, dtype: int, out=None):
    """As densenet_build_pyramid, with the builder's staging in the library's static array: `out` (the
    planes only) is the only device buffer.  Returns (planes tensor, PlanResult)."""
    torch = _torch()
    if images.dim() == 3:
        images = images[None]
    n_img, _, H, W = images.shape
    geom = (dn_scale_geom * n_entries(p))()
    planes = (dn_plane_desc * DN_MAX_PLANES_PER_IMAGE)()
    n = ctypes.c_int32()
    e = ctypes.c_int64()
    need = ctypes.c_size_t()
    L = lib()
    check(L.densenet_build_pyramid_noalloc(None, n_img, H, W, ctypes.byref(p), dtype, None, 0,
                                           ctypes.byref(need), geom, planes, DN_MAX_PLANES_PER_IMAGE,
                                           ctypes.byref(n), ctypes.byref(e), None))
    es = 4 if dtype == DN_F32 else 2
    if out is None:
        out = torch.empty(need.value // es, dtype=_tdtype(dtype), device=images.device)
    check(L.densenet_build_pyramid_noalloc(_ptr(images), n_img, H, W, ctypes.byref(p), dtype, _ptr(out),
                                           out.numel() * out.element_size(), ctypes.byref(need), geom,
                                           planes, DN_MAX_PLANES_PER_IMAGE, ctypes.byref(n),
                                           ctypes.byref(e), _stream()))
    return out, PlanResult(list(geom), list(planes[:n.value]), e.value)


class BatchPlan:
    """Cross-image packing (Sec. 3.1 stitching over a whole batch): the plan of n_img images of H x W,
    its host geometry (entry e of image b at b * E + e) and a device copy of it for the kernels,
    uploaded once."""

    def __init__(self, n_img: int, H: int, W: int, p: dn_pyramid_params, device="cuda"):
        """device=None plans on the host only (no device copy)."""
        self.n_img, self.H, self.W, self.params = n_img, H, W, p
        self.E = n_entries(p)
        self.geom = (dn_scale_geom * (n_img * self.E))()
        n, e = ctypes.c_int32(), ctypes.c_int64()
        cap = n_img * self.E
        planes = (dn_plane_desc * cap)()
        check(lib().densenet_plan_batch(n_img, H, W, ctypes.byref(p), self.geom, planes, cap,
                                        ctypes.byref(n), ctypes.byref(e)))
        self.planes = list(planes[:n.value])
        self.total_elems = e.value
        self.d_geom = None
        if device is not None:
            raw = np.frombuffer(bytes(self.geom), np.uint8).copy()
            self.d_geom = _torch().from_numpy(raw).to(device)

    @property
    def n_planes(self) -> int:
        return len(self.planes)

    def entry(self, b: int, e: int) -> dn_scale_geom:
        return self.geom[b * self.E + e]

    def geom_array(self) -> np.ndarray:
        """[n_img * E][14] int32: k, h, w, plane, y, x, rh, rw, r0, r1, c0, c1, aspect, image."""
        return np.array([[getattr(g, f) for f in ("k", "h", "w", "plane", "y", "x", "rh", "rw", "r0",
                                                   "r1", "c0", "c1", "aspect", "image")]
                         for g in self.geom], np.int32)


def densenet_build_batch(images, plan: BatchPlan, dtype: int, out=None):
    """images: uint8 device tensor [n_img][3][H][W] -> the packed batch's planes (flat tensor; plane j
    at j * 3 * plane_h * pitch, followed by the builder's scratch; views: plane_view(out, plan.planes[j]))."""
    torch = _torch()
    n_img, _, H, W = images.shape
    assert (n_img, H, W) == (plan.n_img, plan.H, plan.W), "images do not match the plan"
    need = ctypes.c_size_t()
    L = lib()
    check(L.densenet_build_batch(None, n_img, H, W, ctypes.byref(plan.params), dtype, plan.geom, None,
                                 plan.n_planes, None, 0, ctypes.byref(need), None))
    es = 4 if dtype == DN_F32 else 2
    if out is None:
        out = torch.empty(need.value // es, dtype=_tdtype(dtype), device=images.device)
    check(L.densenet_build_batch(_ptr(images), n_img, H, W, ctypes.byref(plan.params), dtype, plan.geom,
                                 _ptr(plan.d_geom), plan.n_planes, _ptr(out),
                                 out.numel() * out.element_size(), ctypes.byref(need), _stream()))
    return out


def densenet_region_windows_batch(conv5, conv5_desc, dtype: int, plan: BatchPlan, boxes, box_img=None,
                                  target=227.0, S=6, pooled=False, want_idx=False, out=None, scale=None):
    """Region windows (pooled=False) or max-pooled bins (pooled=True) over a cross-image packed batch."""
    torch = _torch()
    n = boxes.shape[0]
    if out is None:
        out = torch.empty((n, 256 * S * S), dtype=torch.float32, device=boxes.device)
    if scale is None:
        scale = torch.empty(n, dtype=torch.int32, device=boxes.device)
    idx = torch.empty((n, S, S, 4 if pooled else 2), dtype=torch.int32, device=boxes.device) if want_idx \
        else None
    cd = (dn_plane_desc * len(conv5_desc))(*conv5_desc)
    check(lib().densenet_region_windows_batch(_ptr(conv5), cd, len(conv5_desc), dtype, plan.geom,
                                              _ptr(plan.d_geom), plan.n_img, plan.E, plan.params.pad,
                                              int(pooled), _ptr(boxes), _ptr(box_img), n, target, S,
                                              _ptr(out), _ptr(scale), _ptr(idx), _stream()))
    return out, scale, idx


def densenet_pack_weights(weights, dtype: int):
    """weights: [(w, b)] conv1..conv5 as fp32 device tensors (OIHW).  Returns the packed blob."""
    torch = _torch()
    ws = [w.contiguous().float() for w, _ in weights]
    bs = [b.contiguous().float() for _, b in weights]
    wp = (ctypes.c_void_p * 5)(*[w.data_ptr() for w in ws])
    bp = (ctypes.c_void_p * 5)(*[b.data_ptr() for b in bs])
    need = ctypes.c_size_t()
    L = lib()
    check(L.densenet_pack_weights(wp, bp, dtype, None, 0, ctypes.byref(need), None))
    blob = torch.empty(need.value, dtype=torch.uint8, device=ws[0].device)
    check(L.densenet_pack_weights(wp, bp, dtype, _ptr(blob), need.value, ctypes.byref(need),
                                  _stream()))
    return blob


class ConvFeatures:
    """Reusable buffers for densenet_conv_features over a fixed plane list."""

    def __init__(self, planes_desc, dtype: int, net: dn_net_params, device="cuda"):
        torch = _torch()
        self.n = len(planes_desc)
        self.pd = (dn_plane_desc * self.n)(*planes_desc)
        self.dtype, self.net = dtype, net
        self.c5d = (dn_plane_desc * self.n)()
        self.p5d = (dn_plane_desc * self.n)()
        ws, c5, p5 = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        check(lib().densenet_conv_features(None, self.pd, self.n, dtype, None, ctypes.byref(net), None,
                                           0, ctypes.byref(ws), None, 0, ctypes.byref(c5), self.c5d,
                                           None, 0, ctypes.byref(p5), self.p5d, None))
        es = 4 if dtype == DN_F32 else 2
        self.workspace = torch.empty(max(ws.value, 1), dtype=torch.uint8, device=device)
        self.conv5 = torch.empty(c5.value // es, dtype=_tdtype(dtype), device=device)
        self.pool5 = torch.empty(p5.value // es, dtype=_tdtype(dtype), device=device) if net.pool5 else None

    def __call__(self, planes_tensor, packed):
        check(lib().densenet_conv_features(
            _ptr(planes_tensor), self.pd, self.n, self.dtype, _ptr(packed), ctypes.byref(self.net),
            _ptr(self.workspace), self.workspace.numel(), ctypes.byref(ctypes.c_size_t()),
            _ptr(self.conv5), self.conv5.numel() * self.conv5.element_size(),
            ctypes.byref(ctypes.c_size_t()), self.c5d, _ptr(self.pool5),
            0 if self.pool5 is None else self.pool5.numel() * self.pool5.element_size(),
            ctypes.byref(ctypes.c_size_t()), self.p5d, _stream()))
        return self.conv5, self.pool5

    def conv5_maps(self):
        """Per-plane [Hc][Wc][256] views of the conv5 buffer."""
        return [self.conv5[d.offset:d.offset + d.h * d.w * 256].view(d.h, d.w, 256) for d in self.c5d]

    def pool5_maps(self):
        return [self.pool5[d.offset:d.offset + d.h * d.w * 256].view(d.h, d.w, 256) for d in self.p5d]


def densenet_conv_features(planes_tensor, planes_desc, dtype: int, packed, net: dn_net_params):
    cf = ConvFeatures(planes_desc, dtype, net, device=planes_tensor.device)
    cf(planes_tensor, packed)
    return cf


def _regions(fn, conv5, conv5_desc, dtype, plan, pad, planes_per_img, boxes, box_img, target, S, want_idx,
             out, scale, idx_width):
    torch = _torch()
    n = boxes.shape[0]
    if out is None:
        out = torch.empty((n, 256 * S * S), dtype=torch.float32, device=boxes.device)
    if scale is None:
        scale = torch.empty(n, dtype=torch.int32, device=boxes.device)
    idx = torch.empty((n, S, S, idx_width), dtype=torch.int32, device=boxes.device) if want_idx else None
    geom = (dn_scale_geom * len(plan.geom))(*plan.geom)
    cd = (dn_plane_desc * len(conv5_desc))(*conv5_desc)
    check(fn(_ptr(conv5), cd, len(conv5_desc), dtype, geom, len(plan.geom), pad, planes_per_img,
             _ptr(boxes), _ptr(box_img), n, target, S, _ptr(out), _ptr(scale), _ptr(idx), _stream()))
    return out, scale, idx


def densenet_region_windows(conv5, conv5_desc, dtype: int, plan: PlanResult, pad: int, planes_per_img,
                            boxes, box_img=None, target=227.0, S=6, want_idx=False, out=None,
                            scale=None):
    """Region windows (Sec. 4, crop after): bilinear samples at the S x S bin centres of each box."""
    return _regions(lib().densenet_region_windows, conv5, conv5_desc, dtype, plan, pad, planes_per_img,
                    boxes, box_img, target, S, want_idx, out, scale, 2)


def densenet_region_pool(conv5, conv5_desc, dtype: int, plan: PlanResult, pad: int, planes_per_img,
                         boxes, box_img=None, target=227.0, S=6, want_idx=False, out=None, scale=None):
    """Max-pooled region bins: per-channel max over the conv5 cells centred inside each of the S x S
    bins of each box (idx: first/last row, first/last column of each bin)."""
    return _regions(lib().densenet_region_pool, conv5, conv5_desc, dtype, plan, pad, planes_per_img,
                    boxes, box_img, target, S, want_idx, out, scale, 4)


def densenet_warp_regions(images, boxes, dtype: int, S=227, mean=(0.0, 0.0, 0.0), box_img=None, out=None,
                          pitch=0):
    """Crop-before windows (Sec. 3.4 per-window baseline, Sec. 4): uint8 images [n_img][3][H][W], boxes
    [n][4] fp32 -> [n][3][S][pitch or S] mean-centred windows in `dtype` (columns past S are 0)."""
    torch = _torch()
    if images.dim() == 3:
        images = images[None]
    n_img, _, H, W = images.shape
    n = boxes.shape[0]
    P = pitch or S
    if out is None:
        out = torch.empty((n, 3, S, P), dtype=_tdtype(dtype), device=boxes.device)
    m = (ctypes.c_float * 3)(*[float(v) for v in mean])
    check(lib().densenet_warp_regions(_ptr(images), n_img, H, W, _ptr(boxes), _ptr(box_img), n, S, pitch, m,
                                      dtype, _ptr(out), out.numel() * out.element_size(),
                                      ctypes.byref(ctypes.c_size_t()), _stream()))
    return out


class PerWindow:
    """The per-window baseline (Sec. 3.4): every box warped to S x S on its own, then the whole conv stack
    with pool5 on each window as an independent plane (one launch per layer over all windows).  The
    per-window descriptor is the window's pool5 map, [n][Hp][Wp][256] (6 x 6 x 256 at S = 227).
    Window rows are padded to a multiple of 8 elements (zeros past S) so that conv1 loads them straight
    into LDS; the padding never reaches a stored output."""

    def __init__(self, n: int, dtype: int, S=227, device="cuda", net=None):
        torch = _torch()
        self.n, self.S, self.dtype = n, S, dtype
        self.pitch = (S + 7) // 8 * 8
        net = net or net_params(pool5=True)
        net.pool5 = 1
        desc = []
        for i in range(n):
            q = dn_plane_desc()
            q.h, q.w, q.offset, q.pitch = S, S, i * 3 * S * self.pitch, self.pitch
            desc.append(q)
        self.windows = torch.empty((n, 3, S, self.pitch), dtype=_tdtype(dtype), device=device)
        self.conv = ConvFeatures(desc, dtype, net, device=device)
        hp = self.conv.p5d[0]
        self.pool5_shape = (n, hp.h, hp.w, 256)

    def __call__(self, images, boxes, packed, mean=(0.0, 0.0, 0.0), box_img=None):
        densenet_warp_regions(images, boxes, self.dtype, self.S, mean, box_img, out=self.windows,
                              pitch=self.pitch)
        self.conv(self.windows, packed)
        return self.conv.pool5[: self.pool5_shape[0] * self.pool5_shape[1] * self.pool5_shape[2] * 256].view(
            self.pool5_shape)


def densenet_conv_layer(layer: int, x, n: int, H: int, W: int, dtype: int, packed):
    torch = _torch()
    hw = layer_sizes(H, W, strict=False) if layer == 1 else None
    M = (96, 256, 384, 384, 256)[layer - 1]
    Ho, Wo = (hw[0] if layer == 1 else (H, W))
    out = torch.empty((n, Ho, Wo, M), dtype=_tdtype(dtype), device=x.device)
    check(lib().densenet_conv_layer(layer, _ptr(x), n, H, W, dtype, _ptr(packed), _ptr(out), _stream()))
    return out


def _pool_side(v):
    return (v - 2) // 2 + 1 if v >= 2 else 0


def densenet_lrn_pool(x, dtype: int, net: dn_net_params):
    torch = _torch()
    n, H, W, C = x.shape
    out = torch.empty((n, _pool_side(H), _pool_side(W), C), dtype=_tdtype(dtype), device=x.device)
    check(lib().densenet_lrn_pool(_ptr(x), n, H, W, C, dtype, ctypes.byref(net), _ptr(out), _stream()))
    return out


def densenet_maxpool(x, dtype: int):
    torch = _torch()
    n, H, W, C = x.shape
    out = torch.empty((n, _pool_side(H), _pool_side(W), C), dtype=_tdtype(dtype), device=x.device)
    check(lib().densenet_maxpool(_ptr(x), n, H, W, C, dtype, _ptr(out), _stream()))
    return out


def layer_sizes(H: int, W: int, strict=True):
    hw = (ctypes.c_int32 * 16)()
    st = lib().densenet_layer_sizes(H, W, hw)
    if strict:
        check(st)
    return [(hw[2 * i], hw[2 * i + 1]) for i in range(8)]


def profile_start(names=None):
    """Trace launches (all, or those named in `names`) with events on their own streams."""
    check(lib().densenet_profile_start(",".join(names).encode() if names else None))


def profile_stop():
    """Stop tracing; returns {name: (launches, total_ms)} (waits for the traced launches)."""
    out = (dn_profile_entry * 64)()
    n = ctypes.c_int32()
    check(lib().densenet_profile_stop(out, 64, ctypes.byref(n)))
    return {out[i].name.decode(): (out[i].launches, out[i].total_ms) for i in range(min(n.value, 64))}


# ------------------------------------------------------------------------------------------------
# The paper's interface: pyra = convnet_featpyramid(image)
# ------------------------------------------------------------------------------------------------
@dataclass
class Pyramid:
    feat: list            # per scale: [rows][cols][256] view of its plane's conv5 map
    scales: np.ndarray    # [K] scale factors s_k
    plan: PlanResult
    planes: object        # the stitched planes tensor
    conv: ConvFeatures
    n_img: int


def convnet_featpyramid(images, p: dn_pyramid_params, packed, dtype: int, net=None) -> Pyramid:
    """Image(s) (uint8 device tensor [n][3][H][W]) -> per-scale conv5 maps (views) + geometry."""
    if images.dim() == 3:
        images = images[None]
    net = net or net_params()
    planes, plan = densenet_build_pyramid(images, p, dtype)
    n_img = images.shape[0]
    cf = densenet_conv_features(planes, plan.image_descs(n_img), dtype, packed, net)
    maps = cf.conv5_maps()
    feat = []
    npl = len(plan.planes)
    for b in range(n_img):
        for g in plan.geom:
            feat.append(maps[b * npl + g.plane][g.r0:g.r1 + 1, g.c0:g.c1 + 1])
    return Pyramid(feat, np.array([g.s for g in plan.geom]), plan, planes, cf, n_img)


def convnet_featpyramid_batch(images, p: dn_pyramid_params, packed, dtype: int, net=None,
                              plan: BatchPlan | None = None) -> Pyramid:
    """A batch of images stitched together (cross-image packing) -> per-(image, scale) conv5 maps
    (views, image-major) + the batch plan."""
    net = net or net_params()
    n_img, _, H, W = images.shape
    plan = plan or BatchPlan(n_img, H, W, p, device=images.device)
    planes = densenet_build_batch(images, plan, dtype)
    cf = densenet_conv_features(planes, plan.planes, dtype, packed, net)
    maps = cf.conv5_maps()
    feat = [maps[g.plane][g.r0:g.r1 + 1, g.c0:g.c1 + 1] for g in plan.geom]
    return Pyramid(feat, np.array([plan.geom[e].s for e in range(plan.E)]), plan, planes, cf, n_img)
