"""CPU oracle for the DenseNet conv5 descriptor-pyramid path (arXiv 1404.1869).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The GPU library never imports, links or
calls it, and it never imports the GPU library.

The arithmetic lives in ``oracle.cpp`` (plain C++17 + OpenMP, fp64); this module only marshals numpy
arrays through ctypes.  Array conventions are the natural ones of the paper's description: images and
planes are channel-major ``[C][H][W]``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = False) -> str:
    """Compile oracle.cpp into liboracle.so with g++ (no HIP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-fopenmp", "-ffp-contract=off", "-fPIC",
                               "-shared", _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, f64 = ctypes.c_int, ctypes.c_double
        L.oracle_plan.argtypes = [i32, i32, i32, i32, f64, i32, i32, i32, i32, i32, P, P, P]
        L.oracle_plan.restype = i32
        L.oracle_plan_batch.argtypes = [i32] + L.oracle_plan.argtypes
        L.oracle_plan_batch.restype = i32
        L.oracle_resize_center.argtypes = [P, i32, i32, i32, i32, P, P]
        L.oracle_resize_center.restype = None
        L.oracle_build_planes.argtypes = [P, i32, i32, i32, P, P, i32, i32, P, i32, i32, i32, P]
        L.oracle_build_planes.restype = None
        L.oracle_warp_regions.argtypes = [P, i32, i32, i32, P, P, i32, i32, P, P]
        L.oracle_warp_regions.restype = None
        L.oracle_conv2d.argtypes = [P, i32, i32, i32, P, P, i32, i32, i32, i32, i32, i32, P]
        L.oracle_conv2d.restype = i32
        L.oracle_lrn.argtypes = [P, i32, i32, i32, i32, f64, f64, f64, P]
        L.oracle_lrn.restype = i32
        L.oracle_maxpool.argtypes = [P, i32, i32, i32, i32, i32, P]
        L.oracle_maxpool.restype = i32
        L.oracle_net.argtypes = [P, i32, i32, P, P, f64, f64, f64, i32, i32, P, P]
        L.oracle_net.restype = i32
        L.oracle_region_windows.argtypes = [P, P, P, P, i32, i32, P, P, i32, P, P, i32, f64, i32,
                                            i32, P, P, P, P]
        L.oracle_region_windows.restype = i32
        L.oracle_region_pool.argtypes = [P, P, P, P, i32, i32, P, P, i32, P, P, i32, f64, i32, i32,
                                         P, P, P]
        L.oracle_region_pool.restype = i32
        for name in ("oracle_conv5_side", "oracle_pool_side"):
            getattr(L, name).argtypes = [i32]
            getattr(L, name).restype = i32
        L.oracle_threads.argtypes = []
        L.oracle_threads.restype = i32
        L.oracle_conv_side.argtypes = [i32, i32, i32, i32]
        L.oracle_conv_side.restype = i32
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


# ----------------------------------------------------------------------------------------------
# Geometry
# ----------------------------------------------------------------------------------------------
GI_FIELDS = ("k", "h", "w", "plane", "y", "x", "rh", "rw", "r0", "r1", "c0", "c1", "plane_h",
             "plane_w", "aspect", "image")


@dataclass
class Plan:
    gi: np.ndarray          # [K][16] int32, fields GI_FIELDS
    gd: np.ndarray          # [K][3] float64: s, sy, sx
    n_planes: int
    pad: int
    plane_sizes: list       # [(PH, PW)] per plane
    n_aspects: int = 0
    n_img: int = 1          # images whose entries the rows hold (cross-image packing: n_img > 1)
    packed: bool = False    # rows are n_img blocks of entries stitched over the batch

    @property
    def entries(self) -> int:
        """Pyramid entries per image."""
        return self.gi.shape[0] // self.n_img

    def field(self, name):
        return self.gi[:, GI_FIELDS.index(name)]


def plan(H, W, K, spo, base_scale=1.0, base_longest_side=0, pad=0, plane_h=0, plane_w=0,
         aspects=None) -> Plan:
    """Scales, sizes, rectangles, stitching and conv5 windows (Sec. 3.1); with `aspects`, one pyramid
    per aspect ratio, all stitched together (Sec. 3.3), entries aspect-major."""
    asp = np.ascontiguousarray(aspects if aspects is not None else [], np.float64)
    E = K * max(1, len(asp))
    gi = np.zeros((E, 16), np.int32)
    gd = np.zeros((E, 3), np.float64)
    n = lib().oracle_plan(H, W, K, spo, float(base_scale), base_longest_side, pad, plane_h, plane_w,
                          len(asp), _p(asp) if len(asp) else None, _p(gi), _p(gd))
    if n < 0:
        raise ValueError(f"oracle_plan failed with {n}")
    sizes = [None] * n
    for k in range(E):
        sizes[gi[k, 3]] = (int(gi[k, 12]), int(gi[k, 13]))
    return Plan(gi, gd, n, pad, sizes, len(asp))


def plan_batch(n_img, H, W, K, spo, base_scale=1.0, base_longest_side=0, pad=0, plane_h=0, plane_w=0,
               aspects=None) -> Plan:
    """Cross-image packing: the rectangles of all n_img images (each H x W) stitched as one set of items
    (Sec. 3.1 stitching over a batch).  Row b * E + e is entry e of image b; plane indices count over the
    batch."""
    asp = np.ascontiguousarray(aspects if aspects is not None else [], np.float64)
    E = K * max(1, len(asp))
    gi = np.zeros((n_img * E, 16), np.int32)
    gd = np.zeros((n_img * E, 3), np.float64)
    n = lib().oracle_plan_batch(n_img, H, W, K, spo, float(base_scale), base_longest_side, pad, plane_h,
                                plane_w, len(asp), _p(asp) if len(asp) else None, _p(gi), _p(gd))
    if n < 0:
        raise ValueError(f"oracle_plan_batch failed with {n}")
    return Plan(gi, gd, n, pad, [(plane_h, plane_w)] * n, len(asp), n_img, True)


def threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return lib().oracle_threads()


def conv5_side(n: int) -> int:
    return lib().oracle_conv5_side(n)


def pool_side(n: int) -> int:
    return lib().oracle_pool_side(n)


def conv_side(n: int, R: int, s: int, p: int) -> int:
    return lib().oracle_conv_side(n, R, s, p)


# ----------------------------------------------------------------------------------------------
# Pyramid
# ----------------------------------------------------------------------------------------------
def resize_center(img: np.ndarray, h: int, w: int, mean) -> np.ndarray:
    """Bilinear half-pixel resize of a uint8 [3][H][W] image to h x w, minus the mean pixel (fp64)."""
    img = np.ascontiguousarray(img, np.uint8)
    _, H, W = img.shape
    m = np.ascontiguousarray(mean, np.float64)
    out = np.zeros((3, h, w), np.float64)
    lib().oracle_resize_center(_p(img), H, W, h, w, _p(m), _p(out))
    return out


def build_planes(img: np.ndarray, pl: Plan, pad_mode: int, mean) -> list:
    """Stitched, centred, padded planes of one image ([3][H][W]), or of a cross-image packed batch
    ([n_img][3][H][W] with a plan_batch plan), as a list of fp64 [3][PH][PW] arrays."""
    img = np.ascontiguousarray(img, np.uint8)
    if img.ndim == 3:
        img = img[None]
    if img.shape[0] < pl.n_img:
        raise ValueError("fewer images than the plan holds")
    _, _, H, W = img.shape
    PHm = max(s[0] for s in pl.plane_sizes)
    PWm = max(s[1] for s in pl.plane_sizes)
    m = np.ascontiguousarray(mean, np.float64)
    buf = np.zeros((pl.n_planes, 3, PHm, PWm), np.float64)
    lib().oracle_build_planes(_p(img), H, W, pl.gi.shape[0], _p(pl.gi), _p(pl.gd), pl.pad, pad_mode,
                              _p(m), pl.n_planes, PHm, PWm, _p(buf))
    return [np.ascontiguousarray(buf[i, :, :ph, :pw]) for i, (ph, pw) in enumerate(pl.plane_sizes)]


def warp_regions(images: np.ndarray, boxes: np.ndarray, S=227, mean=(0.0, 0.0, 0.0), box_img=None):
    """Crop-before windows (Sec. 3.4, Sec. 4): each box cut from its uint8 [3][H][W] image and warped
    bilinearly to S x S with half-pixel centres, minus the mean pixel.  images: [3][H][W] or
    [n_img][3][H][W]; boxes: [n][4] fp32 (x1, y1, x2, y2).  Returns fp32 [n][3][S][S]."""
    images = np.ascontiguousarray(images, np.uint8)
    if images.ndim == 3:
        images = images[None]
    n_img, _, H, W = images.shape
    boxes = np.ascontiguousarray(boxes, np.float32).reshape(-1, 4)
    n = boxes.shape[0]
    bi = None if box_img is None else np.ascontiguousarray(box_img, np.int32)
    m = np.ascontiguousarray(mean, np.float64)
    out = np.zeros((n, 3, S, S), np.float32)
    lib().oracle_warp_regions(_p(images), n_img, H, W, _p(boxes), None if bi is None else _p(bi), n, S,
                              _p(m), _p(out))
    return out


# ----------------------------------------------------------------------------------------------
# Layers
# ----------------------------------------------------------------------------------------------
def conv2d(x: np.ndarray, w: np.ndarray, b: np.ndarray, stride=1, pad=0, groups=1, relu=True):
    x = np.ascontiguousarray(x, np.float32)
    w = np.ascontiguousarray(w, np.float32)
    b = np.ascontiguousarray(b, np.float32)
    C, Hi, Wi = x.shape
    M, _, R, _ = w.shape
    Ho, Wo = conv_side(Hi, R, stride, pad), conv_side(Wi, R, stride, pad)
    out = np.zeros((M, Ho, Wo), np.float32)
    rc = lib().oracle_conv2d(_p(x), C, Hi, Wi, _p(w), _p(b), M, R, stride, pad, groups, int(relu),
                             _p(out))
    if rc:
        raise ValueError("oracle_conv2d: bad arguments")
    return out


def lrn(x: np.ndarray, n=5, alpha=1e-4, beta=0.75, k=1.0):
    x = np.ascontiguousarray(x, np.float32)
    C, H, W = x.shape
    out = np.zeros_like(x)
    if lib().oracle_lrn(_p(x), C, H, W, n, alpha, beta, k, _p(out)):
        raise ValueError("oracle_lrn: bad arguments")
    return out


def maxpool(x: np.ndarray, R=3, s=2):
    x = np.ascontiguousarray(x, np.float32)
    C, H, W = x.shape
    Ho, Wo = pool_side(H) if (R, s) == (3, 2) else None, pool_side(W) if (R, s) == (3, 2) else None
    if Ho is None:
        raise ValueError("only 3x3/2 pooling has a size helper")
    out = np.zeros((C, Ho, Wo), np.float32)
    if lib().oracle_maxpool(_p(x), C, H, W, R, s, _p(out)):
        raise ValueError("oracle_maxpool: bad arguments")
    return out


def net(plane: np.ndarray, weights, lrn_params=(1e-4, 0.75, 1.0, 5), lrn_before_pool=True,
        pool5=False):
    """conv1..conv5 (+pool5) on one [3][PH][PW] plane.  weights = [(w1,b1),...,(w5,b5)] fp32."""
    plane = np.ascontiguousarray(plane, np.float32)
    _, PH, PW = plane.shape
    Hc, Wc = conv5_side(PH), conv5_side(PW)
    if Hc <= 0 or Wc <= 0:
        raise ValueError("plane too small for the network")
    ws = [np.ascontiguousarray(w, np.float32) for w, _ in weights]
    bs = [np.ascontiguousarray(b, np.float32) for _, b in weights]
    wp = (ctypes.c_void_p * 5)(*[w.ctypes.data for w in ws])
    bp = (ctypes.c_void_p * 5)(*[b.ctypes.data for b in bs])
    c5 = np.zeros((256, Hc, Wc), np.float32)
    p5 = np.zeros((256, pool_side(Hc), pool_side(Wc)), np.float32) if pool5 else None
    a, be, k, n = lrn_params
    rc = lib().oracle_net(_p(plane), PH, PW, wp, bp, a, be, k, n, int(lrn_before_pool), _p(c5),
                          _p(p5) if pool5 else None)
    if rc:
        raise ValueError("oracle_net failed")
    return (c5, p5) if pool5 else c5


# ----------------------------------------------------------------------------------------------
# Region windows
# ----------------------------------------------------------------------------------------------
def region_windows(conv5_planes: list, pl: Plan, boxes: np.ndarray, box_img=None, T=227.0, S=6):
    """conv5_planes: list over (image, plane) of fp32 [256][Hc][Wc] (over the batch's planes for a
    plan_batch plan); returns desc, scale, idx, lam."""
    flat = np.concatenate([np.ascontiguousarray(c, np.float32).ravel() for c in conv5_planes])
    offs = np.cumsum([0] + [c.size for c in conv5_planes[:-1]]).astype(np.int64)
    Hcs = np.array([c.shape[1] for c in conv5_planes], np.int32)
    Wcs = np.array([c.shape[2] for c in conv5_planes], np.int32)
    boxes = np.ascontiguousarray(boxes, np.float32)
    n = boxes.shape[0]
    bi = None if box_img is None else np.ascontiguousarray(box_img, np.int32)
    desc = np.zeros((n, 256 * S * S), np.float32)
    scale = np.zeros(n, np.int32)
    idx = np.zeros((n, S, S, 2), np.int32)
    lam = np.zeros((n, S, S, 2), np.float64)
    rc = lib().oracle_region_windows(_p(flat), _p(offs), _p(Hcs), _p(Wcs), 0 if pl.packed else pl.n_planes,
                                     pl.entries, _p(pl.gi), _p(pl.gd), pl.pad, _p(boxes),
                                     _p(bi) if bi is not None else None, n, float(T), S,
                                     pl.n_aspects, _p(desc), _p(scale), _p(idx), _p(lam))
    if rc:
        raise ValueError("oracle_region_windows: bad arguments")
    return desc, scale, idx, lam


def region_pool(conv5_planes: list, pl: Plan, boxes: np.ndarray, box_img=None, T=227.0, S=6):
    """Max-pooled region bins: the box read at the same entry as region_windows, each of its S x S bins
    the per-channel max over the conv5 cells centred inside it.  Returns desc [n][256*S*S], scale [n],
    idx [n][S][S][4] (i_first, i_last, j_first, j_last)."""
    flat = np.concatenate([np.ascontiguousarray(c, np.float32).ravel() for c in conv5_planes])
    offs = np.cumsum([0] + [c.size for c in conv5_planes[:-1]]).astype(np.int64)
    Hcs = np.array([c.shape[1] for c in conv5_planes], np.int32)
    Wcs = np.array([c.shape[2] for c in conv5_planes], np.int32)
    boxes = np.ascontiguousarray(boxes, np.float32)
    n = boxes.shape[0]
    bi = None if box_img is None else np.ascontiguousarray(box_img, np.int32)
    desc = np.zeros((n, 256 * S * S), np.float32)
    scale = np.zeros(n, np.int32)
    idx = np.zeros((n, S, S, 4), np.int32)
    rc = lib().oracle_region_pool(_p(flat), _p(offs), _p(Hcs), _p(Wcs), 0 if pl.packed else pl.n_planes,
                                  pl.entries,
                                  _p(pl.gi), _p(pl.gd), pl.pad, _p(boxes),
                                  _p(bi) if bi is not None else None, n, float(T), S, pl.n_aspects,
                                  _p(desc), _p(scale), _p(idx))
    if rc:
        raise ValueError("oracle_region_pool: bad arguments")
    return desc, scale, idx
