"""The C-ABI library loads on a machine without a GPU, exports every entry point that
include/densenet.h declares, and rejects bad arguments on the host before any device work."""
import ctypes
import os
import re

import pytest

from paper_1404_1869_amd import densenet as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    text = open(os.path.join(ROOT, "include", "densenet.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(densenet_\w+)\s*\(", text, re.M)))


def test_exports_match_header():
    names = declared()
    assert len(names) >= 10
    L = D.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(D.EXPORTS) == set(names)


def test_plan_errors():
    p = D.pyramid_params(3, 10, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=700, plane_w=700)
    with pytest.raises(D.DenseNetError) as e:
        D.densenet_plan_pyramid(768, 1024, p)
    assert e.value.status == D.DN_E_TOO_LARGE and "larger than" in D.last_error()
    for bad in (dict(n_scales=0), dict(steps_per_octave=0), dict(pad=-1), dict(plane_h=5),
                dict(pad_mode=7), dict(base_scale=0.0)):
        kw = dict(n_scales=3, steps_per_octave=2, pad=16, pad_mode=D.DN_PAD_ZERO)
        kw.update(bad)
        p = D.pyramid_params(**kw)
        with pytest.raises(D.DenseNetError) as e:
            D.densenet_plan_pyramid(100, 100, p)
        assert e.value.status == D.DN_E_INVALID_ARG, bad
    with pytest.raises(D.DenseNetError):
        D.densenet_plan_pyramid(0, 100, D.pyramid_params(2, 2))


def test_size_queries_without_device():
    L = D.lib()
    p = D.pyramid_params(25, 10, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=1200, plane_w=1200)
    geom = (D.dn_scale_geom * 25)()
    planes = (D.dn_plane_desc * 64)()
    n, e, need = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_size_t()
    assert L.densenet_build_pyramid(None, 16, 768, 1024, ctypes.byref(p), D.DN_BF16, None, 0,
                                    ctypes.byref(need), geom, planes, 64, ctypes.byref(n),
                                    ctypes.byref(e), None) == 0
    assert n.value == 6 and e.value == 6 * 3 * 1200 * 1216   # rows padded to 1216 elements
    # the planes, then the builder's scratch (4 bytes per image pixel) 256-byte aligned after them
    full = (16 * e.value * 2 + 255) // 256 * 256 + 16 * 4 * 768 * 1024
    assert need.value == full
    # short buffer: error, needed size still reported (no device work happens)
    fake = ctypes.c_void_p(256)
    assert L.densenet_build_pyramid(fake, 16, 768, 1024, ctypes.byref(p), D.DN_BF16, fake, 10,
                                    ctypes.byref(need), geom, planes, 64, ctypes.byref(n),
                                    ctypes.byref(e), None) == D.DN_E_BUFFER_TOO_SMALL
    assert need.value == full
    assert L.densenet_build_pyramid(None, 1, 768, 1024, ctypes.byref(p), 9, None, 0,
                                    ctypes.byref(need), geom, planes, 64, ctypes.byref(n),
                                    ctypes.byref(e), None) == D.DN_E_UNSUPPORTED
    # packed weights size query
    assert L.densenet_pack_weights(None, None, D.DN_F16, None, 0, ctypes.byref(need), None) == 0
    assert need.value > 2 * 2_300_000


def test_conv_features_size_query_and_validation():
    L = D.lib()
    net = D.net_params(pool5=True)
    pd = (D.dn_plane_desc * 2)()
    pd[0].h, pd[0].w, pd[0].offset = 1200, 1200, 0
    pd[1].h, pd[1].w, pd[1].offset = 1200, 1200, 3 * 1200 * 1200
    c5d, p5d = (D.dn_plane_desc * 2)(), (D.dn_plane_desc * 2)()
    ws, c5, p5 = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    assert L.densenet_conv_features(None, pd, 2, D.DN_F16, None, ctypes.byref(net), None, 0,
                                    ctypes.byref(ws), None, 0, ctypes.byref(c5), c5d, None, 0,
                                    ctypes.byref(p5), p5d, None) == 0
    assert (c5d[0].h, c5d[0].w, c5d[1].offset) == (74, 74, 74 * 74 * 256)
    assert c5.value == 2 * 74 * 74 * 256 * 2 and p5.value == 2 * 37 * 37 * 256 * 2
    assert ws.value >= 2 * 298 * 298 * 96 * 2
    pd[1].h = 20                     # too small for conv5
    assert L.densenet_conv_features(None, pd, 2, D.DN_F16, None, ctypes.byref(net), None, 0,
                                    ctypes.byref(ws), None, 0, ctypes.byref(c5), c5d, None, 0,
                                    ctypes.byref(p5), p5d, None) == D.DN_E_INVALID_ARG
    net.lrn_n = 4
    pd[1].h = 1200
    assert L.densenet_conv_features(None, pd, 2, D.DN_F16, None, ctypes.byref(net), None, 0,
                                    ctypes.byref(ws), None, 0, ctypes.byref(c5), c5d, None, 0,
                                    ctypes.byref(p5), p5d, None) == D.DN_E_INVALID_ARG


def test_layer_sizes_and_layer_validation():
    assert D.layer_sizes(1200, 1200) == [(298, 298), (149, 149), (149, 149), (74, 74), (74, 74),
                                         (74, 74), (74, 74), (37, 37)]
    assert D.layer_sizes(227, 227)[6] == (13, 13) and D.layer_sizes(227, 227)[7] == (6, 6)
    with pytest.raises(D.DenseNetError):
        D.layer_sizes(18, 18)
    L = D.lib()
    fake = ctypes.c_void_p(256)
    assert L.densenet_conv_layer(6, fake, 1, 50, 50, D.DN_F16, fake, fake, None) == D.DN_E_INVALID_ARG
    assert L.densenet_conv_layer(1, fake, 1, 10, 50, D.DN_F16, fake, fake, None) == D.DN_E_INVALID_ARG
    assert L.densenet_conv_layer(2, None, 1, 10, 50, D.DN_F16, fake, fake, None) == D.DN_E_INVALID_ARG
    assert L.densenet_region_windows(fake, None, 1, D.DN_F16, None, 1, 16, 1, fake, None, 1, 227.0,
                                     6, fake, fake, None, None) == D.DN_E_INVALID_ARG
    assert L.densenet_region_pool(fake, None, 1, D.DN_F16, None, 1, 16, 1, fake, None, 1, 227.0,
                                  6, fake, fake, None, None) == D.DN_E_INVALID_ARG
    pd = (D.dn_plane_desc * 1)()
    pd[0].h, pd[0].w = 13, 13
    g = (D.dn_scale_geom * 1)()
    assert L.densenet_region_pool(fake, pd, 1, D.DN_F16, g, 1, 16, 1, fake, None, 1, 227.0,
                                  9, fake, fake, None, None) == D.DN_E_UNSUPPORTED   # S > 8
    assert L.densenet_region_pool(fake, pd, 1, D.DN_F16, g, 1, 16, 1, None, None, 0, 227.0,
                                  6, None, None, None, None) == D.DN_OK               # no boxes


def test_warp_regions_size_query_and_validation():
    L = D.lib()
    need = ctypes.c_size_t()
    m = (ctypes.c_float * 3)(1.0, 2.0, 3.0)
    assert L.densenet_warp_regions(None, 1, 768, 1024, None, None, 2000, 227, 0, m, D.DN_BF16, None, 0,
                                   ctypes.byref(need), None) == D.DN_OK
    assert need.value == 2000 * 3 * 227 * 227 * 2
    fake = ctypes.c_void_p(256)
    assert L.densenet_warp_regions(fake, 1, 768, 1024, fake, None, 2000, 227, 0, m, D.DN_BF16, fake, 10,
                                   ctypes.byref(need), None) == D.DN_E_BUFFER_TOO_SMALL
    assert L.densenet_warp_regions(fake, 1, 768, 1024, fake, None, 1, 0, 0, m, D.DN_F32, fake, 1 << 30,
                                   None, None) == D.DN_E_INVALID_ARG
    assert L.densenet_warp_regions(fake, 1, 768, 1024, fake, None, 1, D.DN_MAX_WARP_SIDE + 1, 0, m,
                                   D.DN_F32, fake, 1 << 40, None, None) == D.DN_E_INVALID_ARG
    assert L.densenet_warp_regions(fake, 0, 768, 1024, fake, None, 1, 227, 0, m, D.DN_F32, fake, 1 << 30,
                                   None, None) == D.DN_E_INVALID_ARG
    assert L.densenet_warp_regions(fake, 1, 768, 1024, fake, None, 1, 227, 0, m, 7, fake, 1 << 30, None,
                                   None) == D.DN_E_UNSUPPORTED
    assert L.densenet_warp_regions(None, 1, 768, 1024, None, None, 10, 227, 232, m, D.DN_BF16, None, 0,
                                   ctypes.byref(need), None) == D.DN_OK
    assert need.value == 10 * 3 * 227 * 232 * 2
    assert L.densenet_warp_regions(fake, 1, 768, 1024, fake, None, 10, 227, 200, m, D.DN_BF16, fake,
                                   1 << 30, None, None) == D.DN_E_INVALID_ARG
    # n == 0 launches nothing and accepts null buffers
    assert L.densenet_warp_regions(None, 1, 768, 1024, None, None, 0, 227, 0, None, D.DN_F32, fake, 0,
                                   None, None) == D.DN_OK


def test_batch_entry_points_validation():
    L = D.lib()
    p = D.pyramid_params(25, 10, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=1200, plane_w=1200)
    E, n_img = 25, 16
    geom = (D.dn_scale_geom * (n_img * E))()
    planes = (D.dn_plane_desc * 200)()
    n, e = ctypes.c_int32(), ctypes.c_int64()
    assert L.densenet_plan_batch(n_img, 768, 1024, ctypes.byref(p), geom, planes, 200, ctypes.byref(n),
                                 ctypes.byref(e)) == D.DN_OK
    assert n.value == 88 and e.value == 88 * 3 * 1200 * 1216
    assert L.densenet_plan_batch(n_img, 768, 1024, ctypes.byref(p), geom, planes, 50, ctypes.byref(n),
                                 ctypes.byref(e)) == D.DN_E_TOO_LARGE and n.value == 88
    q = D.pyramid_params(25, 10, pad=16)                       # no stitching planes
    assert L.densenet_plan_batch(2, 768, 1024, ctypes.byref(q), geom, planes, 200, ctypes.byref(n),
                                 ctypes.byref(e)) == D.DN_E_INVALID_ARG
    assert L.densenet_plan_batch(0, 768, 1024, ctypes.byref(p), geom, planes, 200, ctypes.byref(n),
                                 ctypes.byref(e)) == D.DN_E_INVALID_ARG
    big = D.pyramid_params(64, 10, pad=16, plane_h=4000, plane_w=4000)
    assert L.densenet_plan_batch(1025, 100, 100, ctypes.byref(big), geom, planes, 200, ctypes.byref(n),
                                 ctypes.byref(e)) == D.DN_E_TOO_LARGE   # 1025 * 64 > DN_MAX_BATCH_ITEMS
    assert L.densenet_plan_batch(2, 100, 100, ctypes.byref(big), None, planes, 200, ctypes.byref(n),
                                 ctypes.byref(e)) == D.DN_E_INVALID_ARG            # null geom
    # build: size query (no device work), then host validation of the geometry before any launch
    need = ctypes.c_size_t()
    assert L.densenet_build_batch(None, n_img, 768, 1024, ctypes.byref(p), D.DN_BF16, geom, None, 88,
                                  None, 0, ctypes.byref(need), None) == D.DN_OK
    assert need.value == (88 * 3 * 1200 * 1216 * 2 + 255) // 256 * 256 + n_img * 4 * 768 * 1024 + \
        4 * (88 + 1 + n_img * E)
    fake = ctypes.c_void_p(256)
    assert L.densenet_build_batch(fake, n_img, 768, 1024, ctypes.byref(p), D.DN_BF16, geom, fake, 88, fake,
                                  10, ctypes.byref(need), None) == D.DN_E_BUFFER_TOO_SMALL
    assert L.densenet_build_batch(fake, n_img, 768, 1024, ctypes.byref(p), D.DN_BF16, geom, fake, 87, fake,
                                  1 << 40, ctypes.byref(need), None) == D.DN_E_INVALID_ARG  # plane 87
    geom[3].x = 8                                               # not on the 16-px grid
    assert L.densenet_build_batch(fake, n_img, 768, 1024, ctypes.byref(p), D.DN_BF16, geom, fake, 88, fake,
                                  1 << 40, ctypes.byref(need), None) == D.DN_E_INVALID_ARG
    geom[3].x = 0
    geom[5].image = 3                                           # rows out of order
    assert L.densenet_build_batch(fake, n_img, 768, 1024, ctypes.byref(p), D.DN_BF16, geom, fake, 88, fake,
                                  1 << 40, ctypes.byref(need), None) == D.DN_E_INVALID_ARG
    geom[5].image = 0
    # region reads: maps must be one size and evenly spaced; windows inside them
    cd = (D.dn_plane_desc * 88)()
    for j in range(88):
        cd[j].h, cd[j].w, cd[j].offset = 74, 74, j * 74 * 74 * 256
    args = lambda cdesc, nm, pooled: (fake, cdesc, nm, D.DN_BF16, geom, fake, n_img, E, 16, pooled, fake,
                                      None, 0, 227.0, 6, fake, fake, None, None)
    assert L.densenet_region_windows_batch(*args(cd, 88, 0)) == D.DN_OK            # n = 0: nothing runs
    assert L.densenet_region_windows_batch(*args(cd, 88, 2)) == D.DN_E_INVALID_ARG
    assert L.densenet_region_windows_batch(*args(cd, 87, 1)) == D.DN_E_INVALID_ARG  # plane 87 missing
    cd[7].offset += 256
    assert L.densenet_region_windows_batch(*args(cd, 88, 0)) == D.DN_E_INVALID_ARG
    cd[7].offset -= 256
    cd[0].h = cd[1].h = 20
    assert L.densenet_region_windows_batch(*args(cd, 88, 0)) == D.DN_E_INVALID_ARG


def test_noalloc_builder_size_query_and_limit():
    """The scratch-free builder reports the planes' size alone and rejects a batch whose staged
    images exceed its static array, before any device work."""
    L = D.lib()
    p = D.pyramid_params(25, 10, pad=16, pad_mode=D.DN_PAD_RAMP, plane_h=1200, plane_w=1200)
    geom = (D.dn_scale_geom * 25)()
    planes = (D.dn_plane_desc * 64)()
    n, e, need = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_size_t()
    assert L.densenet_build_pyramid_noalloc(None, 16, 768, 1024, ctypes.byref(p), D.DN_BF16, None, 0,
                                            ctypes.byref(need), geom, planes, 64, ctypes.byref(n),
                                            ctypes.byref(e), None) == 0
    assert need.value == 16 * e.value * 2
    n_img = D.DN_STATIC_SCRATCH_BYTES // (4 * 768 * 1024) + 1
    fake = ctypes.c_void_p(256)
    st = L.densenet_build_pyramid_noalloc(fake, n_img, 768, 1024, ctypes.byref(p), D.DN_F16, fake,
                                          1 << 40, ctypes.byref(need), geom, planes, 64,
                                          ctypes.byref(n), ctypes.byref(e), None)
    assert st == D.DN_E_TOO_LARGE and "DN_STATIC_SCRATCH_BYTES" in D.last_error()


def test_builder_offset_limits():
    """The builder addresses pixel images and planes with 32-bit byte offsets: an image (or a packed
    batch) of 2^30 pixels and a plane of 2^31 bytes are rejected before any device work."""
    L = D.lib()
    geom = (D.dn_scale_geom * 4096)()
    planes = (D.dn_plane_desc * 64)()
    n, e, need = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_size_t()
    p = D.pyramid_params(1, 10, pad=16)
    q = lambda side: L.densenet_build_pyramid(None, 1, side, side, ctypes.byref(p), D.DN_BF16, None, 0,
                                              ctypes.byref(need), geom, planes, 64, ctypes.byref(n),
                                              ctypes.byref(e), None)
    assert q(32768) == D.DN_E_TOO_LARGE and "2^30" in D.last_error()      # 2^30 pixels
    assert q(32767) == D.DN_E_TOO_LARGE and "2^31" in D.last_error()      # one 32799^2 plane, 6.4 GB
    assert q(16384) == D.DN_OK                                            # 16416 x 16448 x 3 x 2 B
    pb = D.pyramid_params(25, 10, pad=16, plane_h=1200, plane_w=1200)
    assert L.densenet_build_batch(None, 1024, 1024, 1024, ctypes.byref(pb), D.DN_BF16, geom, None, 88,
                                  None, 0, ctypes.byref(need), None) == D.DN_E_TOO_LARGE
    assert "2^30" in D.last_error()
    big = D.pyramid_params(25, 10, pad=16, plane_h=16384, plane_w=16384)
    assert L.densenet_build_batch(None, 1, 1024, 1024, ctypes.byref(big), D.DN_F32, geom, None, 1,
                                  None, 0, ctypes.byref(need), None) == D.DN_E_TOO_LARGE
    assert "2^31" in D.last_error()


def test_region_map_size_limit():
    """Region windows address a conv5 map with 32-bit byte offsets: a map of 2^31 bytes is rejected
    before any device work, per image and in a packed batch."""
    L = D.lib()
    fake = ctypes.c_void_p(256)
    geom = (D.dn_scale_geom * 1)()
    geom[0].plane, geom[0].r0, geom[0].r1, geom[0].c0, geom[0].c1 = 0, 0, 0, 0, 0
    d = (D.dn_plane_desc * 1)()
    d[0].h, d[0].w, d[0].offset = 2048, 2048, 0          # 2048 * 2048 * 256 * 2 B = 2^31
    st = L.densenet_region_windows(fake, d, 1, D.DN_BF16, geom, 1, 16, 1, fake, None, 1,
                                   ctypes.c_float(227.0), 6, fake, fake, None, None)
    assert st == D.DN_E_TOO_LARGE and "2^31" in D.last_error()
    d[0].h = 2047
    assert L.densenet_region_windows(fake, d, 1, D.DN_BF16, geom, 1, 16, 1, fake, None, 0,
                                     ctypes.c_float(227.0), 6, fake, fake, None, None) == D.DN_OK


def _conv_query(L, descs, dt, net):
    n = len(descs)
    pd = (D.dn_plane_desc * n)(*descs)
    c5d, p5d = (D.dn_plane_desc * n)(), (D.dn_plane_desc * n)()
    ws, c5, p5 = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    st = L.densenet_conv_features(None, pd, n, dt, None, ctypes.byref(net), None, 0, ctypes.byref(ws),
                                  None, 0, ctypes.byref(c5), c5d, None, 0, ctypes.byref(p5), p5d, None)
    return st, ws.value, c5.value, list(c5d)


def test_conv_features_workspace_for_mixed_plane_sizes():
    """Planes of several sizes (the 480 x 640 image's 8 per-scale planes, twice: 16 runs of one plane)
    share one launch per layer: the workspace holds two buffers, each one layer's maps of all planes
    back to back (plus partial sums where fp32 launches too small for the GPU split), and the conv5
    maps lie back to back in plane order.  Size queries only: no device (the CU count defaults to
    256)."""
    L = D.lib()
    net = D.net_params()
    p = D.pyramid_params(8, 4, base_longest_side=1024, pad=16, pad_mode=D.DN_PAD_ZERO)
    one = list(D.densenet_plan_pyramid(480, 640, p).planes)
    descs = []
    for b in range(2):
        for d in one:
            q = D.dn_plane_desc()
            q.h, q.w, q.pitch = d.h, d.w, d.pitch
            q.offset = b * 10 ** 8 + d.offset
            descs.append(q)
    hw = [D.layer_sizes(d.h, d.w) for d in descs]
    a = max(sum(c * h[i][0] * h[i][1] for h in hw) for c, i in ((96, 0), (256, 2), (384, 4)))
    b = max(sum(c * h[i][0] * h[i][1] for h in hw) for c, i in ((96, 1), (256, 3), (384, 5)))
    for dt, es in ((D.DN_F16, 2), (D.DN_BF16, 2), (D.DN_F32, 4)):
        st, ws, c5, c5d = _conv_query(L, descs, dt, net)
        assert st == 0
        ab = (a * es + 255) // 256 * 256 + (b * es + 255) // 256 * 256
        assert ws == ab  # 16 planes fill the GPU: no launch splits
        off = 0
        for d, h in zip(c5d, hw):
            assert (d.h, d.w, d.offset) == (h[6][0], h[6][1], off)
            off += 256 * d.h * d.w
        assert c5 == off * es
    # one image's 8 planes in fp32: conv4/conv5 launches too small to fill the GPU split their sums
    st, ws, _, _ = _conv_query(L, descs[:8], D.DN_F32, net)
    hw = hw[:8]
    a = max(sum(c * h[i][0] * h[i][1] for h in hw) for c, i in ((96, 0), (256, 2), (384, 4))) * 4
    b = max(sum(c * h[i][0] * h[i][1] for h in hw) for c, i in ((96, 1), (256, 3), (384, 5))) * 4
    assert st == 0 and ws > (a + 255) // 256 * 256 + (b + 255) // 256 * 256
    # one large plane in fp32 fills the GPU: no partial sums
    q = D.dn_plane_desc()
    q.h, q.w, q.pitch, q.offset = 1200, 1200, 1216, 0
    hw = D.layer_sizes(1200, 1200)
    st, ws, _, _ = _conv_query(L, [q] * 4, D.DN_F32, net)
    a = max(c * hw[i][0] * hw[i][1] for c, i in ((96, 0), (256, 2), (384, 4))) * 4
    b = max(c * hw[i][0] * hw[i][1] for c, i in ((96, 1), (256, 3), (384, 5))) * 4
    assert st == 0 and ws == (4 * a + 255) // 256 * 256 + (4 * b + 255) // 256 * 256


def test_host_threads_call_concurrently():
    """Eight host threads plan pyramids at once (valid and invalid parameters in turn): every plan
    equals the one made alone, and each thread's error message is the one its own call left
    (densenet_last_error is per thread)."""
    import threading

    good = D.pyramid_params(25, 10, pad=16, plane_h=1200, plane_w=1200)
    ref = [(g.plane, g.y, g.x, g.rh, g.rw) for g in D.densenet_plan_pyramid(768, 1024, good).geom]
    failures = []
    own_msg = {}
    for t in range(8):  # each thread's invalid call, made alone first
        with pytest.raises(D.DenseNetError):
            D.densenet_plan_pyramid(100 * (1 + t), 100, D.pyramid_params(2, 2, plane_h=8 + t, plane_w=8 + t))
        own_msg[t] = D.last_error()
    assert len(set(own_msg.values())) == 8

    def worker(t):
        try:
            for i in range(40):
                if (i + t) % 2:
                    got = [(g.plane, g.y, g.x, g.rh, g.rw)
                           for g in D.densenet_plan_pyramid(768, 1024, good).geom]
                    if got != ref:
                        failures.append(f"thread {t}: plan differs")
                else:
                    H = 1 + t  # a different invalid call per thread: the plane is too small
                    bad = D.pyramid_params(2, 2, plane_h=8 + t, plane_w=8 + t)
                    try:
                        D.densenet_plan_pyramid(100 * H, 100, bad)
                        failures.append(f"thread {t}: invalid plan accepted")
                    except D.DenseNetError:
                        msg = D.last_error()
                        if msg != own_msg[t]:
                            failures.append(f"thread {t}: error message {msg!r} is not its own")
        except Exception as e:  # noqa: BLE001
            failures.append(f"thread {t}: {e!r}")

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(8)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not failures, failures[:5]
