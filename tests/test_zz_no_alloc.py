"""The scratch-free builder entry point (for callers that cannot allocate device memory): through the
C ABI its planes equal those of densenet_build_pyramid bit for bit, on two calls in a row, the second
with a smaller input (the library's static staging array keeps the first call's contents).  The
size limit is checked on the CPU in test_abi.py."""
import ctypes

import pytest

from paper_1404_1869_amd import configs as C
from paper_1404_1869_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def D():
    from paper_1404_1869_amd import densenet
    assert torch.cuda.is_available()
    densenet.lib()
    return densenet


def call_noalloc(D, imgs, p, dt, out):
    """densenet_build_pyramid_noalloc through the C ABI into `out`; returns (status, plan sizes)."""
    n_img, _, H, W = imgs.shape
    geom = (D.dn_scale_geom * D.n_entries(p))()
    planes = (D.dn_plane_desc * D.DN_MAX_PLANES_PER_IMAGE)()
    n, e, need = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_size_t()
    st = D.lib().densenet_build_pyramid_noalloc(
        D._ptr(imgs), n_img, H, W, ctypes.byref(p), dt, D._ptr(out), out.numel() * out.element_size(),
        ctypes.byref(need), geom, planes, D.DN_MAX_PLANES_PER_IMAGE, ctypes.byref(n), ctypes.byref(e),
        D._stream())
    return st, need.value, e.value


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_noalloc_builder_equals_builder_on_two_calls(D, dt):
    dtc = D.DTYPES[dt]
    cases = [(C.XGA_25SCALE_B16, 16), (C.VGA_8SCALE, 1)]    # the second call is smaller
    for w, n_img in cases:
        seeds = tuple(w.seeds[0] + 31 * i for i in range(n_img))
        imgs = torch.from_numpy(synth.images(seeds, w.H, w.W)).cuda()
        p = D.params_for(w)
        ref, plan = D.densenet_build_pyramid(imgs, p, dtc)
        elems = n_img * plan.image_elems
        out = torch.full((elems,), float("nan"), dtype=ref.dtype, device="cuda")
        st, need, image_elems = call_noalloc(D, imgs, p, dtc, out)
        assert st == D.DN_OK, D.last_error()
        assert need == elems * out.element_size() and image_elems == plan.image_elems
        torch.cuda.synchronize()
        assert torch.equal(out, ref[:elems]), f"{w.name}: planes differ"
    # the binding returns the same
    got, plan2 = D.densenet_build_pyramid_noalloc(imgs, p, dtc)
    torch.cuda.synchronize()
    assert torch.equal(got, ref[:n_img * plan2.image_elems])
