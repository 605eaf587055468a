// C ABI entry points: argument validation, size queries, workspace layout and kernel dispatch.
// Every check happens on the host before any device work is enqueued; launch failures surface as
// DN_E_HIP with the HIP error string in densenet_last_error().
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <sstream>

#include "common.h"

namespace dn {

static thread_local std::string g_error;

void set_error(const std::string& msg) { g_error = msg; }

int fail(int status, const std::string& msg) {
  g_error = msg;
  return status;
}

static int hip_status(int err, const char* what) {
  if (err == 0) return DN_OK;
  std::ostringstream os;
  os << what << ": " << hipGetErrorString((hipError_t)err);
  return fail(DN_E_HIP, os.str());
}

// One traced launch: the launcher's HIP status mapped to a dn_status naming the step.
template <typename F>
static int run_step(const char* name, void* stream, F&& launch) {
  TraceScope trace(name, stream);
  return hip_status(launch(), name);
}

static bool valid_dtype(dn_dtype dt) { return dt == DN_F32 || dt == DN_F16 || dt == DN_BF16; }

// Sizes of the stack for one plane size; false if conv5 would be empty.
struct StackShape {
  int64_t h[8], w[8];
};
static bool stack_shape(int32_t H, int32_t W, StackShape& s) {
  stack_sides(H, s.h);
  stack_sides(W, s.w);
  return s.h[6] > 0 && s.w[6] > 0;
}

// Planes grouped into runs of equal size and pitch and evenly spaced offsets (the runs of a layer
// share its launches).
struct Run {
  int32_t first, count, h, w, pitch;
  int64_t stride;  // elements between consecutive planes (0 for a run of one)
};
static int32_t row_pitch(const dn_plane_desc& d) { return d.pitch ? d.pitch : d.w; }
static std::vector<Run> make_runs(const dn_plane_desc* planes, int32_t n) {
  std::vector<Run> runs;
  for (int32_t i = 0; i < n;) {
    Run r{i, 1, planes[i].h, planes[i].w, row_pitch(planes[i]), 0};
    int32_t j = i + 1;
    if (j < n && planes[j].h == r.h && planes[j].w == r.w && row_pitch(planes[j]) == r.pitch) {
      r.stride = planes[j].offset - planes[i].offset;
      while (j < n && planes[j].h == r.h && planes[j].w == r.w && row_pitch(planes[j]) == r.pitch &&
             planes[j].offset - planes[j - 1].offset == r.stride && r.stride > 0)
        ++j;
      r.count = j - i;
      if (r.count == 1) r.stride = 0;
    }
    runs.push_back(r);
    i += r.count;
  }
  return runs;
}

}  // namespace dn

using namespace dn;

static int region_call(const void* d_conv5, const dn_plane_desc* conv5_desc, int32_t n_maps,
                       dn_dtype conv5_dtype, const dn_scale_geom* geom, int32_t n_scales, int32_t pad,
                       int32_t planes_per_img, const float* d_boxes, const int32_t* d_box_img,
                       int32_t n, float target, int32_t S, float* d_out, int32_t* d_scale,
                       int32_t* d_idx, bool pool, void* stream) {
  try {
    if (!d_conv5 || !conv5_desc || !geom) return fail(DN_E_INVALID_ARG, "null pointer argument");
    if (n > 0 && (!d_boxes || !d_out || !d_scale))
      return fail(DN_E_INVALID_ARG, "null box or output pointer");
    if (!valid_dtype(conv5_dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (n_scales <= 0 || n_scales > DN_MAX_SCALES) return fail(DN_E_INVALID_ARG, "bad n_scales");
    if (planes_per_img <= 0 || planes_per_img > DN_MAX_PLANES_PER_IMAGE || n_maps < planes_per_img ||
        n_maps % planes_per_img)
      return fail(DN_E_INVALID_ARG, "n_maps must be a positive multiple of planes_per_img");
    if (S <= 0 || S > 8) return fail(DN_E_UNSUPPORTED, "S must be in 1..8");
    if (!(target > 0)) return fail(DN_E_INVALID_ARG, "target must be positive");
    if (n < 0) return fail(DN_E_INVALID_ARG, "n must be >= 0");
    if (n == 0) return DN_OK;
    RegArgs a{};
    a.n_scales = n_scales;
    a.n_aspects = 1;
    for (int k = 0; k < n_scales; ++k) a.n_aspects = std::max(a.n_aspects, geom[k].aspect + 1);
    a.pad = pad;
    a.planes_per_img = planes_per_img;
    a.S = S;
    a.C = 256;
    a.target = (double)target;
    const int64_t vec = 16 / (int64_t)dtype_size(conv5_dtype);
    for (int32_t i = 0; i < n_maps; ++i) {
      if (conv5_desc[i].offset < 0 || conv5_desc[i].offset % vec)
        return fail(DN_E_INVALID_ARG, "conv5 map offsets must be multiples of 16 bytes");
      // the kernel addresses a map with 32-bit byte offsets
      if ((int64_t)conv5_desc[i].h * conv5_desc[i].w * 256 * (int64_t)dtype_size(conv5_dtype) >= (1LL << 31))
        return fail(DN_E_TOO_LARGE, "a conv5 map is limited to 2^31 - 1 bytes");
    }
    for (int32_t j = 0; j < planes_per_img; ++j) {
      a.map_off[j] = conv5_desc[j].offset - conv5_desc[0].offset;
      a.map_w[j] = conv5_desc[j].w;
    }
    const int n_img = n_maps / planes_per_img;
    a.n_img = n_img;
    a.image_stride = 0;
    if (n_img > 1) {
      a.image_stride = conv5_desc[planes_per_img].offset - conv5_desc[0].offset;
      for (int b = 1; b < n_img; ++b)
        for (int j = 0; j < planes_per_img; ++j) {
          const dn_plane_desc& d = conv5_desc[b * planes_per_img + j];
          if (d.offset - conv5_desc[0].offset != b * a.image_stride + a.map_off[j] ||
              d.w != conv5_desc[j].w || d.h != conv5_desc[j].h)
            return fail(DN_E_INVALID_ARG, "images' conv5 maps must be laid out identically");
        }
    }
    for (int k = 0; k < n_scales; ++k) {
      const dn_scale_geom& g = geom[k];
      if (g.plane < 0 || g.plane >= planes_per_img) return fail(DN_E_INVALID_ARG, "bad geom plane");
      const dn_plane_desc& d = conv5_desc[g.plane];
      const bool empty = g.r1 < g.r0 || g.c1 < g.c0;
      if (!empty && (g.r0 < 0 || g.c0 < 0 || g.r1 >= d.h || g.c1 >= d.w))
        return fail(DN_E_INVALID_ARG, "scale window outside its conv5 map");
      a.s[k] = RegScale{g.plane, g.y, g.x, g.r0, g.r1, g.c0, g.c1, empty ? 1 : 0, g.sy, g.sx};
    }
    const char* base = (const char*)d_conv5 + conv5_desc[0].offset * dtype_size(conv5_dtype);
    TraceScope trace(pool ? "region_pool" : "region_windows", stream);
    return hip_status(launch_region_windows(base, conv5_dtype, a, nullptr, d_boxes, d_box_img, n, d_out,
                                            d_scale, d_idx, pool, stream),
                      pool ? "region_pool launch" : "region_windows launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}


// Validates a cross-image packed plan's host geometry against the batch and the stitching planes.
static int check_batch_geom(const dn_scale_geom* geom, int32_t n_img, int32_t E, int32_t n_planes,
                            int32_t PH, int32_t PW) {
  for (int32_t b = 0; b < n_img; ++b)
    for (int32_t e = 0; e < E; ++e) {
      const dn_scale_geom& g = geom[(int64_t)b * E + e];
      if (g.image != b || g.k != e) return fail(DN_E_INVALID_ARG, "geom is not a batch plan's entry array");
      if (g.plane < 0 || g.plane >= n_planes) return fail(DN_E_INVALID_ARG, "geom plane out of range");
      if (g.h < 1 || g.w < 1 || g.h > 65535 || g.w > 65535 || g.rh < 16 || g.rw < 16 ||
          ((g.y | g.x | g.rh | g.rw) & 15) || g.y < 0 || g.x < 0 || g.y > PH - g.rh || g.x > PW - g.rw)
        return fail(DN_E_INVALID_ARG, "geom rectangle is not a placement on the batch's planes");
    }
  return DN_OK;
}

static int region_batch_call(const void* d_conv5, const dn_plane_desc* conv5_desc, int32_t n_maps,
                             dn_dtype conv5_dtype, const dn_scale_geom* geom, const dn_scale_geom* d_geom,
                             int32_t n_img, int32_t E, int32_t pad, bool pool, const float* d_boxes,
                             const int32_t* d_box_img, int32_t n, float target, int32_t S, float* d_out,
                             int32_t* d_scale, int32_t* d_idx, void* stream) {
  try {
    if (!d_conv5 || !conv5_desc || !geom || !d_geom) return fail(DN_E_INVALID_ARG, "null pointer argument");
    if (n > 0 && (!d_boxes || !d_out || !d_scale))
      return fail(DN_E_INVALID_ARG, "null box or output pointer");
    if (!valid_dtype(conv5_dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (n_img <= 0 || E <= 0 || E > DN_MAX_SCALES || (int64_t)n_img * E > DN_MAX_BATCH_ITEMS)
      return fail(DN_E_INVALID_ARG, "bad n_img or n_entries");
    if (n_maps <= 0) return fail(DN_E_INVALID_ARG, "n_maps must be positive");
    if (S <= 0 || S > 8) return fail(DN_E_UNSUPPORTED, "S must be in 1..8");
    if (!(target > 0)) return fail(DN_E_INVALID_ARG, "target must be positive");
    if (n < 0) return fail(DN_E_INVALID_ARG, "n must be >= 0");
    const dn_plane_desc& d0 = conv5_desc[0];
    const int64_t vec = 16 / (int64_t)dtype_size(conv5_dtype);
    const int64_t stride = n_maps > 1 ? conv5_desc[1].offset - d0.offset : 0;
    if (d0.h <= 0 || d0.w <= 0 || (n_maps > 1 && stride < (int64_t)d0.h * d0.w * 256))
      return fail(DN_E_INVALID_ARG, "conv5 maps must be non-empty and not overlap");
    if ((int64_t)d0.h * d0.w * 256 * (int64_t)dtype_size(conv5_dtype) >= (1LL << 31))
      return fail(DN_E_TOO_LARGE, "a conv5 map is limited to 2^31 - 1 bytes");
    for (int32_t j = 0; j < n_maps; ++j) {
      const dn_plane_desc& d = conv5_desc[j];
      if (d.h != d0.h || d.w != d0.w || d.offset != d0.offset + j * stride || d.offset < 0 || d.offset % vec)
        return fail(DN_E_INVALID_ARG,
                    "conv5 maps of a packed batch must be of one size, evenly spaced, 16-byte aligned");
    }
    RegArgs a{};
    a.n_scales = E;
    a.n_aspects = 1;
    a.pad = pad;
    a.planes_per_img = 0;
    a.S = S;
    a.C = 256;
    a.n_img = n_img;
    a.target = (double)target;
    for (int32_t b = 0; b < n_img; ++b)
      for (int32_t e = 0; e < E; ++e) {
        const dn_scale_geom& g = geom[(int64_t)b * E + e];
        if (g.image != b || g.k != e) return fail(DN_E_INVALID_ARG, "geom is not a batch plan's entry array");
        if (g.plane < 0 || g.plane >= n_maps) return fail(DN_E_INVALID_ARG, "bad geom plane");
        const bool empty = g.r1 < g.r0 || g.c1 < g.c0;
        if (!empty && (g.r0 < 0 || g.c0 < 0 || g.r1 >= d0.h || g.c1 >= d0.w))
          return fail(DN_E_INVALID_ARG, "scale window outside its conv5 map");
        a.n_aspects = std::max(a.n_aspects, g.aspect + 1);
      }
    if (n == 0) return DN_OK;
    RegBatch bt{d_geom, stride, n_maps, d0.h, d0.w};
    const char* base = (const char*)d_conv5 + d0.offset * dtype_size(conv5_dtype);
    TraceScope trace(pool ? "region_pool" : "region_windows", stream);
    return hip_status(launch_region_windows(base, conv5_dtype, a, &bt, d_boxes, d_box_img, n, d_out,
                                            d_scale, d_idx, pool, stream),
                      pool ? "region_pool launch" : "region_windows launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

extern "C" {

const char* densenet_last_error(void) { return g_error.c_str(); }

int densenet_layer_sizes(int32_t H, int32_t W, int32_t* hw) {
  if (!hw) return fail(DN_E_INVALID_ARG, "hw is NULL");
  if (H <= 0 || W <= 0) return fail(DN_E_INVALID_ARG, "plane sides must be positive");
  StackShape s;
  const bool ok = stack_shape(H, W, s);
  for (int i = 0; i < 8; ++i) {
    hw[2 * i] = (int32_t)s.h[i];
    hw[2 * i + 1] = (int32_t)s.w[i];
  }
  if (!ok) return fail(DN_E_INVALID_ARG, "plane too small: conv5 would be empty");
  return DN_OK;
}

int densenet_plan_pyramid(int32_t H, int32_t W, const dn_pyramid_params* p, dn_scale_geom* geom,
                          dn_plane_desc* planes, int32_t max_planes, int32_t* n_planes,
                          int64_t* image_elems) {
  try {
    if (!p || !geom || !planes || !n_planes || !image_elems)
      return fail(DN_E_INVALID_ARG, "null pointer argument");
    Plan plan;
    int st = make_plan(H, W, *p, plan);
    if (st != DN_OK) return st;
    const int32_t np = (int32_t)plan.planes.size();
    *n_planes = np;
    if (np > max_planes) return fail(DN_E_TOO_LARGE, "more planes than max_planes");
    std::copy(plan.scales.begin(), plan.scales.end(), geom);
    int64_t off = 0;
    for (int32_t j = 0; j < np; ++j) {
      planes[j] = dn_plane_desc{};
      planes[j].h = plan.planes[j].h;
      planes[j].w = plan.planes[j].w;
      planes[j].pitch = plane_pitch(plan.planes[j].w);
      planes[j].offset = off;
      off += 3LL * plan.planes[j].h * planes[j].pitch;
    }
    *image_elems = off;
    return DN_OK;
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

// densenet_build_pyramid (static_scratch = false: the pixel image stages after the planes in the
// caller's buffer) and densenet_build_pyramid_noalloc (true: it stages in the library's static array).
static int build_pyramid(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                         const dn_pyramid_params* p, dn_dtype dtype, void* d_planes, size_t planes_bytes,
                         size_t* bytes_needed, dn_scale_geom* geom, dn_plane_desc* planes,
                         int32_t max_planes, int32_t* n_planes, int64_t* image_elems, void* stream,
                         bool static_scratch_area) {
  try {
    if (!bytes_needed) return fail(DN_E_INVALID_ARG, "bytes_needed is NULL");
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (n_img <= 0) return fail(DN_E_INVALID_ARG, "n_img must be positive");
    int st = densenet_plan_pyramid(H, W, p, geom, planes, max_planes, n_planes, image_elems);
    if (st != DN_OK) return st;
    // the builder addresses an image's pixels (4 bytes each) and a plane with 32-bit byte offsets
    if ((int64_t)H * W >= (1LL << 30)) return fail(DN_E_TOO_LARGE, "an image is limited to 2^30 - 1 pixels");
    for (int j = 0; j < *n_planes; ++j)
      if (3LL * planes[j].h * planes[j].pitch * (int64_t)dtype_size(dtype) >= (1LL << 31))
        return fail(DN_E_TOO_LARGE, "a plane is limited to 2^31 - 1 bytes");
    const size_t planes_end = ((size_t)n_img * (size_t)*image_elems * dtype_size(dtype) + 255) &
                              ~(size_t)255;
    const size_t pix_bytes = (size_t)n_img * 4 * (size_t)H * (size_t)W;
    if (static_scratch_area && pix_bytes > (size_t)DN_STATIC_SCRATCH_BYTES)
      return fail(DN_E_TOO_LARGE, "4 * H * W * n_img exceeds DN_STATIC_SCRATCH_BYTES");
    const size_t need = static_scratch_area ? (size_t)n_img * (size_t)*image_elems * dtype_size(dtype)
                                            : planes_end + pix_bytes;
    *bytes_needed = need;
    if (!d_planes) return DN_OK;
    if (planes_bytes < need) return fail(DN_E_BUFFER_TOO_SMALL, "planes buffer too small");
    if (!d_images) return fail(DN_E_INVALID_ARG, "d_images is NULL");
    if ((int64_t)n_img * *n_planes > 65535) return fail(DN_E_TOO_LARGE, "too many planes in one call");
    const int K = p->n_scales * (p->n_aspects > 0 ? p->n_aspects : 1);  // pyramid entries
    PyrArgs a{};
    a.n_scales = K;
    a.H = H;
    a.W = W;
    a.pad = p->pad;
    a.ramp = p->pad_mode == DN_PAD_RAMP;
    for (int c = 0; c < 3; ++c) a.mean[c] = p->mean[c];
    int e = 0;
    for (int j = 0; j < *n_planes; ++j) {
      a.plane_first[j] = (uint8_t)e;
      for (int k = 0; k < K; ++k)
        if (geom[k].plane == j)
          a.s[e++] = PyrScale{geom[k].plane, geom[k].y, geom[k].x, geom[k].rh, geom[k].rw, geom[k].h,
                              geom[k].w};
      a.plane_count[j] = (uint8_t)(e - a.plane_first[j]);
    }
    PyrPlanes pl{};
    pl.n = *n_planes;
    pl.image_elems = *image_elems;
    int32_t mh = 0, mw = 0;
    for (int j = 0; j < pl.n; ++j) {
      pl.p[j] = PyrPlane{planes[j].h, planes[j].w, planes[j].offset};
      mh = std::max(mh, planes[j].h);
      mw = std::max(mw, planes[j].w);
    }
    int32_t max_scale_w = 0;
    for (int k = 0; k < K; ++k) max_scale_w = std::max(max_scale_w, geom[k].w);
    uint8_t* pix = (uint8_t*)d_planes + planes_end;
    if (static_scratch_area) {
      const int e = static_scratch(&pix);
      if (e != (int)hipSuccess) return hip_status(e, "static scratch lookup");
    }
    TraceScope trace("build_planes", stream);
    return hip_status(launch_build_planes(d_images, n_img, a, pl, nullptr, mh, mw, max_scale_w, dtype,
                                          d_planes, pix, stream),
                      "build_planes launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_build_pyramid(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                           const dn_pyramid_params* p, dn_dtype dtype, void* d_planes,
                           size_t planes_bytes, size_t* bytes_needed, dn_scale_geom* geom,
                           dn_plane_desc* planes, int32_t max_planes, int32_t* n_planes,
                           int64_t* image_elems, void* stream) {
  return build_pyramid(d_images, n_img, H, W, p, dtype, d_planes, planes_bytes, bytes_needed, geom,
                       planes, max_planes, n_planes, image_elems, stream, false);
}

int densenet_build_pyramid_noalloc(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                                   const dn_pyramid_params* p, dn_dtype dtype, void* d_planes,
                                   size_t planes_bytes, size_t* bytes_needed, dn_scale_geom* geom,
                                   dn_plane_desc* planes, int32_t max_planes, int32_t* n_planes,
                                   int64_t* image_elems, void* stream) {
  return build_pyramid(d_images, n_img, H, W, p, dtype, d_planes, planes_bytes, bytes_needed, geom,
                       planes, max_planes, n_planes, image_elems, stream, true);
}

int densenet_plan_batch(int32_t n_img, int32_t H, int32_t W, const dn_pyramid_params* p,
                        dn_scale_geom* geom, dn_plane_desc* planes, int32_t max_planes,
                        int32_t* n_planes, int64_t* total_elems) {
  try {
    if (!p || !geom || !planes || !n_planes || !total_elems)
      return fail(DN_E_INVALID_ARG, "null pointer argument");
    std::vector<dn_scale_geom> items;
    int np = 0;
    const int st = make_plan_batch(n_img, H, W, *p, items, np);
    if (st != DN_OK) return st;
    *n_planes = np;
    if (np > max_planes) return fail(DN_E_TOO_LARGE, "more planes than max_planes");
    std::copy(items.begin(), items.end(), geom);
    const int64_t pe = 3LL * p->plane_h * plane_pitch(p->plane_w);
    for (int32_t j = 0; j < np; ++j) {
      planes[j] = dn_plane_desc{};
      planes[j].h = p->plane_h;
      planes[j].w = p->plane_w;
      planes[j].pitch = plane_pitch(p->plane_w);
      planes[j].offset = j * pe;
    }
    *total_elems = np * pe;
    return DN_OK;
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_build_batch(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                         const dn_pyramid_params* p, dn_dtype dtype, const dn_scale_geom* geom,
                         const dn_scale_geom* d_geom, int32_t n_planes, void* d_planes,
                         size_t planes_bytes, size_t* bytes_needed, void* stream) {
  try {
    if (!bytes_needed || !p) return fail(DN_E_INVALID_ARG, "null pointer argument");
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (n_img <= 0 || H <= 0 || W <= 0 || H > 32768 || W > 32768)
      return fail(DN_E_INVALID_ARG, "bad batch or image size");
    if (p->plane_h <= 0 || p->plane_w <= 0)
      return fail(DN_E_INVALID_ARG, "cross-image packing needs stitching planes (plane_h, plane_w > 0)");
    if (p->pad < 0 || p->pad > 1024 || (p->pad_mode != DN_PAD_ZERO && p->pad_mode != DN_PAD_RAMP))
      return fail(DN_E_INVALID_ARG, "bad pad or pad_mode");
    const int64_t E = (int64_t)p->n_scales * std::max(1, p->n_aspects);
    if (p->n_scales <= 0 || E > DN_MAX_SCALES || n_img * E > DN_MAX_BATCH_ITEMS)
      return fail(DN_E_INVALID_ARG, "bad n_scales, n_aspects or batch size");
    if (n_planes <= 0) return fail(DN_E_INVALID_ARG, "n_planes must be positive");
    if (n_planes > MAX_INDEX_PLANES) {
      std::ostringstream os;
      os << "a packed batch is limited to " << MAX_INDEX_PLANES << " planes";
      return fail(DN_E_TOO_LARGE, os.str());
    }
    // the builder addresses the batch's pixel images (4 bytes per pixel) and a plane with 32-bit
    // byte offsets
    if ((int64_t)n_img * H * W >= (1LL << 30))
      return fail(DN_E_TOO_LARGE, "a packed batch is limited to 2^30 - 1 image pixels");
    const int64_t pe = 3LL * p->plane_h * plane_pitch(p->plane_w);
    if (pe * (int64_t)dtype_size(dtype) >= (1LL << 31))
      return fail(DN_E_TOO_LARGE, "a plane is limited to 2^31 - 1 bytes");
    const size_t planes_end = ((size_t)n_planes * (size_t)pe * dtype_size(dtype) + 255) & ~(size_t)255;
    const size_t need = planes_end + builder_scratch_bytes(n_img, H, W, n_planes, (int32_t)(n_img * E));
    *bytes_needed = need;
    if (!d_planes) return DN_OK;
    if (planes_bytes < need) return fail(DN_E_BUFFER_TOO_SMALL, "planes buffer too small");
    if (!d_images || !geom || !d_geom) return fail(DN_E_INVALID_ARG, "null pointer argument");
    const int st = check_batch_geom(geom, n_img, (int32_t)E, n_planes, p->plane_h, p->plane_w);
    if (st != DN_OK) return st;
    PyrArgs a{};
    a.n_scales = 0;
    a.H = H;
    a.W = W;
    a.pad = p->pad;
    a.ramp = p->pad_mode == DN_PAD_RAMP;
    for (int c = 0; c < 3; ++c) a.mean[c] = p->mean[c];
    PyrPlanes pl{};
    BatchGeom bg{d_geom, (int32_t)(n_img * E), n_img, n_planes, p->plane_h, p->plane_w, nullptr, nullptr};
    int32_t max_scale_w = 0;
    for (int64_t i = 0; i < n_img * E; ++i) max_scale_w = std::max(max_scale_w, geom[i].w);
    TraceScope trace("build_planes", stream);
    return hip_status(launch_build_planes(d_images, n_img, a, pl, &bg, p->plane_h, p->plane_w,
                                          max_scale_w, dtype, d_planes, (uint8_t*)d_planes + planes_end,
                                          stream),
                      "build_planes launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_pack_weights(const float* const* d_w, const float* const* d_b, dn_dtype dtype,
                          void* d_packed, size_t packed_bytes, size_t* bytes_needed, void* stream) {
  try {
    if (!bytes_needed) return fail(DN_E_INVALID_ARG, "bytes_needed is NULL");
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    const PackedLayout L = packed_layout(dtype);
    *bytes_needed = L.total;
    if (!d_packed) return DN_OK;
    if (packed_bytes < L.total) return fail(DN_E_BUFFER_TOO_SMALL, "packed buffer too small");
    if (!d_w || !d_b) return fail(DN_E_INVALID_ARG, "weight pointer arrays are NULL");
    for (int l = 0; l < 5; ++l)
      if (!d_w[l] || !d_b[l]) return fail(DN_E_INVALID_ARG, "a layer's weight or bias is NULL");
    TraceScope trace("pack_weights", stream);
    return hip_status(launch_pack_weights(d_w, d_b, dtype, d_packed, stream), "pack launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_conv_layer(int32_t layer, const void* d_in, int32_t n, int32_t H, int32_t W,
                        dn_dtype dtype, const void* d_packed, void* d_out, void* stream) {
  try {
    if (layer < 1 || layer > 5) return fail(DN_E_INVALID_ARG, "layer must be 1..5");
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (!d_in || !d_out || !d_packed) return fail(DN_E_INVALID_ARG, "null device pointer");
    if (n <= 0 || H <= 0 || W <= 0) return fail(DN_E_INVALID_ARG, "sizes must be positive");
    static const int Cs[5] = {3, 96, 256, 384, 384}, Ms[5] = {96, 256, 384, 384, 256};
    int64_t Ho = H, Wo = W;
    if (layer == 1) {
      if (H < 11 || W < 11) return fail(DN_E_INVALID_ARG, "conv1 needs at least 11 x 11 input");
      Ho = (H - 11) / 4 + 1;
      Wo = (W - 11) / 4 + 1;
    }
    const int64_t in_stride = (int64_t)Cs[layer - 1] * H * W;
    const int64_t out_stride = (int64_t)Ms[layer - 1] * Ho * Wo;
    static const char* names[5] = {"conv1", "conv2", "conv3", "conv4", "conv5"};
    TraceScope trace(names[layer - 1], stream);
    const MapRun run{n, H, W, W, 0, in_stride, 0, out_stride};
    return hip_status(launch_conv(layer, d_in, &run, 1, dtype, d_packed, d_out, nullptr, 0, stream),
                      "conv launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_lrn_pool(const void* d_in, int32_t n, int32_t H, int32_t W, int32_t C, dn_dtype dtype,
                      const dn_net_params* net, void* d_out, void* stream) {
  try {
    if (!net) return fail(DN_E_INVALID_ARG, "net is NULL");
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (!d_in || !d_out) return fail(DN_E_INVALID_ARG, "null device pointer");
    if (n <= 0 || H < 2 || W < 2 || C <= 0) return fail(DN_E_INVALID_ARG, "bad sizes");
    if (net->lrn_n <= 0 || net->lrn_n % 2 == 0 || net->lrn_n > 9)
      return fail(DN_E_INVALID_ARG, "lrn_n must be odd and at most 9");
    if (!(net->lrn_k > 0)) return fail(DN_E_INVALID_ARG, "lrn_k must be positive");
    const int64_t Ho = (H - 2) / 2 + 1, Wo = (W - 2) / 2 + 1;
    TraceScope trace(C == 96 ? "lrn_pool1" : "lrn_pool2", stream);
    const MapRun run{n, H, W, 0, 0, (int64_t)C * H * W, 0, (int64_t)C * Ho * Wo};
    return hip_status(launch_lrn_pool(d_in, &run, 1, C, dtype, true, net->lrn_before_pool != 0,
                                      net->lrn_alpha, net->lrn_beta, net->lrn_k, net->lrn_n, d_out,
                                      stream),
                      "lrn_pool launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_maxpool(const void* d_in, int32_t n, int32_t H, int32_t W, int32_t C, dn_dtype dtype,
                     void* d_out, void* stream) {
  try {
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (!d_in || !d_out) return fail(DN_E_INVALID_ARG, "null device pointer");
    if (n <= 0 || H < 2 || W < 2 || C <= 0) return fail(DN_E_INVALID_ARG, "bad sizes");
    const int64_t Ho = (H - 2) / 2 + 1, Wo = (W - 2) / 2 + 1;
    TraceScope trace("pool5", stream);
    const MapRun run{n, H, W, 0, 0, (int64_t)C * H * W, 0, (int64_t)C * Ho * Wo};
    return hip_status(launch_lrn_pool(d_in, &run, 1, C, dtype, false, false, 0, 0, 1, 1, d_out, stream),
                      "maxpool launch");
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_conv_features(const void* d_planes, const dn_plane_desc* planes, int32_t n_planes,
                           dn_dtype dtype, const void* d_packed, const dn_net_params* net,
                           void* d_workspace, size_t ws_bytes, size_t* ws_needed, void* d_conv5,
                           size_t conv5_bytes, size_t* conv5_needed, dn_plane_desc* conv5_desc,
                           void* d_pool5, size_t pool5_bytes, size_t* pool5_needed,
                           dn_plane_desc* pool5_desc, void* stream) {
  try {
    if (!planes || !net || !ws_needed || !conv5_needed || !conv5_desc)
      return fail(DN_E_INVALID_ARG, "null pointer argument");
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (n_planes <= 0) return fail(DN_E_INVALID_ARG, "n_planes must be positive");
    if (n_planes > MAX_INDEX_PLANES) {
      std::ostringstream os;
      os << "a packed batch is limited to " << MAX_INDEX_PLANES << " planes";
      return fail(DN_E_TOO_LARGE, os.str());
    }
    if (net->lrn_n <= 0 || net->lrn_n % 2 == 0 || net->lrn_n > 9)
      return fail(DN_E_INVALID_ARG, "lrn_n must be odd and at most 9");
    if (!(net->lrn_k > 0)) return fail(DN_E_INVALID_ARG, "lrn_k must be positive");
    if (net->pool5 && (!pool5_needed || !pool5_desc))
      return fail(DN_E_INVALID_ARG, "pool5 requested without pool5_needed / pool5_desc");
    const size_t es = dtype_size(dtype);
    // Output layout: the conv5 (and pool5) maps in plane order.
    int64_t c5_off = 0, p5_off = 0;
    for (int32_t i = 0; i < n_planes; ++i) {
      StackShape s;
      if (planes[i].h <= 0 || planes[i].w <= 0 || planes[i].offset < 0 ||
          (planes[i].pitch != 0 && planes[i].pitch < planes[i].w))
        return fail(DN_E_INVALID_ARG, "bad plane descriptor");
      if (!stack_shape(planes[i].h, planes[i].w, s)) {
        std::ostringstream os;
        os << "plane " << i << " (" << planes[i].h << "x" << planes[i].w
           << ") is too small for conv5";
        return fail(DN_E_INVALID_ARG, os.str());
      }
      conv5_desc[i] = dn_plane_desc{(int32_t)s.h[6], (int32_t)s.w[6], c5_off};
      c5_off += 256 * s.h[6] * s.w[6];
      if (net->pool5) {
        if (s.h[6] < 2 || s.w[6] < 2) return fail(DN_E_INVALID_ARG, "conv5 too small for pool5");
        pool5_desc[i] = dn_plane_desc{(int32_t)s.h[7], (int32_t)s.w[7], p5_off};
        p5_off += 256 * s.h[7] * s.w[7];
      }
    }
    // Each layer is one launch over all runs (planes of different sizes included): the runs' maps of
    // a layer are packed one after another in the workspace's two ping-pong buffers, A (conv1,
    // conv2, conv3 outputs) and B (pool1, pool2, conv4 outputs).
    const std::vector<Run> runs = make_runs(planes, n_planes);
    const size_t nr = runs.size();
    std::vector<StackShape> shp(nr);
    std::vector<int64_t> oa1(nr), ob1(nr), oa2(nr), ob2(nr), oa3(nr), ob4(nr);
    int64_t a1 = 0, b1 = 0, a2 = 0, b2 = 0, a3 = 0, b4 = 0;
    for (size_t i = 0; i < nr; ++i) {
      StackShape& s = shp[i];
      stack_shape(runs[i].h, runs[i].w, s);
      const int64_t n = runs[i].count;
      oa1[i] = a1, a1 += n * 96 * s.h[0] * s.w[0];
      ob1[i] = b1, b1 += n * 96 * s.h[1] * s.w[1];
      oa2[i] = a2, a2 += n * 256 * s.h[2] * s.w[2];
      ob2[i] = b2, b2 += n * 256 * s.h[3] * s.w[3];
      oa3[i] = a3, a3 += n * 384 * s.h[4] * s.w[4];
      ob4[i] = b4, b4 += n * 384 * s.h[5] * s.w[5];
    }
    // Per layer and run: planes, input size, input/output offsets and strides (elements).
    std::vector<MapRun> c1(nr), l1(nr), c2(nr), l2(nr), c3(nr), c4(nr), c5(nr), q5(nr);
    for (size_t i = 0; i < nr; ++i) {
      const Run& r = runs[i];
      const StackShape& s = shp[i];
      const int n = r.count;
      const int64_t s1 = 96 * s.h[0] * s.w[0], p1 = 96 * s.h[1] * s.w[1];
      const int64_t s2 = 256 * s.h[2] * s.w[2], p2 = 256 * s.h[3] * s.w[3];
      const int64_t s3 = 384 * s.h[4] * s.w[4], s4 = 384 * s.h[5] * s.w[5];
      const int64_t s5 = 256 * s.h[6] * s.w[6];
      const int h0 = (int)s.h[0], w0 = (int)s.w[0], h1 = (int)s.h[1], w1 = (int)s.w[1];
      const int h2 = (int)s.h[2], w2 = (int)s.w[2], h3 = (int)s.h[3], w3 = (int)s.w[3];
      const int h4 = (int)s.h[4], w4 = (int)s.w[4], h6 = (int)s.h[6], w6 = (int)s.w[6];
      const int64_t sp = r.count > 1 ? r.stride : 3LL * r.h * r.pitch;
      const int64_t o5 = conv5_desc[r.first].offset;
      c1[i] = MapRun{n, r.h, r.w, r.pitch, planes[r.first].offset, sp, oa1[i], s1};
      l1[i] = MapRun{n, h0, w0, 0, oa1[i], s1, ob1[i], p1};
      c2[i] = MapRun{n, h1, w1, 0, ob1[i], p1, oa2[i], s2};
      l2[i] = MapRun{n, h2, w2, 0, oa2[i], s2, ob2[i], p2};
      c3[i] = MapRun{n, h3, w3, 0, ob2[i], p2, oa3[i], s3};
      c4[i] = MapRun{n, h4, w4, 0, oa3[i], s3, ob4[i], s4};
      c5[i] = MapRun{n, h4, w4, 0, ob4[i], s4, o5, s5};
      if (net->pool5)
        q5[i] = MapRun{n, h6, w6, 0, o5, s5, pool5_desc[r.first].offset, 256 * s.h[7] * s.w[7]};
    }
    const int n_runs = (int)nr;
    // C: partial sums of the fp32 conv launches too small to fill the chip (0 bytes otherwise)
    const size_t ws_c = std::max({conv_part_bytes(2, c2.data(), n_runs, dtype),
                                  conv_part_bytes(3, c3.data(), n_runs, dtype),
                                  conv_part_bytes(4, c4.data(), n_runs, dtype),
                                  conv_part_bytes(5, c5.data(), n_runs, dtype)});
    const size_t ws_a = ((size_t)std::max({a1, a2, a3}) * es + 255) & ~(size_t)255;
    const size_t ws_b = ((size_t)std::max({b1, b2, b4}) * es + 255) & ~(size_t)255;
    *ws_needed = ws_a + ws_b + ws_c;
    *conv5_needed = (size_t)c5_off * es;
    if (net->pool5) *pool5_needed = (size_t)p5_off * es;
    if (!d_conv5) return DN_OK;
    if (!d_planes || !d_packed) return fail(DN_E_INVALID_ARG, "null device pointer");
    if (!d_workspace || ws_bytes < *ws_needed)
      return fail(DN_E_BUFFER_TOO_SMALL, "workspace too small");
    if (conv5_bytes < *conv5_needed) return fail(DN_E_BUFFER_TOO_SMALL, "conv5 buffer too small");
    if (net->pool5 && (!d_pool5 || pool5_bytes < *pool5_needed))
      return fail(DN_E_BUFFER_TOO_SMALL, "pool5 buffer too small");

    char* A = (char*)d_workspace;
    char* B = A + ws_a;
    char* Cp = B + ws_b;
    const bool lf = net->lrn_before_pool != 0;
    const float al = net->lrn_alpha, be = net->lrn_beta, kk = net->lrn_k;
    const int ln = net->lrn_n;
    int st;
    if ((st = run_step("conv1", stream, [&] {
           return launch_conv(1, d_planes, c1.data(), n_runs, dtype, d_packed, A, Cp, ws_c, stream);
         })))
      return st;
    if ((st = run_step("lrn_pool1", stream, [&] {
           return launch_lrn_pool(A, l1.data(), n_runs, 96, dtype, true, lf, al, be, kk, ln, B, stream);
         })))
      return st;
    if ((st = run_step("conv2", stream, [&] {
           return launch_conv(2, B, c2.data(), n_runs, dtype, d_packed, A, Cp, ws_c, stream);
         })))
      return st;
    if ((st = run_step("lrn_pool2", stream, [&] {
           return launch_lrn_pool(A, l2.data(), n_runs, 256, dtype, true, lf, al, be, kk, ln, B, stream);
         })))
      return st;
    if ((st = run_step("conv3", stream, [&] {
           return launch_conv(3, B, c3.data(), n_runs, dtype, d_packed, A, Cp, ws_c, stream);
         })))
      return st;
    if ((st = run_step("conv4", stream, [&] {
           return launch_conv(4, A, c4.data(), n_runs, dtype, d_packed, B, Cp, ws_c, stream);
         })))
      return st;
    if ((st = run_step("conv5", stream, [&] {
           return launch_conv(5, B, c5.data(), n_runs, dtype, d_packed, d_conv5, Cp, ws_c, stream);
         })))
      return st;
    if (net->pool5) {
      if ((st = run_step("pool5", stream, [&] {
             return launch_lrn_pool(d_conv5, q5.data(), n_runs, 256, dtype, false, false, 0, 0, 1, 1,
                                    d_pool5, stream);
           })))
        return st;
    }
    return DN_OK;
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_warp_regions(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                          const float* d_boxes, const int32_t* d_box_img, int32_t n, int32_t S,
                          int32_t pitch, const float* mean, dn_dtype dtype, void* d_out,
                          size_t out_bytes, size_t* bytes_needed, void* stream) {
  try {
    if (!valid_dtype(dtype)) return fail(DN_E_UNSUPPORTED, "unknown dtype");
    if (n < 0) return fail(DN_E_INVALID_ARG, "n must be >= 0");
    if (S <= 0 || S > DN_MAX_WARP_SIDE) return fail(DN_E_INVALID_ARG, "S must be in 1..DN_MAX_WARP_SIDE");
    if (n_img <= 0 || H <= 0 || W <= 0) return fail(DN_E_INVALID_ARG, "bad image batch size");
    if (H > 32768 || W > 32768) return fail(DN_E_TOO_LARGE, "image sides are limited to 32768 px");
    if (pitch == 0) pitch = S;
    if (pitch < S || pitch > 8 * DN_MAX_WARP_SIDE) return fail(DN_E_INVALID_ARG, "pitch must be 0 or >= S");
    const size_t need = (size_t)n * 3 * (size_t)S * pitch * dtype_size(dtype);
    if (bytes_needed) *bytes_needed = need;
    if (!d_out) return DN_OK;
    if (out_bytes < need) return fail(DN_E_BUFFER_TOO_SMALL, "output buffer too small");
    if (n == 0) return DN_OK;
    if (!d_images || !d_boxes || !mean) return fail(DN_E_INVALID_ARG, "null pointer argument");
    if ((int64_t)n * ((S + 15) / 16) > 0x7fffffffLL) return fail(DN_E_TOO_LARGE, "too many boxes");
    return run_step("warp_regions", stream, [&] {
      return launch_warp_regions(d_images, n_img, H, W, d_boxes, d_box_img, n, S, pitch, mean, dtype,
                                 d_out, stream);
    });
  } catch (...) {
    return fail(DN_E_INTERNAL, "unexpected exception");
  }
}

int densenet_region_windows(const void* d_conv5, const dn_plane_desc* conv5_desc, int32_t n_maps,
                            dn_dtype conv5_dtype, const dn_scale_geom* geom, int32_t n_scales,
                            int32_t pad, int32_t planes_per_img, const float* d_boxes,
                            const int32_t* d_box_img, int32_t n, float target, int32_t S,
                            float* d_out, int32_t* d_scale, int32_t* d_idx, void* stream) {
  return region_call(d_conv5, conv5_desc, n_maps, conv5_dtype, geom, n_scales, pad, planes_per_img,
                     d_boxes, d_box_img, n, target, S, d_out, d_scale, d_idx, false, stream);
}

int densenet_region_pool(const void* d_conv5, const dn_plane_desc* conv5_desc, int32_t n_maps,
                         dn_dtype conv5_dtype, const dn_scale_geom* geom, int32_t n_scales,
                         int32_t pad, int32_t planes_per_img, const float* d_boxes,
                         const int32_t* d_box_img, int32_t n, float target, int32_t S, float* d_out,
                         int32_t* d_scale, int32_t* d_idx, void* stream) {
  return region_call(d_conv5, conv5_desc, n_maps, conv5_dtype, geom, n_scales, pad, planes_per_img,
                     d_boxes, d_box_img, n, target, S, d_out, d_scale, d_idx, true, stream);
}

int densenet_region_windows_batch(const void* d_conv5, const dn_plane_desc* conv5_desc,
                                  int32_t n_maps, dn_dtype conv5_dtype, const dn_scale_geom* geom,
                                  const dn_scale_geom* d_geom, int32_t n_img, int32_t n_entries,
                                  int32_t pad, int32_t pooled, const float* d_boxes,
                                  const int32_t* d_box_img, int32_t n, float target, int32_t S,
                                  float* d_out, int32_t* d_scale, int32_t* d_idx, void* stream) {
  if (pooled != 0 && pooled != 1) return fail(DN_E_INVALID_ARG, "pooled must be 0 or 1");
  return region_batch_call(d_conv5, conv5_desc, n_maps, conv5_dtype, geom, d_geom, n_img, n_entries, pad,
                           pooled == 1, d_boxes, d_box_img, n, target, S, d_out, d_scale, d_idx, stream);
}

}  // extern "C"
