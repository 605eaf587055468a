// Host geometry of the pyramid (Sec. 3.1): scale list, scaled sizes, padded rectangles, Bottom-Left
// Fill stitching onto planes, and each scale's window of conv5 cells.  Integer and fp64 arithmetic
// only; no device code.
//
// Stitching works on a 16-px occupancy grid: in stitched mode every rectangle side is a multiple of
// 16 px (the conv5 stride), so every corner a rectangle can take is a grid point and a fit test is a
// scan of grid cells.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <sstream>

#include "common.h"

namespace dn {

static int64_t div_floor(int64_t a, int64_t b) {  // b > 0
  return a >= 0 ? a / b : -((-a + b - 1) / b);
}
static int64_t div_ceil(int64_t a, int64_t b) { return -div_floor(-a, b); }

void stack_sides(int64_t n, int64_t out[8]) {
  auto conv = [](int64_t v, int64_t R, int64_t s, int64_t p) -> int64_t {
    return v + 2 * p >= R ? (v + 2 * p - R) / s + 1 : 0;
  };
  // 3x3/2 pooling, ceil mode: ceil((v-3)/2)+1 windows, the last one starting inside the input.
  auto pool = [](int64_t v) -> int64_t { return v >= 2 ? (v - 2) / 2 + 1 : 0; };
  out[0] = conv(n, 11, 4, 0);
  out[1] = pool(out[0]);
  out[2] = conv(out[1], 5, 1, 2);
  out[3] = pool(out[2]);
  out[4] = conv(out[3], 3, 1, 1);
  out[5] = conv(out[4], 3, 1, 1);
  out[6] = conv(out[5], 3, 1, 1);
  out[7] = pool(out[6]);
}

namespace {

struct Grid {  // occupancy of one plane in 16 x 16 px cells
  int gh, gw;
  int64_t free_cells;
  std::vector<uint8_t> used;
  std::vector<int> tops, lefts;  // candidate corner coordinates in cells
  Grid(int h, int w) : gh(h), gw(w), free_cells((int64_t)h * w), used((size_t)h * w, 0), tops{0}, lefts{0} {}
  bool free_at(int cy, int cx, int nh, int nw) const {
    if (cy + nh > gh || cx + nw > gw) return false;
    for (int r = cy; r < cy + nh; ++r) {
      const uint8_t* row = used.data() + (size_t)r * gw;
      for (int c = cx; c < cx + nw; ++c)
        if (row[c]) return false;
    }
    return true;
  }
  void occupy(int cy, int cx, int nh, int nw) {
    for (int r = cy; r < cy + nh; ++r) std::memset(used.data() + (size_t)r * gw + cx, 1, nw);
    free_cells -= (int64_t)nh * nw;
    tops.insert(std::upper_bound(tops.begin(), tops.end(), cy + nh), cy + nh);
    lefts.insert(std::upper_bound(lefts.begin(), lefts.end(), cx + nw), cx + nw);
  }
  // First corner in (top, left) order where an nh x nw block fits, or false.
  bool place(int nh, int nw, int& cy, int& cx) const {
    if (free_cells < (int64_t)nh * nw) return false;
    for (size_t i = 0; i < tops.size(); ++i) {
      if (i && tops[i] == tops[i - 1]) continue;
      for (size_t j = 0; j < lefts.size(); ++j) {
        if (j && lefts[j] == lefts[j - 1]) continue;
        if (free_at(tops[i], lefts[j], nh, nw)) {
          cy = tops[i];
          cx = lefts[j];
          return true;
        }
      }
    }
    return false;
  }
};

// Bottom-Left Fill of rectangles (sides multiples of 16 px) onto planes of PH x PW: items largest
// first (height, then width, then index), each on the first plane, in creation order, with a fitting
// candidate corner, topmost then leftmost; else on a new plane.  Writes plane, y, x of every item.
int stitch(std::vector<dn_scale_geom>& items, int32_t PH, int32_t PW, int max_planes, int& n_planes) {
  const int N = (int)items.size();
  std::vector<int> order(N);
  for (int i = 0; i < N; ++i) order[i] = i;
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    const dn_scale_geom &A = items[a], &B = items[b];
    if (A.rh != B.rh) return A.rh > B.rh;
    if (A.rw != B.rw) return A.rw > B.rw;
    return a < b;
  });
  std::vector<Grid> grids;
  for (int i : order) {
    dn_scale_geom& g = items[i];
    const int nh = g.rh / 16, nw = g.rw / 16;
    int cy = 0, cx = 0;
    size_t pi = 0;
    for (; pi < grids.size(); ++pi)
      if (grids[pi].place(nh, nw, cy, cx)) break;
    if (pi == grids.size()) {
      if ((int)grids.size() >= max_planes) {
        std::ostringstream os;
        os << "more than " << max_planes << " planes";
        return fail(DN_E_TOO_LARGE, os.str());
      }
      grids.emplace_back(PH / 16, PW / 16);
      cy = cx = 0;
    }
    grids[pi].occupy(cy, cx, nh, nw);
    g.plane = (int32_t)pi;
    g.y = cy * 16;
    g.x = cx * 16;
  }
  n_planes = (int)grids.size();
  return DN_OK;
}

// conv5 window of an entry on a PH x PW plane: cell i is centred at 16 i + 17.5; keep the cells
// centred on rows [y+p, y+p+h) (columns likewise), clipped to the plane's conv5 map.
void set_window(dn_scale_geom& g, int32_t PH, int32_t PW, int32_t pad) {
  int64_t sh[8], sw[8];
  stack_sides(PH, sh);
  stack_sides(PW, sw);
  const int64_t top = g.y + pad, left = g.x + pad;
  // first i with 32 i + 35 >= 2 top; last i with 32 i + 35 <= 2 (top + h) - 1
  g.r0 = (int32_t)std::max<int64_t>(0, div_ceil(2 * top - 35, 32));
  g.r1 = (int32_t)std::min<int64_t>(sh[6] - 1, div_floor(2 * (top + g.h) - 36, 32));
  g.c0 = (int32_t)std::max<int64_t>(0, div_ceil(2 * left - 35, 32));
  g.c1 = (int32_t)std::min<int64_t>(sw[6] - 1, div_floor(2 * (left + g.w) - 36, 32));
}

}  // namespace

int make_plan(int32_t H, int32_t W, const dn_pyramid_params& p, Plan& plan) {
  if (H <= 0 || W <= 0) return fail(DN_E_INVALID_ARG, "image sides must be positive");
  if (H > 32768 || W > 32768) return fail(DN_E_TOO_LARGE, "image sides are limited to 32768");
  if (p.n_scales <= 0 || p.n_scales > DN_MAX_SCALES) {
    std::ostringstream os;
    os << "n_scales must be in 1.." << DN_MAX_SCALES;
    return fail(DN_E_INVALID_ARG, os.str());
  }
  if (p.steps_per_octave <= 0) return fail(DN_E_INVALID_ARG, "steps_per_octave must be positive");
  if (p.pad < 0 || p.pad > 1024) return fail(DN_E_INVALID_ARG, "pad must be in 0..1024");
  if (p.pad_mode != DN_PAD_ZERO && p.pad_mode != DN_PAD_RAMP)
    return fail(DN_E_INVALID_ARG, "pad_mode must be DN_PAD_ZERO or DN_PAD_RAMP");
  if ((p.plane_h == 0) != (p.plane_w == 0) || p.plane_h < 0 || p.plane_w < 0)
    return fail(DN_E_INVALID_ARG, "plane_h and plane_w must both be 0 or both positive");
  const double base = p.base_longest_side > 0 ? (double)p.base_longest_side / (double)std::max(H, W)
                                               : p.base_scale;
  if (!(base > 0.0) || !std::isfinite(base)) return fail(DN_E_INVALID_ARG, "base scale must be > 0");
  if (p.n_aspects < 0 || p.n_aspects > DN_MAX_ASPECTS)
    return fail(DN_E_INVALID_ARG, "n_aspects must be in 0..DN_MAX_ASPECTS");
  for (int a = 0; a < p.n_aspects; ++a)
    if (!(p.aspects[a] > 0.0) || !std::isfinite(p.aspects[a]))
      return fail(DN_E_INVALID_ARG, "aspect ratios must be positive and finite");
  const int NA = p.n_aspects > 0 ? p.n_aspects : 1, NS = p.n_scales;
  if (NA * NS > DN_MAX_SCALES) {
    std::ostringstream os;
    os << "n_aspects * n_scales must be at most " << DN_MAX_SCALES;
    return fail(DN_E_INVALID_ARG, os.str());
  }

  // Entries: one per (aspect ratio, scale), aspect-major (Sec. 3.3: a whole pyramid per ratio).
  const int K = NA * NS;
  const bool stitched = p.plane_h > 0;
  plan.scales.assign(K, dn_scale_geom{});
  plan.planes.clear();
  for (int k = 0; k < K; ++k) {
    dn_scale_geom& g = plan.scales[k];
    g.k = k;
    g.aspect = k / NS;
    g.s = base * std::pow(2.0, -(double)(k % NS) / (double)p.steps_per_octave);
    // Area-keeping warp to ratio r: height over sqrt(r), width times sqrt(r) (r = 1: the plain scale).
    const double q = p.n_aspects > 0 ? std::sqrt(p.aspects[g.aspect]) : 1.0;
    const double fh = std::floor((double)H * (g.s / q) + 0.5), fw = std::floor((double)W * (g.s * q) + 0.5);
    if (!(fh <= 65535.0) || !(fw <= 65535.0))
      return fail(DN_E_TOO_LARGE, "scaled image sides are limited to 65535 px");
    g.h = std::max(1, (int)fh);
    g.w = std::max(1, (int)fw);
    g.sy = (double)g.h / (double)H;
    g.sx = (double)g.w / (double)W;
    g.rh = g.h + 2 * p.pad;
    g.rw = g.w + 2 * p.pad;
    if (stitched) {
      g.rh = (int)(div_ceil(g.rh, 16) * 16);
      g.rw = (int)(div_ceil(g.rw, 16) * 16);
      if (g.rh > p.plane_h || g.rw > p.plane_w) {
        std::ostringstream os;
        os << "scale " << k << " needs a " << g.rh << "x" << g.rw << " rectangle, larger than the "
           << p.plane_h << "x" << p.plane_w << " stitching plane";
        return fail(DN_E_TOO_LARGE, os.str());
      }
    }
  }

  if (!stitched) {
    for (int k = 0; k < K; ++k) {
      dn_scale_geom& g = plan.scales[k];
      g.plane = k;
      g.y = g.x = 0;
      plan.planes.push_back({g.rh, g.rw});
    }
  } else {
    int n_planes = 0;
    const int st = stitch(plan.scales, p.plane_h, p.plane_w, DN_MAX_PLANES_PER_IMAGE, n_planes);
    if (st != DN_OK) return st;
    plan.planes.assign(n_planes, PlaneSize{p.plane_h, p.plane_w});
  }
  if ((int)plan.planes.size() > DN_MAX_PLANES_PER_IMAGE)
    return fail(DN_E_TOO_LARGE, "more planes than DN_MAX_PLANES_PER_IMAGE");
  for (dn_scale_geom& g : plan.scales) {
    const PlaneSize ps = plan.planes[g.plane];
    set_window(g, ps.h, ps.w, p.pad);
  }
  return DN_OK;
}

int make_plan_batch(int32_t n_img, int32_t H, int32_t W, const dn_pyramid_params& p,
                    std::vector<dn_scale_geom>& items, int& n_planes) {
  if (n_img <= 0) return fail(DN_E_INVALID_ARG, "n_img must be positive");
  if (p.plane_h <= 0 || p.plane_w <= 0)
    return fail(DN_E_INVALID_ARG, "cross-image packing needs stitching planes (plane_h, plane_w > 0)");
  Plan one;  // the entries' sizes and rectangles; its own placement is replaced below
  const int st = make_plan(H, W, p, one);
  if (st != DN_OK) return st;
  const int64_t E = (int64_t)one.scales.size();
  if ((int64_t)n_img * E > DN_MAX_BATCH_ITEMS) {
    std::ostringstream os;
    os << "n_img * entries must be at most " << DN_MAX_BATCH_ITEMS;
    return fail(DN_E_TOO_LARGE, os.str());
  }
  items.assign((size_t)(n_img * E), dn_scale_geom{});
  for (int32_t b = 0; b < n_img; ++b)
    for (int64_t e = 0; e < E; ++e) {
      dn_scale_geom& g = items[(size_t)(b * E + e)];
      g = one.scales[(size_t)e];
      g.image = b;
    }
  const int st2 = stitch(items, p.plane_h, p.plane_w, (int)items.size(), n_planes);
  if (st2 != DN_OK) return st2;
  for (dn_scale_geom& g : items) set_window(g, p.plane_h, p.plane_w, p.pad);
  return DN_OK;
}

}  // namespace dn
