// Oracle for the DenseNet conv5 descriptor-pyramid path (Iandola et al., "DenseNet: Implementing
// Efficient ConvNet Descriptor Pyramids", arXiv 1404.1869).
//
// TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check and the benchmark's
// CPU-baseline leg may load this library.  The GPU library shares no source, header, table or helper
// with it, and neither links the other.
//
// What it is: a plain, slow, obviously correct CPU implementation of every step of the path, written
// from the paper (Sec. 3, 3.1, 3.2, 4) and, where the paper is silent, from the readings listed beside
// each function (the same readings are listed in the design notes).  All arithmetic is fp64; conv
// activations are rounded to fp32 only where a caller stores them as fp32 between layers.  Geometry is
// integer and fp64 only.  The library is built with -ffp-contract=off so that fp64 region arithmetic
// is a fixed sequence of correctly rounded + - * / operations.
//
// Parity unpinned (fixed only by a reading, with no external value to check against):
//   * the RAMP padding weights  w(d) = (p+1-d)/(p+1)            (Sec. 3.1, border interpolation)
//   * the Bottom-Left-Fill variant used for stitching           (Sec. 3.1, BLF)
//   * the region-to-scale rule (closest area to T x T, T = 227) (Sec. 4, crop after)
//   * the mean-pixel values (a caller parameter)                (Sec. 3.2)
// Every other function is pinned by closed forms, invariants or independent library routines in the
// CPU test suite.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

#ifdef _OPENMP
#include <omp.h>
#endif

extern "C" {

// Threads the OpenMP loops of this library use.
int oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

// ------------------------------------------------------------------------------------------------
// Geometry (Sec. 3.1): scale selection, scale sizes, padded rectangles, Bottom-Left-Fill stitching,
// and the per-scale window of conv5 cells.
//
// Output per scale k, as 16 int32 and 3 doubles:
//   gi[k*16 + 0..15] = k, h, w, plane, y, x, rh, rw, r0, r1, c0, c1, plane_h, plane_w, 0, 0
//   gd[k*3 + 0..2]   = s_k, sy_k = h/H, sx_k = w/W
// (y, x) is the top-left of the padded rectangle on its plane; the real image starts at (y+p, x+p).
// [r0,r1] x [c0,c1] are the conv5 cells whose receptive-field centre lies on a real pixel of the
// scale (empty when r1 < r0 or c1 < c0).  Returns the number of planes, or a negative error:
// -1 bad argument, -2 a rectangle larger than the stitching plane.
//
// Cross-image packing (oracle_plan_batch): the rectangles of all n_img images of a batch (same size
// H x W, so the same entries) are stitched as one set of items, so that small scales of several images
// share planes instead of leaving each image a half-empty last plane.  Item (b, e) is row b E + e of
// gi/gd (E entries per image), with gi[.. + 0] = e and gi[.. + 15] = b; its plane index counts over the
// whole batch.  The order is the one above with ties going to the smaller item index b E + e; a plane
// whose free area is smaller than the item's rectangle is skipped (it could not hold it anyway).
// oracle_plan is the case n_img = 1.
//
// Readings: s_k = base * 2^(-k/spo) for k = 0..K-1 (Sec. 3.1 scales per octave), base = base_scale or
// longest_side / max(H, W); sizes round half up, minimum 1.
// Aspect-ratio pyramids (Sec. 3.3): with n_aspects > 0 ratios r_a, the image warped to each ratio gets
// a whole pyramid: entry e = a K + k has h = floor(H (s_k / sqrt(r_a)) + 0.5), w = floor(W (s_k
// sqrt(r_a)) + 0.5) (the warp keeps the image's area), and every entry is one item of the stitching
// below; gi[e*16 + 0] = e, gi[e*16 + 14] = a.  n_aspects = 0 is the single pyramid of ratio 1.  Per-scale mode (plane_h == 0): each
// scale padded by p on every side is its own plane.  Stitched mode: rectangle sides rounded up to a
// multiple of 16 (the conv5 stride, so every scale keeps the same cell grid as when run alone); items
// taken largest first (rh desc, rw desc, k asc); on each existing plane, in creation order, the
// candidate corners are x in {0} U {x_j + rw_j}, y in {0} U {y_j + rh_j}; the first fitting corner in
// (y asc, x asc) order is taken; otherwise a new plane is opened.
// ------------------------------------------------------------------------------------------------

static int64_t floor_div(int64_t a, int64_t b) {  // b > 0
  int64_t q = a / b;
  if ((a % b) != 0 && (a < 0)) --q;
  return q;
}
static int64_t ceil_div(int64_t a, int64_t b) { return -floor_div(-a, b); }

// Output size of the conv stack on an n-pixel side, with the layer table of the AlexNet topology:
// conv1 11/4/0, pool 3/2 ceil, conv2 5/1/2, pool 3/2 ceil, conv3..5 3/1/1.  Returns <= 0 if empty.
static int64_t conv_out(int64_t n, int k, int s, int p) {
  int64_t t = n + 2 * p - k;
  if (t < 0) return 0;
  return t / s + 1;
}
static int64_t pool_out_ceil(int64_t n, int k, int s) {
  if (n <= 0) return 0;
  int64_t t = n - k;
  // ceil((n-k)/s) + 1, and the last window must start inside the input
  int64_t o = ceil_div(t, s) + 1;
  while ((o - 1) * s >= n) --o;
  return o;
}
static int64_t conv5_side(int64_t n) {
  int64_t a = conv_out(n, 11, 4, 0);
  a = pool_out_ceil(a, 3, 2);
  a = conv_out(a, 5, 1, 2);
  a = pool_out_ceil(a, 3, 2);
  a = conv_out(a, 3, 1, 1);
  a = conv_out(a, 3, 1, 1);
  a = conv_out(a, 3, 1, 1);
  return a;
}

int oracle_conv5_side(int n) { return (int)conv5_side(n); }

int oracle_plan_batch(int n_img, int H, int W, int K, int spo, double base_scale,
                      int base_longest_side, int pad, int plane_h, int plane_w, int n_aspects,
                      const double* aspects, int32_t* gi, double* gd) {
  if (n_img <= 0 || H <= 0 || W <= 0 || K <= 0 || spo <= 0 || pad < 0 || n_aspects < 0) return -1;
  if (n_img > 1 && plane_h == 0) return -1;  // cross-image packing needs stitching planes
  for (int a = 0; a < n_aspects; ++a)
    if (!(aspects[a] > 0.0) || !std::isfinite(aspects[a])) return -1;
  const int A = n_aspects > 0 ? n_aspects : 1, NS = K;
  K = A * NS;  // items: one per (aspect, scale)
  if ((plane_h == 0) != (plane_w == 0)) return -1;
  double base = base_scale;
  if (base_longest_side > 0) base = (double)base_longest_side / (double)std::max(H, W);
  if (!(base > 0.0)) return -1;

  struct Item { int k, h, w, rh, rw, plane, y, x; };
  const int E = K;    // entries per image
  K = n_img * E;      // items of the whole batch: item b E + e is entry e of image b
  std::vector<Item> it(K);
  for (int k = 0; k < K; ++k) {
    const int a = (k % E) / NS;
    double s = base * std::pow(2.0, -(double)(k % NS) / (double)spo);
    gd[k * 3 + 0] = s;
    const double q = n_aspects > 0 ? std::sqrt(aspects[a]) : 1.0;
    int h = (int)std::floor((double)H * (s / q) + 0.5);
    int w = (int)std::floor((double)W * (s * q) + 0.5);
    if (h < 1) h = 1;
    if (w < 1) w = 1;
    gd[k * 3 + 1] = (double)h / (double)H;
    gd[k * 3 + 2] = (double)w / (double)W;
    it[k].k = k % E; it[k].h = h; it[k].w = w;
    if (plane_h == 0) {
      it[k].rh = h + 2 * pad;
      it[k].rw = w + 2 * pad;
    } else {
      it[k].rh = (int)(ceil_div(h + 2 * pad, 16) * 16);
      it[k].rw = (int)(ceil_div(w + 2 * pad, 16) * 16);
    }
  }

  int n_planes = 0;
  std::vector<int> ph, pw;  // per plane size
  if (plane_h == 0) {
    for (int k = 0; k < K; ++k) {
      it[k].plane = k; it[k].y = 0; it[k].x = 0;
      ph.push_back(it[k].rh); pw.push_back(it[k].rw);
    }
    n_planes = K;
  } else {
    for (int k = 0; k < K; ++k)
      if (it[k].rh > plane_h || it[k].rw > plane_w) return -2;
    std::vector<int> order(K);
    for (int k = 0; k < K; ++k) order[k] = k;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
      if (it[a].rh != it[b].rh) return it[a].rh > it[b].rh;
      if (it[a].rw != it[b].rw) return it[a].rw > it[b].rw;
      return a < b;
    });
    std::vector<std::vector<int>> on_plane;  // item indices placed on each plane
    std::vector<int64_t> free_area;          // plane area not covered by rectangles
    for (int idx : order) {
      Item& r = it[idx];
      bool placed = false;
      for (int p = 0; p < n_planes && !placed; ++p) {
        if (free_area[p] < (int64_t)r.rh * r.rw) continue;
        std::vector<int> ys{0}, xs{0};
        for (int j : on_plane[p]) { ys.push_back(it[j].y + it[j].rh); xs.push_back(it[j].x + it[j].rw); }
        std::sort(ys.begin(), ys.end());
        std::sort(xs.begin(), xs.end());
        for (int y : ys) {
          if (placed) break;
          for (int x : xs) {
            if (y + r.rh > plane_h || x + r.rw > plane_w) continue;
            bool overlap = false;
            for (int j : on_plane[p]) {
              const Item& q = it[j];
              if (y < q.y + q.rh && q.y < y + r.rh && x < q.x + q.rw && q.x < x + r.rw) { overlap = true; break; }
            }
            if (!overlap) {
              r.plane = p; r.y = y; r.x = x;
              on_plane[p].push_back(idx);
              free_area[p] -= (int64_t)r.rh * r.rw;
              placed = true;
              break;
            }
          }
        }
      }
      if (!placed) {
        on_plane.push_back({idx});
        free_area.push_back((int64_t)plane_h * plane_w - (int64_t)r.rh * r.rw);
        r.plane = n_planes; r.y = 0; r.x = 0;
        ph.push_back(plane_h); pw.push_back(plane_w);
        ++n_planes;
      }
    }
  }

  for (int k = 0; k < K; ++k) {
    const Item& r = it[k];
    int PH = ph[r.plane], PW = pw[r.plane];
    int64_t Hc = conv5_side(PH), Wc = conv5_side(PW);
    // Sec. 3.1 unpacking: conv5 cell i has its receptive-field centre at 16 i + 17.5 in continuous
    // plane coordinates; keep the cells whose centre lies on a real pixel [y+p, y+p+h).
    int64_t r0 = ceil_div(2 * (int64_t)(r.y + pad) - 35, 32);
    int64_t r1 = ceil_div(2 * (int64_t)(r.y + pad + r.h) - 35, 32) - 1;
    int64_t c0 = ceil_div(2 * (int64_t)(r.x + pad) - 35, 32);
    int64_t c1 = ceil_div(2 * (int64_t)(r.x + pad + r.w) - 35, 32) - 1;
    r0 = std::max<int64_t>(r0, 0); c0 = std::max<int64_t>(c0, 0);
    r1 = std::min<int64_t>(r1, Hc - 1); c1 = std::min<int64_t>(c1, Wc - 1);
    int32_t* o = gi + k * 16;
    o[0] = r.k; o[1] = r.h; o[2] = r.w; o[3] = r.plane; o[4] = r.y; o[5] = r.x; o[6] = r.rh; o[7] = r.rw;
    o[8] = (int32_t)r0; o[9] = (int32_t)r1; o[10] = (int32_t)c0; o[11] = (int32_t)c1;
    o[12] = PH; o[13] = PW; o[14] = r.k / NS; o[15] = k / E;
  }
  return n_planes;
}

int oracle_plan(int H, int W, int K, int spo, double base_scale, int base_longest_side, int pad,
                int plane_h, int plane_w, int n_aspects, const double* aspects, int32_t* gi,
                double* gd) {
  return oracle_plan_batch(1, H, W, K, spo, base_scale, base_longest_side, pad, plane_h, plane_w,
                           n_aspects, aspects, gi, gd);
}

// ------------------------------------------------------------------------------------------------
// Resize + centring (Sec. 3 pyramid by up/down-sampling; Sec. 3.2 mean-pixel centring).
// Half-pixel-centre bilinear interpolation of the original uint8 image (every scale is sampled from
// the original), source coordinate clamped at 0 below and the neighbour index clamped at the last
// row/column, no antialiasing; then the mean pixel of the channel is subtracted.
// out[c][y][x] for y < h, x < w; all fp64.
// ------------------------------------------------------------------------------------------------
void oracle_resize_center(const uint8_t* img, int H, int W, int h, int w, const double* mean,
                          double* out) {
  const double ry = (double)H / (double)h, rx = (double)W / (double)w;
  for (int c = 0; c < 3; ++c) {
    const uint8_t* I = img + (size_t)c * H * W;
    for (int y = 0; y < h; ++y) {
      double sy = (y + 0.5) * ry - 0.5;
      if (sy < 0) sy = 0;
      int y0 = (int)std::floor(sy);
      if (y0 > H - 1) y0 = H - 1;
      int y1 = std::min(y0 + 1, H - 1);
      double ly = sy - y0;
      for (int x = 0; x < w; ++x) {
        double sx = (x + 0.5) * rx - 0.5;
        if (sx < 0) sx = 0;
        int x0 = (int)std::floor(sx);
        if (x0 > W - 1) x0 = W - 1;
        int x1 = std::min(x0 + 1, W - 1);
        double lx = sx - x0;
        double top = (1 - lx) * I[(size_t)y0 * W + x0] + lx * I[(size_t)y0 * W + x1];
        double bot = (1 - lx) * I[(size_t)y1 * W + x0] + lx * I[(size_t)y1 * W + x1];
        double v = (1 - ly) * top + ly * bot;
        out[((size_t)c * h + y) * w + x] = v - mean[c];
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// Crop-before baseline (Sec. 3.4, Sec. 4): every region is cut out of the image in pixel space and
// warped on its own to the classifier's S x S input, then mean-centred, so that each window can be run
// through the network in isolation.
//   box (x1, y1, x2, y2) in pixel-edge coordinates of image b = box_img[r] (0 when box_img is null);
//   output pixel (i, j) samples the image at
//     sy = y1 + (i + 0.5) (y2 - y1) / S - 0.5,   sx = x1 + (j + 0.5) (x2 - x1) / S - 0.5,
//   i.e. the box is stretched onto the S x S grid with half-pixel centres (no context margin), with
//   bilinear sampling with the coordinate clamped to [0, H - 1] (resp. [0, W - 1]): a box reaching
//   outside the image repeats the edge pixel, with interpolation weights in [0, 1); the top-left
//   neighbour is floor(s), the other one further (clamped).  Then the mean pixel of the channel is
//   subtracted.  A box with a non-finite or non-positive side gives an all-zero
//   window.  out[r][c][i][j], fp32 values of fp64 arithmetic.
// ------------------------------------------------------------------------------------------------
void oracle_warp_regions(const uint8_t* img, int n_img, int H, int W, const float* boxes,
                         const int32_t* box_img, int n, int S, const double* mean, float* out) {
#pragma omp parallel for schedule(dynamic, 4)
  for (int r = 0; r < n; ++r) {
    float* o = out + (size_t)r * 3 * S * S;
    std::fill(o, o + (size_t)3 * S * S, 0.f);
    const double x1 = boxes[r * 4 + 0], y1 = boxes[r * 4 + 1], x2 = boxes[r * 4 + 2], y2 = boxes[r * 4 + 3];
    if (!std::isfinite(x1) || !std::isfinite(y1) || !std::isfinite(x2) || !std::isfinite(y2)) continue;
    if (!(x2 - x1 > 0) || !(y2 - y1 > 0)) continue;
    const int b = box_img ? box_img[r] : 0;
    if (b < 0 || b >= n_img) continue;
    const double fy = (y2 - y1) / S, fx = (x2 - x1) / S;
    for (int c = 0; c < 3; ++c) {
      const uint8_t* I = img + ((size_t)b * 3 + c) * H * W;
      for (int i = 0; i < S; ++i) {
        double sy = y1 + (i + 0.5) * fy - 0.5;
        sy = std::min(std::max(sy, 0.0), (double)(H - 1));
        const int y0 = (int)std::floor(sy);
        const int yb = std::min(y0 + 1, H - 1);
        const double ly = sy - y0;
        for (int j = 0; j < S; ++j) {
          double sx = x1 + (j + 0.5) * fx - 0.5;
          sx = std::min(std::max(sx, 0.0), (double)(W - 1));
          const int x0 = (int)std::floor(sx);
          const int xb = std::min(x0 + 1, W - 1);
          const double lx = sx - x0;
          const double top = (1 - lx) * I[(size_t)y0 * W + x0] + lx * I[(size_t)y0 * W + xb];
          const double bot = (1 - lx) * I[(size_t)yb * W + x0] + lx * I[(size_t)yb * W + xb];
          o[((size_t)c * S + i) * S + j] = (float)((1 - ly) * top + ly * bot - mean[c]);
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------------------
// Plane filling (Sec. 3.1 border and background, Sec. 3.2 background equals the mean pixel, hence 0
// after centring).  For a plane pixel inside scale k's rectangle, with v, u its row/column relative to
// the first real pixel and d the distance outside the image along each axis:
//   value = C_k(clamp(v), clamp(u)) * w(dy) * w(dx)  if dy <= p and dx <= p, else 0,
//   RAMP (pad_mode 1): w(d) = (p+1-d)/(p+1), a linear blend from the edge pixel to the mean;
//   ZERO (pad_mode 0): w(d) = [d == 0].
// Pixels covered by no rectangle are 0.  planes: [n_planes][3][PH][PW] fp64, every plane of size
// (PH_max, PW_max) with the plane's own (plane_h, plane_w) region used; the caller passes the sizes.
// gi/gd as produced by oracle_plan or oracle_plan_batch (K rows); row k samples image gi[k*16 + 15]
// of img ([n_img][3][H][W] uint8).
// ------------------------------------------------------------------------------------------------
void oracle_build_planes(const uint8_t* img, int H, int W, int K, const int32_t* gi, const double* gd,
                         int pad, int pad_mode, const double* mean, int n_planes, int PHmax, int PWmax,
                         double* planes) {
  (void)gd;
  std::memset(planes, 0, sizeof(double) * (size_t)n_planes * 3 * PHmax * PWmax);
  for (int k = 0; k < K; ++k) {
    const int32_t* g = gi + k * 16;
    int h = g[1], w = g[2], pl = g[3], y0 = g[4], x0 = g[5], rh = g[6], rw = g[7];
    std::vector<double> C((size_t)3 * h * w);
    oracle_resize_center(img + (size_t)g[15] * 3 * H * W, H, W, h, w, mean, C.data());
    auto weight = [&](int d) -> double {
      if (d == 0) return 1.0;
      if (pad_mode == 0) return 0.0;
      return (double)(pad + 1 - d) / (double)(pad + 1);
    };
    for (int c = 0; c < 3; ++c)
      for (int yy = 0; yy < rh; ++yy)
        for (int xx = 0; xx < rw; ++xx) {
          int v = yy - pad, u = xx - pad;
          int dy = std::max(0, std::max(-v, v - (h - 1)));
          int dx = std::max(0, std::max(-u, u - (w - 1)));
          double val = 0.0;
          if (dy <= pad && dx <= pad) {
            int vc = std::min(std::max(v, 0), h - 1), uc = std::min(std::max(u, 0), w - 1);
            val = C[((size_t)c * h + vc) * w + uc] * weight(dy) * weight(dx);
          }
          planes[(((size_t)pl * 3 + c) * PHmax + (y0 + yy)) * PWmax + (x0 + xx)] = val;
        }
  }
}

// ------------------------------------------------------------------------------------------------
// Convolution (the conv layers that carry the bulk of the work, Sec. 3), by its definition:
//   out[m,i,j] = b[m] + sum_{c in group(m)} sum_{ky,kx} w[m, c - c0(m), ky, kx] * in[c, s i + ky - p, s j + kx - p]
// with zero outside the input; Ho = floor((Hi + 2p - R)/s) + 1; group g owns input channels
// [g C/G, (g+1) C/G) and output channels [g M/G, (g+1) M/G).  Optional ReLU max(0, x).
// in [C][Hi][Wi], w [M][C/G][R][R], b [M], out [M][Ho][Wo]; fp64 accumulation, fp32 output.
// ------------------------------------------------------------------------------------------------
int oracle_conv2d(const float* in, int C, int Hi, int Wi, const float* w, const float* b, int M, int R,
                  int stride, int pad, int groups, int relu, float* out) {
  if (C % groups || M % groups) return -1;
  const int Ho = (int)conv_out(Hi, R, stride, pad), Wo = (int)conv_out(Wi, R, stride, pad);
  if (Ho <= 0 || Wo <= 0) return -1;
  const int Cg = C / groups, Mg = M / groups;
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const int g = m / Mg;
    std::vector<double> acc((size_t)Ho * Wo, (double)b[m]);
    for (int cl = 0; cl < Cg; ++cl) {
      const int c = g * Cg + cl;
      const float* I = in + (size_t)c * Hi * Wi;
      for (int ky = 0; ky < R; ++ky)
        for (int kx = 0; kx < R; ++kx) {
          const double wv = (double)w[(((size_t)m * Cg + cl) * R + ky) * R + kx];
          for (int i = 0; i < Ho; ++i) {
            const int iy = stride * i + ky - pad;
            if (iy < 0 || iy >= Hi) continue;
            double* a = acc.data() + (size_t)i * Wo;
            for (int j = 0; j < Wo; ++j) {
              const int ix = stride * j + kx - pad;
              if (ix < 0 || ix >= Wi) continue;
              a[j] += wv * (double)I[(size_t)iy * Wi + ix];
            }
          }
        }
    }
    float* o = out + (size_t)m * Ho * Wo;
    for (size_t t = 0; t < (size_t)Ho * Wo; ++t) {
      double v = acc[t];
      if (relu && v < 0) v = 0;
      o[t] = (float)v;
    }
  }
  return 0;
}

// ------------------------------------------------------------------------------------------------
// Local response normalisation across channels (the AlexNet topology the paper runs, Sec. 3):
//   b_c = a_c * (k + (alpha/n) * sum_{j = c - n/2}^{c + n/2, clipped to [0, C)} a_j^2)^(-beta)
// over all C channels of the layer (not per group).  n odd.  fp64 arithmetic, fp32 output.
// ------------------------------------------------------------------------------------------------
int oracle_lrn(const float* in, int C, int H, int W, int n, double alpha, double beta, double k,
               float* out) {
  if (n <= 0 || (n % 2) == 0) return -1;
  const int half = n / 2;
  const size_t HW = (size_t)H * W;
#pragma omp parallel for schedule(static)
  for (long long t = 0; t < (long long)HW; ++t) {
    for (int c = 0; c < C; ++c) {
      double s = 0;
      for (int j = std::max(0, c - half); j <= std::min(C - 1, c + half); ++j) {
        double a = (double)in[(size_t)j * HW + t];
        s += a * a;
      }
      double a = (double)in[(size_t)c * HW + t];
      out[(size_t)c * HW + t] = (float)(a * std::pow(k + (alpha / n) * s, -beta));
    }
  }
  return 0;
}

// ------------------------------------------------------------------------------------------------
// Max pooling R x R / stride s with ceil-mode output size and windows clipped to the input:
//   Ho = ceil((Hi - R)/s) + 1 (last window starts inside the input); out[c,i,j] = max over rows
//   [s i, min(s i + R, Hi)) and columns [s j, min(s j + R, Wi)).
// ------------------------------------------------------------------------------------------------
int oracle_maxpool(const float* in, int C, int Hi, int Wi, int R, int s, float* out) {
  const int Ho = (int)pool_out_ceil(Hi, R, s), Wo = (int)pool_out_ceil(Wi, R, s);
  if (Ho <= 0 || Wo <= 0) return -1;
#pragma omp parallel for schedule(static)
  for (int c = 0; c < C; ++c)
    for (int i = 0; i < Ho; ++i)
      for (int j = 0; j < Wo; ++j) {
        double m = -INFINITY;
        for (int y = s * i; y < std::min(s * i + R, Hi); ++y)
          for (int x = s * j; x < std::min(s * j + R, Wi); ++x)
            m = std::max(m, (double)in[((size_t)c * Hi + y) * Wi + x]);
        out[((size_t)c * Ho + i) * Wo + j] = (float)m;
      }
  return 0;
}

int oracle_pool_side(int n) { return (int)pool_out_ceil(n, 3, 2); }
int oracle_conv_side(int n, int R, int s, int p) { return (int)conv_out(n, R, s, p); }

// ------------------------------------------------------------------------------------------------
// The conv stack on one plane (Sec. 3: the first five conv layers of the AlexNet classifier):
//   conv1 -> ReLU -> LRN -> pool, conv2(g2) -> ReLU -> LRN -> pool, conv3 -> ReLU,
//   conv4(g2) -> ReLU, conv5(g2) -> ReLU [-> pool5].
// lrn_before_pool = 0 swaps each LRN/pool pair (pool then LRN).  plane [3][PH][PW] fp32; weights
// w[l] OIHW fp32 and biases b[l]; conv5 out [256][Hc][Wc]; pool5 out (nullable) [256][Hp][Wp].
// Intermediates are stored as fp32.
// ------------------------------------------------------------------------------------------------
int oracle_net(const float* plane, int PH, int PW, const float* const* w, const float* const* b,
               double lrn_alpha, double lrn_beta, double lrn_k, int lrn_n, int lrn_before_pool,
               float* conv5, float* pool5) {
  struct L { int M, C, R, s, p, G; };
  const L Ls[5] = {{96, 3, 11, 4, 0, 1}, {256, 96, 5, 1, 2, 2}, {384, 256, 3, 1, 1, 1},
                   {384, 384, 3, 1, 1, 2}, {256, 384, 3, 1, 1, 2}};
  std::vector<float> cur(plane, plane + (size_t)3 * PH * PW), nxt, tmp;
  int H = PH, W = PW;
  for (int l = 0; l < 5; ++l) {
    const L& L_ = Ls[l];
    int Ho = (int)conv_out(H, L_.R, L_.s, L_.p), Wo = (int)conv_out(W, L_.R, L_.s, L_.p);
    if (Ho <= 0 || Wo <= 0) return -1;
    nxt.assign((size_t)L_.M * Ho * Wo, 0.f);
    if (oracle_conv2d(cur.data(), L_.C, H, W, w[l], b[l], L_.M, L_.R, L_.s, L_.p, L_.G, 1, nxt.data()))
      return -1;
    H = Ho; W = Wo;
    cur.swap(nxt);
    if (l < 2) {
      int Hp = (int)pool_out_ceil(H, 3, 2), Wp = (int)pool_out_ceil(W, 3, 2);
      if (Hp <= 0 || Wp <= 0) return -1;
      if (lrn_before_pool) {
        tmp.assign(cur.size(), 0.f);
        oracle_lrn(cur.data(), L_.M, H, W, lrn_n, lrn_alpha, lrn_beta, lrn_k, tmp.data());
        nxt.assign((size_t)L_.M * Hp * Wp, 0.f);
        oracle_maxpool(tmp.data(), L_.M, H, W, 3, 2, nxt.data());
      } else {
        tmp.assign((size_t)L_.M * Hp * Wp, 0.f);
        oracle_maxpool(cur.data(), L_.M, H, W, 3, 2, tmp.data());
        nxt.assign(tmp.size(), 0.f);
        oracle_lrn(tmp.data(), L_.M, Hp, Wp, lrn_n, lrn_alpha, lrn_beta, lrn_k, nxt.data());
      }
      cur.swap(nxt);
      H = Hp; W = Wp;
    }
  }
  std::memcpy(conv5, cur.data(), sizeof(float) * cur.size());
  if (pool5) oracle_maxpool(cur.data(), 256, H, W, 3, 2, pool5);
  return 0;
}

// ------------------------------------------------------------------------------------------------
// Region windows ("crop after", Sec. 4): each box of the original image is read out of the conv5
// pyramid at the scale whose scaled box area is closest (in log ratio) to T x T, as S x S bilinear
// samples at bin centres of the box, all 256 channels.
//   box (x1, y1, x2, y2) in original-image pixel-edge coordinates; bw = x2 - x1, bh = y2 - y1; a box
//   with a non-finite or non-positive side gets scale -1 and a zero row.
//   a_k = (sy_k bh)(sx_k bw); cost_k = max(a_k / T^2, T^2 / a_k); k* = argmin, ties to the smaller k,
//   scales with an empty cell window are skipped.  With aspect-ratio pyramids (n_aspects > 1) the
//   cost is multiplied by max(rho_k, 1 / rho_k), rho_k = (sx_k bw) / (sy_k bh) the aspect of the box on
//   entry k, so the box is read where it is closest to a T x T square.
//   X = x * sx + x_k + p (plane coordinates of the scale's real pixels); bin centre
//   U = X1 + f_b (X2 - X1), f_b = (b + 0.5)/S; conv5 coordinate g = (U - 17.5) * 0.0625 (cell i is
//   centred at 16 i + 17.5), clamped to [c0, c1]; j0 = floor(g), j1 = min(j0 + 1, c1), lambda = g - j0.
//   Rows likewise.  The value is the bilinear blend of the four cells, fp64.
// conv5 planes: [n_img * planes_per_img][256][Hc][Wc] fp32, each plane (Hc, Wc) = (Hcs[p], Wcs[p])
// stored at plane_off[p] (elements); the box's image b reads plane b * planes_per_img + plane_k.
// planes_per_img = 0 is a cross-image packed batch (oracle_plan_batch): gi/gd hold K rows per image,
// image b's entries are rows b K .. b K + K - 1, and their plane indices count over the batch.
// desc [n][256 * S * S] flattened (channel, row, col);
// scale [n]; idx (nullable) [n][S][S][2] = (i0, j0) plane cell of the top-left sample;
// lam (nullable) [n][S][S][2] = (lambda_y, lambda_x).
// ------------------------------------------------------------------------------------------------
int oracle_region_windows(const float* conv5, const int64_t* plane_off, const int32_t* Hcs,
                          const int32_t* Wcs, int planes_per_img, int K, const int32_t* gi,
                          const double* gd, int pad, const float* boxes, const int32_t* box_img, int n,
                          double T, int S, int n_aspects, float* desc, int32_t* scale, int32_t* idx,
                          double* lam) {
  if (S <= 0 || !(T > 0)) return -1;
  const int C = 256;
#pragma omp parallel for schedule(dynamic, 16)
  for (int r = 0; r < n; ++r) {
    float* d = desc + (size_t)r * C * S * S;
    std::fill(d, d + (size_t)C * S * S, 0.f);
    scale[r] = -1;
    if (idx) std::fill(idx + (size_t)r * S * S * 2, idx + (size_t)(r + 1) * S * S * 2, 0);
    if (lam) std::fill(lam + (size_t)r * S * S * 2, lam + (size_t)(r + 1) * S * S * 2, 0.0);
    const double x1 = boxes[r * 4 + 0], y1 = boxes[r * 4 + 1], x2 = boxes[r * 4 + 2], y2 = boxes[r * 4 + 3];
    const double bw = x2 - x1, bh = y2 - y1;
    if (!std::isfinite(x1) || !std::isfinite(y1) || !std::isfinite(x2) || !std::isfinite(y2)) continue;
    if (!(bw > 0) || !(bh > 0)) continue;
    const int img = box_img ? box_img[r] : 0;
    const int32_t* gi_b = planes_per_img ? gi : gi + (size_t)img * K * 16;
    const double* gd_b = planes_per_img ? gd : gd + (size_t)img * K * 3;
    const double T2 = T * T;
    int best = -1;
    double best_cost = 0;
    for (int k = 0; k < K; ++k) {
      const int32_t* g = gi_b + k * 16;
      if (g[9] < g[8] || g[11] < g[10]) continue;
      const double a = (gd_b[k * 3 + 1] * bh) * (gd_b[k * 3 + 2] * bw);
      double cost = std::max(a / T2, T2 / a);
      if (n_aspects > 1) {
        const double rho = (gd_b[k * 3 + 2] * bw) / (gd_b[k * 3 + 1] * bh);
        cost = cost * std::max(rho, 1.0 / rho);
      }
      if (best < 0 || cost < best_cost) { best = k; best_cost = cost; }
    }
    if (best < 0) continue;
    const int32_t* g = gi_b + best * 16;
    const double sy = gd_b[best * 3 + 1], sx = gd_b[best * 3 + 2];
    const int pl = img * planes_per_img + g[3];
    const int Hc = Hcs[pl], Wc = Wcs[pl];
    (void)Hc;
    const float* F = conv5 + plane_off[pl];
    const double X1 = x1 * sx + g[5] + pad, X2 = x2 * sx + g[5] + pad;
    const double Y1 = y1 * sy + g[4] + pad, Y2 = y2 * sy + g[4] + pad;
    const int r0 = g[8], r1 = g[9], c0 = g[10], c1 = g[11];
    scale[r] = best;
    for (int a = 0; a < S; ++a) {
      const double fa = (a + 0.5) / S;
      double gy = ((Y1 + fa * (Y2 - Y1)) - 17.5) * 0.0625;
      gy = std::min(std::max(gy, (double)r0), (double)r1);
      const int i0 = (int)std::floor(gy), i1 = std::min(i0 + 1, r1);
      const double ly = gy - i0;
      for (int bb = 0; bb < S; ++bb) {
        const double fb = (bb + 0.5) / S;
        double gx = ((X1 + fb * (X2 - X1)) - 17.5) * 0.0625;
        gx = std::min(std::max(gx, (double)c0), (double)c1);
        const int j0 = (int)std::floor(gx), j1 = std::min(j0 + 1, c1);
        const double lx = gx - j0;
        if (idx) { idx[((size_t)r * S * S + a * S + bb) * 2 + 0] = i0; idx[((size_t)r * S * S + a * S + bb) * 2 + 1] = j0; }
        if (lam) { lam[((size_t)r * S * S + a * S + bb) * 2 + 0] = ly; lam[((size_t)r * S * S + a * S + bb) * 2 + 1] = lx; }
        for (int c = 0; c < C; ++c) {
          const float* Fc = F + (size_t)c * Hc * Wc;
          const double v00 = Fc[(size_t)i0 * Wc + j0], v01 = Fc[(size_t)i0 * Wc + j1];
          const double v10 = Fc[(size_t)i1 * Wc + j0], v11 = Fc[(size_t)i1 * Wc + j1];
          const double top = (1 - lx) * v00 + lx * v01, bot = (1 - lx) * v10 + lx * v11;
          d[(size_t)c * S * S + a * S + bb] = (float)((1 - ly) * top + ly * bot);
        }
      }
    }
  }
  return 0;
}

// ------------------------------------------------------------------------------------------------
// Max-pooled region bins (descriptor post-processing after the region windows, the pool5-style
// alternative to bilinear samples): the box is read at the same entry as above (same cost, same
// ties), and its S x S bins take, per channel, the maximum over the conv5 cells whose receptive-field
// centre (16 i + 17.5 in plane coordinates) lies inside the bin.
//   Bin a spans plane rows [Y1 + a (Y2 - Y1) / S, Y1 + (a + 1)(Y2 - Y1) / S); its cells are
//   i in [ceil((lo - 17.5) / 16), ceil((hi - 17.5) / 16) - 1], clipped to the entry's window [r0, r1];
//   a bin left with no cell takes the one cell nearest its centre: clamp(floor(g + 0.5), r0, r1) with
//   g = (centre - 17.5) / 16.  Columns likewise.  Everything is fp64 with + - * / only.
// idx (nullable) [n][S][S][4] = (i_first, i_last, j_first, j_last) of each bin.  Same layouts (and the
// same cross-image packed mode, planes_per_img = 0) as oracle_region_windows otherwise.
// ------------------------------------------------------------------------------------------------
static void pool_bin_range(double lo, double hi, int cmin, int cmax, int& first, int& last) {
  // cells with lo <= 16 i + 17.5 < hi
  int f = (int)std::ceil((lo - 17.5) / 16.0);
  int l = (int)std::ceil((hi - 17.5) / 16.0) - 1;
  f = std::max(f, cmin);
  l = std::min(l, cmax);
  if (l < f) {
    const double g = ((lo + hi) * 0.5 - 17.5) / 16.0;
    int c = (int)std::floor(g + 0.5);
    c = std::min(std::max(c, cmin), cmax);
    f = l = c;
  }
  first = f;
  last = l;
}

int oracle_region_pool(const float* conv5, const int64_t* plane_off, const int32_t* Hcs,
                       const int32_t* Wcs, int planes_per_img, int K, const int32_t* gi,
                       const double* gd, int pad, const float* boxes, const int32_t* box_img, int n,
                       double T, int S, int n_aspects, float* desc, int32_t* scale, int32_t* idx) {
  if (S <= 0 || !(T > 0)) return -1;
  const int C = 256;
#pragma omp parallel for schedule(dynamic, 16)
  for (int r = 0; r < n; ++r) {
    float* d = desc + (size_t)r * C * S * S;
    std::fill(d, d + (size_t)C * S * S, 0.f);
    scale[r] = -1;
    if (idx) std::fill(idx + (size_t)r * S * S * 4, idx + (size_t)(r + 1) * S * S * 4, 0);
    const double x1 = boxes[r * 4 + 0], y1 = boxes[r * 4 + 1], x2 = boxes[r * 4 + 2], y2 = boxes[r * 4 + 3];
    const double bw = x2 - x1, bh = y2 - y1;
    if (!std::isfinite(x1) || !std::isfinite(y1) || !std::isfinite(x2) || !std::isfinite(y2)) continue;
    if (!(bw > 0) || !(bh > 0)) continue;
    const int img = box_img ? box_img[r] : 0;
    const int32_t* gi_b = planes_per_img ? gi : gi + (size_t)img * K * 16;
    const double* gd_b = planes_per_img ? gd : gd + (size_t)img * K * 3;
    const double T2 = T * T;
    int best = -1;
    double best_cost = 0;
    for (int k = 0; k < K; ++k) {
      const int32_t* g = gi_b + k * 16;
      if (g[9] < g[8] || g[11] < g[10]) continue;
      const double a = (gd_b[k * 3 + 1] * bh) * (gd_b[k * 3 + 2] * bw);
      double cost = std::max(a / T2, T2 / a);
      if (n_aspects > 1) {
        const double rho = (gd_b[k * 3 + 2] * bw) / (gd_b[k * 3 + 1] * bh);
        cost = cost * std::max(rho, 1.0 / rho);
      }
      if (best < 0 || cost < best_cost) { best = k; best_cost = cost; }
    }
    if (best < 0) continue;
    const int32_t* g = gi_b + best * 16;
    const double sy = gd_b[best * 3 + 1], sx = gd_b[best * 3 + 2];
    const int pl = img * planes_per_img + g[3];
    const int Hc = Hcs[pl], Wc = Wcs[pl];
    const float* F = conv5 + plane_off[pl];
    const double X1 = x1 * sx + g[5] + pad, X2 = x2 * sx + g[5] + pad;
    const double Y1 = y1 * sy + g[4] + pad, Y2 = y2 * sy + g[4] + pad;
    scale[r] = best;
    for (int a = 0; a < S; ++a) {
      int i0, i1;
      pool_bin_range(Y1 + a * (Y2 - Y1) / S, Y1 + (a + 1) * (Y2 - Y1) / S, g[8], g[9], i0, i1);
      for (int b = 0; b < S; ++b) {
        int j0, j1;
        pool_bin_range(X1 + b * (X2 - X1) / S, X1 + (b + 1) * (X2 - X1) / S, g[10], g[11], j0, j1);
        if (idx) {
          int32_t* q = idx + ((size_t)r * S * S + a * S + b) * 4;
          q[0] = i0; q[1] = i1; q[2] = j0; q[3] = j1;
        }
        for (int c = 0; c < C; ++c) {
          const float* Fc = F + (size_t)c * Hc * Wc;
          float m = Fc[(size_t)i0 * Wc + j0];
          for (int i = i0; i <= i1; ++i)
            for (int j = j0; j <= j1; ++j) m = std::max(m, Fc[(size_t)i * Wc + j]);
          d[(size_t)c * S * S + a * S + b] = m;
        }
      }
    }
  }
  return 0;
}

}  // extern "C"
