// Plane builder: bilinear resampling of the uint8 image to every scale (Sec. 3.1 pyramid), mean-pixel
// centring (Sec. 3.2), the 16-px border (ramp to the mean, or the mean itself) and stitching onto
// planes with a zero background (Sec. 3.1), fused into one pass that writes every plane pixel once.
//
// A pre-pass rewrites each image pixel-interleaved, 4 bytes per pixel (R, G, B, 0), so that one
// bilinear tap of all three channels is a single 4-byte load, and one image (3 MB at 768 x 1024) fits
// an XCD's L2.  The builder then produces 4 plane pixels per thread, 64 columns apart, so that each
// of a wave's gathers reads the taps of 64 consecutive pixels and each store writes 64 consecutive
// pixels of a channel; a wave covers 256 columns.  Plane rows are padded to a multiple of 64 elements
// (written as 0), so every store instruction fills whole cache lines.  Workgroups are ordered so that
// each XCD works through a contiguous range of images and planes.  The half-pixel source coordinate
// ((2 y + 1) H - h) / (2 h) is formed exactly in 32-bit integers, the horizontal blend of a source
// row is exact in integers (v_dot2_u32_u16 of the two taps with the weights 2 w - r and r), and only
// the vertical blend, the centring and the border weight are fp32.
#include "common.h"

#include <mutex>
#include <type_traits>

namespace dn {
namespace {

// Plane pixels per thread, a compile-time setting chosen by timing the 96-plane batch (2 or 8 pixels
// per thread were slower).
#ifndef DN_BUILD_PX
#define DN_BUILD_PX 4
#endif
constexpr int PX = DN_BUILD_PX;  // plane pixels per thread

// floor(n / d) and the remainder for n, d < 2^32 with d > 0: a double-precision reciprocal estimate,
// corrected to the exact quotient with integer arithmetic.
__device__ inline uint32_t udiv_exact(uint32_t n, uint32_t d, double inv_d, uint32_t& rem) {
  uint32_t q = (uint32_t)((double)n * inv_d);
  if ((uint64_t)q * d > n) --q;
  else if ((uint64_t)(q + 1) * d <= n) ++q;
  rem = n - q * d;
  return q;
}

// Source row (or column) of output index o of a scale of size h out of H: the half-pixel coordinate
// ((2 o + 1) H - h) / (2 h), clamped at 0, split into the integer part and the fraction.
__device__ inline void src_coord(int o, int H, int h, double inv2h, int& i0, int& i1, float& frac) {
  const int64_t num = (int64_t)(2 * o + 1) * H - h;
  const uint32_t n = num > 0 ? (uint32_t)num : 0u, d = 2u * (uint32_t)h;
  uint32_t rem;
  i0 = (int)udiv_exact(n, d, inv2h, rem);
  i1 = min(i0 + 1, H - 1);
  frac = (float)((double)rem * inv2h);
}

__device__ inline float border_weight(int d, int pad, bool ramp) {
  if (d == 0) return 1.f;
  if (!ramp || d > pad) return 0.f;
  return (float)(pad + 1 - d) / (float)(pad + 1);
}

// Workgroup tile: NBANDS bands of 16 plane rows x 64 * PX columns (4 bands on large launches, 1 where
// a launch has too few tiles to fill the chip).  In stitched planes every rectangle edge
// is a multiple of 16 px, and a per-scale plane is its scale's rectangle, so each 16 x 16 cell of a
// band has a single owner scale (or none).  Per tile the workgroup finds the owners of its cells and
// tabulates, per (cell, row), the two source rows, the row fraction and the row's border weight.  The
// four waves take the tile's rows in turn (wave w: rows w, w + 4, ...), so at any time they read the
// same few source rows; a lane computes its columns' taps for the first band and again only where
// a later band's owner differs.
// f(integral_constant<I>) for I = B .. E - 1, in order.
template <int B, int E, typename F>
__device__ inline void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

constexpr int BAND = 16;                 // rows per band (one row of 16-px cells)
constexpr int TCELLS = 64 * PX / 16;     // 16-px cells per tile row

// Pixel image: pix[b][y][x] = R | G << 8 | B << 16, one thread per pixel (any width), or per 4 pixels
// (width a multiple of 4: three 4-byte channel loads, one 16-byte store).
__global__ __launch_bounds__(256) void pixel_image_kernel(const uint8_t* __restrict__ img, int H, int W,
                                                          uint32_t* __restrict__ pix) {
  const int x = blockIdx.x * 256 + threadIdx.x, y = blockIdx.y, b = blockIdx.z;
  if (x >= W) return;
  const int64_t HW = (int64_t)H * W;
  const uint8_t* row = img + (int64_t)b * 3 * HW + (int64_t)y * W;
  const uint32_t r0 = row[x], g0 = row[HW + x], b0 = row[2 * HW + x];
  pix[(int64_t)b * HW + (int64_t)y * W + x] = r0 | (g0 << 8) | (b0 << 16);
}

__global__ __launch_bounds__(256) void pixel_image4_kernel(const uint8_t* __restrict__ img, int H, int W,
                                                           uint32_t* __restrict__ pix) {
  const int x = 4 * (blockIdx.x * 256 + threadIdx.x), y = blockIdx.y, b = blockIdx.z;
  if (x >= W) return;
  const int64_t HW = (int64_t)H * W;
  const uint8_t* row = img + (int64_t)b * 3 * HW + (int64_t)y * W + x;
  const uint32_t r = *(const uint32_t*)row, g = *(const uint32_t*)(row + HW),
                 bl = *(const uint32_t*)(row + 2 * HW);
  uint4 o;
  o.x = (r & 0xffu) | ((g & 0xffu) << 8) | ((bl & 0xffu) << 16);
  o.y = ((r >> 8) & 0xffu) | (g & 0xff00u) | ((bl & 0xff00u) << 8);
  o.z = ((r >> 16) & 0xffu) | ((g >> 8) & 0xff00u) | (bl & 0xff0000u);
  o.w = (r >> 24) | ((g >> 16) & 0xff00u) | ((bl >> 8) & 0xff0000u);
  *(uint4*)(pix + (int64_t)b * HW + (int64_t)y * W + x) = o;
}

struct RowEntry {
  uint32_t r0, r1;  // byte offsets of source rows sy0, sy1 (plus image * 4 H W in a packed batch)
  float ly, wy;     // row fraction, row border weight (0: background)
};

// Per-plane item lists of a packed plan, so that a builder workgroup scans only its plane's items:
// items of plane j are list[first[j]] .. list[first[j + 1] - 1] (their order within a plane is
// unspecified; rectangles do not overlap, so the builder's result does not depend on it).  One
// workgroup: per-plane counts in LDS, an exclusive scan, then a scatter.  Items whose plane is out of
// range are left out.
constexpr int IDX_THREADS = 1024;
__global__ __launch_bounds__(IDX_THREADS) void index_items_kernel(const dn_scale_geom* __restrict__ geom,
                                                                  int n_items, int n_planes,
                                                                  int32_t* __restrict__ first,
                                                                  int32_t* __restrict__ list) {
  extern __shared__ int s_cnt[];          // n_planes counts, then cursors
  __shared__ int s_part[IDX_THREADS];     // per-thread chunk sums, scanned
  const int tid = threadIdx.x;
  for (int j = tid; j < n_planes; j += IDX_THREADS) s_cnt[j] = 0;
  __syncthreads();
  for (int e = tid; e < n_items; e += IDX_THREADS) {
    const int pl = geom[e].plane;
    if (pl >= 0 && pl < n_planes) atomicAdd(&s_cnt[pl], 1);
  }
  __syncthreads();
  // exclusive scan: thread t owns planes [t C, (t + 1) C)
  const int C = (n_planes + IDX_THREADS - 1) / IDX_THREADS, j0 = min(tid * C, n_planes),
            j1 = min(j0 + C, n_planes);
  int sum = 0;
  for (int j = j0; j < j1; ++j) sum += s_cnt[j];
  s_part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < IDX_THREADS; off <<= 1) {  // inclusive Hillis-Steele scan of the chunk sums
    const int v = tid >= off ? s_part[tid - off] : 0;
    __syncthreads();
    s_part[tid] += v;
    __syncthreads();
  }
  int run = s_part[tid] - sum;
  for (int j = j0; j < j1; ++j) {
    const int c = s_cnt[j];
    first[j] = run;
    s_cnt[j] = run;  // cursor
    run += c;
  }
  if (tid == IDX_THREADS - 1) first[n_planes] = s_part[tid];
  __syncthreads();
  for (int e = tid; e < n_items; e += IDX_THREADS) {
    const int pl = geom[e].plane;
    if (pl >= 0 && pl < n_planes) list[atomicAdd(&s_cnt[pl], 1)] = e;
  }
}

// Whether a placement read from a device copy of a packed plan is a rectangle of 16-px cells inside a
// PH x PW plane of image < n_img with a real size; other entries are ignored (background).
__device__ inline bool valid_item(const dn_scale_geom& g, const BatchGeom& bg) {
  return g.image >= 0 && g.image < bg.n_img && g.h >= 1 && g.w >= 1 && g.h <= 65535 &&
         g.w <= 65535 && g.rh >= 16 && g.rw >= 16 && ((g.y | g.x | g.rh | g.rw) & 15) == 0 &&
         g.y >= 0 && g.x >= 0 && g.y <= bg.PH - g.rh && g.x <= bg.PW - g.rw;
}


// PAIR (source width at least 2): the two taps of a source row are one 8-byte load.

// BATCH = false: planes of each image (a.s, pl), blocks z = image * pl.n + plane.  BATCH = true: the
// planes of a cross-image packed batch (bg), blocks z = plane, each cell sampling its owner's image.
// Two consecutive pixels of the pixel image: 4-byte aligned (a dword-aligned 8-byte load).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2), aligned(4)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Horizontal taps of one source row, exact in integers: for the 4-byte pixels q0 (left) and q1
// (right), channel c gives I0 (Dx - rx) + I1 rx = Dx ((1 - lx) I0 + lx I1), with the column fraction
// lx = rx / Dx, Dx = 2 w (at most 65535) and the weights packed as u16 pairs (Dx - rx) | rx << 16.
// v_perm_b32 places byte c of q0 and of q1 in the two 16-bit halves of one dword.
template <int C>
__device__ inline uint32_t taps_x(uint32_t q0, uint32_t q1, uint32_t wts) {
  constexpr uint32_t sel = 0x0c000c00u | ((4u + C) << 16) | (uint32_t)C;
  const uint32_t pair = __builtin_amdgcn_perm(q1, q0, sel);
  return __builtin_amdgcn_udot2(__builtin_bit_cast(u16x2, pair), __builtin_bit_cast(u16x2, wts), 0u,
                                false);
}

// PAIR (source width at least 2): the two taps of a source row are one 8-byte load.  XDOT (every
// scale at most 32767 px wide): horizontal taps in exact integers (taps_x); otherwise an fp32 lerp.
template <typename T, bool BATCH, bool PAIR, bool XDOT, int NBANDS>
__global__ __launch_bounds__(256) void build_planes_kernel(const uint32_t* __restrict__ pix,
                                                           PyrArgs a, PyrPlanes pl, BatchGeom bg,
                                                           T* __restrict__ out, int tiles_x,
                                                           int tiles_y) {
  constexpr int TROWS = NBANDS * BAND;    // rows of the tile
  constexpr int NCELL = NBANDS * TCELLS;  // cells of the tile, band-major
  static_assert(NCELL <= 256 && (NCELL * BAND) % 256 == 0, "one cell per thread");
  __shared__ int s_own[NCELL];
  __shared__ PyrScale s_sc[NCELL];   // owner's rectangle, per cell
  __shared__ double s_inv[NCELL];    // 1 / (2 h) of the owner, per cell
  __shared__ uint32_t s_img[NCELL];  // owner's image offset (pixels), per cell
  __shared__ RowEntry s_row[NCELL * BAND];
  // XCD-aware order over a flat grid: XCD x takes a contiguous range of (image, plane, row tile,
  // column tile) indices, so the tiles in flight on one XCD read the same image from its L2.
  const int nbk = gridDim.x, xcd = blockIdx.x % 8, per = nbk / 8, rem = nbk % 8;
  int bid = xcd * per + min(xcd, rem) + blockIdx.x / 8;
  const int gx = bid % tiles_x;
  bid /= tiles_x;
  const int gy = bid % tiles_y;
  const int z = bid / tiles_y;
  const int b = BATCH ? 0 : z / pl.n, j = BATCH ? z : z - b * pl.n;
  const int PH = BATCH ? bg.PH : pl.p[j].h, PW = BATCH ? bg.PW : pl.p[j].w;
  const int PP = plane_pitch(PW);  // row pitch; columns PW .. PP - 1 are written as 0
  const int ty0 = gy * TROWS;
  const int tx0 = gx * 64 * PX;
  if (tx0 >= PP || ty0 >= PH) return;  // uniform per workgroup
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave

  // Owners of the tile's cells (cell c = band * TCELLS + column).
  if constexpr (BATCH) {
    // Rectangles never overlap and their edges are multiples of 16, so each cell has at most one
    // owner among the items on plane j.
    if (tid < NCELL) s_own[tid] = -1;
    __syncthreads();
    for (int i = bg.first[j] + tid; i < bg.first[j + 1]; i += 256) {
      const int e = bg.list[i];
      const dn_scale_geom& g = bg.geom[e];
      if (g.plane != j || !valid_item(g, bg)) continue;
      const int r_lo = max(0, (g.y - ty0) / 16), r_hi = min(NBANDS, (g.y + g.rh - ty0) / 16);
      const int c_lo = max(0, (g.x - tx0) / 16), c_hi = min(TCELLS, (g.x + g.rw - tx0) / 16);
      for (int r = r_lo; r < r_hi; ++r)
        for (int c = c_lo; c < c_hi; ++c) s_own[r * TCELLS + c] = e;
    }
    __syncthreads();
    if (tid < NCELL) {
      const int e = s_own[tid];
      const int cy = ty0 + 16 * (tid / TCELLS), cx = tx0 + 16 * (tid % TCELLS);
      if (e >= 0 && cx < PW && cy < PH) {
        const dn_scale_geom& g = bg.geom[e];
        s_sc[tid] = PyrScale{g.plane, g.y, g.x, g.rh, g.rw, g.h, g.w};
        s_img[tid] = (uint32_t)g.image * (uint32_t)a.H * (uint32_t)a.W;
        s_inv[tid] = 1.0 / (2.0 * g.h);
      } else {
        s_own[tid] = -1;
      }
    }
  } else {
    const int f0 = a.plane_first[j], f1 = f0 + a.plane_count[j];
    if (tid < NCELL) {
      const int cy = ty0 + 16 * (tid / TCELLS), cx = tx0 + 16 * (tid % TCELLS);
      int owner = -1;
      for (int e = f0; e < f1 && cx < PW && cy < PH; ++e) {
        const PyrScale& s = a.s[e];
        if (cy >= s.y && cy < s.y + s.rh && cx >= s.x && cx < s.x + s.rw) {
          owner = e;
          break;
        }
      }
      s_own[tid] = owner;
      if (owner >= 0) {
        s_sc[tid] = a.s[owner];
        s_img[tid] = 0u;
        s_inv[tid] = 1.0 / (2.0 * a.s[owner].h);
      }
    }
  }
  __syncthreads();
  // Row table: entry (cell, r) for row 16 band + r of the tile.
#pragma unroll
  for (int k = 0; k < NCELL * BAND / 256; ++k) {
    const int ent = k * 256 + tid, cell = ent / BAND, r = ent % BAND;
    const int y = ty0 + 16 * (cell / TCELLS) + r;
    RowEntry re{0u, 0u, 0.f, 0.f};
    if (s_own[cell] >= 0 && y < PH) {
      const PyrScale& s = s_sc[cell];
      const int vy = y - s.y - a.pad;
      const int dy = max(0, max(-vy, vy - (s.h - 1)));
      re.wy = border_weight(dy, a.pad, a.ramp);
      int sy0, sy1;
      src_coord(min(max(vy, 0), s.h - 1), a.H, s.h, s_inv[cell], sy0, sy1, re.ly);
      // a packed batch reads the owner's image: its offset is folded into the row offsets, so the
      // pixel loads keep one buffer descriptor for the whole workgroup
      re.r0 = 4u * (s_img[cell] + (uint32_t)sy0 * (uint32_t)a.W);
      re.r1 = 4u * (s_img[cell] + (uint32_t)sy1 * (uint32_t)a.W);
    }
    s_row[ent] = re;
  }
  __syncthreads();

  // This lane's columns: pairs of neighbours, x_i = tx0 + 128 (i / 2) + 2 lane + i % 2, so each
  // store instruction of a wave writes a pair of one channel per lane (128 consecutive pixels), the
  // two pixels of a pair share their cell's row entry, and each gather instruction reads the taps of
  // 64 pixels two columns apart.  Per column: its owner, border weight, first source column and the
  // horizontal weights (XDOT: u16 pair and 1 / Dx; else the fp32 fraction lx).
  static_assert(PX % 2 == 0, "pairs of neighbouring columns");
  auto col_of = [&](int i) { return tx0 + 128 * (i / 2) + 2 * lane + (i % 2); };
  auto cell_of = [&](int band, int i) { return band * TCELLS + ((128 * (i / 2) + 2 * lane) >> 4); };
  bool inside[PX];
  int own[PX];
  float wx[PX], hx[PX];  // border weight; 1 / Dx (XDOT) or the column fraction lx
  uint32_t sx0[PX], sx1[PX], wts[PX];
  auto column_taps = [&](int i, int cell) {
    const int x = col_of(i);
    wx[i] = 0.f;
    hx[i] = XDOT ? 1.f : 0.f;
    sx0[i] = sx1[i] = 0u;
    wts[i] = 0u;
    if (own[i] >= 0) {
      const PyrScale& s = s_sc[cell];
      const int ux = x - s.x - a.pad;
      const int dx = max(0, max(-ux, ux - (s.w - 1)));
      wx[i] = border_weight(dx, a.pad, a.ramp);
      // half-pixel source column ((2 u + 1) W - w) / (2 w), clamped at 0: c0 and remainder rx
      const int u = min(max(ux, 0), s.w - 1);
      const int64_t num = (int64_t)(2 * u + 1) * a.W - s.w;
      const uint32_t n = num > 0 ? (uint32_t)num : 0u, d = 2u * (uint32_t)s.w;
      uint32_t rx;
      int c0 = (int)udiv_exact(n, d, 1.0 / (double)d, rx);
      const int c1 = min(c0 + 1, a.W - 1);
      // On the last source column (c1 = c0) the pair starts one column earlier with all the weight
      // on its right tap, the value the clamped tap gives.
      if (PAIR && c1 == c0) {
        c0 -= 1;
        rx = d;
      }
      sx0[i] = 4u * (uint32_t)c0;  // byte offsets
      sx1[i] = 4u * (uint32_t)c1;
      if constexpr (XDOT) {
        wts[i] = (d - rx) | (rx << 16);
        hx[i] = 1.f / (float)d;
      } else {
        hx[i] = (float)((double)rx / (double)d);
      }
    }
  };
#pragma unroll
  for (int i = 0; i < PX; ++i) {
    inside[i] = col_of(i) < PP;
    own[i] = -2;  // nothing computed yet
  }
  constexpr uint32_t OOB = 0x80000000u;  // a store offset past any plane: dropped by the hardware
  uint32_t soff_lane[PX / 2];  // byte offset of pair p in a plane row (OOB past the pitch)
#pragma unroll
  for (int i = 0; i < PX; i += 2)
    soff_lane[i / 2] = inside[i] ? (uint32_t)((tx0 + 128 * (i / 2) + 2 * lane) * (int)sizeof(T)) : OOB;
  // Buffer descriptors: the pixel image(s) (below 2^32 bytes, so 32-bit byte offsets reach every
  // pixel) and this plane (below 2^31 bytes).  A store lane past the row pitch takes an offset past
  // the plane's size, which the hardware drops.
  const uint32_t* P = pix + (BATCH ? 0 : (int64_t)b * a.H * a.W);
  T* o = out + (BATCH ? (int64_t)j * 3 * PH * PP : (int64_t)b * pl.image_elems + pl.p[j].offset);
  const int64_t plane = (int64_t)PH * PP;
  const __amdgpu_buffer_rsrc_t rp =
      uniform_rsrc(P, 4u * (uint32_t)(BATCH ? bg.n_img : 1) * (uint32_t)a.H * (uint32_t)a.W);
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(o, (uint32_t)(3 * plane * (int64_t)sizeof(T)));
  const float mean[3] = {a.mean[0], a.mean[1], a.mean[2]};

  // A row's taps (4 pixels per lane) and its per-pixel row fraction and weight.
  struct RowTaps {
    uint32_t q[PX][4];  // (row 0, col 0), (row 0, col 1), (row 1, col 0), (row 1, col 1)
    float ly[PX], wgt[PX];
  };
  // live[p]: some lane of the wave has a pixel of pair p in a scale's rectangle (wave-uniform); a
  // pair that is background in every lane of the wave loads nothing and stores zeros.  A row is
  // emitted by a variant compiled for its wave's live pattern (LIVE bit p: pair p), so no value is
  // merged across live and background paths.
  bool live[PX / 2];
  auto fetch = [&](auto live_c, int band, int r, RowTaps& t) {
    constexpr int LIVE = decltype(live_c)::value;
    RowEntry re;
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      if (!((LIVE >> (i / 2)) & 1)) continue;
      if (i % 2 == 0) re = s_row[cell_of(band, i) * BAND + r];  // one entry per pair
      t.ly[i] = re.ly;
      t.wgt[i] = re.wy * wx[i];
      if constexpr (PAIR) {
        const u32x2 a0 = __builtin_amdgcn_raw_buffer_load_b64(rp, re.r0 + sx0[i], 0, 0);
        const u32x2 a1 = __builtin_amdgcn_raw_buffer_load_b64(rp, re.r1 + sx0[i], 0, 0);
        t.q[i][0] = a0.x, t.q[i][1] = a0.y, t.q[i][2] = a1.x, t.q[i][3] = a1.y;
      } else {
        t.q[i][0] = __builtin_amdgcn_raw_buffer_load_b32(rp, re.r0 + sx0[i], 0, 0);
        t.q[i][1] = __builtin_amdgcn_raw_buffer_load_b32(rp, re.r0 + sx1[i], 0, 0);
        t.q[i][2] = __builtin_amdgcn_raw_buffer_load_b32(rp, re.r1 + sx0[i], 0, 0);
        t.q[i][3] = __builtin_amdgcn_raw_buffer_load_b32(rp, re.r1 + sx1[i], 0, 0);
      }
    }
  };
  //   XDOT: the two rows' taps T0, T1 are exact integers below 2^24 (so exact in fp32); the value is
  //   ((T0 + ly (T1 - T0)) / Dx - mean) * weight, as fma(ly, T1 - T0, T0), fma(., 1 / Dx, -mean)
  //   and a product.  Otherwise the fp32 lerps run on the fraction lx.
  auto emit = [&](auto live_c, int y, const RowTaps& t) {
    constexpr int LIVE = decltype(live_c)::value;
    float v[PX][3];
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      if (!((LIVE >> (i / 2)) & 1)) {
        v[i][0] = v[i][1] = v[i][2] = 0.f;
        continue;
      }
      const uint32_t q00 = t.q[i][0], q01 = t.q[i][1], q10 = t.q[i][2], q11 = t.q[i][3];
      if constexpr (XDOT) {
        const uint32_t t0[3] = {taps_x<0>(q00, q01, wts[i]), taps_x<1>(q00, q01, wts[i]),
                                taps_x<2>(q00, q01, wts[i])};
        const uint32_t t1[3] = {taps_x<0>(q10, q11, wts[i]), taps_x<1>(q10, q11, wts[i]),
                                taps_x<2>(q10, q11, wts[i])};
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          const float f0 = (float)t0[c], f1 = (float)t1[c];
          const float vr = __builtin_fmaf(t.ly[i], f1 - f0, f0);
          v[i][c] = __builtin_fmaf(vr, hx[i], -mean[c]) * t.wgt[i];
        }
      } else {
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          const int sh = 8 * c;
          const float i00 = (float)((q00 >> sh) & 255u), i01 = (float)((q01 >> sh) & 255u);
          const float i10 = (float)((q10 >> sh) & 255u), i11 = (float)((q11 >> sh) & 255u);
          const float top = i00 + hx[i] * (i01 - i00), bot = i10 + hx[i] * (i11 - i10);
          v[i][c] = (top + t.ly[i] * (bot - top) - mean[c]) * t.wgt[i];
        }
      }
    }
    typedef T pair_t __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      // uniform per wave (plane, row and channel are): a scalar offset, not a per-lane one
      const uint32_t soff =
          __builtin_amdgcn_readfirstlane((uint32_t)((c * plane + (int64_t)y * PP) * (int64_t)sizeof(T)));
#pragma unroll
      for (int i = 0; i < PX; i += 2) {
        const pair_t pv = from_f32x2<T>(v[i][c], v[i + 1][c]);
        // non-temporal (aux 2): conv1 reads the planes only after the whole batch is built
        if constexpr (sizeof(T) == 2)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, pv), ro, soff_lane[i / 2], soff, 2);
        else
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, pv), ro, soff_lane[i / 2], soff, 2);
      }
    }
  };

  // Per band: refresh the columns whose owner changed, then the wave's 4 rows of the band.
  for (int band = 0; band < NBANDS; ++band) {
    const int yb = ty0 + BAND * band;
    if (yb >= PH) break;  // uniform
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      const int cell = cell_of(band, i);
      const int o_new = inside[i] ? s_own[cell] : -1;
      if (o_new != own[i]) {
        own[i] = o_new;
        column_taps(i, cell);
      }
    }
    int lm = 0;  // live pattern of the band (wave-uniform)
#pragma unroll
    for (int i = 0; i < PX; i += 2) {
      live[i / 2] = __builtin_amdgcn_ballot_w64(own[i] >= 0 || own[i + 1] >= 0) != 0;
      lm |= live[i / 2] ? 1 << (i / 2) : 0;
    }
    auto rows = [&](auto live_c) {
#pragma unroll
      for (int k = 0; k < BAND / 4; ++k) {
        const int r = wave + 4 * k;
        if (yb + r < PH) {
          RowTaps t;
          fetch(live_c, band, r, t);
          emit(live_c, yb + r, t);
        }
      }
    };
    static_for<0, 1 << (PX / 2)>([&](auto c) {
      if (lm == decltype(c)::value) rows(c);
    });
  }
}

}  // namespace

// Staging array of the scratch-free builder entry point (the pixel-interleaved images).  Each device
// holds its own copy at its own address; host code never passes this name to a kernel or a copy (in
// host code it is only a stand-in), it uses the address hipGetSymbolAddress returns for the device.
static __device__ __align__(256) uint8_t scratch[DN_STATIC_SCRATCH_BYTES];

int static_scratch(uint8_t** out) {
  constexpr int MAX_DEVICES = 64;
  static std::mutex mu;
  static uint8_t* addr[MAX_DEVICES] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= MAX_DEVICES) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {  // once per device, with that device current
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    if (!ptr) return (int)hipErrorInvalidSymbol;
    addr[dev] = (uint8_t*)ptr;
  }
  *out = addr[dev];
  return (int)hipSuccess;
}

int launch_build_planes(const uint8_t* d_img, int32_t n_img, const PyrArgs& a, const PyrPlanes& pl,
                        const BatchGeom* batch, int32_t max_h, int32_t max_w, int32_t max_scale_w,
                        dn_dtype dt, void* d_out, uint8_t* d_scratch, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  uint32_t* pix = (uint32_t*)d_scratch;
  if (a.W % 4 == 0)
    pixel_image4_kernel<<<dim3((a.W / 4 + 255) / 256, a.H, n_img), 256, 0, s>>>(d_img, a.H, a.W, pix);
  else
    pixel_image_kernel<<<dim3((a.W + 255) / 256, a.H, n_img), 256, 0, s>>>(d_img, a.H, a.W, pix);
  // 64-row tiles (4 bands) where that still gives at least 4096 workgroups, else 16-row tiles
  const int tiles_x = (plane_pitch(max_w) + 64 * PX - 1) / (64 * PX);
  const int64_t n_pl = batch ? batch->n_planes : (int64_t)n_img * pl.n;
  const bool tall = (int64_t)tiles_x * ((max_h + 4 * BAND - 1) / (4 * BAND)) * n_pl >= 4096;
  const int tiles_y = tall ? (max_h + 4 * BAND - 1) / (4 * BAND) : (max_h + BAND - 1) / BAND;
  const int64_t nblk = (int64_t)tiles_x * tiles_y * n_pl;
  if (nblk > 0x7fffffff) return (int)hipErrorInvalidValue;
  const unsigned grid = (unsigned)nblk;
  BatchGeom bg = batch ? *batch : BatchGeom{};
  if (batch) {
    // per-plane item lists in the scratch after the pixel image
    if (bg.n_planes > MAX_INDEX_PLANES) return (int)hipErrorInvalidValue;
    int32_t* first = (int32_t*)(d_scratch + index_offset(n_img, a.H, a.W));
    int32_t* list = first + bg.n_planes + 1;
    index_items_kernel<<<1, IDX_THREADS, sizeof(int) * bg.n_planes, s>>>(bg.geom, bg.n_items, bg.n_planes,
                                                                        first, list);
    bg.first = first;
    bg.list = list;
  }
  // exact integer horizontal taps need 2 w <= 65535 (u16 weights) for every scale
  const bool xdot = max_scale_w <= 32767;
  auto go4 = [&](auto tag, auto pair, auto xd, auto nbands) {
    using T = decltype(tag);
    constexpr bool PAIR = decltype(pair)::value, XDOT = decltype(xd)::value;
    constexpr int NB = decltype(nbands)::value;
    if (batch)
      build_planes_kernel<T, true, PAIR, XDOT, NB>
          <<<grid, 256, 0, s>>>(pix, a, pl, bg, (T*)d_out, tiles_x, tiles_y);
    else
      build_planes_kernel<T, false, PAIR, XDOT, NB>
          <<<grid, 256, 0, s>>>(pix, a, pl, bg, (T*)d_out, tiles_x, tiles_y);
  };
  auto go3 = [&](auto tag, auto pair, auto xd) {
    if (tall)
      go4(tag, pair, xd, std::integral_constant<int, 4>{});
    else
      go4(tag, pair, xd, std::integral_constant<int, 1>{});
  };
  auto go2 = [&](auto tag, auto pair) {
    if (xdot)
      go3(tag, pair, std::true_type{});
    else
      go3(tag, pair, std::false_type{});
  };
  auto go = [&](auto tag) {
    if (a.W >= 2)
      go2(tag, std::true_type{});
    else
      go2(tag, std::false_type{});
  };
  switch (dt) {
    case DN_F32: go(float{}); break;
    case DN_F16: go(_Float16{}); break;
    case DN_BF16: go(__bf16{}); break;
  }
  return (int)hipGetLastError();
}

}  // namespace dn
