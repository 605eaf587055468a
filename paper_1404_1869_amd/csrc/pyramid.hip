// Plane builder: bilinear resampling of the uint8 image to every scale (Sec. 3.1 pyramid), mean-pixel
// centring (Sec. 3.2), the 16-px border (ramp to the mean, or the mean itself) and stitching onto
// planes with a zero background (Sec. 3.1), fused into one pass that writes every plane pixel once.
//
// A pre-pass rewrites each image pixel-interleaved, 4 bytes per pixel (R, G, B, 0), so that one
// bilinear tap of all three channels is a single 4-byte load, and one image (3 MB at 768 x 1024) fits
// an XCD's L2.  The builder then produces 4 plane pixels per thread, 64 columns apart, so that each
// of a wave's gathers reads the taps of 64 consecutive pixels and each store writes 64 consecutive
// pixels of a channel; a wave covers 256 columns.  Workgroups are ordered so that each XCD works
// through a contiguous range of images and planes.  The half-pixel source coordinate
// ((2 y + 1) H - h) / (2 h) is formed exactly in 32-bit integers; only the blend is fp32.
#include "common.h"

#include <mutex>
#include <type_traits>

namespace dn {
namespace {

// Tile shape (plane pixels per thread, rows per workgroup tile), compile-time settings chosen by
// timing the 96-plane batch (2 or 8 pixels per thread and 8-row tiles were slower).
#ifndef DN_BUILD_PX
#define DN_BUILD_PX 4
#endif
#ifndef DN_BUILD_ROWS
#define DN_BUILD_ROWS 16
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

// Workgroup tile: 16 plane rows x 64 * PX columns; each lane owns PX consecutive columns and the
// four waves take the tile's rows in turn.  In stitched planes every rectangle edge is a multiple of
// 16 px, and a per-scale plane is its scale's rectangle, so each 16 x 16 cell of a 16-row-aligned tile
// has a single owner scale (or none).  Per tile the workgroup finds the owner of each of its 16 cells
// and tabulates, per (cell, row), the two source rows, the row fraction and the row's border weight;
// each lane computes its columns' source coordinates and border weights once and then only blends
// per row.
constexpr int TROWS = DN_BUILD_ROWS;     // rows per tile
static_assert(16 % TROWS == 0 && TROWS % 4 == 0, "a tile's rows lie in one row of 16-px cells");
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
  uint32_t r0, r1;  // source row offsets sy0 * W, sy1 * W (pixels; plus image * H * W in a packed batch)
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

// BATCH = false: planes of each image (a.s, pl), blocks z = image * pl.n + plane.  BATCH = true: the
// planes of a cross-image packed batch (bg), blocks z = plane, each cell sampling its owner's image.
// Two consecutive pixels of the pixel image: 4-byte aligned (a dword-aligned 8-byte load).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2), aligned(4)));

// PAIR (source width at least 2): the two taps of a source row are one 8-byte load.
template <typename T, bool BATCH, bool PAIR>
__global__ __launch_bounds__(256) void build_planes_kernel(const uint32_t* __restrict__ pix,
                                                           PyrArgs a, PyrPlanes pl, BatchGeom bg,
                                                           T* __restrict__ out, int tiles_x,
                                                           int tiles_y) {
  static_assert(TCELLS <= 256, "one owner search per thread");
  __shared__ int s_own[TCELLS];
  __shared__ PyrScale s_sc[TCELLS];  // owner's rectangle, per cell
  __shared__ int s_img[TCELLS];      // owner's image, per cell
  __shared__ RowEntry s_row[TCELLS * TROWS];
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
  const int tx0 = gx * 64 * PX, ty0 = gy * TROWS;
  if (tx0 >= PW || ty0 >= PH) return;  // uniform per workgroup
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave

  if constexpr (BATCH) {
    // Rectangles never overlap and their edges are multiples of 16, so each cell of this 16-row band
    // has at most one owner among the items on plane j.
    if (tid < TCELLS) s_own[tid] = -1;
    __syncthreads();
    for (int i = bg.first[j] + tid; i < bg.first[j + 1]; i += 256) {
      const int e = bg.list[i];
      const dn_scale_geom& g = bg.geom[e];
      if (g.plane != j || !valid_item(g, bg) || ty0 < g.y || ty0 >= g.y + g.rh) continue;
      const int c_lo = max(0, (g.x - tx0) / 16), c_hi = min(TCELLS, (g.x + g.rw - tx0) / 16);
      for (int c = c_lo; c < c_hi; ++c) s_own[c] = e;
    }
    __syncthreads();
    if (tid < TCELLS) {
      const int e = s_own[tid];
      if (e >= 0 && tx0 + 16 * tid < PW) {
        const dn_scale_geom& g = bg.geom[e];
        s_sc[tid] = PyrScale{g.plane, g.y, g.x, g.rh, g.rw, g.h, g.w};
        s_img[tid] = g.image;
      } else {
        s_own[tid] = -1;
      }
    }
  } else {
    const int f0 = a.plane_first[j], f1 = f0 + a.plane_count[j];
    if (tid < TCELLS) {
      const int cx = tx0 + 16 * tid;
      int owner = -1;
      for (int e = f0; e < f1 && cx < PW; ++e) {
        const PyrScale& s = a.s[e];
        if (ty0 >= s.y && ty0 < s.y + s.rh && cx >= s.x && cx < s.x + s.rw) {
          owner = e;
          break;
        }
      }
      s_own[tid] = owner;
      if (owner >= 0) {
        s_sc[tid] = a.s[owner];
        s_img[tid] = b;
      }
    }
  }
  __syncthreads();
  for (int ent = tid; ent < TCELLS * TROWS; ent += 256) {
    const int cell = ent / TROWS, r = ent % TROWS, y = ty0 + r;
    RowEntry re{0u, 0u, 0.f, 0.f};
    if (s_own[cell] >= 0 && y < PH) {
      const PyrScale& s = s_sc[cell];
      const int vy = y - s.y - a.pad;
      const int dy = max(0, max(-vy, vy - (s.h - 1)));
      re.wy = border_weight(dy, a.pad, a.ramp);
      int sy0, sy1;
      src_coord(min(max(vy, 0), s.h - 1), a.H, s.h, 1.0 / (2.0 * s.h), sy0, sy1, re.ly);
      // a packed batch reads the owner's image: its offset is folded into the row offsets, so the
      // pixel loads keep one base address for the whole workgroup
      const uint32_t img_off = BATCH ? (uint32_t)s_img[cell] * (uint32_t)a.H * (uint32_t)a.W : 0u;
      re.r0 = img_off + (uint32_t)sy0 * (uint32_t)a.W;
      re.r1 = img_off + (uint32_t)sy1 * (uint32_t)a.W;
    }
    s_row[ent] = re;
  }
  __syncthreads();

  // This lane's columns x_i = tx0 + lane + 64 i: each gather instruction of a wave then reads the
  // taps of 64 consecutive plane pixels (few cache lines), and each store writes 64 consecutive
  // pixels of one channel.  Per column: its cell, border weight, source columns and fraction.
  int cl[PX];
  bool inside[PX];
  float wx[PX], lx[PX];
  uint32_t sx0[PX], sx1[PX];
#pragma unroll
  for (int i = 0; i < PX; ++i) {
    const int xl = lane + 64 * i, x = tx0 + xl;
    cl[i] = xl >> 4;
    inside[i] = x < PW;
    wx[i] = 0.f;
    lx[i] = 0.f;
    sx0[i] = sx1[i] = 0u;
    if (inside[i] && s_own[cl[i]] >= 0) {
      const PyrScale& s = s_sc[cl[i]];
      const int ux = x - s.x - a.pad;
      const int dx = max(0, max(-ux, ux - (s.w - 1)));
      wx[i] = border_weight(dx, a.pad, a.ramp);
      int c0, c1;  // c1 = min(c0 + 1, W - 1)
      src_coord(min(max(ux, 0), s.w - 1), a.W, s.w, 1.0 / (2.0 * s.w), c0, c1, lx[i]);
      // On the last source column (c1 = c0) the pair starts one column earlier with fraction 1:
      // a + 1 (b - a) is exactly b for these small integers, the value the clamped tap gives.
      if (PAIR && c1 == c0) {
        c0 -= 1;
        lx[i] = 1.f;
      }
      sx0[i] = (uint32_t)c0;
      sx1[i] = (uint32_t)c1;
    }
  }
  const uint32_t* P = pix + (BATCH ? 0 : (int64_t)b * a.H * a.W);
  T* o = out + (BATCH ? (int64_t)j * 3 * PH * PW : (int64_t)b * pl.image_elems + pl.p[j].offset);
  const int64_t plane = (int64_t)PH * PW;

  // Rows wave, wave + 4, ... of the tile, unrolled so that the taps of several rows are in flight.
  // Every pixel reads its four taps (background pixels and pixels outside a scale's border read valid
  // pixels, with weight 0), so the loads carry no per-pixel branch.
#pragma unroll
  for (int rr = 0; rr < TROWS / 4; ++rr) {
    const int r = wave + 4 * rr;
    const int y = ty0 + r;
    if (y >= PH) break;  // uniform per wave
    float v[PX][3];
#pragma unroll
    for (int i = 0; i < PX; ++i) {
      const RowEntry re = s_row[cl[i] * TROWS + r];
      const float wgt = re.wy * wx[i];
      uint32_t q00, q01, q10, q11;
      if constexpr (PAIR) {
        const u32x2 t = *(const u32x2*)(P + re.r0 + sx0[i]), u = *(const u32x2*)(P + re.r1 + sx0[i]);
        q00 = t.x, q01 = t.y, q10 = u.x, q11 = u.y;
      } else {
        q00 = P[re.r0 + sx0[i]], q01 = P[re.r0 + sx1[i]];
        q10 = P[re.r1 + sx0[i]], q11 = P[re.r1 + sx1[i]];
      }
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        const int sh = 8 * c;
        const float i00 = (float)((q00 >> sh) & 255u), i01 = (float)((q01 >> sh) & 255u);
        const float i10 = (float)((q10 >> sh) & 255u), i11 = (float)((q11 >> sh) & 255u);
        const float top = i00 + lx[i] * (i01 - i00), bot = i10 + lx[i] * (i11 - i10);
        v[i][c] = (top + re.ly * (bot - top) - a.mean[c]) * wgt;
      }
    }
    T* orow = o + (int64_t)y * PW + tx0 + lane;
#pragma unroll
    for (int c = 0; c < 3; ++c)
#pragma unroll
      for (int i = 0; i < PX; ++i)
        if (inside[i]) orow[c * plane + 64 * i] = from_f32<T>(v[i][c]);
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
                        const BatchGeom* batch, int32_t max_h, int32_t max_w, dn_dtype dt, void* d_out,
                        uint8_t* d_scratch, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  uint32_t* pix = (uint32_t*)d_scratch;
  if (a.W % 4 == 0)
    pixel_image4_kernel<<<dim3((a.W / 4 + 255) / 256, a.H, n_img), 256, 0, s>>>(d_img, a.H, a.W, pix);
  else
    pixel_image_kernel<<<dim3((a.W + 255) / 256, a.H, n_img), 256, 0, s>>>(d_img, a.H, a.W, pix);
  const int tiles_x = (max_w + 64 * PX - 1) / (64 * PX), tiles_y = (max_h + TROWS - 1) / TROWS;
  const int64_t nblk = (int64_t)tiles_x * tiles_y * (batch ? batch->n_planes : n_img * pl.n);
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
  auto go2 = [&](auto tag, auto pair) {
    using T = decltype(tag);
    constexpr bool PAIR = decltype(pair)::value;
    if (batch)
      build_planes_kernel<T, true, PAIR><<<grid, 256, 0, s>>>(pix, a, pl, bg, (T*)d_out, tiles_x, tiles_y);
    else
      build_planes_kernel<T, false, PAIR><<<grid, 256, 0, s>>>(pix, a, pl, bg, (T*)d_out, tiles_x, tiles_y);
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
