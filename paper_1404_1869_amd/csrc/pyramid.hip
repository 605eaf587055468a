// Plane builder: bilinear resampling of the uint8 image to every scale (Sec. 3.1 pyramid), mean-pixel
// centring (Sec. 3.2), the 16-px border (ramp to the mean, or the mean itself) and stitching onto
// planes with a zero background (Sec. 3.1), fused into one pass that writes every plane pixel once.
//
// Each thread produces 4 consecutive pixels of a plane row and stores them as one vector per channel;
// a wave covers 256 columns.  The owner scale is found among the scales of the workgroup's plane
// (a uniform skip of the others).  The source image (a few MB) stays in L2 / MALL for the gathers.
// The half-pixel source coordinate ((2 y + 1) H - h) / (2 h) is formed exactly in 32-bit integers;
// only the blend is fp32.
#include "common.h"

namespace dn {
namespace {

constexpr int PX = 4;  // consecutive plane pixels per thread

// Value of plane pixel (y, x) of plane j: owner scale lookup, border weight, bilinear sample.
// Writes the three centred channel values; 0 for background and alignment slack.
__device__ inline void plane_pixel(const uint8_t* __restrict__ I, const PyrArgs& a, int j, int y,
                                   int x, float v[3]) {
  v[0] = v[1] = v[2] = 0.f;
  int owner = -1;
  for (int k = 0; k < a.n_scales; ++k) {
    if (a.s[k].plane != j) continue;  // uniform across the workgroup
    const PyrScale& s = a.s[k];
    if (y >= s.y && y < s.y + s.rh && x >= s.x && x < s.x + s.rw) {
      owner = k;
      break;
    }
  }
  if (owner < 0) return;
  const PyrScale s = a.s[owner];
  const int vy = y - s.y - a.pad, ux = x - s.x - a.pad;
  const int dy = max(0, max(-vy, vy - (s.h - 1)));
  const int dx = max(0, max(-ux, ux - (s.w - 1)));
  if (dy > a.pad || dx > a.pad) return;
  float wgt = 1.f;
  if (dy | dx) {
    if (!a.ramp) return;
    const float den = (float)(a.pad + 1);
    const float wy = dy ? (float)(a.pad + 1 - dy) / den : 1.f;
    const float wx = dx ? (float)(a.pad + 1 - dx) / den : 1.f;
    wgt = wy * wx;
  }
  const int yc = min(max(vy, 0), s.h - 1), xc = min(max(ux, 0), s.w - 1);
  // half-pixel source coordinate ((2 yc + 1) H - h) / (2 h), clamped at 0; exact in 32 bits
  // (sides are limited so that (2 h + 1) H < 2^32)
  const uint32_t dh = 2u * (uint32_t)s.h, dw = 2u * (uint32_t)s.w;
  const int64_t nys = (int64_t)(2 * yc + 1) * a.H - s.h, nxs = (int64_t)(2 * xc + 1) * a.W - s.w;
  const uint32_t ny = nys > 0 ? (uint32_t)nys : 0u, nx = nxs > 0 ? (uint32_t)nxs : 0u;
  const uint32_t y0 = ny / dh, x0 = nx / dw;
  const float ly = (float)(ny - y0 * dh) / (float)dh;
  const float lx = (float)(nx - x0 * dw) / (float)dw;
  const int y1 = min((int)y0 + 1, a.H - 1), x1 = min((int)x0 + 1, a.W - 1);
  const int64_t HW = (int64_t)a.H * a.W;
  const int r0 = (int)y0 * a.W, r1 = y1 * a.W;
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const uint8_t* P = I + c * HW;
    const float i00 = P[r0 + (int)x0], i01 = P[r0 + x1];
    const float i10 = P[r1 + (int)x0], i11 = P[r1 + x1];
    const float top = i00 + lx * (i01 - i00), bot = i10 + lx * (i11 - i10);
    v[c] = (top + ly * (bot - top) - a.mean[c]) * wgt;
  }
}

// One thread per PX consecutive pixels of a plane row; a wave covers 64 * PX columns.
template <typename T>
__global__ __launch_bounds__(256) void build_planes_kernel(const uint8_t* __restrict__ img,
                                                           PyrArgs a, PyrPlanes pl,
                                                           T* __restrict__ out) {
  typedef T vec_t __attribute__((ext_vector_type(PX)));
  const int z = blockIdx.z;
  const int b = z / pl.n, j = z - b * pl.n;
  const int PH = pl.p[j].h, PW = pl.p[j].w;
  const int x0 = (blockIdx.x * 64 + (threadIdx.x & 63)) * PX;
  const int y = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (x0 >= PW || y >= PH) return;
  const uint8_t* I = img + (int64_t)b * 3 * a.H * a.W;
  float v[PX][3];
#pragma unroll
  for (int i = 0; i < PX; ++i) {
    if (x0 + i < PW) {
      plane_pixel(I, a, j, y, x0 + i, v[i]);
    } else {
      v[i][0] = v[i][1] = v[i][2] = 0.f;
    }
  }
  T* o = out + (int64_t)b * pl.image_elems + pl.p[j].offset;
  const int64_t plane = (int64_t)PH * PW, at = (int64_t)y * PW + x0;
  if ((PW % PX) == 0) {  // whole, aligned vectors (uniform per plane)
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      vec_t r;
#pragma unroll
      for (int i = 0; i < PX; ++i) r[i] = from_f32<T>(v[i][c]);
      *(vec_t*)(o + c * plane + at) = r;
    }
  } else {
#pragma unroll
    for (int c = 0; c < 3; ++c)
#pragma unroll
      for (int i = 0; i < PX; ++i)
        if (x0 + i < PW) o[c * plane + at + i] = from_f32<T>(v[i][c]);
  }
}

}  // namespace

int launch_build_planes(const uint8_t* d_img, int32_t n_img, const PyrArgs& a, const PyrPlanes& pl,
                        int32_t max_h, int32_t max_w, dn_dtype dt, void* d_out, void* stream) {
  dim3 grid((max_w + 64 * PX - 1) / (64 * PX), (max_h + 3) / 4, n_img * pl.n);
  hipStream_t s = (hipStream_t)stream;
  switch (dt) {
    case DN_F32:
      build_planes_kernel<float><<<grid, 256, 0, s>>>(d_img, a, pl, (float*)d_out);
      break;
    case DN_F16:
      build_planes_kernel<_Float16><<<grid, 256, 0, s>>>(d_img, a, pl, (_Float16*)d_out);
      break;
    case DN_BF16:
      build_planes_kernel<__bf16><<<grid, 256, 0, s>>>(d_img, a, pl, (__bf16*)d_out);
      break;
  }
  return (int)hipGetLastError();
}

}  // namespace dn
