// Plane builder: bilinear resampling of the uint8 image to every scale (Sec. 3.1 pyramid), mean-pixel
// centring (Sec. 3.2), the 16-px border (ramp to the mean, or the mean itself) and stitching onto
// planes with a zero background (Sec. 3.1), fused into one pass that writes every plane pixel once.
//
// One thread per plane pixel, 64 consecutive columns per wave so every channel row is written with
// contiguous stores; the source image (a few MB) stays in L2 / MALL for the gathers.  The half-pixel
// source coordinate ((2 y + 1) H - h) / (2 h) is formed exactly in integers; only the blend is fp32.
#include "common.h"

namespace dn {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void build_planes_kernel(const uint8_t* __restrict__ img,
                                                           PyrArgs a, PyrPlanes pl,
                                                           T* __restrict__ out) {
  const int z = blockIdx.z;
  const int b = z / pl.n, j = z - b * pl.n;
  const int PH = pl.p[j].h, PW = pl.p[j].w;
  const int x = blockIdx.x * 64 + (threadIdx.x & 63);
  const int y = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (x >= PW || y >= PH) return;

  int owner = -1;
  for (int k = 0; k < a.n_scales; ++k) {
    const PyrScale& s = a.s[k];
    if (s.plane == j && y >= s.y && y < s.y + s.rh && x >= s.x && x < s.x + s.rw) {
      owner = k;
      break;
    }
  }
  float v0 = 0.f, v1 = 0.f, v2 = 0.f;
  if (owner >= 0) {
    const PyrScale s = a.s[owner];
    const int vy = y - s.y - a.pad, ux = x - s.x - a.pad;
    const int dy = max(0, max(-vy, vy - (s.h - 1)));
    const int dx = max(0, max(-ux, ux - (s.w - 1)));
    if (dy <= a.pad && dx <= a.pad) {
      float wgt = 1.f;
      if (dy | dx) {
        if (a.ramp) {
          const float den = (float)(a.pad + 1);
          const float wy = dy ? (float)(a.pad + 1 - dy) / den : 1.f;
          const float wx = dx ? (float)(a.pad + 1 - dx) / den : 1.f;
          wgt = wy * wx;
        } else {
          wgt = 0.f;
        }
      }
      if (wgt != 0.f) {
        const int yc = min(max(vy, 0), s.h - 1), xc = min(max(ux, 0), s.w - 1);
        int64_t ny = (int64_t)(2 * yc + 1) * a.H - s.h;
        int64_t nx = (int64_t)(2 * xc + 1) * a.W - s.w;
        if (ny < 0) ny = 0;
        if (nx < 0) nx = 0;
        const int64_t dh = 2 * (int64_t)s.h, dw = 2 * (int64_t)s.w;
        const int y0 = (int)(ny / dh), x0 = (int)(nx / dw);
        const float ly = (float)(ny - y0 * dh) / (float)dh;
        const float lx = (float)(nx - x0 * dw) / (float)dw;
        const int y1 = min(y0 + 1, a.H - 1), x1 = min(x0 + 1, a.W - 1);
        const int64_t HW = (int64_t)a.H * a.W;
        const uint8_t* I = img + (int64_t)b * 3 * HW;
        float r[3];
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          const uint8_t* P = I + c * HW;
          const float i00 = P[(int64_t)y0 * a.W + x0], i01 = P[(int64_t)y0 * a.W + x1];
          const float i10 = P[(int64_t)y1 * a.W + x0], i11 = P[(int64_t)y1 * a.W + x1];
          const float top = i00 + lx * (i01 - i00), bot = i10 + lx * (i11 - i10);
          r[c] = (top + ly * (bot - top) - a.mean[c]) * wgt;
        }
        v0 = r[0];
        v1 = r[1];
        v2 = r[2];
      }
    }
  }
  T* o = out + (int64_t)b * pl.image_elems + pl.p[j].offset;
  const int64_t plane = (int64_t)PH * PW, at = (int64_t)y * PW + x;
  o[at] = from_f32<T>(v0);
  o[plane + at] = from_f32<T>(v1);
  o[2 * plane + at] = from_f32<T>(v2);
}

}  // namespace

int launch_build_planes(const uint8_t* d_img, int32_t n_img, const PyrArgs& a, const PyrPlanes& pl,
                        int32_t max_h, int32_t max_w, dn_dtype dt, void* d_out, void* stream) {
  dim3 grid((max_w + 63) / 64, (max_h + 3) / 4, n_img * pl.n);
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
