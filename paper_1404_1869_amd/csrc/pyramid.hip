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

// One thread per PX consecutive pixels of a plane row; a wave covers 64 * PX columns.  In stitched
// planes every rectangle edge is a multiple of 16 px, and a per-scale plane is its scale's rectangle,
// so an aligned group of PX pixels has a single owner (or none), found among the plane's own scales.
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

  float v[PX][3];
#pragma unroll
  for (int i = 0; i < PX; ++i) v[i][0] = v[i][1] = v[i][2] = 0.f;

  int owner = -1;
  const int f0 = a.plane_first[j], f1 = f0 + a.plane_count[j];
  for (int e = f0; e < f1; ++e) {
    const PyrScale& s = a.s[e];
    if (y >= s.y && y < s.y + s.rh && x0 >= s.x && x0 < s.x + s.rw) {
      owner = e;
      break;
    }
  }
  if (owner >= 0) {
    const PyrScale s = a.s[owner];
    const int vy = y - s.y - a.pad;
    const int dy = max(0, max(-vy, vy - (s.h - 1)));
    const float wy = border_weight(dy, a.pad, a.ramp);
    if (wy != 0.f) {
      const uint8_t* I = img + (int64_t)b * 3 * a.H * a.W;
      const int64_t HW = (int64_t)a.H * a.W;
      int sy0, sy1;
      float ly;
      src_coord(min(max(vy, 0), s.h - 1), a.H, s.h, 1.0 / (2.0 * s.h), sy0, sy1, ly);
      const double inv2w = 1.0 / (2.0 * s.w);
      const int r0 = sy0 * a.W, r1 = sy1 * a.W;
#pragma unroll
      for (int i = 0; i < PX; ++i) {
        const int ux = x0 + i - s.x - a.pad;
        const int dx = max(0, max(-ux, ux - (s.w - 1)));
        const float wgt = wy * border_weight(dx, a.pad, a.ramp);
        if (wgt == 0.f || x0 + i >= PW) continue;
        int sx0, sx1;
        float lx;
        src_coord(min(max(ux, 0), s.w - 1), a.W, s.w, inv2w, sx0, sx1, lx);
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          const uint8_t* P = I + c * HW;
          const float i00 = P[r0 + sx0], i01 = P[r0 + sx1];
          const float i10 = P[r1 + sx0], i11 = P[r1 + sx1];
          const float top = i00 + lx * (i01 - i00), bot = i10 + lx * (i11 - i10);
          v[i][c] = (top + ly * (bot - top) - a.mean[c]) * wgt;
        }
      }
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
