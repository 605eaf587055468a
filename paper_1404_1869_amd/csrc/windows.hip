// Crop-before windows: the per-window baseline the paper measures its dense pyramid against (Sec. 3.4)
// and the "crop before" pipeline of Sec. 4.  Every region is cut out of its image in pixel space and
// warped on its own to the classifier's S x S input (bilinear, half-pixel centres, the box stretched
// onto the grid with no context margin), then mean-centred, so that each window can run through the
// conv stack as an independent plane.
//
// Output pixel (i, j) of box (x1, y1, x2, y2) samples the image at
//   sy = y1 + (i + 0.5) (y2 - y1) / S - 0.5,  sx = x1 + (j + 0.5) (x2 - x1) / S - 0.5,
// each clamped to the image ([0, H - 1], [0, W - 1]), so a box reaching outside the image repeats the
// edge pixel with interpolation weights in [0, 1); the top-left neighbour is floor(s), the other one
// lies one further (clamped).  Coordinates and fractions are fp64
// with + - * / only and contraction off, in the order written, so the taps are reproducible bit for
// bit; the blend is fp32.  A workgroup owns RB output rows of one box: it tabulates the S columns'
// taps and fractions and its rows' taps in LDS once, then each thread produces one pixel per row
// (three channels, 12 byte gathers that hit L2) and stores it channel by channel, coalesced along the
// row.  Rows are `pitch` elements apart; the columns from S to pitch - 1 are written as zeros (a
// pitch that is a multiple of 8 lets conv1 load the rows straight into LDS).
#include <cmath>

#include "common.h"

namespace dn {
namespace {

constexpr int RB = 16;  // output rows per workgroup

struct Tap {
  int32_t i0, i1;
  float frac;
};

#pragma clang fp contract(off)
__device__ inline Tap warp_tap(double lo, double step, int o, int n) {
  double s = lo + (o + 0.5) * step - 0.5;
  s = fmin(fmax(s, 0.0), (double)(n - 1));
  const int i0 = (int)floor(s);
  Tap t;
  t.i0 = i0;
  t.i1 = min(i0 + 1, n - 1);
  t.frac = (float)(s - (double)i0);
  return t;
}

template <typename T>
__global__ __launch_bounds__(256) void warp_regions_kernel(const uint8_t* __restrict__ img, int n_img,
                                                           int H, int W, const float* __restrict__ boxes,
                                                           const int32_t* __restrict__ box_img, int S,
                                                           int pitch, int row_blocks, float m0, float m1,
                                                           float m2, T* __restrict__ out) {
  __shared__ Tap s_col[DN_MAX_WARP_SIDE];
  __shared__ Tap s_row[RB];
  const int r = blockIdx.x / row_blocks, i_first = (blockIdx.x % row_blocks) * RB;
  const int rows = min(RB, S - i_first);
  const double x1 = boxes[4 * r + 0], y1 = boxes[4 * r + 1], x2 = boxes[4 * r + 2], y2 = boxes[4 * r + 3];
  const int b = box_img ? box_img[r] : 0;
  const bool ok = isfinite(x1) && isfinite(y1) && isfinite(x2) && isfinite(y2) && x2 - x1 > 0 &&
                  y2 - y1 > 0 && b >= 0 && b < n_img;
  const int64_t SS = (int64_t)S * pitch;
  T* o = out + (int64_t)r * 3 * SS;
  if (!ok) {
    for (int i = 0; i < rows; ++i)
      for (int j = threadIdx.x; j < pitch; j += 256)
#pragma unroll
        for (int c = 0; c < 3; ++c) o[c * SS + (int64_t)(i_first + i) * pitch + j] = from_f32<T>(0.f);
    return;
  }
  const double fx = (x2 - x1) / S, fy = (y2 - y1) / S;
  for (int j = threadIdx.x; j < S; j += 256) s_col[j] = warp_tap(x1, fx, j, W);
  if (threadIdx.x < rows) s_row[threadIdx.x] = warp_tap(y1, fy, i_first + threadIdx.x, H);
  __syncthreads();
  const int64_t HW = (int64_t)H * W;
  const uint8_t* I = img + (int64_t)b * 3 * HW;
  const float mean[3] = {m0, m1, m2};
  for (int i = 0; i < rows; ++i) {
    const Tap ty = s_row[i];
    const uint8_t* r0 = I + (int64_t)ty.i0 * W;
    const uint8_t* r1 = I + (int64_t)ty.i1 * W;
    T* orow = o + (int64_t)(i_first + i) * pitch;
    for (int j = threadIdx.x; j < pitch; j += 256) {
      if (j >= S) {
#pragma unroll
        for (int c = 0; c < 3; ++c) orow[c * SS + j] = from_f32<T>(0.f);
        continue;
      }
      const Tap tx = s_col[j];
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        const float a = r0[c * HW + tx.i0], bq = r0[c * HW + tx.i1];
        const float cq = r1[c * HW + tx.i0], d = r1[c * HW + tx.i1];
        const float top = (1.f - tx.frac) * a + tx.frac * bq;
        const float bot = (1.f - tx.frac) * cq + tx.frac * d;
        orow[c * SS + j] = from_f32<T>((1.f - ty.frac) * top + ty.frac * bot - mean[c]);
      }
    }
  }
}

}  // namespace

int launch_warp_regions(const uint8_t* d_img, int32_t n_img, int32_t H, int32_t W, const float* d_boxes,
                        const int32_t* d_box_img, int32_t n, int32_t S, int32_t pitch, const float* mean,
                        dn_dtype dt, void* d_out, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int row_blocks = (S + RB - 1) / RB;
  const int64_t blocks = (int64_t)n * row_blocks;
  if (blocks <= 0 || blocks > 0x7fffffff) return (int)hipErrorInvalidValue;
#define DN_WARP_ARGS \
  d_img, n_img, H, W, d_boxes, d_box_img, S, pitch, row_blocks, mean[0], mean[1], mean[2]
  switch (dt) {
    case DN_F32:
      warp_regions_kernel<float><<<(unsigned)blocks, 256, 0, s>>>(DN_WARP_ARGS, (float*)d_out);
      break;
    case DN_F16:
      warp_regions_kernel<_Float16><<<(unsigned)blocks, 256, 0, s>>>(DN_WARP_ARGS, (_Float16*)d_out);
      break;
    case DN_BF16:
      warp_regions_kernel<__bf16><<<(unsigned)blocks, 256, 0, s>>>(DN_WARP_ARGS, (__bf16*)d_out);
      break;
  }
#undef DN_WARP_ARGS
  return (int)hipGetLastError();
}

}  // namespace dn
