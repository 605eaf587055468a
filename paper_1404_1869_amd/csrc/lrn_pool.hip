// Cross-channel LRN and 3x3 / stride-2 max-pooling with ceil-mode output size and clipped windows,
// on channels-last maps (the normalisation and pooling that follow conv1 and conv2 of the AlexNet
// topology, and the optional pool after conv5).
//
// One thread per output element, channels fastest, so a wave reads and writes 64 consecutive
// channels of one pixel.  LRN of the pooling window's pixels is recomputed per output: inputs come
// from L1/L2 (each is reused by neighbouring windows and channels), and HBM sees each input once.
// (k + alpha/n * s)^-beta is evaluated as exp2(-beta * log2(.)) with the hardware transcendental
// units; the argument is >= k > 0.
#include "common.h"

namespace dn {
namespace {

__device__ inline float lrn_scale(float s, float alpha_n, float beta, float k) {
  return __builtin_amdgcn_exp2f(-beta * __builtin_amdgcn_logf(k + alpha_n * s));
}

template <typename T, bool LRN, bool LRN_FIRST>
__global__ __launch_bounds__(256) void lrn_pool_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                       int H, int W, int C, int Ho, int Wo,
                                                       int64_t in_stride, int64_t out_stride,
                                                       int64_t total, float alpha_n, float beta,
                                                       float k, int half_n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int c = (int)(i % C);
  int64_t r = i / C;
  const int ox = (int)(r % Wo);
  r /= Wo;
  const int oy = (int)(r % Ho);
  const int plane = (int)(r / Ho);
  const T* src = in + plane * in_stride;
  const int y0 = 2 * oy, y1 = min(y0 + 3, H), x0 = 2 * ox, x1 = min(x0 + 3, W);
  const int clo = max(0, c - half_n), chi = min(C - 1, c + half_n);
  float best = -INFINITY;
  if (!LRN) {
    for (int y = y0; y < y1; ++y)
      for (int x = x0; x < x1; ++x) best = fmaxf(best, to_f32(src[((int64_t)y * W + x) * C + c]));
  } else if (LRN_FIRST) {
    for (int y = y0; y < y1; ++y)
      for (int x = x0; x < x1; ++x) {
        const T* px = src + ((int64_t)y * W + x) * C;
        float s = 0.f;
        for (int j = clo; j <= chi; ++j) {
          const float v = to_f32(px[j]);
          s += v * v;
        }
        best = fmaxf(best, to_f32(px[c]) * lrn_scale(s, alpha_n, beta, k));
      }
  } else {
    float s = 0.f, mine = 0.f;
    for (int j = clo; j <= chi; ++j) {
      float m = -INFINITY;
      for (int y = y0; y < y1; ++y)
        for (int x = x0; x < x1; ++x) m = fmaxf(m, to_f32(src[((int64_t)y * W + x) * C + j]));
      s += m * m;
      if (j == c) mine = m;
    }
    best = mine * lrn_scale(s, alpha_n, beta, k);
  }
  out[plane * out_stride + ((int64_t)oy * Wo + ox) * C + c] = from_f32<T>(best);
}

template <typename T>
int run(const void* d_in, int32_t n, int32_t H, int32_t W, int32_t C, int64_t in_stride, bool lrn,
        bool lrn_first, float alpha, float beta, float k, int32_t lrn_n, void* d_out,
        int64_t out_stride, hipStream_t s) {
  const int Ho = H >= 2 ? (H - 2) / 2 + 1 : 0, Wo = W >= 2 ? (W - 2) / 2 + 1 : 0;
  const int64_t total = (int64_t)n * Ho * Wo * C;
  if (total <= 0) return (int)hipErrorInvalidValue;
  const int64_t blocks = (total + 255) / 256;
  if (blocks > 0x7fffffff) return (int)hipErrorInvalidValue;
  const float an = alpha / (float)lrn_n;
  const int hn = lrn_n / 2;
  const T* in = (const T*)d_in;
  T* out = (T*)d_out;
  if (!lrn)
    lrn_pool_kernel<T, false, false><<<(unsigned)blocks, 256, 0, s>>>(
        in, out, H, W, C, Ho, Wo, in_stride, out_stride, total, an, beta, k, hn);
  else if (lrn_first)
    lrn_pool_kernel<T, true, true><<<(unsigned)blocks, 256, 0, s>>>(
        in, out, H, W, C, Ho, Wo, in_stride, out_stride, total, an, beta, k, hn);
  else
    lrn_pool_kernel<T, true, false><<<(unsigned)blocks, 256, 0, s>>>(
        in, out, H, W, C, Ho, Wo, in_stride, out_stride, total, an, beta, k, hn);
  return (int)hipGetLastError();
}

}  // namespace

int launch_lrn_pool(const void* d_in, int32_t n, int32_t H, int32_t W, int32_t C, int64_t in_stride,
                    dn_dtype dt, bool lrn, bool lrn_first, float alpha, float beta, float k,
                    int32_t lrn_n, void* d_out, int64_t out_stride, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  switch (dt) {
    case DN_F32:
      return run<float>(d_in, n, H, W, C, in_stride, lrn, lrn_first, alpha, beta, k, lrn_n, d_out,
                        out_stride, s);
    case DN_F16:
      return run<_Float16>(d_in, n, H, W, C, in_stride, lrn, lrn_first, alpha, beta, k, lrn_n, d_out,
                           out_stride, s);
    case DN_BF16:
      return run<__bf16>(d_in, n, H, W, C, in_stride, lrn, lrn_first, alpha, beta, k, lrn_n, d_out,
                         out_stride, s);
  }
  return (int)hipErrorInvalidValue;
}

}  // namespace dn
