// Cross-channel LRN and 3x3 / stride-2 max-pooling with ceil-mode output size and clipped windows,
// on channels-last maps (the normalisation and pooling that follow conv1 and conv2 of the AlexNet
// topology, and the optional pool after conv5).  Bandwidth-bound: every input element should cross
// HBM once and every output once.
//
// Tiled kernel (LRN then pool, or pool only): a workgroup owns TPH x TPW pooled outputs and all C
// channels.  Phase 1 reads the (2 TPH + 1) x (2 TPW + 1) input pixels of its windows with 16-byte
// channel vectors, computes the LRN of each input element once (the channel window is taken from
// the neighbouring vectors, zero beyond the channel range, which equals clipping the window), and
// stores the results in LDS in the storage type.  Phase 2 takes the max over each clipped window
// from LDS and writes 16-byte vectors.  Rounding to the storage type before the max gives the same
// result as after it, since rounding is monotone.
//
// (k + alpha/n * s)^-beta is evaluated as exp2(-beta * log2(.)) on the hardware transcendental units;
// the argument is >= k > 0.
//
// With 16-bit storage, C = 256 (after conv2) walks column strips instead of tiles on large launches,
// so that each input element's LRN is computed about once rather than once per tile whose windows
// reach it.
//
// The pool-then-LRN order uses a simple kernel with one thread per output element.
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace dn {
namespace {

__device__ inline float lrn_scale(float s, float alpha_n, float beta, float k) {
  return __builtin_amdgcn_exp2f(-beta * __builtin_amdgcn_logf(k + alpha_n * s));
}

constexpr int VECB = 16;  // bytes per channel vector

#ifndef DN_LRN96_CPT
#define DN_LRN96_CPT 96
#endif
#ifndef DN_LRN96_TH
#define DN_LRN96_TH 8
#endif
#ifndef DN_LRN96_TW
#define DN_LRN96_TW 7
#endif
#ifndef DN_LRN96_WPE
#define DN_LRN96_WPE 3
#endif
// The tile kernel's configuration at C = 96 for 16-bit storage (channels per thread, output tile rows
// and columns, waves per SIMD), chosen by timing on the 96-plane batch: a whole pixel per thread.
// Strip kernel configuration for C = 256 and 16-bit storage: channels per thread, pooled columns and
// rows per workgroup, waves per SIMD (the LDS ring admits 4 workgroups per CU).  Chosen by timing on
// the 96-plane batch (lrn_pool2 0.334 -> 0.313 ms against the tile kernel; 16 rows 0.315 ms).  At
// C = 96 the tile kernel stays: a whole pixel per thread (12 loads in flight, no neighbour vectors)
// with 1.14x recomputation beat the strips (0.43 against 0.46-0.50 ms).
#ifndef DN_STRIP256
#define DN_STRIP256 32, 7, 8, 4
#endif
// Compute units of the device current at the first call (256 if the query fails), queried once;
// the initialisation is thread-safe.
int device_cus() {
  static const int n = [] {
    int dev = 0, v = 0;
    const bool ok = hipGetDevice(&dev) == hipSuccess &&
                    hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess;
    return ok && v > 0 ? v : 256;
  }();
  return n;
}
constexpr int MAX_HALF = 8;

template <typename T>
struct Vec {
  static constexpr int N = VECB / sizeof(T);
  typedef T type __attribute__((ext_vector_type(N)));
};

template <typename T, bool LRN, int HN>
__global__ __launch_bounds__(256) void lrn_pool_tile_kernel(const T* __restrict__ in,
                                                            T* __restrict__ out, KRuns runs, int C,
                                                            int TPH, int TPW, float alpha_n,
                                                            float beta, float k) {
  constexpr int N = Vec<T>::N;
  static_assert(HN <= N && HN <= MAX_HALF, "the channel window must fit one neighbouring vector");
  typedef typename Vec<T>::type vec_t;
  extern __shared__ __align__(16) unsigned char smem[];
  T* s = (T*)smem;
  const int CS = C + N;  // LDS pixel stride (elements), keeps 16-byte alignment
  const int G = C / N;   // channel vectors per pixel

  int bid = blockIdx.x;
  const KRun& rn = runs.r[run_of(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, Ho = rn.Ho, Wo = rn.Wo, tiles_x = rn.tiles_x, tiles_y = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  const int tx = bid % tiles_x;
  bid /= tiles_x;
  const int ty = bid % tiles_y;
  const int plane = bid / tiles_y;
  const int oy0 = ty * TPH, ox0 = tx * TPW;
  const int iy0 = 2 * oy0, ix0 = 2 * ox0;
  const int IH = 2 * TPH + 1, IW = 2 * TPW + 1;
  const T* src = in + plane * in_stride;

  // Phase 1: LRN of every input element of the tile's windows, into LDS.
  for (int e = threadIdx.x; e < IH * IW * G; e += blockDim.x) {
    const int g = e % G, p = e / G;
    const int hy = p / IW, hx = p % IW;
    const int y = iy0 + hy, x = ix0 + hx;
    if (y >= H || x >= W) continue;  // outside the map: never inside a clipped window
    const T* px = src + ((int64_t)y * W + x) * C;
    const vec_t v = *(const vec_t*)(px + g * N);
    vec_t r;
    if constexpr (LRN) {
      float f[N + 2 * MAX_HALF];
#pragma unroll
      for (int i = 0; i < N + 2 * MAX_HALF; ++i) f[i] = 0.f;
#pragma unroll
      for (int i = 0; i < N; ++i) f[MAX_HALF + i] = to_f32(v[i]);
      if (g > 0) {
        const vec_t l = *(const vec_t*)(px + (g - 1) * N);
#pragma unroll
        for (int i = 0; i < N; ++i)
          if (i >= N - MAX_HALF) f[MAX_HALF - N + i] = to_f32(l[i]);
      }
      if (g + 1 < G) {
        const vec_t q = *(const vec_t*)(px + (g + 1) * N);
#pragma unroll
        for (int i = 0; i < N; ++i)
          if (i < MAX_HALF) f[MAX_HALF + N + i] = to_f32(q[i]);
      }
#pragma unroll
      for (int i = 0; i < N; ++i) {
        float sq = 0.f;
#pragma unroll
        for (int j = -HN; j <= HN; ++j) {
          const float a = f[MAX_HALF + i + j];
          sq += a * a;
        }
        r[i] = from_f32<T>(f[MAX_HALF + i] * lrn_scale(sq, alpha_n, beta, k));
      }
    } else {
      r = v;
    }
    *(vec_t*)(s + p * CS + g * N) = r;
  }
  __syncthreads();

  // Phase 2: max over each clipped 3x3 window.
  for (int e = threadIdx.x; e < TPH * TPW * G; e += blockDim.x) {
    const int g = e % G, q = e / G;
    const int qy = q / TPW, qx = q % TPW;
    const int oy = oy0 + qy, ox = ox0 + qx;
    if (oy >= Ho || ox >= Wo) continue;
    const int y1 = min(2 * oy + 3, H) - iy0, x1 = min(2 * ox + 3, W) - ix0;
    float m[N];
#pragma unroll
    for (int i = 0; i < N; ++i) m[i] = -INFINITY;
    for (int hy = 2 * qy; hy < y1; ++hy)
      for (int hx = 2 * qx; hx < x1; ++hx) {
        const vec_t v = *(const vec_t*)(s + (hy * IW + hx) * CS + g * N);
#pragma unroll
        for (int i = 0; i < N; ++i) m[i] = fmaxf(m[i], to_f32(v[i]));
      }
    vec_t r;
#pragma unroll
    for (int i = 0; i < N; ++i) r[i] = from_f32<T>(m[i]);
    *(vec_t*)(out + plane * out_stride + ((int64_t)oy * Wo + ox) * C + g * N) = r;
  }
}

// LRN (window n = 5) of CPT consecutive channels c0 .. c0 + CPT - 1 of one pixel: v holds them, lv
// the vector just below c0 and rv the vector just above (zero beyond the channel range, which equals
// clipping the window).  The results go to d in the storage type.
template <typename T, int CPT>
__device__ inline void lrn_channels(const typename Vec<T>::type* v, const typename Vec<T>::type& lv,
                                    const typename Vec<T>::type& rv, T* d, float alpha_n, float beta,
                                    float k) {
  constexpr int N = Vec<T>::N, NV = CPT / N;
  typedef typename Vec<T>::type vec_t;
  // xs[1 + c] = channel c of this thread (c = -1 .. CPT, the outer ones from the neighbours or
  // zero); win[c] = sum of squares over channels c - 2 .. c + 2.
  float win[CPT], xs[CPT + 2];
  xs[0] = to_f32(lv[N - 1]);
  xs[CPT + 1] = to_f32(rv[0]);
#pragma unroll
  for (int c = 0; c < CPT; ++c) xs[1 + c] = to_f32(v[c / N][c % N]);
  if constexpr (sizeof(T) == 2) {
    // Pair sums P_j = x_2j^2 + x_2j+1^2 (j = -1 .. CPT / 2, counting the neighbours' pairs), their
    // neighbour sums Q_j = P_j + P_j+1, then window(2 i) = Q_i-1 + x_2i+2^2 and window(2 i + 1) =
    // Q_i + x_2i-1^2: two and a half operations per channel.
    constexpr int NP = CPT / 2;
    float pp[NP + 2];  // pp[1 + j] = P_j
    {
      const float a = to_f32(lv[N - 2]), b = to_f32(rv[1]);
      pp[0] = __builtin_fmaf(a, a, xs[0] * xs[0]);
      pp[NP + 1] = __builtin_fmaf(b, b, xs[CPT + 1] * xs[CPT + 1]);
    }
#pragma unroll
    for (int j = 0; j < NP; ++j) pp[1 + j] = __builtin_fmaf(xs[1 + 2 * j], xs[1 + 2 * j], xs[2 + 2 * j] * xs[2 + 2 * j]);
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      win[2 * i] = __builtin_fmaf(xs[2 * i + 3], xs[2 * i + 3], pp[i] + pp[i + 1]);
      win[2 * i + 1] = __builtin_fmaf(xs[2 * i], xs[2 * i], pp[i + 1] + pp[i + 2]);
    }
  } else {
    // sq[2 + i] = a_i^2, pr[i] = sq[i] + sq[i + 1]: window(c) = pr[c] + pr[c + 2] + sq[c + 4]
    float sq[CPT + 4], pr[CPT + 3];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const float a = to_f32(lv[N - 2 + i]), b = to_f32(rv[i]);
      sq[i] = a * a;
      sq[CPT + 2 + i] = b * b;
    }
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const float a = to_f32(v[i / N][i % N]);
      sq[2 + i] = a * a;
    }
#pragma unroll
    for (int i = 0; i < CPT + 3; ++i) pr[i] = sq[i] + sq[i + 1];
#pragma unroll
    for (int c = 0; c < CPT; ++c) win[c] = pr[c] + pr[c + 2] + sq[c + 4];
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    vec_t r;
#pragma unroll
    for (int e = 0; e < N; ++e) {
      const int c = i * N + e;
      r[e] = from_f32<T>(xs[1 + c] * lrn_scale(win[c], alpha_n, beta, k));
    }
    *(vec_t*)(d + i * N) = r;
  }
}

// LRN then pool for C = CPT * TPP channels (96 = 96 x 1; 256 = 64 x 4 at 16-bit storage, 128 x 2 at
// fp32) with the default window n = 5: every thread owns CPT consecutive channels of one input pixel.  It issues all of their
// 16-byte loads at once (plus one neighbouring vector on each inner side when a pixel is split over
// several threads), forms the five-channel sums of squares from pair sums, and stores the LRN result
// to LDS.  Pixels of the tile outside the map are stored as
// -inf, so every pooled output then takes the max over its full 3 x 3 window from LDS, unrolled, with
// no clipping tests.  Channel count and tile shape are compile-time constants, so no index
// arithmetic needs a division.  With 16-bit storage, a tile whose LRN values are all >= +0 (the usual
// case after ReLU) takes its maxima on the raw 16-bit patterns, two per instruction (for such values,
// and the -inf fill, signed-integer order is the float order); any other tile takes them in fp32.
// The tile's sign is read from the inputs' sign bits (LRN keeps the sign; -0 counts as negative).
template <typename T, int C, int CPT, int TPH, int TPW, int WPE, bool MULTI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE, WPE))) void lrn_pool_pixel_kernel(
                                                             const T* __restrict__ in,
                                                             T* __restrict__ out, KRuns runs,
                                                             float alpha_n, float beta, float k) {
  constexpr int N = Vec<T>::N;
  constexpr int NV = CPT / N, TPP = C / CPT, G = C / N, CS = C + N;
  constexpr int IW = 2 * TPW + 1, NP = (2 * TPH + 1) * IW;
  static_assert(CPT % N == 0 && C % CPT == 0 && N >= 2, "channel split must be whole vectors");
  static_assert(NP * TPP <= 256, "one thread per (pixel, part)");
  typedef typename Vec<T>::type vec_t;
  __shared__ __align__(16) T s[NP * CS];

  int bid = blockIdx.x;
  const KRun& rn = runs.r[run_of<MULTI>(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, Ho = rn.Ho, Wo = rn.Wo, tiles_x = rn.tiles_x, tiles_y = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  const int tx = bid % tiles_x;
  bid /= tiles_x;
  const int ty = bid % tiles_y;
  const int plane = bid / tiles_y;
  const int oy0 = ty * TPH, ox0 = tx * TPW;
  const int iy0 = 2 * oy0, ix0 = 2 * ox0;

  const int p = threadIdx.x / TPP, part = threadIdx.x % TPP;
  bool neg = false;
  if (p < NP) {
    const int y = iy0 + p / IW, x = ix0 + p % IW;
    T* d = s + p * CS + part * CPT;
    if (y < H && x < W) {
      const T* px = in + plane * in_stride + ((int64_t)y * W + x) * C + part * CPT;
      vec_t v[NV], lv = vec_t{}, rv = vec_t{};
#pragma unroll
      for (int i = 0; i < NV; ++i) v[i] = *(const vec_t*)(px + i * N);
      if (TPP > 1 && part > 0) lv = *(const vec_t*)(px - N);
      if (TPP > 1 && part + 1 < TPP) rv = *(const vec_t*)(px + CPT);
      if constexpr (sizeof(T) == 2) {
        typedef uint32_t uvec_t __attribute__((ext_vector_type(N / 2)));
        uint32_t bits = 0;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const uvec_t u = __builtin_bit_cast(uvec_t, v[i]);
#pragma unroll
          for (int j = 0; j < N / 2; ++j) bits |= u[j];
        }
        neg = (bits & 0x80008000u) != 0;
      }
      lrn_channels<T, CPT>(v, lv, rv, d, alpha_n, beta, k);
    } else {
      vec_t f;
#pragma unroll
      for (int e = 0; e < N; ++e) f[e] = from_f32<T>(-INFINITY);
#pragma unroll
      for (int i = 0; i < NV; ++i) *(vec_t*)(d + i * N) = f;
    }
  }
  const bool any_neg = __syncthreads_or(neg);

  if constexpr (sizeof(T) == 2) {
    if (!any_neg) {
      typedef short svec_t __attribute__((ext_vector_type(N)));
      for (int e = threadIdx.x; e < TPH * TPW * G; e += 256) {
        const int g = e % G, q = e / G;
        const int qy = q / TPW, qx = q % TPW;
        const int oy = oy0 + qy, ox = ox0 + qx;
        if (oy >= Ho || ox >= Wo) continue;
        const T* b = s + ((2 * qy) * IW + 2 * qx) * CS + g * N;
        svec_t m = *(const svec_t*)b;
#pragma unroll
        for (int wy = 0; wy < 3; ++wy)
#pragma unroll
          for (int wx = 0; wx < 3; ++wx)
            if (wy || wx) m = __builtin_elementwise_max(m, *(const svec_t*)(b + (wy * IW + wx) * CS));
        *(svec_t*)(out + plane * out_stride + ((int64_t)oy * Wo + ox) * C + g * N) = m;
      }
      return;
    }
  }
  for (int e = threadIdx.x; e < TPH * TPW * G; e += 256) {
    const int g = e % G, q = e / G;
    const int qy = q / TPW, qx = q % TPW;
    const int oy = oy0 + qy, ox = ox0 + qx;
    if (oy >= Ho || ox >= Wo) continue;
    const T* b = s + ((2 * qy) * IW + 2 * qx) * CS + g * N;
    float m[N];
#pragma unroll
    for (int i = 0; i < N; ++i) m[i] = -INFINITY;
#pragma unroll
    for (int wy = 0; wy < 3; ++wy)
#pragma unroll
      for (int wx = 0; wx < 3; ++wx) {
        const vec_t v = *(const vec_t*)(b + (wy * IW + wx) * CS);
#pragma unroll
        for (int i = 0; i < N; ++i) m[i] = fmaxf(m[i], to_f32(v[i]));
      }
    vec_t r;
#pragma unroll
    for (int i = 0; i < N; ++i) r[i] = from_f32<T>(m[i]);
    *(vec_t*)(out + plane * out_stride + ((int64_t)oy * Wo + ox) * C + g * N) = r;
  }
}

// LRN then pool on column strips, for 16-bit storage and the default window (n = 5).  A workgroup
// owns TPW pooled columns and SR pooled rows of one plane; it walks its output rows top to bottom.
// For output row oy it computes the LRN of input rows 2 oy + 1 and 2 oy + 2 over the strip's 2 TPW + 1
// input columns (one thread per (row, pixel, CPT channels)) into a ring of five LDS rows, and pools
// rows 2 oy .. 2 oy + 2 of the ring; row 2 oy came from the previous output row.  Each input element's
// LRN is thus computed once per strip, apart from the one column two strips share and the one row two
// row blocks share ((2 TPW + 1) / (2 TPW) x (2 SR + 1) / (2 SR) of the map's elements, against
// (2 TPH + 1)(2 TPW + 1) / (4 TPH TPW) for a workgroup tile of TPH x TPW outputs).  One barrier per
// output row: the ring's five rows keep the rows being written apart from the three being pooled.
// The next output row's input vectors are loaded into registers before the current row's LRN, so
// their latency overlaps the LRN, the barrier and the pooling.  Every thread issues the same loads
// and one store per output row, with no branches around them (addresses outside the map are
// clamped into it and their values discarded; threads without a pooling task repeat the strip's
// last one), so the compiler's vector-memory waits count exactly.  Pixels outside the map are stored
// as -inf.  The maxima are taken on the raw 16-bit patterns when the pooled rows' LRN values are all
// >= +0, else in fp32, as in the tile kernel.
template <typename T, int C, int CPT, int TPW, int SR, int WPE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE, WPE))) void lrn_pool_strip_kernel(
    const T* __restrict__ in, T* __restrict__ out, KRuns runs, float alpha_n, float beta, float k) {
  constexpr int N = Vec<T>::N;
  constexpr int NV = CPT / N, TPP = C / CPT, G = C / N, CS = C + N;
  constexpr int IW = 2 * TPW + 1, NSLOT = 5;
  static_assert(sizeof(T) == 2, "16-bit storage");
  static_assert(CPT % N == 0 && C % CPT == 0, "channel split must be whole vectors");
  static_assert(2 * IW * TPP <= 256 && TPW * G <= 256, "one thread per (row, pixel, part) and per task");
  typedef typename Vec<T>::type vec_t;
  typedef short svec_t __attribute__((ext_vector_type(N)));
  typedef uint32_t uvec_t __attribute__((ext_vector_type(N / 2)));
  __shared__ __align__(16) T s[NSLOT * IW * CS];

  int bid = blockIdx.x;
  const KRun& rn = runs.r[run_of(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, Ho = rn.Ho, Wo = rn.Wo, strips_x = rn.tiles_x, strips_y = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  const int sx = bid % strips_x;
  bid /= strips_x;
  const int sy = bid % strips_y;
  const int plane = bid / strips_y;
  const int ox0 = sx * TPW, oy0 = sy * SR, ix0 = 2 * ox0;
  const int nrows = min(SR, Ho - oy0);
  const T* src = in + plane * in_stride;
  T* dst = out + plane * out_stride;

  const int tid = threadIdx.x;
  const int r = min(tid / (IW * TPP), 1), rem = tid % (IW * TPP), px = rem / TPP, part = rem % TPP;
  const bool worker = tid < 2 * IW * TPP;
  const int x = ix0 + px, xc = min(x, W - 1);
  const bool col_ok = worker && x < W;
  // This thread's input vectors of one row: its CPT channels and the vectors just below and above
  // them (zero at the ends of the channel range).
  struct Row {
    vec_t v[NV], lv, rv;
  };
  auto load_row = [&](int y) {
    Row a;
    const T* p = src + ((int64_t)min(y, H - 1) * W + xc) * C + part * CPT;
#pragma unroll
    for (int i = 0; i < NV; ++i) a.v[i] = *(const vec_t*)(p + i * N);
    a.lv = *(const vec_t*)(p - (part > 0 ? N : 0));
    a.rv = *(const vec_t*)(p + (part + 1 < TPP ? CPT : 0));
    return a;
  };
  // LRN of row y's vectors into ring row `slot` (-inf outside the map).  Returns whether an input
  // sign bit was set (LRN keeps the sign; -0 counts as negative).
  auto lrn_row = [&](const Row& a, int y, int slot) -> bool {
    T* d = s + (slot * IW + px) * CS + part * CPT;
    if (col_ok && y < H) {
      uint32_t bits = 0;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const uvec_t u = __builtin_bit_cast(uvec_t, a.v[i]);
#pragma unroll
        for (int j = 0; j < N / 2; ++j) bits |= u[j];
      }
      const vec_t lv = part > 0 ? a.lv : vec_t{}, rv = part + 1 < TPP ? a.rv : vec_t{};
      lrn_channels<T, CPT>(a.v, lv, rv, d, alpha_n, beta, k);
      return (bits & 0x80008000u) != 0;
    }
    if (worker) {
      vec_t f;
#pragma unroll
      for (int e = 0; e < N; ++e) f[e] = from_f32<T>(-INFINITY);
#pragma unroll
      for (int i = 0; i < NV; ++i) *(vec_t*)(d + i * N) = f;
    }
    return false;
  };
  // Pooling task of this thread: pooled column q of the strip, channel vector g (threads past the
  // tasks, and columns past the map, repeat the strip's last column in the map).
  const int task = min(tid, TPW * G - 1);
  const int q = min(task / G, Wo - 1 - ox0), g = task % G;

  // Ring rows of input rows 2 oy, 2 oy + 1, 2 oy + 2 (input row y sits in ring row y mod 5).
  int s0 = (2 * oy0) % NSLOT;
  bool neg;
  {
    const Row top = load_row(2 * oy0);  // the first window's top row (threads of row 0)
    neg = r == 0 ? lrn_row(top, 2 * oy0, s0) : false;
  }
  Row cur = load_row(2 * oy0 + 1 + r);
  bool prev_any = false;
  for (int i = 0; i < nrows; ++i) {
    const int oy = oy0 + i;
    const Row nxt = load_row(2 * oy + 3 + r);
    const int s1 = s0 == NSLOT - 1 ? 0 : s0 + 1, s2 = s1 == NSLOT - 1 ? 0 : s1 + 1;
    neg |= lrn_row(cur, 2 * oy + 1 + r, r ? s2 : s1);
    const bool any = __syncthreads_or(neg) != 0;
    const bool fp = any || prev_any;  // rows 2 oy + 1, 2 oy + 2 and (previous pass) row 2 oy
    prev_any = any;
    neg = false;
    const T* b[3] = {s + (s0 * IW + 2 * q) * CS + g * N, s + (s1 * IW + 2 * q) * CS + g * N,
                     s + (s2 * IW + 2 * q) * CS + g * N};
    vec_t res;
    if (!fp) {
      svec_t m = *(const svec_t*)b[0];
#pragma unroll
      for (int wy = 0; wy < 3; ++wy)
#pragma unroll
        for (int wx = 0; wx < 3; ++wx)
          if (wy || wx) m = __builtin_elementwise_max(m, *(const svec_t*)(b[wy] + wx * CS));
      res = __builtin_bit_cast(vec_t, m);
    } else {
      float m[N];
#pragma unroll
      for (int e = 0; e < N; ++e) m[e] = -INFINITY;
#pragma unroll
      for (int wy = 0; wy < 3; ++wy)
#pragma unroll
        for (int wx = 0; wx < 3; ++wx) {
          const vec_t v = *(const vec_t*)(b[wy] + wx * CS);
#pragma unroll
          for (int e = 0; e < N; ++e) m[e] = fmaxf(m[e], to_f32(v[e]));
        }
#pragma unroll
      for (int e = 0; e < N; ++e) res[e] = from_f32<T>(m[e]);
    }
    *(vec_t*)(dst + ((int64_t)oy * Wo + ox0 + q) * C + g * N) = res;
    cur = nxt;
    s0 = s2;
  }
}

// Pool first, then LRN of the pooled vector: one thread per output element.
template <typename T>
__global__ __launch_bounds__(256) void pool_lrn_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                       KRuns runs, int C, float alpha_n, float beta,
                                                       float k, int half_n) {
  // run r: tiles_x workgroups of 256 output elements per plane
  int bid = blockIdx.x;
  const KRun& rn = runs.r[run_of(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, Ho = rn.Ho, Wo = rn.Wo, tiles_x = rn.tiles_x, tiles_y_unused = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  (void)tiles_y_unused;
  const int plane = bid / tiles_x, i = (bid % tiles_x) * 256 + (int)threadIdx.x;
  if (i >= Ho * Wo * C) return;
  const int c = i % C, ox = (i / C) % Wo, oy = i / C / Wo;
  const T* src = in + plane * in_stride;
  const int y0 = 2 * oy, y1 = min(y0 + 3, H), x0 = 2 * ox, x1 = min(x0 + 3, W);
  const int clo = max(0, c - half_n), chi = min(C - 1, c + half_n);
  float s = 0.f, mine = 0.f;
  for (int j = clo; j <= chi; ++j) {
    float m = -INFINITY;
    for (int y = y0; y < y1; ++y)
      for (int x = x0; x < x1; ++x) m = fmaxf(m, to_f32(src[((int64_t)y * W + x) * C + j]));
    s += m * m;
    if (j == c) mine = m;
  }
  out[plane * out_stride + ((int64_t)oy * Wo + ox) * C + c] =
      from_f32<T>(mine * lrn_scale(s, alpha_n, beta, k));
}

// Output tile so that the LDS tile stays within 64 KB.
template <typename T>
void pick_tile(int C, int& TPH, int& TPW) {
  const size_t es = sizeof(T), cs = (size_t)C + VECB / es;
  const int cand[][2] = {{8, 8}, {4, 8}, {4, 6}, {4, 4}, {2, 4}, {2, 2}, {1, 2}, {1, 1}};
  for (auto& c : cand) {
    const size_t bytes = (size_t)(2 * c[0] + 1) * (2 * c[1] + 1) * cs * es;
    if (bytes <= 65536) {
      TPH = c[0];
      TPW = c[1];
      return;
    }
  }
  TPH = TPW = 0;
}

// The per-pixel kernel over the runs of kr: the single-run variant when there is one.
template <typename T, int C, int CPT, int TPH, int TPW, int WPE>
void pixel(int64_t blocks, hipStream_t s, const T* in, T* out, const KRuns& kr, float an, float beta,
           float k) {
  if (kr.count == 1)
    lrn_pool_pixel_kernel<T, C, CPT, TPH, TPW, WPE, false><<<(unsigned)blocks, 256, 0, s>>>(in, out, kr, an,
                                                                                          beta, k);
  else
    lrn_pool_pixel_kernel<T, C, CPT, TPH, TPW, WPE, true><<<(unsigned)blocks, 256, 0, s>>>(in, out, kr, an,
                                                                                         beta, k);
}

template <typename T>
int run(const void* d_in, const MapRun* runs, int n_runs, int32_t C, bool lrn, bool lrn_first,
        float alpha, float beta, float k, int32_t lrn_n, void* d_out, hipStream_t s) {
  for (int i = 0; i < n_runs; ++i)
    if (runs[i].n <= 0 || runs[i].H < 2 || runs[i].W < 2) return (int)hipErrorInvalidValue;
  const float an = alpha / (float)lrn_n;
  const int hn = lrn_n / 2;
  const T* in = (const T*)d_in;
  T* out = (T*)d_out;
  KRuns kr;
  // Per run: the pooled size and tiles of TPH x TPW output pixels.
  auto tiles = [&](int TPH, int TPW) {
    return fill_kruns(runs, n_runs, kr, [=](KRun& q) {
      q.Ho = (q.H - 2) / 2 + 1, q.Wo = (q.W - 2) / 2 + 1;
      q.tiles_x = (q.Wo + TPW - 1) / TPW, q.tiles_y = (q.Ho + TPH - 1) / TPH;
      return (int64_t)q.tiles_x * q.tiles_y;
    });
  };
  if (lrn && !lrn_first) {
    const int64_t blocks = fill_kruns(runs, n_runs, kr, [=](KRun& q) {
      q.Ho = (q.H - 2) / 2 + 1, q.Wo = (q.W - 2) / 2 + 1;
      q.tiles_x = (int)(((int64_t)q.Ho * q.Wo * C + 255) / 256), q.tiles_y = 1;
      return (int64_t)q.tiles_x;
    });
    if (blocks <= 0) return (int)hipErrorInvalidValue;
    pool_lrn_kernel<T><<<(unsigned)blocks, 256, 0, s>>>(in, out, kr, C, an, beta, k, hn);
    return (int)hipGetLastError();
  }
  constexpr int N = Vec<T>::N;
  if (C % N || hn > 4) return (int)hipErrorInvalidValue;
  // Per-pixel kernel for the two channel counts of the network with the default window (n = 5).
  // Tiles: the largest whose input pixels fit one thread each (per part) and whose LDS tile stays
  // within 64 KB.
  if constexpr (sizeof(T) == 2) {
    if (lrn && hn == 2 && C == 256) {
      const int cfg[4] = {DN_STRIP256};
      const int TPW = cfg[1], SR = cfg[2];
      const int64_t blocks = tiles(SR, TPW);  // strips of SR rows x TPW columns
      if (blocks <= 0) return (int)hipErrorInvalidValue;
      // Launches of fewer strips than two rounds of the chip's resident slots (one image's planes:
      // about 660) take the tile kernel's 2850 shorter workgroups instead (29 against 31-37 us).
      if (blocks < 2LL * 4 * device_cus()) {
        const int64_t tb = tiles(3, 4);
        if (tb <= 0) return (int)hipErrorInvalidValue;
        pixel<T, 256, 64, 3, 4, 4>(tb, s, in, out, kr, an, beta, k);
        return (int)hipGetLastError();
      }
      lrn_pool_strip_kernel<T, 256, DN_STRIP256><<<(unsigned)blocks, 256, 0, s>>>(in, out, kr, an, beta, k);
      return (int)hipGetLastError();
    }
  }
  if (lrn && hn == 2 && (C == 96 || C == 256)) {
    // (16-bit storage reaches this only for C = 96: C = 256 takes the strip kernel above)
    constexpr bool F32 = sizeof(T) == 4;
    constexpr int TH96 = F32 ? 4 : DN_LRN96_TH, TW96 = F32 ? 7 : DN_LRN96_TW, TH256 = 2, TW256 = 5;
    const int64_t blocks = C == 96 ? tiles(TH96, TW96) : tiles(TH256, TW256);
    if (blocks <= 0) return (int)hipErrorInvalidValue;
    // Waves per SIMD the LDS tile allows (3 and 2 workgroups of 4 waves per CU): the compiler may use
    // the registers that occupancy leaves free for more independent work in flight.
    if (C == 96) {
      pixel<T, 96, F32 ? 96 : DN_LRN96_CPT, TH96, TW96, F32 ? 3 : DN_LRN96_WPE>(blocks, s, in, out, kr, an,
                                                                               beta, k);
    } else if constexpr (F32) {
      pixel<T, 256, 128, TH256, TW256, 2>(blocks, s, in, out, kr, an, beta, k);
    } else {
      return (int)hipErrorInvalidValue;
    }
    return (int)hipGetLastError();
  }
  int TPH, TPW;
  pick_tile<T>(C, TPH, TPW);
  if (!TPH) return (int)hipErrorInvalidValue;
  const int64_t blocks = tiles(TPH, TPW);
  if (blocks <= 0) return (int)hipErrorInvalidValue;
  const size_t lds = (size_t)(2 * TPH + 1) * (2 * TPW + 1) * (C + N) * sizeof(T);
#define DN_TILE_ARGS in, out, kr, C, TPH, TPW, an, beta, k
  if (!lrn) {
    lrn_pool_tile_kernel<T, false, 0><<<(unsigned)blocks, 256, lds, s>>>(DN_TILE_ARGS);
  } else {
    switch (hn) {
      case 0: lrn_pool_tile_kernel<T, true, 0><<<(unsigned)blocks, 256, lds, s>>>(DN_TILE_ARGS); break;
      case 1: lrn_pool_tile_kernel<T, true, 1><<<(unsigned)blocks, 256, lds, s>>>(DN_TILE_ARGS); break;
      case 2: lrn_pool_tile_kernel<T, true, 2><<<(unsigned)blocks, 256, lds, s>>>(DN_TILE_ARGS); break;
      case 3: lrn_pool_tile_kernel<T, true, 3><<<(unsigned)blocks, 256, lds, s>>>(DN_TILE_ARGS); break;
      case 4: lrn_pool_tile_kernel<T, true, 4><<<(unsigned)blocks, 256, lds, s>>>(DN_TILE_ARGS); break;
      default: return (int)hipErrorInvalidValue;
    }
  }
#undef DN_TILE_ARGS
  return (int)hipGetLastError();
}

}  // namespace

int launch_lrn_pool(const void* d_in, const MapRun* runs, int32_t n_runs, int32_t C, dn_dtype dt,
                    bool lrn, bool lrn_first, float alpha, float beta, float k, int32_t lrn_n,
                    void* d_out, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (n_runs <= 0) return (int)hipErrorInvalidValue;
  for (int i0 = 0; i0 < n_runs; i0 += MAX_RUNS) {  // one launch per MAX_RUNS runs
    const int nr = std::min(MAX_RUNS, n_runs - i0);
    int st = (int)hipErrorInvalidValue;
    switch (dt) {
      case DN_F32:
        st = run<float>(d_in, runs + i0, nr, C, lrn, lrn_first, alpha, beta, k, lrn_n, d_out, s);
        break;
      case DN_F16:
        st = run<_Float16>(d_in, runs + i0, nr, C, lrn, lrn_first, alpha, beta, k, lrn_n, d_out, s);
        break;
      case DN_BF16:
        st = run<__bf16>(d_in, runs + i0, nr, C, lrn, lrn_first, alpha, beta, k, lrn_n, d_out, s);
        break;
    }
    if (st) return st;
  }
  return 0;
}

}  // namespace dn
