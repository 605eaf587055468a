// Convolution engine for conv1..conv5 of the AlexNet topology (the bulk of the path's work, Sec. 3),
// as implicit GEMMs on gfx950 MFMA: fp16 / bf16 inputs with fp32 accumulation (32x32x16 tiles) or an
// fp32 path (32x32x2 tiles).  Bias and ReLU are applied in the epilogue.
//
// GEMM view: rows = output pixels of a 2-D spatial tile, columns = output channels of one group,
// k = (input channel, kernel tap).  A workgroup stages the input tile with its halo in LDS once per
// chunk of 16 input channels and reuses it for every kernel tap, so each input element is read from
// L2 once per output-channel block instead of once per tap.
//
//  conv1 (11x11, stride 4, 3 channels) reads channel-major planes.  Per input channel its 144 k
//  values cover a 12 x 12 tap square (taps with ky = 11 or kx = 11 carry zero weights): k-step s
//  (16 k) covers rows 4 (s / 3) .. + 3 and columns 4 (s % 3) .. + 3, and each lane's 8 k values are
//  4 consecutive input pixels of one row and the 4 below them, read as two 8-byte LDS loads at
//  offsets that do not depend on the lane.
//  conv2..conv5 (stride 1, R x R, pad (R-1)/2, groups) read channels-last maps; k = (tap, channel),
//  each lane's 8 k values are 8 consecutive channels of one pixel (one 16-byte LDS load).
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace dn {
namespace {

// ------------------------------------------------------------------------------------------------
// Packed weight layout
//   conv1: [96][3][144] in dtype, k = 16 s + 8 h + 4 j + e holds tap ky = 4 (s / 3) + 2 h + j,
//          kx = 4 (s % 3) + e (zero where ky or kx is 11)
//   conv2..5: [M][R*R][C/G] in dtype (tap-major, channels contiguous)
//   conv2..5, 16-bit types, stage-major copy for conv_s1_direct_kernel: per channel block (group g,
//          block of BM output channels) and stage (chunk of 16 input channels, kernel row ky), one
//          contiguous block of R * BM * 2 16-byte pieces, piece (kx BM + m) 2 + p holding input
//          channels 8 (p ^ ((m >> 4) & 1)) .. + 7 of the chunk at tap (ky, kx) of channel m: exactly
//          the order of the LDS weight-row buffer, so each direct load reads 1 KB of contiguous memory
//   biases: fp32 [M]
// ------------------------------------------------------------------------------------------------
constexpr int L_M[5] = {96, 256, 384, 384, 256};
constexpr int L_C[5] = {3, 96, 256, 384, 384};
constexpr int L_R[5] = {11, 5, 3, 3, 3};
constexpr int L_G[5] = {1, 2, 1, 2, 2};
constexpr int K1 = 144;  // conv1 packed k per input channel
__host__ __device__ constexpr int conv1_ky(int k) {
  return 4 * ((k >> 4) / 3) + 2 * ((k >> 3) & 1) + ((k >> 2) & 1);
}
__host__ __device__ constexpr int conv1_kx(int k) { return 4 * ((k >> 4) % 3) + (k & 3); }

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

template <typename T>
__global__ void pack_conv1_kernel(const float* __restrict__ w, T* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 96 * 3 * K1) return;
  const int k = i % K1, mc = i / K1;  // mc = m * 3 + c
  const int ky = conv1_ky(k), kx = conv1_kx(k);
  float v = 0.f;
  if (ky < 11 && kx < 11) v = w[(mc * 11 + ky) * 11 + kx];
  out[i] = from_f32<T>(v);
}

template <typename T>
__global__ void pack_conv_kernel(const float* __restrict__ w, T* __restrict__ out, int M, int Cg,
                                 int RR) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * Cg * RR) return;
  const int c = (int)(i % Cg);
  const int t = (int)((i / Cg) % RR);
  const int m = (int)(i / ((int64_t)Cg * RR));
  out[i] = from_f32<T>(w[((int64_t)m * Cg + c) * RR + t]);
}

// conv1, 16-bit types, for conv1_resident_kernel: the 3 x 11 x 11 taps of an output channel as 99
// units of 4 taps (input channel c, kernel row r, columns 4 cb .. 4 cb + 3, the column 11 of the last
// block zero), unit u = 33 c + 11 cb + r, packed into 25 k-steps of 16: k-step j holds units 4 j .. 4 j
// + 3 (a zero unit past 98), k = 8 h + 4 s + e taking unit 4 j + 2 h + s, column 4 cb + e.  Layout
// [25][96][16] in the order of the kernel's LDS weights: the two 16-byte slots of a channel's k-step
// are swapped for channels 16..31 of every 32-channel group.
constexpr int C1_UNITS = 99, C1_KSTEPS = (C1_UNITS + 3) / 4;
template <typename T>
__global__ void pack_conv1_resident_kernel(const float* __restrict__ w, T* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= C1_KSTEPS * 96 * 16) return;
  const int j = i / (96 * 16), m = (i / 16) % 96, kk = i % 16;
  const int h = (kk / 8) ^ ((m >> 4) & 1), sx = (kk % 8) / 4, e = kk % 4;
  const int u = 4 * j + 2 * h + sx;
  float v = 0.f;
  if (u < C1_UNITS) {
    const int c = u / 33, cb = (u % 33) / 11, r = (u % 33) % 11, kx = 4 * cb + e;
    if (kx < 11) v = w[((m * 3 + c) * 11 + r) * 11 + kx];
  }
  out[i] = from_f32<T>(v);
}

template <typename T>
__global__ void pack_stage_kernel(const float* __restrict__ w, T* __restrict__ out, int Mg, int Cg,
                                  int R, int BM, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int e = (int)(i % 8), p = (int)((i / 8) % 2), m = (int)((i / 16) % BM);
  int64_t r = i / (16 * (int64_t)BM);
  const int kx = (int)(r % R);
  r /= R;
  const int ky = (int)(r % R);
  r /= R;
  const int nchunks = Cg / 16;
  const int chunk = (int)(r % nchunks);
  const int64_t blk = r / nchunks;  // channel block: group * (Mg / BM) + block within the group
  const int mpg = Mg / BM;
  const int g = (int)(blk / mpg), mb = (int)(blk % mpg);
  const int v = p ^ ((m >> 4) & 1);
  const int64_t oc = (int64_t)g * Mg + (int64_t)mb * BM + m;
  const int c = chunk * 16 + v * 8 + e;
  out[i] = from_f32<T>(w[((oc * Cg + c) * R + ky) * R + kx]);
}

__global__ void copy_f32_kernel(const float* __restrict__ a, float* __restrict__ b, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) b[i] = a[i];
}

// ------------------------------------------------------------------------------------------------
// LDS fragment loads
// ------------------------------------------------------------------------------------------------
template <typename T>
__device__ inline typename Mfma<T>::frag lds_frag16(const T* p) {  // 8 consecutive halves, 16 B
  return *(const typename Mfma<T>::frag*)p;
}
template <>
__device__ inline float lds_frag16<float>(const float* p) {
  return *p;
}

// ------------------------------------------------------------------------------------------------
// conv1: 11x11 / stride 4 / no padding, 3 -> 96 channels, channel-major input planes.
// Workgroup: 16 x 16 output pixels x all 96 output channels, 4 waves of 96 channels x 64 pixels.
// ------------------------------------------------------------------------------------------------
template <typename T>
struct Conv1Cfg {
  static_assert(std::is_same<T, float>::value, "16-bit storage uses the direct or persistent kernel");
  static constexpr int TH = 16, TW = 16;
  static constexpr int HR = 72;  // halo rows / cols (4*15+12)
  static constexpr int HS = 72;  // halo row stride
  static constexpr int WS = K1 + 1;
};

// ksplit > 1: as conv_s1_kernel's split, over the three input channels.
template <typename T>
__global__ __launch_bounds__(256) void conv1_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                    const T* __restrict__ wp,
                                                    const float* __restrict__ bias, KRuns runs,
                                                    int ksplit, int base, float* __restrict__ part,
                                                    int64_t part_slice) {
  using C = Conv1Cfg<T>;
  using Op = Mfma<T>;
  __shared__ T s_in[C::HR * C::HS];
  __shared__ T s_w[96 * C::WS];

  int bid = blockIdx.x;
  const int copy = bid / base;  // split copy: input channels [3 copy / ksplit, 3 (copy + 1) / ksplit)
  bid -= copy * base;
  const KRun& rn = runs.r[run_of(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, tiles_x = rn.tiles_x, tiles_y = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  const int P = rn.pitch, Ho = rn.Ho, Wo = rn.Wo;
  const int tx = bid % tiles_x;
  bid /= tiles_x;
  const int ty = bid % tiles_y;
  const int plane = bid / tiles_y;
  const int oy0 = ty * C::TH, ox0 = tx * C::TW;
  const int iy0 = oy0 * 4, ix0 = ox0 * 4;
  const T* src = in + plane * in_stride;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  int prow[2], pcol[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int idx = wave * 64 + t * 32 + l32;
    prow[t] = idx / C::TW;
    pcol[t] = idx % C::TW;
  }
  f32x16 acc[3][2];
#pragma unroll
  for (int a = 0; a < 3; ++a)
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[a][t] = f32x16{};

  for (int c = copy * 3 / ksplit; c < (copy + 1) * 3 / ksplit; ++c) {
    __syncthreads();
    const T* sc = src + (int64_t)c * H * P;
    for (int e = threadIdx.x; e < C::HR * C::HR; e += 256) {
      const int hy = e / C::HR, hx = e % C::HR;
      const int iy = iy0 + hy, ix = ix0 + hx;
      T v = from_f32<T>(0.f);
      if (iy < H && ix < W) v = sc[(int64_t)iy * P + ix];
      s_in[hy * C::HS + hx] = v;
    }
    for (int e = threadIdx.x; e < 96 * K1; e += 256) {
      const int m = e / K1, k = e % K1;
      s_w[m * C::WS + k] = wp[(m * 3 + c) * K1 + k];
    }
    __syncthreads();
#pragma unroll 3
    for (int ks = 0; ks < K1 / Op::KS; ++ks) {
      typename Op::frag a[2], b[3];
      const int k = ks * 2 + half, ky = conv1_ky(k), kx = conv1_kx(k);
#pragma unroll
      for (int t = 0; t < 2; ++t) a[t] = s_in[(4 * prow[t] + ky) * C::HS + 4 * pcol[t] + kx];
#pragma unroll
      for (int mt = 0; mt < 3; ++mt) b[mt] = s_w[(mt * 32 + l32) * C::WS + k];
#pragma unroll
      for (int mt = 0; mt < 3; ++mt)
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[mt][t] = Op::mma(a[t], b[mt], acc[mt][t]);
    }
  }

  if (ksplit > 1) {  // raw partial sums of this split
    float* pd = part + copy * part_slice + rn.out_off + plane * out_stride;
#pragma unroll
    for (int mt = 0; mt < 3; ++mt)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = 8 * (r >> 2) + 4 * half + (r & 3);
          const int idx = wave * 64 + t * 32 + i;
          const int oy = oy0 + idx / C::TW, ox = ox0 + idx % C::TW;
          if (oy < Ho && ox < Wo) pd[((int64_t)oy * Wo + ox) * 96 + mt * 32 + l32] = acc[mt][t][r];
        }
    return;
  }
  T* dst = out + plane * out_stride;
#pragma unroll
  for (int mt = 0; mt < 3; ++mt) {
    const int m = mt * 32 + l32;
    const float bv = bias[m];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 8 * (r >> 2) + 4 * half + (r & 3);
        const int idx = wave * 64 + t * 32 + i;
        const int oy = oy0 + idx / C::TW, ox = ox0 + idx % C::TW;
        if (oy < Ho && ox < Wo)
          dst[((int64_t)oy * Wo + ox) * 96 + m] = from_f32<T>(fmaxf(acc[mt][t][r] + bv, 0.f));
      }
  }
}

// ------------------------------------------------------------------------------------------------
// conv1 for 16-bit storage: persistent workgroups (one per CU).  All 96 x 432 packed weights stay in
// LDS for the whole launch; each workgroup walks output tiles of 16 x 16 pixels, and while it
// computes one tile the next tile's 3 x 72 x 72 input halo is already loading into registers (16-byte
// loads of plane rows), to be written to the other LDS halo buffer after the tile's MFMAs.
// Waves: 4 x (96 channels x 64 pixels); A = weights, B = pixels, so each lane stores 4 consecutive
// output channels of one pixel per store.
// ------------------------------------------------------------------------------------------------
template <typename T>
struct Conv1P {
  static constexpr int TH = 16, TW = 16, HR = 72, HS = 80;
  static constexpr int KT = 3 * K1, WS = KT + 8;
  static constexpr int HV = 3 * HR * (HR / 8);  // 16-byte vectors per halo
  static constexpr int HPER = (HV + 255) / 256;
  static constexpr size_t LDS = sizeof(T) * (96 * WS + 2 * 3 * HR * HS);
};

template <typename T>
__global__ __launch_bounds__(256) void conv1_persistent_kernel(
    const T* __restrict__ in, T* __restrict__ out, const T* __restrict__ wp,
    const float* __restrict__ bias, KRuns runs, int ntiles) {
  using P = Conv1P<T>;
  using Op = Mfma<T>;
  typedef T vec8 __attribute__((ext_vector_type(8)));
  typedef T out4_t __attribute__((ext_vector_type(4)));
  __shared__ __align__(16) T s_w[96 * P::WS];
  __shared__ __align__(16) T s_in[2][3 * P::HR * P::HS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  for (int e = tid; e < 96 * (P::KT / 8); e += 256) {
    const int m = e / (P::KT / 8), v = e % (P::KT / 8);
    *(vec8*)(s_w + m * P::WS + v * 8) = *(const vec8*)(wp + (int64_t)m * P::KT + v * 8);
  }
  int lpix[2];  // LDS offset of this lane's pixel (row 4 * prow, column 4 * pcol) per pixel tile
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int idx = wave * 64 + t * 32 + l32;
    lpix[t] = 4 * (idx / P::TW) * P::HS + 4 * (idx % P::TW);
  }
  vec8 hreg[P::HPER];
  auto load_halo = [&](int t) {
    const KRun& rn = runs.r[run_of(runs, t)];
    const int H = rn.H, W = rn.W, pitch = rn.pitch, tl = t - rn.first;
    const bool vec_ok = (W % 8) == 0 && (pitch % 8) == 0;
    const int tx = tl % rn.tiles_x, r = tl / rn.tiles_x, ty = r % rn.tiles_y, plane = r / rn.tiles_y;
    const T* src = in + rn.in_off + plane * rn.in_stride;
    const int iy0 = 4 * P::TH * ty, ix0 = 4 * P::TW * tx;
#pragma unroll
    for (int i = 0; i < P::HPER; ++i) {
      const int e = tid + i * 256;
      vec8 val = vec8{};
      if (e < P::HV) {
        const int c = e / (P::HR * 9), rem = e % (P::HR * 9);
        const int iy = iy0 + rem / 9, ix = ix0 + 8 * (rem % 9);
        if (iy < H) {
          const T* rowp = src + ((int64_t)c * H + iy) * pitch;
          if (vec_ok && ix + 8 <= W) {
            val = *(const vec8*)(rowp + ix);
          } else {
#pragma unroll
            for (int q = 0; q < 8; ++q)
              if (ix + q < W) val[q] = rowp[ix + q];
          }
        }
      }
      hreg[i] = val;
    }
  };
  auto store_halo = [&](int buf) {
#pragma unroll
    for (int i = 0; i < P::HPER; ++i) {
      const int e = tid + i * 256;
      if (e < P::HV) {
        const int c = e / (P::HR * 9), rem = e % (P::HR * 9);
        *(vec8*)(s_in[buf] + (c * P::HR + rem / 9) * P::HS + 8 * (rem % 9)) = hreg[i];
      }
    }
  };

  int t = blockIdx.x;
  if (t < ntiles) {
    load_halo(t);
    store_halo(0);
  }
  __syncthreads();
  int buf = 0;
  for (; t < ntiles; t += gridDim.x) {
    const int tn = t + gridDim.x;
    if (tn < ntiles) load_halo(tn);
    f32x16 acc[3][2];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
    const T* hs = s_in[buf];
#pragma unroll 1
    for (int c = 0; c < 3; ++c) {
#pragma unroll
      for (int ks = 0; ks < K1 / 16; ++ks) {
        // k-step ks of channel c: rows ky, ky + 1 (ky = 4 (ks / 3) + 2 half), columns 4 (ks % 3) + 0..3
        const int o0 = (c * P::HR + 4 * (ks / 3) + 2 * half) * P::HS + 4 * (ks % 3);
        typename Op::frag x[2], w[3];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const typename Op::half_frag lo = *(const typename Op::half_frag*)(hs + lpix[b] + o0);
          const typename Op::half_frag hi = *(const typename Op::half_frag*)(hs + lpix[b] + o0 + P::HS);
          x[b] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
#pragma unroll
        for (int mt = 0; mt < 3; ++mt)
          w[mt] = *(const typename Op::frag*)(s_w + (mt * 32 + l32) * P::WS + c * K1 + ks * 16 + half * 8);
#pragma unroll
        for (int mt = 0; mt < 3; ++mt)
#pragma unroll
          for (int b = 0; b < 2; ++b) acc[mt][b] = Op::mma(w[mt], x[b], acc[mt][b]);
      }
    }
    if (tn < ntiles) store_halo(buf ^ 1);
    // epilogue: bias + ReLU, 4 consecutive channels per store
    const KRun& rn = runs.r[run_of(runs, t)];
    const int Ho = rn.Ho, Wo = rn.Wo, tl = t - rn.first;
    const int tx = tl % rn.tiles_x, r = tl / rn.tiles_x, ty = r % rn.tiles_y, plane = r / rn.tiles_y;
    T* dst = out + rn.out_off + plane * rn.out_stride;
#pragma unroll
    for (int mt = 0; mt < 3; ++mt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m = mt * 32 + 8 * q + 4 * half;
        const f32x4 bv = *(const f32x4*)(bias + m);
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int idx = wave * 64 + b * 32 + l32;
          const int oy = ty * P::TH + idx / P::TW, ox = tx * P::TW + idx % P::TW;
          if (oy < Ho && ox < Wo) {
            out4_t v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = from_f32<T>(fmaxf(acc[mt][b][4 * q + e] + bv[e], 0.f));
            *(out4_t*)(dst + ((int64_t)oy * Wo + ox) * 96 + m) = v;
          }
        }
      }
    __syncthreads();
    buf ^= 1;
  }
}

// Compute units of the device current at the first call (256 if the query fails), queried once;
// the initialisation is thread-safe.
int device_cu_count() {
  static const int n = [] {
    int dev = 0, v = 0;
    const bool ok = hipGetDevice(&dev) == hipSuccess &&
                    hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess;
    return ok && v > 0 ? v : 256;
  }();
  return n;
}

// ------------------------------------------------------------------------------------------------
// Stride-1 R x R conv with zero padding (R-1)/2, grouped, channels-last.
// Workgroup: TH x TW = 16 x 16 output pixels x BM output channels of one group.  Waves: BM/(32 TM)
// along channels x 2 along pixels; each wave owns 32 TM channels x 128 pixels (TM x 4 MFMA tiles).  The MFMA
// A operand is the weights and B the pixels, so each lane's accumulator holds 4 consecutive output
// channels of one pixel per register group and the epilogue stores 4 channels at a time.
// Pipeline: a stage is (chunk of 16 input channels, kernel row ky).  LDS holds two halo buffers
// ((TH+R-1) x (TW+R-1) x 16 channels, one per chunk) and two weight-row buffers (R taps x BM x 16).
// While a stage computes from LDS, the next stage's weight row (and, during a chunk's first row, the
// next chunk's halo) is already in flight into registers; it is written to the other buffers after
// the stage's MFMAs, and one barrier per stage publishes it.
// ------------------------------------------------------------------------------------------------
// Slots (16 bytes) that collide modulo 512 bytes when the 32 lanes of a half-wave read pixels
// (r, c), r < 16, c < 2, of a halo whose rows are rs slots apart (two slots per pixel).
constexpr int colpair_collisions(int rs) {
  int n = 0;
  for (int a = 0; a < 32; ++a)
    for (int b = 0; b < a; ++b)
      if ((((a & 15) * rs + 2 * (a >> 4)) - ((b & 15) * rs + 2 * (b >> 4))) % 32 == 0) {
        ++n;
        break;
      }
  return n;
}
// Padding slots per 16-bit halo row: odd (so the two rows of a 2 x 16 MFMA tile fall on slots of
// opposite parity), and of 1 and 3 the one with fewer collisions for 16 x 2 MFMA tiles.
constexpr int halo_row_pad(int hw) {
  return colpair_collisions(2 * hw + 3) < colpair_collisions(2 * hw + 1) ? 3 : 1;
}

template <typename T, int R, int BM, int TM, int TS, int TN_ = 4>
struct ConvCfg {
  // Tile of TH x TW output pixels, TS = 100 TH + TW (TW 16 or 32, TH TW a multiple of 256) for 16-bit
  // storage; fp32 uses 16 x 16.
  static constexpr bool F32_ = std::is_same<T, float>::value;
  static constexpr int TH = F32_ ? 16 : TS / 100, TW = F32_ ? 16 : TS % 100, CC = 16;
  static_assert((TW == 16 || TW == 32) && TH % 2 == 0 && (TH * TW) % 256 == 0, "tile shape");
  static constexpr int TN = TN_;                   // 32-pixel MFMA tiles per wave (32 TN pixels)
  static constexpr int HH = TH + R - 1, HW = TW + R - 1;
  static constexpr bool F32 = std::is_same<T, float>::value;
  static constexpr int WM = BM / (32 * TM), WN = (TH * TW) / (32 * TN);
  static constexpr int NT = 64 * WM * WN;
  static constexpr int VEC = 16 / sizeof(T);  // elements per 16-byte global load
  static constexpr int VPP = CC / VEC;
  static constexpr int HALO_V = HH * HW * VPP, HALO_PER = (HALO_V + NT - 1) / NT;
  static constexpr int W_V = R * BM * VPP, W_PER = (W_V + NT - 1) / NT;
  static_assert(WM * 32 * TM == BM, "channel block must be whole wave tiles");
  // LDS layout.  16-bit types: a pixel (or an output channel's weight row) is 32 bytes, two 16-byte
  // slots.  The 32 lanes of a half-wave read 16 bytes each and must hit distinct slots modulo 512
  // bytes: a halo row is padded by an odd number of slots (RP), so the two tile rows a half-wave
  // reads land on slots of opposite parity; the weight rows of channels 16..31 of a 32-channel group
  // swap their two slots.  fp32: a pixel or channel row is CC + 1 floats.
  static constexpr int PS = F32 ? CC + 1 : CC;          // pixel stride (elements)
  static constexpr int RP = F32 ? 0 : halo_row_pad(HW);  // halo row padding (16-byte slots)
  static constexpr int RSS = 2 * HW + RP;                // 16-bit halo row stride (slots)
  static constexpr int RS = F32 ? HW * PS : HW * PS + 8 * RP;  // halo row stride (elements)
  static constexpr int HALO_E = HH * RS, W_E = R * BM * PS;
  static constexpr int STAGE_E = F32 ? 0 : WM * WN * 32 * TN * 64;  // epilogue staging
  static constexpr int LDS_E = (2 * HALO_E + 2 * W_E) > STAGE_E ? (2 * HALO_E + 2 * W_E) : STAGE_E;
  __device__ static inline int halo_off(int hy, int hx, int v) { return hy * RS + hx * PS + v * VEC; }
  // Tile pixel of index idx: each 32-pixel MFMA tile is 2 rows x 16 columns (the two rows a half-wave
  // reads then fall on LDS slots of opposite parity); with 32-column tiles, MFMA tiles 2 p and 2 p + 1
  // are the left and right halves of row pair p.
  __device__ static inline int pix_row(int idx) { return 2 * ((idx >> 5) / (TW / 16)) + ((idx >> 4) & 1); }
  __device__ static inline int pix_col(int idx) { return 16 * ((idx >> 5) % (TW / 16)) + (idx & 15); }
  __device__ static inline int w_off(int kx, int m, int v) {
    return (kx * BM + m) * PS + (F32 ? v * VEC : ((v ^ ((m >> 4) & 1)) * VEC));
  }
};

template <typename T, int BM, int TM, int TS, int TN = 4>
constexpr int conv_threads() {
  return 64 * (BM / (32 * TM)) * (std::is_same<T, float>::value ? 256 : (TS / 100) * (TS % 100)) / (32 * TN);
}

// ksplit > 1 (fp32 launches too small to fill the chip): the launch is ksplit copies of its base
// workgroups; copy ks runs the input-channel chunks [ks nchunks / ksplit, (ks + 1) nchunks / ksplit)
// and writes its raw sums (no bias, no ReLU) to part + ks part_slice at the output's element offsets;
// split_reduce_kernel then adds the copies in order.
// (fp32 instances run one wave per SIMD whatever the configuration asks: their registers need it)
template <typename T, int OCC>
constexpr int conv_s1_occ() {
  return std::is_same<T, float>::value ? 1 : OCC;
}

template <typename T, int R, int BM, int TM, int OCC, int TS>
__global__ __launch_bounds__((conv_threads<T, BM, TM, TS>()), (conv_s1_occ<T, OCC>())) void conv_s1_kernel(
    const T* __restrict__ in, T* __restrict__ out, const T* __restrict__ wp,
    const float* __restrict__ bias, KRuns runs, int C, int Cg, int M, int Mg, int mblocks, int ksplit,
    int base, float* __restrict__ part, int64_t part_slice) {
  using Cf = ConvCfg<T, R, BM, TM, TS>;
  using Op = Mfma<T>;
  constexpr int pad = (R - 1) / 2;
  constexpr int VEC = Cf::VEC, VPP = Cf::VPP, NT = Cf::NT, TN = Cf::TN;
  typedef T vec_t __attribute__((ext_vector_type(VEC)));
  typedef T out4_t __attribute__((ext_vector_type(4)));
  constexpr int HALO_E = Cf::HALO_E, W_E = Cf::W_E;
  __shared__ __align__(16) T s_mem[Cf::LDS_E];
  auto halo_buf = [&](int b) { return s_mem + b * HALO_E; };
  auto wrow_buf = [&](int b) { return s_mem + 2 * HALO_E + b * W_E; };

  // XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs, so the i-th block of XCD
  // x takes logical index x * (blocks per XCD) + i; consecutive logical blocks (the channel blocks of
  // one tile first, then neighbouring tiles) then share that XCD's L2.
  const int nb = gridDim.x, xcd = blockIdx.x % 8, per = nb / 8, rem = nb % 8;
  int bid = xcd * per + min(xcd, rem) + blockIdx.x / 8;
  const int ks = bid / base;
  bid -= ks * base;
  const KRun& rn = runs.r[run_of(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, tiles_x = rn.tiles_x, tiles_y = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  const int mb = bid % mblocks;
  bid /= mblocks;
  const int tx = bid % tiles_x;
  bid /= tiles_x;
  const int ty = bid % tiles_y;
  const int plane = bid / tiles_y;
  const int mpg = Mg / BM;
  const int g = mb / mpg, m0 = (mb % mpg) * BM;
  const int oy0 = ty * Cf::TH, ox0 = tx * Cf::TW;
  const T* src = in + plane * in_stride + g * Cg;
  const T* wg = wp + ((int64_t)g * Mg + m0) * R * R * Cg;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % Cf::WM, wn = wave / Cf::WM;
  const int half = lane >> 5, l32 = lane & 31;
  int pix[TN];  // LDS element offset of this lane's pixel (tap 0, 0) in each pixel tile
#pragma unroll
  for (int t = 0; t < TN; ++t) {
    const int idx = wn * 32 * TN + t * 32 + l32;
    pix[t] = Cf::halo_off(Cf::pix_row(idx), Cf::pix_col(idx), 0);
  }
  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int t = 0; t < TN; ++t) acc[a][t] = f32x16{};

  vec_t hreg[Cf::HALO_PER], wreg[Cf::W_PER];
  auto load_halo = [&](int c0) {
#pragma unroll
    for (int i = 0; i < Cf::HALO_PER; ++i) {
      const int e = tid + i * NT;
      vec_t val = vec_t{};
      if (e < Cf::HALO_V) {
        const int v = e % VPP, p = e / VPP;
        const int iy = oy0 - pad + p / Cf::HW, ix = ox0 - pad + p % Cf::HW;
        if (iy >= 0 && iy < H && ix >= 0 && ix < W)
          val = *(const vec_t*)(src + ((int64_t)iy * W + ix) * C + c0 + v * VEC);
      }
      hreg[i] = val;
    }
  };
  auto store_halo = [&](int buf) {
#pragma unroll
    for (int i = 0; i < Cf::HALO_PER; ++i) {
      const int e = tid + i * NT;
      if (e < Cf::HALO_V) {
        const int p = e / VPP;
        T* d = halo_buf(buf) + Cf::halo_off(p / Cf::HW, p % Cf::HW, e % VPP);
        if constexpr (Cf::F32) {
#pragma unroll
          for (int q = 0; q < VEC; ++q) d[q] = hreg[i][q];
        } else {
          *(vec_t*)d = hreg[i];
        }
      }
    }
  };
  auto load_w = [&](int c0, int ky) {
#pragma unroll
    for (int i = 0; i < Cf::W_PER; ++i) {
      const int e = tid + i * NT;
      vec_t val = vec_t{};
      if (e < Cf::W_V) {
        const int v = e % VPP, t = e / VPP;
        const int m = t % BM, kx = t / BM;
        val = *(const vec_t*)(wg + ((int64_t)m * R * R + ky * R + kx) * Cg + c0 + v * VEC);
      }
      wreg[i] = val;
    }
  };
  auto store_w = [&](int buf) {
#pragma unroll
    for (int i = 0; i < Cf::W_PER; ++i) {
      const int e = tid + i * NT;
      if (e < Cf::W_V) {
        const int v = e % VPP, t = e / VPP;
        const int m = t % BM, kx = t / BM;
        T* d = wrow_buf(buf) + Cf::w_off(kx, m, v);
        if constexpr (Cf::F32) {
#pragma unroll
          for (int q = 0; q < VEC; ++q) d[q] = wreg[i][q];
        } else {
          *(vec_t*)d = wreg[i];
        }
      }
    }
  };
  auto compute = [&](int hb, int wb, int ky) {
    const T* hs = halo_buf(hb);
    const T* ws = wrow_buf(wb);
#pragma unroll
    for (int kx = 0; kx < R; ++kx) {
#pragma unroll
      for (int kk = 0; kk < Cf::CC / Op::KS; ++kk) {
        const int koff = kk * Op::KS + half * Op::KPL;
        typename Op::frag x[TN], w[TM];
        // k offset of this lane: element koff of the 16-channel chunk (16-bit: slot `half`)
#pragma unroll
        for (int t = 0; t < TN; ++t)
          x[t] = lds_frag16<T>(hs + pix[t] + ky * Cf::RS + kx * Cf::PS + koff);
#pragma unroll
        for (int mt = 0; mt < TM; ++mt) {
          const int m = wm * 32 * TM + mt * 32 + l32;
          if constexpr (Cf::F32)
            w[mt] = lds_frag16<T>(ws + Cf::w_off(kx, m, 0) + koff);
          else
            w[mt] = lds_frag16<T>(ws + Cf::w_off(kx, m, half));
        }
#pragma unroll
        for (int mt = 0; mt < TM; ++mt)
#pragma unroll
          for (int t = 0; t < TN; ++t) acc[mt][t] = Op::mma(w[mt], x[t], acc[mt][t]);
      }
    }
  };

  // this workgroup's chunks [c_lo, c_hi) (all of them without a split): stages c_lo R .. c_hi R - 1
  const int nchunks = Cg / Cf::CC;
  const int c_lo = ks * nchunks / ksplit, c_hi = (ks + 1) * nchunks / ksplit;
  const int st0 = c_lo * R, st1 = c_hi * R;
  load_halo(c_lo * Cf::CC);
  load_w(c_lo * Cf::CC, 0);
  store_halo(c_lo & 1);
  store_w(st0 & 1);
  __syncthreads();
  for (int st = st0; st < st1; ++st) {
    const int chunk = st / R, ky = st - chunk * R;
    const bool more = st + 1 < st1, next_chunk = chunk + 1 < c_hi;
    if (more) load_w(((st + 1) / R) * Cf::CC, (st + 1) % R);
    if (ky == 0 && next_chunk) load_halo((chunk + 1) * Cf::CC);
    compute(chunk & 1, st & 1, ky);
    if (more) store_w((st + 1) & 1);
    if (ky == R - 1 && next_chunk) store_halo((chunk + 1) & 1);
    __syncthreads();
  }

  if constexpr (Cf::F32) {
    if (ksplit > 1) {  // raw partial sums of this split
      float* pd = part + ks * part_slice + rn.out_off + plane * out_stride;
#pragma unroll
      for (int mt = 0; mt < TM; ++mt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = g * Mg + m0 + wm * 32 * TM + mt * 32 + 8 * q + 4 * half;
#pragma unroll
          for (int t = 0; t < TN; ++t) {
            const int idx = wn * 32 * TN + t * 32 + l32;
            const int oy = oy0 + Cf::pix_row(idx), ox = ox0 + Cf::pix_col(idx);
            if (oy < H && ox < W) {
              f32x4 r;
#pragma unroll
              for (int e = 0; e < 4; ++e) r[e] = acc[mt][t][4 * q + e];
              *(f32x4*)(pd + ((int64_t)oy * W + ox) * M + m) = r;
            }
          }
        }
      return;
    }
  }

  // Epilogue: D[m][pixel]; register group q of MFMA tile mt holds channels 32 mt + 8 q + 4 half + 0..3
  // of pixel l32.
  T* dst = out + plane * out_stride;
  if constexpr (!Cf::F32 && TM == 2) {
    // Stage each wave's 128 pixels x 64 channels (one 128-byte line per pixel) in LDS, 16-byte chunks
    // XOR-swizzled by the pixel index, then write whole lines: 8 lanes per pixel, 16 bytes each.
    typedef T vec8_t __attribute__((ext_vector_type(8)));
    static_assert(Cf::STAGE_E <= Cf::LDS_E, "staging must fit in LDS");
    T* stg = s_mem + wave * (32 * TN * 64);
#pragma unroll
    for (int mt = 0; mt < TM; ++mt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = 4 * mt + q;
        const f32x4 bv = *(const f32x4*)(bias + g * Mg + m0 + wm * 64 + 8 * j + 4 * half);
#pragma unroll
        for (int t = 0; t < TN; ++t) {
          const int p = t * 32 + l32;
          out4_t r;
#pragma unroll
          for (int e = 0; e < 4; ++e) r[e] = from_f32<T>(fmaxf(acc[mt][t][4 * q + e] + bv[e], 0.f));
          const int key = (p & 7) ^ ((p >> 3) & 3);
          *(out4_t*)(stg + p * 64 + ((j ^ key) * 8) + 4 * half) = r;
        }
      }
    __syncthreads();
    const int j = lane & 7;
#pragma unroll
    for (int it = 0; it < (32 * TN) / 8; ++it) {
      const int p = it * 8 + (lane >> 3);
      const int key = (p & 7) ^ ((p >> 3) & 3);
      const vec8_t v = *(const vec8_t*)(stg + p * 64 + ((j ^ key) * 8));
      const int idx = wn * 32 * TN + p;
      const int oy = oy0 + Cf::pix_row(idx), ox = ox0 + Cf::pix_col(idx);
      if (oy < H && ox < W)
        *(vec8_t*)(dst + ((int64_t)oy * W + ox) * M + g * Mg + m0 + wm * 64 + 8 * j) = v;
    }
  } else {
#pragma unroll
    for (int mt = 0; mt < TM; ++mt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m = g * Mg + m0 + wm * 32 * TM + mt * 32 + 8 * q + 4 * half;
        const f32x4 bv = *(const f32x4*)(bias + m);
#pragma unroll
        for (int t = 0; t < TN; ++t) {
          const int idx = wn * 32 * TN + t * 32 + l32;
          const int oy = oy0 + Cf::pix_row(idx), ox = ox0 + Cf::pix_col(idx);
          if (oy < H && ox < W) {
            out4_t r;
#pragma unroll
            for (int e = 0; e < 4; ++e) r[e] = from_f32<T>(fmaxf(acc[mt][t][4 * q + e] + bv[e], 0.f));
            *(out4_t*)(dst + ((int64_t)oy * W + ox) * M + m) = r;
          }
        }
      }
  }
}

// Sum of the ksplit partial copies of a split fp32 conv launch, in copy order, plus bias, then ReLU:
// run r has tiles_x workgroups of 256 four-channel groups per plane (Ho x Wo x M outputs).
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part,
                                                           int64_t part_slice, int ksplit,
                                                           const float* __restrict__ bias,
                                                           float* __restrict__ out, KRuns runs, int M) {
  int bid = blockIdx.x;
  const KRun& rn = runs.r[run_of(runs, bid)];
  bid -= rn.first;
  const int plane = bid / rn.tiles_x, v = (bid % rn.tiles_x) * 256 + (int)threadIdx.x;
  if ((int64_t)v * 4 >= (int64_t)rn.Ho * rn.Wo * M) return;
  const int64_t o = rn.out_off + plane * rn.out_stride + (int64_t)v * 4;
  f32x4 acc = *(const f32x4*)(part + o);
  for (int k = 1; k < ksplit; ++k) {
    const f32x4 p = *(const f32x4*)(part + k * part_slice + o);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] += p[e];
  }
  const f32x4 b = *(const f32x4*)(bias + (v * 4) % M);
#pragma unroll
  for (int e = 0; e < 4; ++e) acc[e] = fmaxf(acc[e] + b[e], 0.f);
  *(f32x4*)(out + o) = acc;
}

// ------------------------------------------------------------------------------------------------
// Stride-1 conv for 16-bit storage with direct global->LDS loads.  Same tiling, stages, LDS layout and
// epilogue as conv_s1_kernel, but every stage buffer is filled by buffer_load_dwordx4 ... lds: one
// wave instruction writes 64 consecutive 16-byte LDS slots, each lane choosing the global address of
// its slot (padding slots and halo pixels outside the map use an offset past the buffer's end, which
// the hardware returns as zeros).  No registers hold staged data and no LDS store instructions are
// issued; a stage's loads are waited for (vmcnt) just before the barrier that publishes them.
// ------------------------------------------------------------------------------------------------
template <int BYTES>
struct Pieces {  // 1 KB LDS pieces, rounded up to a whole number per wave
  static constexpr int count(int slots, int waves) { return ((slots + 63) / 64 + waves - 1) / waves; }
};

// Wait until every vector-memory access of this wave has completed (vmcnt 0; other counters left
// free), as an instruction the compiler's own wait bookkeeping sees.
__device__ inline void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// Wait until at most N (< 16) vector-memory accesses of this wave are outstanding.
template <int N>
__device__ inline void wait_vmem_but() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// Output stores are non-temporal: the next layer reads a batch's maps only after this launch has
// written all of them, so they need not stay in the caches next to this layer's inputs.
template <typename V>
__device__ inline void store_out(const V& v, V* p) {
  __builtin_nontemporal_store(v, p);
}

__device__ inline void lds_direct16(__amdgpu_buffer_rsrc_t rsrc, void* lds_piece, uint32_t voff,
                                    uint32_t soff = 0) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)lds_piece,
                                           16, voff, soff, 0, 0);
}

// BMP: the channel block the stage-major weight copy is cut in (a multiple of BM); a workgroup's BM
// channels are a sub-block of one such block.  TN_: 32-pixel MFMA tiles per wave.  MULTI: the launch
// holds several runs (else run 0 only).
template <typename T, int R, int BM, int TM, int OCC, int TS, int BMP, int TN_, bool MULTI>
__global__ __launch_bounds__((conv_threads<T, BM, TM, TS, TN_>()), OCC) void conv_s1_direct_kernel(
    const T* __restrict__ in, T* __restrict__ out, const T* __restrict__ wp,
    const float* __restrict__ bias, KRuns runs, int C, int Cg, int M, int Mg, int mblocks) {
  using Cf = ConvCfg<T, R, BM, TM, TS, TN_>;
  using Op = Mfma<T>;
  static_assert(!Cf::F32 && (TM == 2 || TM == 3), "direct-load path is for 16-bit storage");
  constexpr int pad = (R - 1) / 2;
  constexpr int TN = Cf::TN, NW = Cf::WM * Cf::WN;
  static_assert(BMP % BM == 0, "a channel block is a sub-block of the weight copy's block");
  constexpr int HSLOTS = Cf::HH * Cf::RSS, WSLOTS = R * BM * 2, WSLOTS_P = R * BMP * 2;
  constexpr int DH = Pieces<16>::count(HSLOTS, NW), DW = Pieces<16>::count(WSLOTS, NW);
  constexpr int HALO_E = DH * NW * 512, W_E = DW * NW * 512;  // elements (2 bytes)
  constexpr int PIPE_E = 2 * HALO_E + 2 * W_E;
  // TM = 2: the epilogue stages 16 KB per wave; when that would set the LDS size, it runs in two
  // rounds of half the waves each.  TM = 3 stages 32 pixels per wave at a time (below).
  constexpr int ROUNDS = (TM == 2 && Cf::STAGE_E > PIPE_E && NW % 2 == 0) ? 2 : 1;
  constexpr int STG_E = TM == 2 ? Cf::STAGE_E / ROUNDS : 0;
  constexpr int LDS_E = PIPE_E > STG_E ? PIPE_E : STG_E;
  typedef T out4_t __attribute__((ext_vector_type(4)));
  __shared__ __align__(1024) T s_mem[LDS_E];
  auto halo_buf = [&](int b) { return s_mem + b * HALO_E; };
  auto wrow_buf = [&](int b) { return s_mem + 2 * HALO_E + b * W_E; };

  const int nb = gridDim.x, xcd = blockIdx.x % 8, per = nb / 8, rem = nb % 8;
  int bid = xcd * per + min(xcd, rem) + blockIdx.x / 8;
  const KRun& rn = runs.r[run_of<MULTI>(runs, bid)];
  bid -= rn.first;
  const int H = rn.H, W = rn.W, tiles_x = rn.tiles_x, tiles_y = rn.tiles_y;
  const int64_t in_stride = rn.in_stride, out_stride = rn.out_stride;
  in += rn.in_off;
  out += rn.out_off;
  const int mb = bid % mblocks;
  bid /= mblocks;
  const int tx = bid % tiles_x;
  bid /= tiles_x;
  const int ty = bid % tiles_y;
  const int plane = bid / tiles_y;
  const int mpg = Mg / BM;
  const int g = mb / mpg, m0 = (mb % mpg) * BM;
  const int oy0 = ty * Cf::TH, ox0 = tx * Cf::TW;
  const T* src = in + plane * in_stride + g * Cg;
  // The stage-major weights of the enclosing BMP-channel block: per stage one contiguous block of
  // WSLOTS_P 16-byte pieces, [kernel column][BMP channels][2 slots]; this workgroup's channels start
  // msub channels into it.
  const int mbp = g * (Mg / BMP) + m0 / BMP, msub = m0 % BMP;
  const T* wg = wp + (int64_t)mbp * (Cg / Cf::CC) * R * (WSLOTS_P * 8);
  const __amdgpu_buffer_rsrc_t rsrc_in =
      uniform_rsrc(src, (uint32_t)(((int64_t)H * W * C - g * Cg) * sizeof(T)));
  const __amdgpu_buffer_rsrc_t rsrc_w = uniform_rsrc(wg, (uint32_t)((Cg / Cf::CC) * R * WSLOTS_P * 16));
  constexpr uint32_t OOB = 0x80000000u;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % Cf::WM, wn = wave / Cf::WM;
  const int half = lane >> 5, l32 = lane & 31;
  // MFMA pixel tile t of wave wn is the tile's (t WN + wn)-th 32-pixel tile: the waves along pixels
  // take the tiles in turn, so a partly filled bottom band splits its rows over them.
  auto gtile = [&](int t) { return t * Cf::WN + wn; };
  // Two layouts of the tile's pixels over the MFMA tiles.  Row layout: each MFMA tile is 2 rows x 16
  // columns (pix_row / pix_col).  Column-pair layout, for a tile cut by the map's right edge (cv < TW
  // columns in the map): MFMA tile m is the 16 rows of columns 2 m and 2 m + 1 (lane l: row l % 16,
  // column 2 m + l / 16), so only ceil(cv / 2) MFMA tiles are computed instead of all TW / 16 column
  // blocks.  A tile takes the layout with fewer MFMA tiles holding a map pixel (ties: rows).
  const int cv = min(Cf::TW, W - ox0), rv = min(Cf::TH, H - oy0);
  const int n_rows = ((rv + 1) / 2) * (Cf::TW / 16), n_cols = (cv + 1) / 2;
  const bool colpair = Cf::TH == 16 && n_cols < n_rows;
  const int n_mt = colpair ? n_cols : n_rows;  // MFMA tiles holding a map pixel: tiles 0 .. n_mt - 1
  auto out_row = [&](int idx) { return colpair ? (idx & 15) : Cf::pix_row(idx); };
  auto out_col = [&](int idx) { return colpair ? 2 * (idx >> 5) + ((idx >> 4) & 1) : Cf::pix_col(idx); };
  // LDS offset of this lane's pixel in MFMA pixel tile t: pix0 + t DPIX (tile t of the wave lies
  // t WN tiles further: 2 t WN / (TW / 16) halo rows down, or 2 t WN columns right), so the reads
  // take immediate offsets.
  static_assert(Cf::WN % (Cf::TW / 16) == 0, "a wave's MFMA tiles are whole row pairs apart");
  constexpr int DPIX_R = 2 * (Cf::WN / (Cf::TW / 16)) * Cf::RS, DPIX_C = 2 * Cf::WN * Cf::PS;
  const int pix0 = Cf::halo_off(out_row(gtile(0) * 32 + l32), out_col(gtile(0) * 32 + l32), 0);
  // Byte offsets (chunk 0) of this lane's halo slot in each of its wave's LDS pieces; the chunk's
  // offset goes in the scalar offset (a lane past the plane keeps an offset the hardware drops).
  uint32_t hoff[DH];
#pragma unroll
  for (int i = 0; i < DH; ++i) {
    const int q = (wave * DH + i) * 64 + lane;
    const int row = q / Cf::RSS, r = q % Cf::RSS;
    const int iy = oy0 - pad + row, ix = ox0 - pad + r / 2;
    const bool ok = row < Cf::HH && r < 2 * Cf::HW && iy >= 0 && iy < H && ix >= 0 && ix < W;
    hoff[i] = ok ? (uint32_t)((((int64_t)iy * W + ix) * C + (r & 1) * 8) * sizeof(T)) : OOB;
  }
  auto load_halo = [&](int buf, int c0) {
#pragma unroll
    for (int i = 0; i < DH; ++i)
      lds_direct16(rsrc_in, halo_buf(buf) + (wave * DH + i) * 512, hoff[i], (uint32_t)(c0 * sizeof(T)));
  };
  // Weight piece p of a stage block lands in LDS piece p: lane offset 16 lane, the piece's and the
  // stage's offsets in the scalar offset; the wave skips pieces past the block.
  static_assert(WSLOTS % 64 == 0, "a stage's weights are whole 1 KB pieces");
  const uint32_t lane16 = (uint32_t)lane * 16u;
  // (the wave index as a scalar: the piece offsets go in the scalar offset operand)
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  auto load_w = [&](int buf, int c0, int ky) {  // stage (chunk c0 / 16, kernel row ky)
    const uint32_t add = (uint32_t)(((c0 / Cf::CC) * R + ky) * WSLOTS_P * 16);
#pragma unroll
    for (int i = 0; i < DW; ++i) {
      const int p = wave_s * DW + i;  // piece p: kernel column p / (BM / 32), channels 32 (p % (BM / 32))
      const uint32_t src = BMP == BM ? (uint32_t)p * 1024u
                                     : (uint32_t)(((p / (BM / 32)) * BMP + msub + 32 * (p % (BM / 32))) * 32);
      if (p * 64 < WSLOTS) lds_direct16(rsrc_w, wrow_buf(buf) + p * 512, lane16, add + src);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int t = 0; t < TN; ++t) acc[a][t] = f32x16{};

  const int nchunks = Cg / Cf::CC, nst = nchunks * R;
  // MFMA pixel tiles of this wave that hold a pixel of the map: a prefix of its TN tiles.  In a
  // tile cut by the map's bottom or right edge the wave runs a stage loop that skips the empty
  // tiles' reads and MFMAs; every wave still issues its share of the loads and reaches the same
  // barriers.
  int tnv = 0;
#pragma unroll
  for (int t = 0; t < TN; ++t) tnv += gtile(t) < n_mt ? 1 : 0;
  tnv = __builtin_amdgcn_readfirstlane(tnv);
  auto stage_loop = [&](auto tnv_c, auto dpix_c) {
    constexpr int TNV = decltype(tnv_c)::value, DPIX = decltype(dpix_c)::value;
    load_halo(0, 0);
    load_w(0, 0, 0);
    wait_vmem();
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
      const int chunk = st / R, ky = st - chunk * R;
      const bool next_w = st + 1 < nst, next_h = ky == 0 && chunk + 1 < nchunks;
      const int wbuf = (st + 1) & 1, wc0 = ((st + 1) / R) * Cf::CC, wky = (st + 1) % R;
      const int hbuf = (chunk + 1) & 1, hc0 = (chunk + 1) * Cf::CC;
      const T* hs = halo_buf(chunk & 1);
      const T* ws = wrow_buf(st & 1);
      if (next_w) load_w(wbuf, wc0, wky);
      if (next_h) load_halo(hbuf, hc0);
      if constexpr (TNV > 0) {
#pragma unroll
        for (int kx = 0; kx < R; ++kx) {
          typename Op::frag x[TNV], w[TM];
#pragma unroll
          for (int t = 0; t < TNV; ++t)
            x[t] = lds_frag16<T>(hs + pix0 + t * DPIX + ky * Cf::RS + kx * Cf::PS + half * 8);
#pragma unroll
          for (int mt = 0; mt < TM; ++mt)
            w[mt] = lds_frag16<T>(ws + Cf::w_off(kx, wm * 32 * TM + mt * 32 + l32, half));
#pragma unroll
          for (int mt = 0; mt < TM; ++mt)
#pragma unroll
            for (int t = 0; t < TNV; ++t) acc[mt][t] = Op::mma(w[mt], x[t], acc[mt][t]);
        }
      }
      wait_vmem();
      __syncthreads();
    }
  };
  static_assert(TN >= 1 && TN <= 4, "stage loop variants cover 0..4 tiles");
  using RowL = std::integral_constant<int, DPIX_R>;
  using ColL = std::integral_constant<int, DPIX_C>;
  auto run_layout = [&](auto layout) {
    switch (tnv) {
      case 4: if constexpr (TN >= 4) stage_loop(std::integral_constant<int, 4>{}, layout); break;
      case 3: if constexpr (TN >= 3) stage_loop(std::integral_constant<int, 3>{}, layout); break;
      case 2: if constexpr (TN >= 2) stage_loop(std::integral_constant<int, 2>{}, layout); break;
      case 1: stage_loop(std::integral_constant<int, 1>{}, layout); break;
      default: stage_loop(std::integral_constant<int, 0>{}, layout); break;
    }
  };
  if (colpair)
    run_layout(ColL{});
  else
    run_layout(RowL{});

  typedef T vec8_t __attribute__((ext_vector_type(8)));
  T* dst = out + plane * out_stride;
  if constexpr (TM == 2) {
    // Epilogue as in conv_s1_kernel: stage 128 pixels x 64 channels per wave, write whole lines.
    constexpr int WPR = NW / ROUNDS;  // waves staging per round
  #pragma unroll
    for (int round = 0; round < ROUNDS; ++round) {
      if (round) __syncthreads();
      const bool mine = wave / WPR == round;
      T* stg = s_mem + (wave % WPR) * (32 * TN * 64);
      if (mine) {
  #pragma unroll
        for (int mt = 0; mt < TM; ++mt)
  #pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int j = 4 * mt + q;
            const f32x4 bv = *(const f32x4*)(bias + g * Mg + m0 + wm * 64 + 8 * j + 4 * half);
  #pragma unroll
            for (int t = 0; t < TN; ++t) {
              const int p = t * 32 + l32;
              out4_t r;
  #pragma unroll
              for (int e = 0; e < 4; ++e)
                r[e] = from_f32<T>(fmaxf(acc[mt][t][4 * q + e] + bv[e], 0.f));
              const int key = (p & 7) ^ ((p >> 3) & 3);
              *(out4_t*)(stg + p * 64 + ((j ^ key) * 8) + 4 * half) = r;
            }
          }
      }
      __syncthreads();
      if (mine) {
        const int j = lane & 7;
  #pragma unroll
        for (int it = 0; it < (32 * TN) / 8; ++it) {
          const int p = it * 8 + (lane >> 3);
          const int key = (p & 7) ^ ((p >> 3) & 3);
          const vec8_t v = *(const vec8_t*)(stg + p * 64 + ((j ^ key) * 8));
          const int idx = gtile(p >> 5) * 32 + (p & 31);
          const int oy = oy0 + out_row(idx), ox = ox0 + out_col(idx);
          if (oy < H && ox < W)
            store_out(v, (vec8_t*)(dst + ((int64_t)oy * W + ox) * M + g * Mg + m0 + wm * 64 + 8 * j));
        }
      }
    }
  } else {
    // TM = 3: each wave owns 96 channels (192 bytes) of each of its 128 pixels.  After the loop's
    // last barrier no wave reads the stage buffers, so each wave stages one 32-pixel MFMA tile at a
    // time in a private LDS region (rows of 96 channels + one 16-byte slot: conflict-free 8-byte
    // writes), then writes each pixel's 192 bytes as 16-byte chunks.
    constexpr int SROW = 32 * TM + 8, NCH = 4 * TM;
    static_assert(NW * 32 * SROW <= LDS_E, "per-wave staging fits the stage buffers");
    T* stg = s_mem + wave * (32 * SROW);
    const int mw = g * Mg + m0 + wm * 32 * TM;  // this wave's first output channel
#pragma unroll
    for (int t = 0; t < TN; ++t) {
#pragma unroll
      for (int mt = 0; mt < TM; ++mt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = mt * 32 + 8 * q + 4 * half;
          const f32x4 bv = *(const f32x4*)(bias + mw + m);
          out4_t o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = from_f32<T>(fmaxf(acc[mt][t][4 * q + e] + bv[e], 0.f));
          *(out4_t*)(stg + l32 * SROW + m) = o;
        }
#pragma unroll
      for (int it = 0; it < NCH / 2; ++it) {  // 32 pixels x NCH chunks over 64 lanes
        const int u = it * 64 + lane, p = u / NCH, ch = u % NCH;
        const vec8_t v = *(const vec8_t*)(stg + p * SROW + 8 * ch);
        const int idx = gtile(t) * 32 + p;
        const int oy = oy0 + out_row(idx), ox = ox0 + out_col(idx);
        if (oy < H && ox < W) store_out(v, (vec8_t*)(dst + ((int64_t)oy * W + ox) * M + mw + 8 * ch));
      }
    }
  }
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int OUT_CPOL = 2;  // cache policy of conv1's output stores: non-temporal
// conv1's MFMA pixel tiles per wave (Conv1R): 2, chosen by timing on the 96-plane batch (4, one wave per
// SIMD with 30 % fewer LDS bytes per MFMA, took 0.82-0.84 ms against 0.646: a lone wave does not hide
// its own LDS and load latency).
#ifndef DN_CONV1_PT
#define DN_CONV1_PT 2
#endif
// Wait until at most N (< 64) vector-memory accesses of this wave are outstanding.
template <int N>
__device__ inline void wait_vmem_upto() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// ------------------------------------------------------------------------------------------------
// conv1 for 16-bit storage with direct global->LDS loads (plane width a multiple of 8, 16-byte
// aligned planes), weights resident, one independent pipeline per wave.  A workgroup of 8 waves (one
// per CU, two waves per SIMD) loads all weights (75 KB) into LDS once, as 25 k-steps of 16 (the 363
// taps of an output channel as 99 units of 4 taps: see pack_conv1_resident_kernel) x 96 channels x
// two 16-byte slots, the slots swapped for channels 16..31 of every 32-channel group, so that the 32
// lanes of a half-wave reading one k-step's 16 bytes of 32 channels hit distinct slots modulo 512
// bytes.  After that every wave is its own worker with no workgroup barrier: it walks wave tiles of 4
// x 16 output pixels x 96 channels, and per stage (one input channel of one tile) loads the tile's 24
// x 72 input halo (rows of nine 16-byte slots of plane data and one zero slot) into one of its two
// private LDS buffers while it computes from the other, reading k-step j + 1's fragments while k-step
// j's MFMAs run.  Stage c runs k-steps 0..7, 8..15 or 16..24; k-steps 8 and 16 hold units of two
// input channels, so they run first in their stage, from both buffers, before the next stage's halo
// load reuses the older one.  A wave that writes out a tile, or waits for a load, stalls only
// itself; the other wave on its SIMD keeps the MFMAs busy.  A tile's outputs leave through LDS, as
// whole 192-byte pixel rows.
// ------------------------------------------------------------------------------------------------
// PT: 32-pixel MFMA tiles per wave (2: wave tiles of 4 x 16 pixels, 8 waves per workgroup, two per
// SIMD; 4: 8 x 16 pixels, 4 waves, one per SIMD, 30 % fewer LDS bytes per MFMA).
template <int PT>
struct Conv1R {
  static constexpr int NWV = PT == 2 ? 8 : 4;    // waves (workers) per workgroup
  static constexpr int TH = 2 * PT, TW = 16, HR = 4 * (TH - 1) + 12;  // wave tile; halo rows (k 0..11)
  static constexpr int EPI_STORES = PT * 6;      // 16-byte stores per lane in a tile's epilogue
  static constexpr int HSL = 10, HS = HSL * 8;   // halo row: slots, elements
  static constexpr int NH = (HR * HSL + 63) / 64;  // 1 KB pieces of a halo
  static constexpr int KSE = 96 * 16;            // elements of one k-step's weights
  static constexpr int WP = C1_KSTEPS * KSE / 512;  // 1 KB pieces of all weights
  static constexpr int DWL = (WP + NWV - 1) / NWV;  // weight pieces per wave (all weights, once)
  static constexpr int HALO_E = NH * 512;
  static constexpr int SROW = 104, SPX = 16;     // staging: elements per pixel row, pixels per round
  static constexpr int HALO_OFF = WP * 512, BIAS_OFF = HALO_OFF + NWV * 2 * HALO_E;
  static constexpr int LDS_E = BIAS_OFF + 2 * 96;  // the biases as 96 floats
  // unit u of a tile's k-steps: input channel, and its LDS offset (row r, columns 4 cb ..) in the halo
  __host__ __device__ static constexpr int uchan(int u) { return u < C1_UNITS ? u / 33 : 2; }
  __host__ __device__ static constexpr int uoff(int u) {
    return u < C1_UNITS ? ((u % 33) % 11) * HS + 4 * ((u % 33) / 11) : uoff(C1_UNITS - 1);
  }
  __host__ __device__ static constexpr int kchan(int j) { return j < 8 ? 0 : (j < 16 ? 1 : 2); }  // stage
};
static_assert(Conv1R<2>::WP * 512 == C1_KSTEPS * Conv1R<2>::KSE, "the weights are whole pieces");
static_assert(Conv1R<2>::uchan(4 * 8) == 0 && Conv1R<2>::uchan(4 * 8 + 1) == 1 &&
                  Conv1R<2>::uchan(4 * 16 + 1) == 1 && Conv1R<2>::uchan(4 * 16 + 2) == 2,
              "k-steps 8 and 16 are the only ones that span two input channels");
static_assert(Conv1R<2>::SPX * Conv1R<2>::SROW <= Conv1R<2>::HALO_E, "epilogue staging fits a halo buffer");
static_assert((size_t)Conv1R<2>::LDS_E * 2 <= 160 * 1024, "one workgroup's LDS fits the CU");
static_assert((size_t)Conv1R<4>::LDS_E * 2 <= 160 * 1024, "one workgroup's LDS fits the CU");

// Keeps the compiler from moving this wave's LDS accesses across it (a wave's own LDS operations
// execute in order).
__device__ inline void wave_lds_order() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

// f(integral_constant<I>) for I = B .. E - 1, in order.
template <int B, int E, typename F>
__device__ inline void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

template <typename T, int PT, bool MULTI>
__global__ __launch_bounds__(64 * Conv1R<PT>::NWV, 1) void conv1_resident_kernel(
    const T* __restrict__ in, T* __restrict__ out, const T* __restrict__ wp,
    const float* __restrict__ bias, KRuns runs, int ntiles) {
  using P = Conv1R<PT>;
  constexpr int NWV = P::NWV;
  using Op = Mfma<T>;
  using frag = typename Op::frag;
  using hfrag = typename Op::half_frag;
  typedef T out4_t __attribute__((ext_vector_type(4)));
  typedef T vec8_t __attribute__((ext_vector_type(8)));
  __shared__ __align__(1024) T s_mem[P::LDS_E];
  float* s_bias = (float*)(s_mem + P::BIAS_OFF);
  if (threadIdx.x < 96) s_bias[threadIdx.x] = bias[threadIdx.x];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, l32 = lane & 31;
  constexpr uint32_t OOB = 0x80000000u;

  // Workers: workgroups are dispatched round-robin over the 8 XCDs, and rank r = x * (workgroups
  // per XCD) + i of XCD x has the workers NWV r .. NWV r + NWV - 1; worker w takes wave tiles w,
  // w + NWV G, ...: the workers in flight on one XCD hold neighbouring tiles, whose halos overlap in
  // its L2.
  const int G = gridDim.x, xcd = blockIdx.x % 8, per = G / 8, rem = G % 8;
  const int rank = xcd * per + min(xcd, rem) + blockIdx.x / 8;
  const int NWK = NWV * G, wk = NWV * rank + wave;
  const int ntile = wk < ntiles ? (ntiles - wk + NWK - 1) / NWK : 0;

  // All weights, once: piece q of the k-step blob lands in LDS piece q.
  {
    const __amdgpu_buffer_rsrc_t rsrc_w = uniform_rsrc(wp, (uint32_t)(C1_KSTEPS * P::KSE * sizeof(T)));
#pragma unroll
    for (int i = 0; i < P::DWL; ++i) {
      const int q = wave + NWV * i;
      if (q < P::WP) lds_direct16(rsrc_w, s_mem + q * 512, (uint32_t)(q * 1024 + lane * 16));
    }
  }
  uint32_t chan_bytes = 0;  // bytes of one input channel of the current tile's plane
  auto hbuf = [&](int b) { return s_mem + P::HALO_OFF + (2 * wave + b) * P::HALO_E; };
  uint32_t hoff[P::NH];
  __amdgpu_buffer_rsrc_t rsrc_in;
  // Column W of the plane is the zero-weight tap (kx = 11) of the last output column when
  // (W - 11) % 4 == 0.  With W % 8 != 0 its 16-byte slot starts inside the row and is loaded, so when
  // rows are padded (pitch > W) the padding value would enter as 0 * x; zcol is then that column's
  // position in the tile's halo (else -1) and the halo copy of it is overwritten with zeros.
  int zcol = -1;
  auto set_tile = [&](int t) {  // input descriptor and halo slot offsets of wave tile t
    const KRun& rn = runs.r[run_of<MULTI>(runs, t)];
    const int H = rn.H, W = rn.W, pitch = rn.pitch, tl = t - rn.first;
    const int tx = tl % rn.tiles_x, rr = tl / rn.tiles_x, ty = rr % rn.tiles_y, plane = rr / rn.tiles_y;
    chan_bytes = (uint32_t)((int64_t)H * pitch * sizeof(T));
    rsrc_in = uniform_rsrc(in + rn.in_off + plane * rn.in_stride, 3 * chan_bytes);
    const int iy0 = 4 * P::TH * ty, ix0 = 4 * P::TW * tx;
    const bool zero_col_w = W % 8 != 0 && pitch > W;
    zcol = __builtin_amdgcn_readfirstlane(zero_col_w && W >= ix0 && W < ix0 + 72 ? W - ix0 : -1);
#pragma unroll
    for (int i = 0; i < P::NH; ++i) {
      const int q = i * 64 + lane;
      const int row = q / P::HSL, r = q % P::HSL;
      const int iy = iy0 + row, ix = ix0 + 8 * r;
      const bool ok = row < P::HR && r < 9 && iy < H && ix < W;
      hoff[i] = ok ? (uint32_t)(((int64_t)iy * pitch + ix) * sizeof(T)) : OOB;
    }
  };
  auto load_halo = [&](int b, int c) {  // channel c of the current tile into buffer b
#pragma unroll
    for (int i = 0; i < P::NH; ++i) lds_direct16(rsrc_in, hbuf(b) + i * 512, hoff[i], c * chan_bytes);
  };
  auto zero_col = [&](int b) {  // after buffer b's loads have landed
    if (zcol >= 0) {
      wave_lds_order();
      if (lane < P::HR) hbuf(b)[lane * P::HS + zcol] = from_f32<T>(0.f);
      wave_lds_order();
    }
  };

  int lpix[PT], lpix2[PT];
#pragma unroll
  for (int b = 0; b < PT; ++b) {
    const int idx = b * 32 + l32;
    lpix[b] = 4 * (idx / P::TW) * P::HS + 4 * (idx % P::TW);
    lpix2[b] = lpix[b] + 2 * half * P::HS;
  }
  const int lw = 16 * l32 + 8 * (half ^ ((l32 >> 4) & 1));
  // Lane bases: this lane's pixel (input row 4 prow, column 4 pcol) per pixel tile (lpix2: two rows
  // further in the upper half-wave), and its output channel's weight slot (half ^ swap).  k-step J:
  // lane half h reads units 4 J + 2 h (the fragment's low 8 bytes) and 4 J + 2 h + 1 (high); hp holds
  // the previous input channel's halo, hs the stage's.
  auto read = [&](auto jc, const T* hp, const T* hs, frag* x, frag* w) {
    constexpr int J = decltype(jc)::value, CS = P::kchan(J);
    hfrag hv[PT][2];
#pragma unroll
    for (int sx = 0; sx < 2; ++sx) {
      const int u0 = 4 * J + sx, u1 = 4 * J + 2 + sx;
      const bool p0 = P::uchan(u0) != CS, p1 = P::uchan(u1) != CS;
      const int o0 = P::uoff(u0), o1 = P::uoff(u1);
      if (!p0 && !p1 && o1 - o0 == 2 * P::HS) {  // the usual case: the upper half two rows down
#pragma unroll
        for (int b = 0; b < PT; ++b) hv[b][sx] = *(const hfrag*)(hs + lpix2[b] + o0);
      } else {
        const T* bh = half ? (p1 ? hp : hs) + o1 : (p0 ? hp : hs) + o0;
#pragma unroll
        for (int b = 0; b < PT; ++b) hv[b][sx] = *(const hfrag*)(bh + lpix[b]);
      }
    }
#pragma unroll
    for (int b = 0; b < PT; ++b) x[b] = __builtin_shufflevector(hv[b][0], hv[b][1], 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
    for (int mt = 0; mt < 3; ++mt) w[mt] = *(const frag*)(s_mem + J * P::KSE + 512 * mt + lw);
  };

  f32x16 acc[3][PT];
#pragma unroll
  for (int a = 0; a < 3; ++a)
#pragma unroll
    for (int b = 0; b < PT; ++b) acc[a][b] = f32x16{};

  if (ntile > 0) {
    set_tile(wk);
    load_halo(0, 0);
  }
  wait_vmem();
  __syncthreads();  // weights and biases are in LDS; from here on each wave runs on its own
  zero_col(0);
  // One tile per iteration, its three stages in straight-line code.  Channel 0 and channel 2 of tile
  // j sit in buffer X = j & 1, channel 1 in the other, Y; a stage's load of the next stage's channel
  // goes to the buffer its own k-steps no longer read.
  for (int j = 0; j < ntile; ++j) {
    T* hx = hbuf(j & 1);
    T* hy = hbuf((j + 1) & 1);
    // k-steps J0 .. J1 - 1 of stage J0's channel (halo in hs, the previous channel's in hp); the next
    // stage's load (issue) follows k-step J0's MFMAs, which have then consumed any fragment of hp.
    auto ksteps = [&](auto j0c, auto j1c, const T* hp, const T* hs, auto&& issue) {
      constexpr int J0 = decltype(j0c)::value, J1 = decltype(j1c)::value;
      frag xr[2][PT], wr[2][3];
      read(std::integral_constant<int, J0>{}, hp, hs, xr[0], wr[0]);
      auto body = [&](auto jc) {
        constexpr int J = decltype(jc)::value, B = (J - J0) & 1;
        if constexpr (J + 1 < J1) read(std::integral_constant<int, J + 1>{}, hp, hs, xr[B ^ 1], wr[B ^ 1]);
        // raised wave priority while this k-step's MFMAs issue: the SIMD's other wave then issues
        // its LDS reads, loads and epilogue work in between rather than ahead of them
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int mt = 0; mt < 3; ++mt)
#pragma unroll
          for (int b = 0; b < PT; ++b) acc[mt][b] = Op::mma(wr[B][mt], xr[B][b], acc[mt][b]);
        __builtin_amdgcn_s_setprio(0);
        if constexpr (J == J0) {
          wave_lds_order();
          issue();
        }
      };
      static_for<J0, J1>(body);
    };
    // stage 0: channel 0 in X; channel 1 loads into Y
    ksteps(std::integral_constant<int, 0>{}, std::integral_constant<int, 8>{}, hy, hx, [&] { load_halo((j + 1) & 1, 1); });
    wait_vmem();
    zero_col((j + 1) & 1);
    // stage 1: channel 1 in Y (k-step 8 also reads channel 0 in X); channel 2 loads into X
    ksteps(std::integral_constant<int, 8>{}, std::integral_constant<int, 16>{}, hx, hy, [&] { load_halo(j & 1, 2); });
    wait_vmem();
    zero_col(j & 1);
    // stage 2: channel 2 in X (k-step 16 also reads channel 1 in Y); the next tile's channel 0
    // loads into Y, the next tile's X
    ksteps(std::integral_constant<int, 16>{}, std::integral_constant<int, C1_KSTEPS>{}, hy, hx, [&] {
      if (j + 1 < ntile) {
        set_tile(wk + (j + 1) * NWK);
        load_halo((j + 1) & 1, 0);
      }
    });
    {
      // Epilogue of the tile: bias + ReLU; per 32-pixel MFMA tile, two rounds of 16 pixels staged
      // in X, just consumed (rows of 104 channels), read back as whole pixel rows and written with
      // 16-byte buffer stores that every lane issues (a pixel outside the map stores at an offset
      // past the plane, which the hardware drops): P::EPI_STORES stores per lane.
      T* hs = hx;
      const int t = wk + j * NWK;
      const KRun& rn = runs.r[run_of<MULTI>(runs, t)];
      const int Ho = rn.Ho, Wo = rn.Wo, tl = t - rn.first;
      const int tx = tl % rn.tiles_x, rr = tl / rn.tiles_x, ty = rr % rn.tiles_y, plane = rr / rn.tiles_y;
      const __amdgpu_buffer_rsrc_t rsrc_out =
          uniform_rsrc(out + rn.out_off + plane * rn.out_stride, (uint32_t)((int64_t)Ho * Wo * 96 * sizeof(T)));
#pragma unroll
      for (int b = 0; b < PT; ++b) {
        out4_t v[3][4];
#pragma unroll
        for (int mt = 0; mt < 3; ++mt)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 bv = *(const f32x4*)(s_bias + mt * 32 + 8 * q + 4 * half);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[mt][q][e] = from_f32<T>(fmaxf(acc[mt][b][4 * q + e] + bv[e], 0.f));
          }
#pragma unroll
        for (int ph = 0; ph < 2; ++ph) {
          wave_lds_order();
          if ((l32 >> 4) == ph) {
#pragma unroll
            for (int mt = 0; mt < 3; ++mt)
#pragma unroll
              for (int q = 0; q < 4; ++q)
                *(out4_t*)(hs + (l32 & 15) * P::SROW + mt * 32 + 8 * q + 4 * half) = v[mt][q];
          }
          wave_lds_order();
#pragma unroll
          for (int it = 0; it < 3; ++it) {  // 16 pixels x 12 chunks of 8 channels
            const int u = it * 64 + lane, p = u / 12, ch = u % 12;
            const vec8_t o = *(const vec8_t*)(hs + p * P::SROW + 8 * ch);
            const int idx = b * 32 + 16 * ph + p;
            const int oy = ty * P::TH + idx / P::TW, ox = tx * P::TW + idx % P::TW;
            const uint32_t off = oy < Ho && ox < Wo
                                     ? (uint32_t)((((int64_t)oy * Wo + ox) * 96 + 8 * ch) * sizeof(T))
                                     : OOB;
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o), rsrc_out, off, 0, OUT_CPOL);
          }
        }
      }
      wave_lds_order();
#pragma unroll
      for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < PT; ++b) acc[a][b] = f32x16{};
      // Vector-memory operations retire in issue order: once no more than the epilogue's stores
      // are outstanding, the next tile's halo loads (issued before them) have landed in LDS.
      wait_vmem_upto<P::EPI_STORES>();
    }
    zero_col((j + 1) & 1);
  }
}

// Copies an fp32 launch of `blocks` workgroups splits its input channels over (at most max_copies):
// the ks minimising rounds(ks) / ks + 0.15 [ks > 1] + 0.02 ks blocks / CUs, rounds(ks) =
// ceil(ks blocks / CUs) (one fp32 workgroup per CU at a time): the launch's rounds of shorter
// workgroups, plus the reduction and the partial sums' traffic, which grows with the copies and the
// launch's output (fitted to timed launches of the 227 x 227 and the 8-scale 480 x 640 pyramids).
// Launches of at least one workgroup per CU do not split: a lone workgroup's whole K loop sets a
// small launch's time, not a large one's.
int split_copies(int64_t blocks, int max_copies) {
  const int64_t cus = device_cu_count();
  int ks = 1;
  if (blocks < cus) {
    double best = 1.0;
    for (int k = 2; k <= max_copies; ++k) {
      const double cost = (double)((k * blocks + cus - 1) / cus) / k + 0.15 + 0.02 * k * (double)blocks / cus;
      if (cost < best) best = cost, ks = k;
    }
  }
  return ks;
}

// Elements of one partial copy of a launch over `runs`: its output extent, rounded to 64.
int64_t split_span(const MapRun* runs, int n_runs) {
  int64_t span = 0;
  for (int i = 0; i < n_runs; ++i) span = std::max(span, runs[i].out_off + runs[i].n * runs[i].out_stride);
  return (span + 63) / 64 * 64;
}

// part / part_bytes: workspace for the partial sums of a split fp32 launch (may be NULL: no split);
// part_need non-NULL: only report the bytes this launch would use there (0 without a split).
template <typename T, int R, int BM, int TM, int OCC, int TS, int BMP = BM, int TN = 4>
int run_conv_s1(const T* in, T* out, const T* wp, const T* wstage, const float* bias, const MapRun* runs,
                int n_runs, int C, int G, int M, float* part, size_t part_bytes, size_t* part_need,
                hipStream_t s) {
  using Cf = ConvCfg<T, R, BM, TM, TS, TN>;
  const int Cg = C / G, Mg = M / G;
  if (Mg % BM) return (int)hipErrorInvalidValue;  // whole channel blocks per group
  const int mblocks = G * (Mg / BM);
  KRuns kr;
  const int64_t blocks = fill_kruns(runs, n_runs, kr, [&](KRun& k) {
    k.Ho = k.H, k.Wo = k.W;
    k.tiles_x = (k.W + Cf::TW - 1) / Cf::TW, k.tiles_y = (k.H + Cf::TH - 1) / Cf::TH;
    return (int64_t)k.tiles_x * k.tiles_y * mblocks;
  });
  if (blocks <= 0) return (int)hipErrorInvalidValue;
  if constexpr (Cf::F32 || (TM != 2 && TM != 3)) {
    // fp32 launches too small to fill the chip split their input chunks over ks copies
    int ks = 1;
    int64_t span = 0;  // elements of one partial copy
    if constexpr (Cf::F32) {
      ks = split_copies(blocks, Cg / Cf::CC);
      span = split_span(runs, n_runs);
    }
    const size_t need = ks > 1 ? (size_t)ks * (size_t)span * sizeof(float) : 0;
    if (part_need) {
      *part_need = need;
      return 0;
    }
    if (ks > 1 && (!part || part_bytes < need)) ks = 1;
    conv_s1_kernel<T, R, BM, TM, OCC, TS><<<(unsigned)(blocks * ks), Cf::NT, 0, s>>>(
        in, out, wp, bias, kr, C, Cg, M, Mg, mblocks, ks, (int)blocks, part, span);
    if constexpr (Cf::F32) {
      if (ks > 1) {
        KRuns rr;
        const int64_t rb = fill_kruns(runs, n_runs, rr, [&](KRun& k) {
          k.Ho = k.H, k.Wo = k.W;
          k.tiles_x = (int)(((int64_t)k.H * k.W * M / 4 + 255) / 256), k.tiles_y = 1;
          return (int64_t)k.tiles_x;
        });
        if (rb <= 0) return (int)hipErrorInvalidValue;
        split_reduce_kernel<<<(unsigned)rb, 256, 0, s>>>(part, span, ks, bias, out, rr, M);
      }
    }
  } else {
    if (part_need) {
      *part_need = 0;
      return 0;
    }
    // buffer descriptors address one plane with 32-bit byte offsets
    for (int i = 0; i < n_runs; ++i)
      if ((int64_t)runs[i].H * runs[i].W * C * (int64_t)sizeof(T) >= 0x7fffffffLL)
        return (int)hipErrorInvalidValue;
    if (wstage == wp) return (int)hipErrorInvalidValue;  // the stage-major weight copy is required
    if (n_runs == 1)
      conv_s1_direct_kernel<T, R, BM, TM, OCC, TS, BMP, TN, false><<<(unsigned)blocks, Cf::NT, 0, s>>>(
          in, out, wstage, bias, kr, C, Cg, M, Mg, mblocks);
    else
      conv_s1_direct_kernel<T, R, BM, TM, OCC, TS, BMP, TN, true><<<(unsigned)blocks, Cf::NT, 0, s>>>(
          in, out, wstage, bias, kr, C, Cg, M, Mg, mblocks);
  }
  return (int)hipGetLastError();
}

// Per layer: channel block BM, MFMA tiles per wave along channels TM, waves per SIMD requested, and
// the tile shape (100 rows + columns).  Chosen by timing each layer at the 96-plane batch shapes: two waves per
// SIMD matter most; conv3/conv5 run best at three waves per SIMD; conv4's 192 channels per group run
// best as one block of 3 x 32 channels per wave (7 LDS fragment reads per 12 MFMAs instead of 6 per 8).
// conv2 takes 16 x 32 tiles of 64 channels (four waves of 64 channels x 128 pixels): each stage's
// weight row then serves 512 pixels, which halves the weight loads per output against 16 x 16 tiles
// of 128 channels (2 % faster; with 128 channels, eight waves per workgroup, 10 % slower).  On the
// 74-wide maps of conv3..conv5, 32-wide tiles waste 20 % more MFMA work and were 25-30 % slower.
#ifndef DN_CONV2_CFG
#define DN_CONV2_CFG 64, 2, 2, 1632
#endif
#ifndef DN_CONV3_CFG
#define DN_CONV3_CFG 128, 2, 3, 1616
#endif
#ifndef DN_CONV5_CFG
#define DN_CONV5_CFG 128, 2, 3, 1616
#endif
#ifndef DN_CONV4_CFG
#define DN_CONV4_CFG 192, 3, 2, 1616
#endif

template <int BM_, int TM_, int OCC_, int TS_>
struct CfgBM {
  static constexpr int BM = BM_;
};
// Channel block of the direct-load kernel per layer (the stage-major weight copy is cut in these).
constexpr int L_BM[5] = {0, CfgBM<DN_CONV2_CFG>::BM, CfgBM<DN_CONV3_CFG>::BM, CfgBM<DN_CONV4_CFG>::BM,
                         CfgBM<DN_CONV5_CFG>::BM};

// A launch of the per-layer configuration with fewer workgroups than two rounds of the chip's
// resident slots (CUs x workgroups per CU) leaves CUs idle; such launches (one image's planes) take
// 64-channel blocks of 16 x 16 pixels instead, three to six times as many workgroups.
// Small launches: 64-channel blocks of 16 x 16 pixels whose waves own DN_SMALL_TN MFMA pixel tiles.
#ifndef DN_SMALL_TN
#define DN_SMALL_TN 2
#endif
#ifndef DN_SMALL_OCC
#define DN_SMALL_OCC 3
#endif
template <int BM_, int TM_, int OCC_, int TS_>
bool small_launch(const MapRun* runs, int n_runs, int M) {
  int64_t blocks = 0;
  for (int i = 0; i < n_runs; ++i)
    blocks += (int64_t)((runs[i].W + TS_ % 100 - 1) / (TS_ % 100)) *
              ((runs[i].H + TS_ / 100 - 1) / (TS_ / 100)) * (M / BM_) * runs[i].n;
  const int per_cu = OCC_ * 4 / (BM_ / (32 * TM_) * (TS_ / 100) * (TS_ % 100) / 128);
  return blocks < 2LL * device_cu_count() * (per_cu > 0 ? per_cu : 1);
}

template <typename T>
int conv_dispatch(int layer, const void* d_in, const MapRun* runs, int n_runs, const void* d_packed,
                  void* d_out, float* part, size_t part_bytes, size_t* part_need, const PackedLayout& L,
                  hipStream_t s) {
  const T* in = (const T*)d_in;
  T* out = (T*)d_out;
  const T* wp = (const T*)((const char*)d_packed + L.w_off[layer - 1]);
  // the direct-load kernels (16-bit storage) stream the stage-major copy
  const T* ws = L.s_off[layer - 1] ? (const T*)((const char*)d_packed + L.s_off[layer - 1]) : wp;
  const float* bias = (const float*)((const char*)d_packed + L.b_off[layer - 1]);
  if (layer == 1) {
    if (part_need) *part_need = 0;
    KRuns kr;
    auto tiles16 = [](KRun& k) {  // tiles of 16 x 16 output pixels
      k.Ho = (k.H - 11) / 4 + 1, k.Wo = (k.W - 11) / 4 + 1;
      k.tiles_x = (k.Wo + 15) / 16, k.tiles_y = (k.Ho + 15) / 16;
      return (int64_t)k.tiles_x * k.tiles_y;
    };
    if constexpr (std::is_same<T, float>::value) {
      const int64_t blocks = fill_kruns(runs, n_runs, kr, tiles16);
      if (blocks <= 0) return (int)hipErrorInvalidValue;
      // launches too small to fill the chip split the three input channels (as conv2-5 do)
      int ks = split_copies(blocks, 3);
      const int64_t span = split_span(runs, n_runs);
      const size_t need = ks > 1 ? (size_t)ks * (size_t)span * sizeof(float) : 0;
      if (part_need) {
        *part_need = need;
        return 0;
      }
      if (ks > 1 && (!part || part_bytes < need)) ks = 1;
      conv1_kernel<T><<<(unsigned)(blocks * ks), 256, 0, s>>>(in, out, wp, bias, kr, ks, (int)blocks, part,
                                                            span);
      if (ks > 1) {
        KRuns rr;
        const int64_t rb = fill_kruns(runs, n_runs, rr, [](KRun& k) {
          k.Ho = (k.H - 11) / 4 + 1, k.Wo = (k.W - 11) / 4 + 1;
          k.tiles_x = (int)(((int64_t)k.Ho * k.Wo * 96 / 4 + 255) / 256), k.tiles_y = 1;
          return (int64_t)k.tiles_x;
        });
        if (rb <= 0) return (int)hipErrorInvalidValue;
        split_reduce_kernel<<<(unsigned)rb, 256, 0, s>>>(part, span, ks, bias, (float*)out, rr, 96);
      }
    } else {
      if (part_need) return 0;
      // Direct loads take 16-byte slots of plane rows at 32-bit byte offsets within one plane.
      bool direct = ((uintptr_t)in & 15) == 0;
      for (int i = 0; i < n_runs; ++i) {
        const MapRun& r = runs[i];
        const int64_t Ho = (r.H - 11) / 4 + 1, Wo = (r.W - 11) / 4 + 1;
        const int64_t pitch = r.pitch > 0 ? r.pitch : r.W;
        direct = direct && pitch % 8 == 0 && r.in_stride % 8 == 0 && r.in_off % 8 == 0 &&
                 3 * r.H * pitch * (int64_t)sizeof(T) < 0x7fffffffLL &&
                 Ho * Wo * 96 * (int64_t)sizeof(T) < 0x7fffffffLL;
      }
      if (direct) {
        if (ws == wp) return (int)hipErrorInvalidValue;  // the stage-major weight copy is required
        // wave tiles of 4 x 16 output pixels, 8 workers per workgroup, one workgroup per CU
        using R1 = Conv1R<DN_CONV1_PT>;
        const int64_t wtiles = fill_kruns(runs, n_runs, kr, [](KRun& k) {
          k.Ho = (k.H - 11) / 4 + 1, k.Wo = (k.W - 11) / 4 + 1;
          k.tiles_x = (k.Wo + R1::TW - 1) / R1::TW, k.tiles_y = (k.Ho + R1::TH - 1) / R1::TH;
          return (int64_t)k.tiles_x * k.tiles_y;
        });
        if (wtiles <= 0) return (int)hipErrorInvalidValue;
        const int grid = (int)std::min<int64_t>((wtiles + R1::NWV - 1) / R1::NWV, device_cu_count());
        if (n_runs == 1)
          conv1_resident_kernel<T, DN_CONV1_PT, false><<<grid, 64 * R1::NWV, 0, s>>>(in, out, ws, bias, kr,
                                                                                    (int)wtiles);
        else
          conv1_resident_kernel<T, DN_CONV1_PT, true><<<grid, 64 * R1::NWV, 0, s>>>(in, out, ws, bias, kr,
                                                                                   (int)wtiles);
      } else {
        const int64_t blocks = fill_kruns(runs, n_runs, kr, tiles16);
        if (blocks <= 0) return (int)hipErrorInvalidValue;
        const int grid = (int)std::min<int64_t>(blocks, device_cu_count());
        conv1_persistent_kernel<T><<<grid, 256, 0, s>>>(in, out, wp, bias, kr, (int)blocks);
      }
    }
    return (int)hipGetLastError();
  }
  const int li = layer - 1;
  constexpr bool F32 = std::is_same<T, float>::value;
#define DN_RUN_ARGS in, out, wp, ws, bias, runs, n_runs, L_C[li], L_G[li], L_M[li], part, part_bytes, part_need, s
#define DN_SMALL_CFG(l) 3, 64, 2, DN_SMALL_OCC, 1616, L_BM[l], DN_SMALL_TN
  switch (layer) {
    case 2:
      return run_conv_s1<T, 5, DN_CONV2_CFG>(DN_RUN_ARGS);
    case 3:
      if (!F32 && small_launch<DN_CONV3_CFG>(runs, n_runs, L_M[li]))
        return run_conv_s1<T, DN_SMALL_CFG(2)>(DN_RUN_ARGS);
      return run_conv_s1<T, 3, DN_CONV3_CFG>(DN_RUN_ARGS);
    case 4:
      if (!F32 && small_launch<DN_CONV4_CFG>(runs, n_runs, L_M[li]))
        return run_conv_s1<T, DN_SMALL_CFG(3)>(DN_RUN_ARGS);
      return run_conv_s1<T, 3, DN_CONV4_CFG>(DN_RUN_ARGS);
    case 5:
      if (!F32 && small_launch<DN_CONV5_CFG>(runs, n_runs, L_M[li]))
        return run_conv_s1<T, DN_SMALL_CFG(4)>(DN_RUN_ARGS);
      return run_conv_s1<T, 3, DN_CONV5_CFG>(DN_RUN_ARGS);
  }
#undef DN_SMALL_CFG
#undef DN_RUN_ARGS
  return (int)hipErrorInvalidValue;
}

}  // namespace

PackedLayout packed_layout(dn_dtype dt) {
  PackedLayout L{};
  const size_t es = dtype_size(dt);
  size_t off = 0;
  for (int l = 0; l < 5; ++l) {
    L.w_off[l] = off;
    const size_t n = l == 0 ? (size_t)96 * 3 * K1
                            : (size_t)L_M[l] * (L_C[l] / L_G[l]) * L_R[l] * L_R[l];
    off = align256(off + n * es);
  }
  for (int l = 0; l < 5; ++l) {
    L.b_off[l] = off;
    off = align256(off + (size_t)L_M[l] * 4);
  }
  for (int l = 0; l < 5; ++l) {
    L.s_off[l] = 0;
    if (dt == DN_F32) continue;
    L.s_off[l] = off;
    off = align256(off + (l == 0 ? (size_t)C1_KSTEPS * 96 * 16
                                  : (size_t)L_M[l] * (L_C[l] / L_G[l]) * L_R[l] * L_R[l]) * es);
  }
  L.total = off;
  return L;
}

int launch_pack_weights(const float* const* d_w, const float* const* d_b, dn_dtype dt, void* d_packed,
                        void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const PackedLayout L = packed_layout(dt);
  char* base = (char*)d_packed;
  for (int l = 0; l < 5; ++l) {
    void* dst = base + L.w_off[l];
    if (l == 0) {
      const int n = 96 * 3 * K1;
      if (dt == DN_F32) pack_conv1_kernel<float><<<(n + 255) / 256, 256, 0, s>>>(d_w[0], (float*)dst);
      if (dt == DN_F16)
        pack_conv1_kernel<_Float16><<<(n + 255) / 256, 256, 0, s>>>(d_w[0], (_Float16*)dst);
      if (dt == DN_BF16) pack_conv1_kernel<__bf16><<<(n + 255) / 256, 256, 0, s>>>(d_w[0], (__bf16*)dst);
    } else {
      const int Cg = L_C[l] / L_G[l], RR = L_R[l] * L_R[l];
      const int64_t n = (int64_t)L_M[l] * Cg * RR;
      const unsigned nb = (unsigned)((n + 255) / 256);
      if (dt == DN_F32) pack_conv_kernel<float><<<nb, 256, 0, s>>>(d_w[l], (float*)dst, L_M[l], Cg, RR);
      if (dt == DN_F16)
        pack_conv_kernel<_Float16><<<nb, 256, 0, s>>>(d_w[l], (_Float16*)dst, L_M[l], Cg, RR);
      if (dt == DN_BF16)
        pack_conv_kernel<__bf16><<<nb, 256, 0, s>>>(d_w[l], (__bf16*)dst, L_M[l], Cg, RR);
    }
    copy_f32_kernel<<<(L_M[l] + 255) / 256, 256, 0, s>>>(d_b[l], (float*)(base + L.b_off[l]), L_M[l]);
    if (L.s_off[l] && l == 0) {
      const int n = C1_KSTEPS * 96 * 16;
      void* sd = base + L.s_off[0];
      if (dt == DN_F16)
        pack_conv1_resident_kernel<_Float16><<<(n + 255) / 256, 256, 0, s>>>(d_w[0], (_Float16*)sd);
      if (dt == DN_BF16)
        pack_conv1_resident_kernel<__bf16><<<(n + 255) / 256, 256, 0, s>>>(d_w[0], (__bf16*)sd);
    } else if (L.s_off[l]) {
      const int Cg = L_C[l] / L_G[l], Mg = L_M[l] / L_G[l];
      const int64_t n = (int64_t)L_M[l] * Cg * L_R[l] * L_R[l];
      const unsigned nb = (unsigned)((n + 255) / 256);
      void* sd = base + L.s_off[l];
      if (dt == DN_F16)
        pack_stage_kernel<_Float16><<<nb, 256, 0, s>>>(d_w[l], (_Float16*)sd, Mg, Cg, L_R[l], L_BM[l], n);
      if (dt == DN_BF16)
        pack_stage_kernel<__bf16><<<nb, 256, 0, s>>>(d_w[l], (__bf16*)sd, Mg, Cg, L_R[l], L_BM[l], n);
    }
  }
  return (int)hipGetLastError();
}

// One launch per MAX_RUNS runs (the partial-sum workspace is reused by each in turn), or with
// part_need: the largest workspace any of them would use.
static int conv_part_bytes_or_launch(int layer, const void* d_in, const MapRun* runs, int32_t n_runs,
                                     dn_dtype dt, const void* d_packed, void* d_out, void* d_part,
                                     size_t part_bytes, size_t* part_need, void* stream) {
  const PackedLayout L = packed_layout(dt);
  hipStream_t s = (hipStream_t)stream;
  if (layer < 1 || layer > 5 || n_runs <= 0) return (int)hipErrorInvalidValue;
  if (part_need) *part_need = 0;
  float* part = (float*)d_part;
  for (int i0 = 0; i0 < n_runs; i0 += MAX_RUNS) {
    const int nr = std::min(MAX_RUNS, n_runs - i0);
    size_t need = 0;
    size_t* q = part_need ? &need : nullptr;
    int st = (int)hipErrorInvalidValue;
    switch (dt) {
      case DN_F32:
        st = conv_dispatch<float>(layer, d_in, runs + i0, nr, d_packed, d_out, part, part_bytes, q, L, s);
        break;
      case DN_F16:
        st = conv_dispatch<_Float16>(layer, d_in, runs + i0, nr, d_packed, d_out, part, part_bytes, q, L, s);
        break;
      case DN_BF16:
        st = conv_dispatch<__bf16>(layer, d_in, runs + i0, nr, d_packed, d_out, part, part_bytes, q, L, s);
        break;
    }
    if (st) return st;
    if (part_need) *part_need = std::max(*part_need, need);
  }
  return 0;
}

int launch_conv(int layer, const void* d_in, const MapRun* runs, int32_t n_runs, dn_dtype dt,
                const void* d_packed, void* d_out, void* d_part, size_t part_bytes, void* stream) {
  return conv_part_bytes_or_launch(layer, d_in, runs, n_runs, dt, d_packed, d_out, d_part, part_bytes,
                                   nullptr, stream);
}

size_t conv_part_bytes(int layer, const MapRun* runs, int32_t n_runs, dn_dtype dt) {
  size_t need = 0;
  if (conv_part_bytes_or_launch(layer, nullptr, runs, n_runs, dt, nullptr, nullptr, nullptr, 0, &need,
                                nullptr))
    return 0;
  return need;
}

}  // namespace dn
