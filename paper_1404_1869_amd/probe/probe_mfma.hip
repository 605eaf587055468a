// Matrix-core rate probe (measurement only; not part of the descriptor path).  Built into its own
// library, libprobe.so, which only the benchmark's ceiling measurement loads.
//
// Each wave runs four independent accumulation chains of v_mfma_f32_32x32x16_bf16 with no memory
// traffic, two workgroups of four waves per CU (two waves per SIMD), so the matrix pipe never waits
// on a dependency.  The sustained rate then depends only on the clock, and the clock on the power the
// operands draw:
//   mode 0: every MFMA reads the same A and B registers, A varying smoothly across lanes and B the
//           same on every lane (the most favourable case: near the datasheet peak);
//   mode 1: A and B are hashed bit patterns (random sign, exponent 2^-8..2^7 and mantissa), four
//           register sets used in turn;
//   mode 2: the values of mode 0, copied into four register sets used in turn as in mode 1.
// Modes 0 and 2 run at the same rate and mode 1 at well under half of it: the operand values, not
// the registers read, set the clock.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int CHAINS = 4;
constexpr int ITERS = 2048;  // k-steps per chain and launch
constexpr int THREADS = 256;

__device__ inline uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  return x;
}

__device__ inline __bf16 hashed_bf16(uint32_t h) {
  const uint16_t bits =
      (uint16_t)(((h & 1u) << 15) | ((119u + ((h >> 1) & 15u)) << 7) | ((h >> 8) & 0x7fu));
  return __builtin_bit_cast(__bf16, bits);
}

template <int MODE>
__global__ __launch_bounds__(THREADS, 2) void mfma_chain_kernel(float* out, uint32_t seed) {
  const uint32_t t = blockIdx.x * THREADS + threadIdx.x;
  f32x16 acc[CHAINS];
  for (int c = 0; c < CHAINS; ++c) acc[c] = f32x16{};
  if constexpr (MODE == 0) {
    bf16x8 a, b;
    for (int i = 0; i < 8; ++i) {
      a[i] = (__bf16)(1e-3f * (float)(threadIdx.x + i));
      b[i] = (__bf16)(1e-3f * (float)(i + 1));
    }
    for (int it = 0; it < ITERS; ++it)
#pragma unroll
      for (int c = 0; c < CHAINS; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  } else {
    bf16x8 a[4], b[4];
    for (int v = 0; v < 4; ++v)
      for (int i = 0; i < 8; ++i) {
        if constexpr (MODE == 1) {
          const uint32_t key = t * 64u + (uint32_t)(v * 8 + i);
          a[v][i] = hashed_bf16(mix32(seed ^ key));
          b[v][i] = hashed_bf16(mix32(~seed ^ key));
        } else {
          // the same values in every set; seed (never 0 here) keeps the compiler from merging the sets
          a[v][i] = (__bf16)(1e-3f * (float)(threadIdx.x + i) + (seed == 0u ? (float)v : 0.f));
          b[v][i] = (__bf16)(1e-3f * (float)(i + 1) + (seed == 0u ? (float)v : 0.f));
        }
      }
    for (int it = 0; it < ITERS; it += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int c = 0; c < CHAINS; ++c)
          acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(c + u) % 4], b[(c + 2 * u + 1) % 4], acc[c],
                                                           0, 0, 0);
    }
  }
  float s = 0.f;
  for (int c = 0; c < CHAINS; ++c)
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[t] = s;  // keeps the chains live
}

}  // namespace

extern "C" {

// Launch `launches` probe kernels on `stream` (a hipStream_t, NULL = default stream).  d_out: device
// buffer of out_floats floats, at least 512 x (compute units) (one per thread).  *flop_per_launch
// receives the dense FLOPs of one launch.  Returns 0, or -1 on a bad argument or launch error.
int densenet_probe_mfma_bf16(int mode, int launches, float* d_out, int64_t out_floats,
                             double* flop_per_launch, void* stream) {
  int dev = 0, cus = 0;
  if (mode < 0 || mode > 2 || launches < 1 || !d_out || !flop_per_launch) return -1;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return -1;
  const int grid = 2 * cus;
  if (out_floats < (int64_t)grid * THREADS) return -1;
  *flop_per_launch = (double)grid * (THREADS / 64) * ITERS * CHAINS * (2.0 * 32 * 32 * 16);
  const hipStream_t s = (hipStream_t)stream;
  for (int l = 0; l < launches; ++l) {
    const uint32_t seed = 12345u + (uint32_t)l;
    if (mode == 0)
      mfma_chain_kernel<0><<<grid, THREADS, 0, s>>>(d_out, seed);
    else if (mode == 1)
      mfma_chain_kernel<1><<<grid, THREADS, 0, s>>>(d_out, seed);
    else
      mfma_chain_kernel<2><<<grid, THREADS, 0, s>>>(d_out, seed);
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // extern "C"
