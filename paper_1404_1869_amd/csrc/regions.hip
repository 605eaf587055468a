// Region windows ("crop after", Sec. 4): a box of the original image is read out of the conv5
// pyramid at the scale whose scaled area is closest to target^2, as S x S bilinear samples at the
// bin centres of the box, all channels.  With several aspect-ratio pyramids (Sec. 3.3) the cost of an
// entry is multiplied by max(rho, 1 / rho), rho the aspect of the box on that entry, so the box is
// read where it is closest to a target x target square.
//
// One workgroup per box; each thread blends one 16-byte vector of channels of one bin at a time.
// The scale choice and the sample positions are computed in fp64 with + - * / only and FP
// contraction off, in the same order as the definition, so the chosen scale and cell indices are
// reproducible bit for bit on any IEEE fp64 implementation.  Samples of one bin read 4 cells x C
// contiguous channels (coalesced); the descriptor row is transposed through LDS into its
// channel-major order and written with coalesced non-temporal stores (the rows are not read back by
// this path, so they need not displace the conv5 maps from the caches).
#include "common.h"

namespace dn {
namespace {

constexpr int MAX_S = 8;

// Max-pooled bins: the cells of a bin spanning [lo, hi) in plane coordinates are those whose
// receptive-field centre 16 i + 17.5 lies inside it, clipped to [cmin, cmax]; a bin left with no cell
// takes the cell nearest its centre.
__device__ inline void pool_bin_range(double lo, double hi, int cmin, int cmax, int& first, int& last) {
#pragma clang fp contract(off)
  int f = (int)ceil((lo - 17.5) / 16.0);
  int l = (int)ceil((hi - 17.5) / 16.0) - 1;
  f = f < cmin ? cmin : f;
  l = l > cmax ? cmax : l;
  if (l < f) {
    const double g = ((lo + hi) * 0.5 - 17.5) / 16.0;
    int c = (int)floor(g + 0.5);
    c = c < cmin ? cmin : (c > cmax ? cmax : c);
    f = l = c;
  }
  first = f;
  last = l;
}

// Entry k of image img: from the kernel arguments (per-image maps), or from the device copy of a
// cross-image packed plan, where an entry whose window does not lie inside a map is taken as empty.
template <bool BATCH>
__device__ inline RegScale entry(const RegArgs& a, const RegBatch& bt, int img, int k) {
  if constexpr (!BATCH) {
    return a.s[k];
  } else {
    const dn_scale_geom& g = bt.geom[(int64_t)img * a.n_scales + k];
    RegScale r{g.plane, g.y, g.x, g.r0, g.r1, g.c0, g.c1, 0, g.sy, g.sx};
    const bool inside = g.plane >= 0 && g.plane < bt.n_maps && g.r0 >= 0 && g.c0 >= 0 &&
                        g.r1 < bt.map_h && g.c1 < bt.map_w;
    r.empty = (!inside || g.r1 < g.r0 || g.c1 < g.c0) ? 1 : 0;
    return r;
  }
}

// POOL = false: bilinear samples at the bin centres; POOL = true: per-channel max over each bin's cells.
// BATCH = true: the maps of a cross-image packed batch (bt), else per-image maps (a).  SC: the window
// side S as a compile-time constant (6, the paper's windows), or 0 to take it from a.S.
template <typename T, bool POOL, bool BATCH, int SC>
__global__ __launch_bounds__(256) void region_windows_kernel(const T* __restrict__ maps, RegArgs a,
                                                             RegBatch bt,
                                                             const float* __restrict__ boxes,
                                                             const int32_t* __restrict__ box_img,
                                                             float* __restrict__ out,
                                                             int32_t* __restrict__ scale_out,
                                                             int32_t* __restrict__ idx_out) {
#pragma clang fp contract(off)
  extern __shared__ __align__(16) float s_row[];  // S * S rows of C + 2 floats
  __shared__ int s_i0[MAX_S], s_j0[MAX_S], s_i1[MAX_S], s_j1[MAX_S];
  __shared__ float s_ly[MAX_S], s_lx[MAX_S];
  // byte offsets of the sample rows i0, i1 and columns j0, j1 within the map (below 2^31 bytes)
  __shared__ uint32_t s_ro0[MAX_S], s_ro1[MAX_S], s_co0[MAX_S], s_co1[MAX_S];
  const int r = blockIdx.x;
  const int S = SC ? SC : a.S, C = a.C, SS = S * S;
  const int tid = threadIdx.x;
  const double x1 = boxes[4 * r + 0], y1 = boxes[4 * r + 1], x2 = boxes[4 * r + 2],
               y2 = boxes[4 * r + 3];
  const double bw = x2 - x1, bh = y2 - y1;
  const int img = box_img ? box_img[r] : 0;
  const bool valid = img >= 0 && img < a.n_img && isfinite(x1) && isfinite(y1) && isfinite(x2) &&
                     isfinite(y2) && bw > 0 && bh > 0;
  // Scale choice: lane k of wave 0 evaluates scale k (k < n_scales <= 64), then the wave takes the
  // minimum cost, ties to the smaller k, which is the first minimum in increasing k.
  __shared__ int s_best;
  if (tid < 64) {
    double cost = INFINITY;
    int k = tid;
    const RegScale ek = valid && k < a.n_scales ? entry<BATCH>(a, bt, img, k) : RegScale{};
    if (valid && k < a.n_scales && !ek.empty) {
      const double T2 = a.target * a.target;
      const double area = (ek.sy * bh) * (ek.sx * bw);
      const double p = area / T2, q = T2 / area;
      cost = p < q ? q : p;
      if (a.n_aspects > 1) {
        const double rho = (ek.sx * bw) / (ek.sy * bh), irho = 1.0 / rho;
        cost = cost * (rho < irho ? irho : rho);
      }
    } else {
      k = 1 << 30;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const double oc = __shfl_xor(cost, off);
      const int ok = __shfl_xor(k, off);
      if (oc < cost || (oc == cost && ok < k)) {
        cost = oc;
        k = ok;
      }
    }
    if (tid == 0) s_best = k < a.n_scales ? k : -1;
  }
  __syncthreads();
  const int best = s_best;
  float* dst = out + (int64_t)r * C * SS;
  constexpr int IDXW = POOL ? 4 : 2;  // idx_out entries per bin
  if (best < 0) {
    for (int e = tid; e < C * SS; e += blockDim.x) dst[e] = 0.f;
    if (tid == 0) scale_out[r] = -1;
    if (idx_out)
      for (int e = tid; e < IDXW * SS; e += blockDim.x) idx_out[(int64_t)r * IDXW * SS + e] = 0;
    return;
  }
  const RegScale sc = entry<BATCH>(a, bt, img, best);
  const int Wc = BATCH ? bt.map_w : a.map_w[sc.plane];
  if (POOL && tid < 2 * S) {
    const bool row = tid < S;
    const int t = row ? tid : tid - S;
    const double lo = row ? y1 * sc.sy + (double)sc.y + (double)a.pad : x1 * sc.sx + (double)sc.x + (double)a.pad;
    const double hi = row ? y2 * sc.sy + (double)sc.y + (double)a.pad : x2 * sc.sx + (double)sc.x + (double)a.pad;
    int first, last;
    pool_bin_range(lo + ((double)t * (hi - lo)) / (double)S, lo + ((double)(t + 1) * (hi - lo)) / (double)S,
                   row ? sc.r0 : sc.c0, row ? sc.r1 : sc.c1, first, last);
    if (row) {
      s_i0[t] = first;
      s_i1[t] = last;
    } else {
      s_j0[t] = first;
      s_j1[t] = last;
    }
  }
  if (!POOL && tid < 2 * S) {
    // tid < S: row sample a = tid; S <= tid < 2S: column sample b = tid - S
    const bool row = tid < S;
    const int t = row ? tid : tid - S;
    const double f = ((double)t + 0.5) / (double)S;
    double lo, hi, cmin, cmax;
    if (row) {
      lo = y1 * sc.sy + (double)sc.y + (double)a.pad;
      hi = y2 * sc.sy + (double)sc.y + (double)a.pad;
      cmin = sc.r0;
      cmax = sc.r1;
    } else {
      lo = x1 * sc.sx + (double)sc.x + (double)a.pad;
      hi = x2 * sc.sx + (double)sc.x + (double)a.pad;
      cmin = sc.c0;
      cmax = sc.c1;
    }
    double g = ((lo + f * (hi - lo)) - 17.5) * 0.0625;
    g = g < cmin ? cmin : (g > cmax ? cmax : g);
    const int i0 = (int)floor(g);
    const int i1 = min(i0 + 1, (int)cmax);
    const float lam = (float)(g - (double)i0);
    if (row) {
      s_i0[t] = i0;
      s_i1[t] = i1;
      s_ly[t] = lam;
      s_ro0[t] = (uint32_t)i0 * (uint32_t)Wc * (uint32_t)(C * sizeof(T));
      s_ro1[t] = (uint32_t)i1 * (uint32_t)Wc * (uint32_t)(C * sizeof(T));
    } else {
      s_j0[t] = i0;
      s_j1[t] = i1;
      s_lx[t] = lam;
      s_co0[t] = (uint32_t)i0 * (uint32_t)(C * sizeof(T));
      s_co1[t] = (uint32_t)i1 * (uint32_t)(C * sizeof(T));
    }
  }
  __syncthreads();
  const T* F = BATCH ? maps + (int64_t)sc.plane * bt.map_stride
                     : maps + (int64_t)img * a.image_stride + a.map_off[sc.plane];
  // Each thread blends VT consecutive channels (one 16-byte vector per neighbour cell); C / VT
  // threads cover a bin, and the workgroup's groups of C / VT threads take different bins.  The
  // results are staged bin-major, one row of C + 2 floats per bin in channel order (8-byte writes),
  // then read out in the output's channel-major order: each thread gathers 4 consecutive bins of one
  // channel and writes them with one 16-byte store.  With the row stride C + 2, the lanes of a read
  // (up to 8 channels x bins 4 apart) fall on distinct banks.
  constexpr int VT = 16 / sizeof(T);
  typedef T vec_t __attribute__((ext_vector_type(VT)));
  const int per_bin = C / VT, groups = blockDim.x / per_bin;
  const int lt = tid % per_bin, grp = tid / per_bin;
  const int RSTR = C + 2;
  constexpr int NQ = VT / 4;  // 16-byte float chunks per thread and bin
  constexpr int MAXIT = 5;  // bins per thread whose loads are all issued before any blend
  if (!POOL && grp < groups && SS <= MAXIT * groups) {
    // Bilinear bins, up to MAXIT per thread (S <= 6 with 16-bit maps): all 4 MAXIT cell vectors are
    // in flight at once (buffer loads at the bins' byte offsets: one add each), then blended with the
    // four bilinear weights of the bin.
    const int c0 = lt * VT;
    const uint32_t cb = (uint32_t)(c0 * sizeof(T));
    const __amdgpu_buffer_rsrc_t rf = __builtin_amdgcn_make_buffer_rsrc((void*)F, 0, 0x7fffffff, 0x00020000);
    vec_t a[MAXIT][4];
#pragma unroll
    for (int it = 0; it < MAXIT; ++it) {
      const int bin = grp + it * groups;
      if (bin < SS) {
        const int u = bin / S, v = bin - u * S;
        const uint32_t r0 = s_ro0[u] + cb, r1 = s_ro1[u] + cb, q0 = s_co0[v], q1 = s_co1[v];
        a[it][0] = __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(rf, r0 + q0, 0, 0));
        a[it][1] = __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(rf, r0 + q1, 0, 0));
        a[it][2] = __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(rf, r1 + q0, 0, 0));
        a[it][3] = __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(rf, r1 + q1, 0, 0));
      }
    }
#pragma unroll
    for (int it = 0; it < MAXIT; ++it) {
      const int bin = grp + it * groups;
      if (bin < SS) {
        const int u = bin / S, v = bin - u * S;
        const float ly = s_ly[u], lx = s_lx[v], my = 1.f - ly, mx = 1.f - lx;
        const float w00 = my * mx, w01 = my * lx, w10 = ly * mx, w11 = ly * lx;
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
          f32x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int q = 4 * k + e;
            const float v00 = to_f32(a[it][0][q]), v01 = to_f32(a[it][1][q]);
            const float v10 = to_f32(a[it][2][q]), v11 = to_f32(a[it][3][q]);
            o[e] = __builtin_fmaf(w11, v11, __builtin_fmaf(w10, v10, __builtin_fmaf(w01, v01, w00 * v00)));
          }
          float* d = s_row + bin * RSTR + c0 + 4 * k;
          *(float2*)d = make_float2(o[0], o[1]);
          *(float2*)(d + 2) = make_float2(o[2], o[3]);
        }
      }
    }
  } else if (grp < groups) {
    const int c0 = lt * VT;
    for (int bin = grp; bin < SS; bin += groups) {
      const int u = bin / S, v = bin - u * S;
      const int i0 = s_i0[u], i1 = s_i1[u], j0 = s_j0[v], j1 = s_j1[v];
      if constexpr (POOL) {
        float m[VT];
        const vec_t f = *(const vec_t*)(F + ((int64_t)i0 * Wc + j0) * C + c0);
#pragma unroll
        for (int q = 0; q < VT; ++q) m[q] = to_f32(f[q]);
        for (int i = i0; i <= i1; ++i)
          for (int j = j0; j <= j1; ++j) {
            const vec_t x = *(const vec_t*)(F + ((int64_t)i * Wc + j) * C + c0);
#pragma unroll
            for (int q = 0; q < VT; ++q) m[q] = fmaxf(m[q], to_f32(x[q]));
          }
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
          float* d = s_row + bin * RSTR + c0 + 4 * k;
          *(float2*)d = make_float2(m[4 * k], m[4 * k + 1]);
          *(float2*)(d + 2) = make_float2(m[4 * k + 2], m[4 * k + 3]);
        }
        continue;
      }
      const float ly = s_ly[u], lx = s_lx[v];
      const vec_t a00 = *(const vec_t*)(F + ((int64_t)i0 * Wc + j0) * C + c0);
      const vec_t a01 = *(const vec_t*)(F + ((int64_t)i0 * Wc + j1) * C + c0);
      const vec_t a10 = *(const vec_t*)(F + ((int64_t)i1 * Wc + j0) * C + c0);
      const vec_t a11 = *(const vec_t*)(F + ((int64_t)i1 * Wc + j1) * C + c0);
#pragma unroll
      for (int k = 0; k < NQ; ++k) {
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int q = 4 * k + e;
          const float v00 = to_f32(a00[q]), v01 = to_f32(a01[q]);
          const float v10 = to_f32(a10[q]), v11 = to_f32(a11[q]);
          const float top = __builtin_fmaf(lx, v01 - v00, v00), bot = __builtin_fmaf(lx, v11 - v10, v10);
          o[e] = __builtin_fmaf(ly, bot - top, top);
        }
        float* d = s_row + bin * RSTR + c0 + 4 * k;  // natural channel order, 8-byte aligned
        *(float2*)d = make_float2(o[0], o[1]);
        *(float2*)(d + 2) = make_float2(o[2], o[3]);
      }
    }
  }
  __syncthreads();
  if ((SS & 3) == 0 && ((uintptr_t)dst & 15) == 0) {
    // four consecutive bins of one channel per thread, one 16-byte store
    for (int e4 = tid; e4 < (C * SS) / 4; e4 += blockDim.x) {
      const int e = 4 * e4, c = e / SS, bin = e - c * SS;
      f32x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = s_row[(bin + i) * RSTR + c];
      __builtin_nontemporal_store(o, (f32x4*)(dst + e));  // written once, not read back here
    }
  } else {
    for (int e = tid; e < C * SS; e += blockDim.x) {
      const int c = e / SS, bin = e - c * SS;
      dst[e] = s_row[bin * RSTR + c];
    }
  }
  if (tid == 0) scale_out[r] = best;
  if (idx_out)
    for (int e = tid; e < SS; e += blockDim.x) {
      int32_t* q = idx_out + ((int64_t)r * SS + e) * IDXW;
      if constexpr (POOL) {
        q[0] = s_i0[e / S];
        q[1] = s_i1[e / S];
        q[2] = s_j0[e % S];
        q[3] = s_j1[e % S];
      } else {
        q[0] = s_i0[e / S];
        q[1] = s_j0[e % S];
      }
    }
}

template <bool POOL, bool BATCH>
int launch(const void* d_conv5, dn_dtype dt, const RegArgs& a, const RegBatch& bt, const float* d_boxes,
           const int32_t* d_box_img, int32_t n, float* d_out, int32_t* d_scale, int32_t* d_idx,
           hipStream_t s) {
  if (a.S > MAX_S || a.S <= 0) return (int)hipErrorInvalidValue;
  const size_t lds = sizeof(float) * (size_t)(a.C + 2) * a.S * a.S;
  auto go = [&](auto tag) {
    using T = decltype(tag);
    if (a.S == 6)
      region_windows_kernel<T, POOL, BATCH, 6><<<n, 256, lds, s>>>((const T*)d_conv5, a, bt, d_boxes,
                                                                   d_box_img, d_out, d_scale, d_idx);
    else
      region_windows_kernel<T, POOL, BATCH, 0><<<n, 256, lds, s>>>((const T*)d_conv5, a, bt, d_boxes,
                                                                   d_box_img, d_out, d_scale, d_idx);
  };
  switch (dt) {
    case DN_F32: go(float{}); break;
    case DN_F16: go(_Float16{}); break;
    case DN_BF16: go(__bf16{}); break;
  }
  return (int)hipGetLastError();
}

}  // namespace

int launch_region_windows(const void* d_conv5, dn_dtype dt, const RegArgs& a, const RegBatch* batch,
                          const float* d_boxes, const int32_t* d_box_img, int32_t n, float* d_out,
                          int32_t* d_scale, int32_t* d_idx, bool pool, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const RegBatch bt = batch ? *batch : RegBatch{};
  if (batch)
    return pool ? launch<true, true>(d_conv5, dt, a, bt, d_boxes, d_box_img, n, d_out, d_scale, d_idx, s)
                : launch<false, true>(d_conv5, dt, a, bt, d_boxes, d_box_img, n, d_out, d_scale, d_idx, s);
  return pool ? launch<true, false>(d_conv5, dt, a, bt, d_boxes, d_box_img, n, d_out, d_scale, d_idx, s)
              : launch<false, false>(d_conv5, dt, a, bt, d_boxes, d_box_img, n, d_out, d_scale, d_idx, s);
}

}  // namespace dn
