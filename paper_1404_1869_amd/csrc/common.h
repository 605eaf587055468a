// Internal declarations shared by the library's translation units: status helpers, the host plan,
// device type traits for the three storage types and the MFMA tiles of gfx950, and the launchers.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "densenet.h"

#if defined(__HIPCC__)
#include <hip/hip_runtime.h>
#endif

namespace dn {

// ---------------------------------------------------------------------------------------------
// Errors
// ---------------------------------------------------------------------------------------------
void set_error(const std::string& msg);
int fail(int status, const std::string& msg);

// ---------------------------------------------------------------------------------------------
// Host geometry (plan.cpp)
// ---------------------------------------------------------------------------------------------
struct PlaneSize {
  int32_t h, w;
};

struct Plan {
  std::vector<dn_scale_geom> scales;
  std::vector<PlaneSize> planes;  // planes of one image
};

// Sizes after conv1, pool1, conv2, pool2, conv3, conv4, conv5, pool5 of an n-px side (0 = empty).
void stack_sides(int64_t n, int64_t out[8]);

// Scale list, rectangles, stitching and conv5 windows.  Returns DN_OK or an error status (message
// set).
int make_plan(int32_t H, int32_t W, const dn_pyramid_params& p, Plan& plan);

// Cross-image packing: the entries of n_img images stitched as one set of items (item b * E + e is
// entry e of image b, .image = b, batch-wide plane indices).  Returns DN_OK or an error status.
int make_plan_batch(int32_t n_img, int32_t H, int32_t W, const dn_pyramid_params& p,
                    std::vector<dn_scale_geom>& items, int& n_planes);

// ---------------------------------------------------------------------------------------------
// Launchers (device code in the .hip files).  Every launcher enqueues on `stream` and returns
// hipGetLastError() as an int (0 = success).
// ---------------------------------------------------------------------------------------------
struct PyrScale {  // per-scale parameters of the plane builder, passed by value
  int32_t plane, y, x, rh, rw, h, w;
};
struct PyrArgs {
  int32_t n_scales;
  int32_t H, W, pad, ramp;
  float mean[3];
  PyrScale s[DN_MAX_SCALES];                    // grouped by plane
  uint8_t plane_first[DN_MAX_PLANES_PER_IMAGE];  // first entry of s[] on each plane
  uint8_t plane_count[DN_MAX_PLANES_PER_IMAGE];  // entries of s[] on each plane
};
// Row pitch of a plane w pixels wide: w rounded up to a multiple of DN_PLANE_ROW_ALIGN elements.
__host__ __device__ inline int32_t plane_pitch(int32_t w) {
  return (w + DN_PLANE_ROW_ALIGN - 1) / DN_PLANE_ROW_ALIGN * DN_PLANE_ROW_ALIGN;
}
struct PyrPlane {
  int32_t h, w;
  int64_t offset;
};
struct PyrPlanes {
  int32_t n;
  int64_t image_elems;
  PyrPlane p[DN_MAX_PLANES_PER_IMAGE];
};

// A cross-image packed batch: placements read from a device copy of the plan (n_items entries),
// planes all PH x PW, plane j at j * 3 * PH * PW elements.  first/list: per-plane item lists the
// launcher builds in the scratch (set by the launcher).
struct BatchGeom {
  const dn_scale_geom* geom;
  int32_t n_items, n_img, n_planes, PH, PW;
  const int32_t* first;
  const int32_t* list;
};
constexpr int32_t MAX_INDEX_PLANES = 16384;  // planes of one packed batch (per-plane lists in LDS)

// Builder scratch: the pixel-interleaved image (4 * H * W * n_img bytes), then for a packed batch the
// per-plane item lists (4 * (n_planes + 1 + n_items) bytes), each part 256-byte aligned.
inline size_t index_offset(int32_t n_img, int32_t H, int32_t W) {
  return ((size_t)n_img * 4 * (size_t)H * (size_t)W + 255) & ~(size_t)255;
}
inline size_t builder_scratch_bytes(int32_t n_img, int32_t H, int32_t W, int32_t n_planes, int32_t n_items) {
  return index_offset(n_img, H, W) + 4 * ((size_t)n_planes + 1 + (size_t)n_items);
}

// d_scratch: builder_scratch_bytes (256-byte aligned; n_planes = n_items = 0 without a batch).  batch:
// NULL for per-image planes (a.s / pl), else the packed batch's placements (a.s and pl unused but H,
// W, pad, ramp, mean).
// Device address of the scratch-free builder's static staging array on the current device (looked up
// once per device).  Returns a hipError_t.
int static_scratch(uint8_t** out);
// max_h, max_w: largest plane; max_scale_w: widest scaled image (selects the exact-integer
// horizontal taps when at most 32767).
int launch_build_planes(const uint8_t* d_img, int32_t n_img, const PyrArgs& a, const PyrPlanes& pl,
                        const BatchGeom* batch, int32_t max_h, int32_t max_w, int32_t max_scale_w,
                        dn_dtype dt, void* d_out, uint8_t* d_scratch, void* stream);

// Crop-before windows: n boxes warped to S x S channel-major planes (windows.hip).
int launch_warp_regions(const uint8_t* d_img, int32_t n_img, int32_t H, int32_t W, const float* d_boxes,
                        const int32_t* d_box_img, int32_t n, int32_t S, int32_t pitch, const float* mean,
                        dn_dtype dt, void* d_out, void* stream);

// Packed weight blob: offsets in bytes of each layer's weights and fp32 biases, and (16-bit types)
// of a second, stage-major copy of the weights that the direct-load conv kernels stream as
// contiguous blocks (0 when absent).
struct PackedLayout {
  size_t w_off[5], b_off[5], s_off[5], total;
};
PackedLayout packed_layout(dn_dtype dt);
int launch_pack_weights(const float* const* d_w, const float* const* d_b, dn_dtype dt, void* d_packed,
                        void* stream);

// A run of a layer launch: n planes of one size, H x W at the layer's input; plane i reads at in_off +
// i in_stride and writes at out_off + i out_stride (elements from the launch's base pointers).  pitch:
// row pitch of conv1's channel-major input planes (>= W, or 0 for W); ignored by the other layers.
struct MapRun {
  int32_t n, H, W, pitch;
  int64_t in_off, in_stride, out_off, out_stride;
};

// The runs of one launch as the kernels see them (passed by value): run r owns the launch's
// workgroups (or wave tiles) first .. first of run r + 1 - 1, its planes' tiles in the kernel's own
// order; Ho x Wo is the layer's output size.  A launch of more runs than MAX_RUNS is issued as
// several launches.
constexpr int MAX_RUNS = 16;
struct KRun {
  int32_t first, H, W, pitch, Ho, Wo, tiles_x, tiles_y;
  int64_t in_off, in_stride, out_off, out_stride;
};
struct KRuns {
  int32_t count;
  KRun r[MAX_RUNS];
};
#if defined(__HIPCC__)
// Buffer resource for `bytes` bytes from p (raw buffer, 32-bit offsets; an offset at or past `bytes`
// reads 0 and drops a store).  p and bytes must be wave-uniform: they are taken from the first active
// lane, so the descriptor stays in scalar registers.  Built from values the compiler cannot prove
// uniform, a descriptor lands in vector registers and every buffer instruction that uses it is
// wrapped in a loop over the distinct descriptors of the wave (one pass when they agree).
__device__ inline __amdgpu_buffer_rsrc_t uniform_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)p;
  // The builtin returns a signed int: each word goes back through uint32_t, so the low word is
  // zero-extended (sign-extending it would corrupt the high word of an address with bit 31 set).
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  return __builtin_amdgcn_make_buffer_rsrc((void*)(lo | hi << 32), 0,
                                           __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000);
}

// Run of workgroup (or tile) index b: the last run whose first index is at most b.  The table sits in
// the kernel arguments; a wave-uniform index reads its fields with scalar loads.  MULTI = false: a
// launch of one run, whose fields then sit at fixed offsets like plain scalar arguments (no loads
// per tile, whose waits would also drain a kernel's LDS pipeline).
template <bool MULTI = true>
__device__ inline int run_of(const KRuns& t, int b) {
  if constexpr (!MULTI) {
    return 0;
  } else {
    int k = 0;
#pragma unroll
    for (int i = 1; i < MAX_RUNS; ++i) k = (i < t.count && b >= t.r[i].first) ? i : k;
    return __builtin_amdgcn_readfirstlane(k);
  }
}
#endif
// The kernel table of runs [0, n) (1 <= n <= MAX_RUNS): geometry(k) sets k's Ho, Wo, tiles_x and
// tiles_y from its input size and returns the workgroups (or tiles) of one plane.  Returns the
// launch's total, or -1 when n is out of range, a run is empty or the total passes 2^31 - 1.
template <typename G>
inline int64_t fill_kruns(const MapRun* runs, int n, KRuns& t, G&& geometry) {
  t = KRuns{};
  if (n <= 0 || n > MAX_RUNS) return -1;  // callers issue one launch per MAX_RUNS runs
  t.count = n;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    KRun& k = t.r[i];
    k.first = (int32_t)total;
    k.H = runs[i].H, k.W = runs[i].W, k.pitch = runs[i].pitch > 0 ? runs[i].pitch : runs[i].W;
    k.in_off = runs[i].in_off, k.in_stride = runs[i].in_stride;
    k.out_off = runs[i].out_off, k.out_stride = runs[i].out_stride;
    const int64_t per = geometry(k);
    if (per <= 0 || runs[i].n <= 0) return -1;
    total += per * runs[i].n;
    if (total > 0x7fffffffLL) return -1;
  }
  return total > 0 ? total : -1;
}

// One conv layer (1..5) with bias and ReLU over the planes of `runs` (any number of runs; one launch
// per MAX_RUNS of them).  d_part: conv_part_bytes(...) bytes of device workspace for the partial sums
// of fp32 launches too small to fill the chip, which then split their input channels (NULL or too
// small: no split).
int launch_conv(int layer, const void* d_in, const MapRun* runs, int32_t n_runs, dn_dtype dt,
                const void* d_packed, void* d_out, void* d_part, size_t part_bytes, void* stream);
size_t conv_part_bytes(int layer, const MapRun* runs, int32_t n_runs, dn_dtype dt);

// LRN + pool (order by lrn_first), or plain pool when lrn == false, over the channels-last maps of
// `runs` (one launch per MAX_RUNS runs).
int launch_lrn_pool(const void* d_in, const MapRun* runs, int32_t n_runs, int32_t C, dn_dtype dt,
                    bool lrn, bool lrn_first, float alpha, float beta, float k, int32_t lrn_n,
                    void* d_out, void* stream);

struct RegScale {
  int32_t plane, y, x, r0, r1, c0, c1;
  int32_t empty;
  double sy, sx;
};
struct RegArgs {
  int32_t n_scales, pad, planes_per_img, S, C, n_img;
  int32_t n_aspects;  // > 1: several aspect-ratio pyramids, the scale cost includes the box aspect
  double target;
  RegScale s[DN_MAX_SCALES];
  int64_t map_off[DN_MAX_PLANES_PER_IMAGE];  // offset of plane j's map within an image's maps
  int32_t map_w[DN_MAX_PLANES_PER_IMAGE];
  int64_t image_stride;                       // elements between images' maps
};
// Conv5 maps of a cross-image packed batch: entry e of image b at geom[b * a.n_scales + e] (device),
// map j at j * map_stride elements, every map map_h x map_w.
struct RegBatch {
  const dn_scale_geom* geom;
  int64_t map_stride;
  int32_t n_maps, map_h, map_w;
};
// pool = false: bilinear samples at bin centres (d_idx [n][S][S][2]); true: per-bin max over the cells
// centred inside each bin (d_idx [n][S][S][4]).  batch: NULL for per-image maps (a.s, a.map_*).
int launch_region_windows(const void* d_conv5, dn_dtype dt, const RegArgs& a, const RegBatch* batch,
                          const float* d_boxes, const int32_t* d_box_img, int32_t n, float* d_out,
                          int32_t* d_scale, int32_t* d_idx, bool pool, void* stream);

inline size_t dtype_size(dn_dtype dt) { return dt == DN_F32 ? 4 : 2; }

// Brackets one kernel launch with trace events when tracing is on and the name is selected.
class TraceScope {
 public:
  TraceScope(const char* name, void* stream);
  ~TraceScope();
  TraceScope(const TraceScope&) = delete;
  TraceScope& operator=(const TraceScope&) = delete;

 private:
  int idx_;
  void* stream_;
};

}  // namespace dn

#if defined(__HIPCC__)
namespace dn {
// ---------------------------------------------------------------------------------------------
// Device side: storage types and the gfx950 MFMA tiles used by the conv kernels.
//   32x32x16 f16 / bf16: each lane holds 8 consecutive k of row (lane % 32) of A and column
//   (lane % 32) of B, k offset 8 * (lane / 32); 32x32x2 f32: one k, offset lane / 32.  The
//   accumulator register r of lane l holds D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
// ---------------------------------------------------------------------------------------------
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T>
struct Mfma;
template <>
struct Mfma<_Float16> {
  static constexpr int KPL = 8, KS = 16;
  typedef f16x8 frag;
  typedef f16x4 half_frag;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<__bf16> {
  static constexpr int KPL = 8, KS = 16;
  typedef bf16x8 frag;
  typedef bf16x4 half_frag;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<float> {
  static constexpr int KPL = 1, KS = 2;
  typedef float frag;
  typedef float half_frag;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

template <typename T>
__device__ inline T from_f32(float x) {
  return (T)x;  // round to nearest even for _Float16 and __bf16
}
template <typename T>
__device__ inline float to_f32(T x) {
  return (float)x;
}
// Two values rounded to T (nearest even) as a packed pair: one v_cvt_pk_bf16_f32 for bf16.
template <typename T>
__device__ inline T __attribute__((ext_vector_type(2))) from_f32x2(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef T t2 __attribute__((ext_vector_type(2)));
  return __builtin_convertvector(f2{a, b}, t2);
}

}  // namespace dn
#endif
