/* densenet.h — C ABI of the DenseNet conv5 descriptor-pyramid library for one MI355X (gfx950).
 *
 * Method: Iandola et al., "DenseNet: Implementing Efficient ConvNet Descriptor Pyramids",
 * arXiv 1404.1869.  An image is resampled to a multiscale pyramid (Sec. 3.1), centred on one mean
 * pixel (Sec. 3.2), each scale is padded by a 16-px border and the scales are stitched onto large
 * planes (Sec. 3.1, Bottom-Left Fill); conv1..conv5 of the AlexNet topology then run on every plane,
 * and the conv5 maps are unpacked per scale (Sec. 3.1) and read out as fixed-size region windows
 * ("crop after", Sec. 4).  The paper's own interface is pyra = convnet_featpyramid(image) (Sec. 3.5):
 * image in, per-scale feature maps plus the scale-to-plane geometry out.
 *
 * Conventions for every entry point:
 *  - Return value: a dn_status.  Arguments are validated on the host before any device work; no
 *    C++ exception crosses the ABI.  densenet_last_error() returns a thread-local message for the
 *    last failing call on this thread.
 *  - Ownership: the caller owns every buffer.  d_* pointers are device pointers (256-byte aligned,
 *    as returned by hipMalloc or the torch caching allocator); other pointers are host memory.
 *    The library allocates no device memory.  Its only device state is the staging array of
 *    densenet_build_pyramid_noalloc (DN_STATIC_SCRATCH_BYTES per GPU, part of the code object).
 *  - Size queries: where an output or workspace pointer may be NULL, the call only writes the
 *    required byte count to *_needed and returns DN_OK.  A buffer that is too small returns
 *    DN_E_BUFFER_TOO_SMALL (the needed size is still written).
 *  - Streams: `stream` is a hipStream_t passed as void* (NULL = the default stream).  Device work is
 *    enqueued asynchronously on it; outputs are valid once the stream reaches that point.
 *  - dtypes: DN_F32, DN_F16, DN_BF16 select the storage and MFMA input type of planes and
 *    activations; accumulation is always fp32.  Region descriptors are always fp32.
 *  - Layouts: images are uint8 [n_img][3][H][W].  Planes are channel-major [3][PH][pitch] per plane,
 *    packed back to back, with rows of pitch = PW rounded up to a multiple of DN_PLANE_ROW_ALIGN
 *    elements (columns PW .. pitch-1 hold 0).  Activations and conv5 maps are channels-last [Hc][Wc][C] per plane, packed
 *    back to back.
 */
#ifndef DENSENET_H
#define DENSENET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DN_OK = 0,
  DN_E_INVALID_ARG = -1,      /* null pointer, non-positive size, inconsistent parameters */
  DN_E_TOO_LARGE = -2,        /* a padded scale does not fit the stitching plane, or a limit below */
  DN_E_BUFFER_TOO_SMALL = -3, /* caller buffer shorter than *_needed */
  DN_E_UNSUPPORTED = -4,      /* dtype or mode not implemented */
  DN_E_HIP = -5,              /* a HIP runtime call or kernel launch failed */
  DN_E_INTERNAL = -6
} dn_status;

typedef enum { DN_F32 = 0, DN_F16 = 1, DN_BF16 = 2 } dn_dtype;
typedef enum { DN_PAD_ZERO = 0, DN_PAD_RAMP = 1 } dn_pad_mode;

#define DN_MAX_SCALES 64 /* pyramid entries (scales x aspect ratios) */
/* Row alignment of the planes the library plans and builds, in elements: every row of a plane then
 * starts on a 128-byte boundary (256 at fp32) of a 256-byte aligned buffer, so no two workgroups of
 * the builder write parts of one cache line. */
#define DN_PLANE_ROW_ALIGN 64
#define DN_MAX_PLANES_PER_IMAGE 64
#define DN_MAX_ASPECTS 8

/* Pyramid recipe (Sec. 3.1, 3.2).
 *  scales: s_k = base * 2^(-k / steps_per_octave), k = 0 .. n_scales-1, where base = base_scale, or
 *          base_longest_side / max(H, W) when base_longest_side > 0; scaled sides round half up
 *          (minimum 1).
 *  pad:    border width p around every scale (the paper uses 16).  pad_mode RAMP blends linearly
 *          from the edge pixel to the mean pixel: weight (p+1-d)/(p+1) at distance d, product of the
 *          row and column weights at corners; ZERO fills the border with the mean pixel.
 *  plane_h, plane_w: 0,0 => every padded scale is its own plane; otherwise the scales, padded and
 *          rounded up to multiples of 16 px, are stitched onto planes of this size by Bottom-Left
 *          Fill (largest first; first plane, then topmost, then leftmost candidate corner).
 *  mean:   the mean pixel subtracted from input channels 0, 1, 2 (the background of every plane
 *          is the mean pixel, i.e. 0 after centring).
 *  n_aspects, aspects: aspect-ratio pyramids (Sec. 3.3).  0 => one pyramid of the image.  Otherwise
 *          the image warped to each ratio r = aspects[a] > 0 gets a whole pyramid, keeping its area:
 *          entry e = a * n_scales + k has sides floor(H (s_k / sqrt(r)) + 0.5) x floor(W (s_k sqrt(r))
 *          + 0.5) (minimum 1), and all n_aspects * n_scales entries (at most DN_MAX_SCALES) are
 *          stitched together; geometry arrays then hold one dn_scale_geom per entry. */
typedef struct {
  int32_t n_scales;
  int32_t steps_per_octave;
  double base_scale;
  int32_t base_longest_side;
  int32_t pad;
  int32_t pad_mode;
  int32_t plane_h, plane_w;
  float mean[3];
  int32_t n_aspects;
  double aspects[DN_MAX_ASPECTS];
} dn_pyramid_params;

/* Geometry of pyramid entry k (a scale of one aspect ratio), identical for every image of a batch
 * (Sec. 3.1 unpacking).  k: entry index (aspect * n_scales + scale); aspect: index into aspects (0
 * for a single pyramid); s: the scale factor s_k of the entry's scale.  image: the image the entry
 * belongs to in a cross-image packed batch (densenet_plan_batch), else 0.
 *  (h, w): scaled image size; sy = h/H, sx = w/W are the effective factors.
 *  plane:  index of the scale's plane within one image's planes (within the whole batch's planes for
 *          a cross-image packed batch).
 *  (y, x, rh, rw): padded rectangle on that plane; the real pixels start at (y+pad, x+pad).
 *  [r0, r1] x [c0, c1]: conv5 cells of that plane whose receptive-field centre (16 i + 17.5 in
 *          continuous plane coordinates) lies on a real pixel of the scale; the scale's feature map
 *          is that window of the plane's conv5 map.  Empty when r1 < r0 or c1 < c0. */
typedef struct {
  int32_t k, h, w, plane;
  int32_t y, x, rh, rw;
  int32_t r0, r1, c0, c1;
  int32_t aspect, image;
  double s, sy, sx;
} dn_scale_geom;

/* One plane or map: h x w pixels at `offset` elements from the start of its buffer.
 * pitch: elements between consecutive rows of a channel-major plane (channels are h * pitch apart);
 * 0 means w.  The planners and builders write pitch = w rounded up to a multiple of
 * DN_PLANE_ROW_ALIGN; densenet_conv_features takes any pitch >= w (a multiple of 8 lets conv1 load
 * plane rows directly into LDS whatever the width); the columns between w and pitch are never read
 * into a stored output.  Maps (conv5, pool5) and every other use ignore pitch and write 0. */
typedef struct {
  int32_t h, w;
  int64_t offset;
  int32_t pitch;
  int32_t reserved; /* 0 */
} dn_plane_desc;

/* Network options (Sec. 3: conv1..conv5 of the AlexNet topology, with ReLU, cross-channel LRN and
 * 3x3/2 max-pooling after conv1 and conv2).  LRN: b_c = a_c (k + alpha/n sum_{|j-c|<=n/2} a_j^2)^-beta
 * over all channels of the layer; pooling uses ceil-mode sizes with windows clipped to the input.
 * lrn_n must be odd and at most 9.  lrn_before_pool = 1 applies LRN then pool, 0 pool then LRN.  pool5 = 1 also emits 3x3/2 max-pooled
 * conv5 maps. */
typedef struct {
  float lrn_alpha, lrn_beta, lrn_k;
  int32_t lrn_n;
  int32_t lrn_before_pool;
  int32_t pool5;
} dn_net_params;

/* Geometry only (host, no device work): scales, sizes, stitching and conv5 windows for an H x W image.
 * Image sides are limited to 32768 px and scaled sides to 65535 px (DN_E_TOO_LARGE beyond).
 * geom: [n_scales] out.  planes: [max_planes] out, the planes of ONE image (h, w, pitch and offset in
 * elements of the packed [3][h][pitch] planes); *image_elems = elements per image.  Returns DN_E_TOO_LARGE when a padded
 * scale exceeds the stitching plane or the plane count exceeds max_planes. */
int densenet_plan_pyramid(int32_t H, int32_t W, const dn_pyramid_params* p, dn_scale_geom* geom,
                          dn_plane_desc* planes, int32_t max_planes, int32_t* n_planes,
                          int64_t* image_elems);

/* Image(s) in -> centred, padded, stitched planes out (Sec. 3.1, 3.2), one fused kernel.
 * d_images: uint8 [n_img][3][H][W].  d_planes: n_img consecutive blocks of *image_elems elements of
 * `dtype`, image b's plane j at b * image_elems + planes[j].offset, or NULL for a size query.
 * *bytes_needed (and so planes_bytes) also covers a trailing scratch region after the planes
 * (4 * H * W * n_img bytes, 256-byte aligned) that the call uses while it runs; its contents
 * afterwards are unspecified.  geom/planes/n_planes/image_elems as densenet_plan_pyramid.  An image is
 * limited to 2^30 - 1 pixels and a plane (3 * h * pitch elements) to 2^31 - 1 bytes (DN_E_TOO_LARGE). */
int densenet_build_pyramid(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                           const dn_pyramid_params* p, dn_dtype dtype, void* d_planes,
                           size_t planes_bytes, size_t* bytes_needed, dn_scale_geom* geom,
                           dn_plane_desc* planes, int32_t max_planes, int32_t* n_planes,
                           int64_t* image_elems, void* stream);

/* Scratch-free variant of densenet_build_pyramid, for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops and harnesses that forbid hipMalloc).  Same arguments,
 * validation and planes as densenet_build_pyramid, but d_planes holds the planes only: *bytes_needed
 * is the planes' size, with no trailing scratch region.  The builder's pixel-interleaved image stages
 * in a library-owned device array of DN_STATIC_SCRATCH_BYTES on each GPU, which that GPU holds until
 * the process ends; 4 * H * W * n_img above DN_STATIC_SCRATCH_BYTES returns DN_E_TOO_LARGE (checked
 * before any device work).  The call allocates nothing; its first call on a GPU looks the array up
 * (a runtime query, no allocation).  Every call on one GPU shares that GPU's array: calls that overlap
 * on one GPU (different streams or threads with no ordering between them) race and give wrong planes;
 * calls ordered on one stream are safe.  No part of the array needs to start at zero. */
#define DN_STATIC_SCRATCH_BYTES (64u << 20)
int densenet_build_pyramid_noalloc(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                                   const dn_pyramid_params* p, dn_dtype dtype, void* d_planes,
                                   size_t planes_bytes, size_t* bytes_needed, dn_scale_geom* geom,
                                   dn_plane_desc* planes, int32_t max_planes, int32_t* n_planes,
                                   int64_t* image_elems, void* stream);

/* Cross-image packing: Bottom-Left Fill stitching (Sec. 3.1) applied to a whole batch, so that the
 * small scales of several images share planes instead of each image leaving a half-empty last plane
 * (16 images of 768 x 1024, 25 scales at 2^-0.1 on 1200 x 1200 planes: 88 planes instead of 96).
 * Geometry only (host, no device work).  The E = n_scales * max(1, n_aspects) entries of each of the
 * n_img images (all H x W) are n_img * E items, stitched as densenet_plan_pyramid stitches one
 * image's entries, ties going to the smaller item index b * E + e.  p->plane_h and plane_w must be
 * positive.  geom: [n_img * E] out, entry e of image b at b * E + e, with .image = b, .k = e and .plane
 * counting over the batch.  planes: [max_planes] out, plane j of plane_h x plane_w at offset
 * j * 3 * plane_h * pitch elements, pitch = plane_w rounded up to a multiple of DN_PLANE_ROW_ALIGN;
 * *total_elems = elements of all planes.  Returns DN_E_TOO_LARGE
 * when more than max_planes planes are needed (*n_planes still receives the count) or n_img * E
 * exceeds DN_MAX_BATCH_ITEMS. */
#define DN_MAX_BATCH_ITEMS 65536
int densenet_plan_batch(int32_t n_img, int32_t H, int32_t W, const dn_pyramid_params* p,
                        dn_scale_geom* geom, dn_plane_desc* planes, int32_t max_planes,
                        int32_t* n_planes, int64_t* total_elems);

/* Planes of a cross-image packed batch: the fused resize + centre + pad + stitch of
 * densenet_build_pyramid, with every rectangle sampled from its own image.
 * geom: the host array of n_img * E entries that densenet_plan_batch wrote for (n_img, H, W, *p), and
 * d_geom: a device copy of it (the kernel reads the placements there; upload it once per plan).
 * The host array is validated; an entry of d_geom that is not a placement inside a plane of this
 * batch is ignored by the kernel (its pixels stay background), so a stale copy gives wrong planes but
 * no out-of-bounds access.  d_planes: [n_planes][3][plane_h][pitch] in `dtype`, followed by the
 * builder's scratch (the pixel image, 4 * H * W * n_img bytes, then per-plane item lists,
 * 4 * (n_planes + 1 + n_img * E) bytes, each part 256-byte aligned; contents afterwards unspecified),
 * or NULL for a size query into *bytes_needed.  n_img * H * W must be below 2^30, a plane's
 * 3 * plane_h * pitch elements below 2^31 bytes, and n_planes at most 16384 (DN_E_TOO_LARGE). */
int densenet_build_batch(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                         const dn_pyramid_params* p, dn_dtype dtype, const dn_scale_geom* geom,
                         const dn_scale_geom* d_geom, int32_t n_planes, void* d_planes,
                         size_t planes_bytes, size_t* bytes_needed, void* stream);

/* Repack conv1..conv5 weights for the kernels.  d_w[l]: device fp32 OIHW weights of layer l
 * (96x3x11x11, 256x48x5x5, 384x256x3x3, 384x192x3x3, 256x192x3x3); d_b[l]: device fp32 biases.
 * d_packed: output blob in `dtype` (biases stay fp32), or NULL for a size query. */
int densenet_pack_weights(const float* const* d_w, const float* const* d_b, dn_dtype dtype,
                          void* d_packed, size_t packed_bytes, size_t* bytes_needed, void* stream);

/* Planes -> conv5 maps (+ pool5), the whole conv stack (Sec. 3).  planes: [n_planes] descriptors of
 * the planes to run (offsets into d_planes, elements of `dtype`), of any sizes.  Consecutive planes
 * of equal size whose offsets are evenly spaced form a run; each layer is one launch over up to 16
 * runs (more runs take more launches), so planes of different sizes (one plane per scale, several
 * images) share their launches.  d_packed from densenet_pack_weights with the same dtype.
 * d_workspace: scratch of ws_bytes (NULL => size query into *ws_needed): two buffers, each holding
 * one layer's maps of all planes back to back, and for fp32 launches too small to fill the GPU
 * (whose workgroups then split the input channels) room for their partial sums.
 * d_conv5: out, per plane [Hc][Wc][256] packed back to back (descs in conv5_desc[n_planes]).
 * d_pool5: nullable; when net->pool5 it receives [Hp][Wp][256] per plane (descs in pool5_desc).
 * *conv5_needed / *pool5_needed receive the output sizes in bytes (size query when d_conv5 == NULL). */
int densenet_conv_features(const void* d_planes, const dn_plane_desc* planes, int32_t n_planes,
                           dn_dtype dtype, const void* d_packed, const dn_net_params* net,
                           void* d_workspace, size_t ws_bytes, size_t* ws_needed, void* d_conv5,
                           size_t conv5_bytes, size_t* conv5_needed, dn_plane_desc* conv5_desc,
                           void* d_pool5, size_t pool5_bytes, size_t* pool5_needed,
                           dn_plane_desc* pool5_desc, void* stream);

/* Region windows ("crop after", Sec. 4).  For each box (x1, y1, x2, y2) of original-image pixel-edge
 * coordinates (fp32), the scale k whose scaled box area (sy bh)(sx bw) is closest to target^2 in log
 * ratio (ties to the smaller k; scales with an empty window skipped) is chosen, and S x S bilinear
 * samples at the bin centres of the box are read from that scale's conv5 window (coordinates clamped
 * to the window), all 256 channels: d_out[n][256 * S * S] fp32, flattened (channel, row, column).
 * S must be in 1..8 (DN_E_UNSUPPORTED otherwise; the paper's windows are 6 x 6).
 * geom/n_scales: all pyramid entries; when they span several aspect ratios (geom[k].aspect > 0 for
 * some k, Sec. 3.3) the cost of entry k is multiplied by max(rho, 1/rho), rho = (sx bw)/(sy bh) the
 * box's aspect on that entry, so each box is read where it is closest to a target x target square.
 * conv5_desc: [n_img * planes_per_img] maps from densenet_conv_features (image b's plane j at index
 * b * planes_per_img + j), channels-last with 256 channels, offsets multiples of 16 bytes, each map
 * below 2^31 bytes (DN_E_TOO_LARGE).  d_box_img: nullable [n] image index per box (NULL => image 0).
 * d_scale: [n] chosen scale, -1 for a box with a non-finite or non-positive side (its row is 0).
 * d_idx: nullable [n][S][S][2] int32 (i0, j0) conv5 cell of each sample's top-left neighbour.
 * With n == 0 nothing is launched and d_boxes, d_out, d_scale may be NULL.
 * Index arithmetic is fp64 with + - * / only, so scales and indices are reproducible bit for bit. */
int densenet_region_windows(const void* d_conv5, const dn_plane_desc* conv5_desc, int32_t n_maps,
                            dn_dtype conv5_dtype, const dn_scale_geom* geom, int32_t n_scales,
                            int32_t pad, int32_t planes_per_img, const float* d_boxes,
                            const int32_t* d_box_img, int32_t n, float target, int32_t S,
                            float* d_out, int32_t* d_scale, int32_t* d_idx, void* stream);

/* Max-pooled region bins: descriptor post-processing after the region windows, the pool5-style
 * read-out of a box.  Same arguments, entry choice (scale and aspect) and output layout as
 * densenet_region_windows, but bin (a, b) of the box takes, per channel, the maximum over the conv5
 * cells whose receptive-field centre (16 i + 17.5) lies inside the bin (rows [Y1 + a (Y2-Y1)/S,
 * Y1 + (a+1)(Y2-Y1)/S) in plane coordinates, columns likewise), clipped to the entry's window; a bin
 * holding no cell centre takes the cell nearest its centre.  d_idx: nullable [n][S][S][4] int32
 * (first row, last row, first column, last column) of each bin's cells.  Values are exact maxima of
 * the stored conv5 values; ranges are fp64 with + - * / only, reproducible bit for bit. */
int densenet_region_pool(const void* d_conv5, const dn_plane_desc* conv5_desc, int32_t n_maps,
                         dn_dtype conv5_dtype, const dn_scale_geom* geom, int32_t n_scales,
                         int32_t pad, int32_t planes_per_img, const float* d_boxes,
                         const int32_t* d_box_img, int32_t n, float target, int32_t S, float* d_out,
                         int32_t* d_scale, int32_t* d_idx, void* stream);

/* Region windows (pooled = 0, as densenet_region_windows) or max-pooled bins (pooled = 1, as
 * densenet_region_pool) over the conv5 maps of a cross-image packed batch: a box of image b chooses
 * among entries b * n_entries .. b * n_entries + n_entries - 1 of geom and is read from the map of
 * that entry's (batch-wide) plane.  geom: the host array densenet_plan_batch wrote (n_img * n_entries
 * entries, validated here); d_geom: its device copy (read by the kernel; entries that fall outside
 * the maps are skipped as empty).  conv5_desc: [n_maps] maps of one size, evenly spaced, as
 * densenet_conv_features writes them for the batch's planes.  Outputs and d_idx as the per-image
 * calls. */
int densenet_region_windows_batch(const void* d_conv5, const dn_plane_desc* conv5_desc,
                                  int32_t n_maps, dn_dtype conv5_dtype, const dn_scale_geom* geom,
                                  const dn_scale_geom* d_geom, int32_t n_img, int32_t n_entries,
                                  int32_t pad, int32_t pooled, const float* d_boxes,
                                  const int32_t* d_box_img, int32_t n, float target, int32_t S,
                                  float* d_out, int32_t* d_scale, int32_t* d_idx, void* stream);

/* Crop-before windows: the per-window baseline the paper measures the dense pyramid against
 * (Sec. 3.4: 2000 window proposals, each run through the network on its own) and the "crop before"
 * pipeline of Sec. 4.  Each box (x1, y1, x2, y2) of original-image pixel-edge coordinates (fp32) is
 * cut out of image d_box_img[i] (NULL => image 0) and warped to S x S by bilinear sampling with
 * half-pixel centres, the box stretched onto the grid with no context margin: output pixel (i, j)
 * samples sy = y1 + (i + 0.5)(y2 - y1)/S - 0.5, sx = x1 + (j + 0.5)(x2 - x1)/S - 0.5, each clamped
 * to the image ([0, H-1], [0, W-1]: a box reaching outside repeats the edge pixel), top-left neighbour
 * floor(s), the other one further (clamped); mean[c] (host, 3 floats) is then subtracted.  A box with a non-finite or non-positive side, or an
 * image index outside [0, n_img), gives an all-zero window.
 * d_images: uint8 [n_img][3][H][W].  d_out: [n][3][S][pitch] in `dtype` (n channel-major S x S planes
 * with rows `pitch` elements apart, packed back to back, ready for densenet_conv_features with plane
 * descriptors {S, S, i * 3 * S * pitch, pitch}), or NULL for a size query into *bytes_needed.
 * pitch: 0 => S, else >= S; columns S .. pitch-1 are written as 0.  S in 1 .. DN_MAX_WARP_SIDE.
 * With n == 0 nothing is launched.
 * Coordinates are fp64 with + - * / only, so the taps are reproducible bit for bit. */
#define DN_MAX_WARP_SIDE 1024
int densenet_warp_regions(const uint8_t* d_images, int32_t n_img, int32_t H, int32_t W,
                          const float* d_boxes, const int32_t* d_box_img, int32_t n, int32_t S,
                          int32_t pitch, const float* mean, dn_dtype dtype, void* d_out,
                          size_t out_bytes, size_t* bytes_needed, void* stream);

/* Single layers of the conv stack, for callers composing their own schedule.  All on channels-last
 * maps of n planes of equal size, packed back to back.
 * densenet_conv_layer: layer 1..5 with bias and ReLU.  Layer 1 reads channel-major planes
 * [n][3][H][W]; layers 2..5 read [n][H][W][C].  Output [n][Ho][Wo][M].
 * densenet_lrn_pool: LRN + 3x3/2 ceil max-pool (order per net->lrn_before_pool), [n][H][W][C] ->
 * [n][Hp][Wp][C].  densenet_maxpool: 3x3/2 ceil max-pool only. */
int densenet_conv_layer(int32_t layer, const void* d_in, int32_t n, int32_t H, int32_t W,
                        dn_dtype dtype, const void* d_packed, void* d_out, void* stream);
int densenet_lrn_pool(const void* d_in, int32_t n, int32_t H, int32_t W, int32_t C, dn_dtype dtype,
                      const dn_net_params* net, void* d_out, void* stream);
int densenet_maxpool(const void* d_in, int32_t n, int32_t H, int32_t W, int32_t C, dn_dtype dtype,
                     void* d_out, void* stream);

/* Output sizes of the conv stack for an H x W plane: conv1, pool1, conv2, pool2, conv3..5, pool5
 * (8 pairs written to hw[16]).  Returns DN_E_INVALID_ARG when the plane is too small for conv5. */
int densenet_layer_sizes(int32_t H, int32_t W, int32_t* hw);

/* Launch tracing.  While tracing is on, every kernel launch whose name matches `filter` (a
 * comma-separated list of names; NULL or "" = all) is bracketed by two hipEvents recorded on the
 * launch's own stream.  densenet_profile_stop() waits for the recorded events, writes per-name
 * totals (launches, summed elapsed ms) to out[max_entries] (*n_entries = number of names) and turns
 * tracing off.  Kernel names: build_planes, conv1..conv5, lrn_pool1, lrn_pool2, pool5, warp_regions,
 * region_windows, region_pool, pack_weights (a cross-image packed batch traces as build_planes,
 * region_windows, region_pool).  Events come from a pool owned by the library (no device memory). */
typedef struct {
  char name[32];
  int32_t launches;
  double total_ms;
} dn_profile_entry;
int densenet_profile_start(const char* filter);
int densenet_profile_stop(dn_profile_entry* out, int32_t max_entries, int32_t* n_entries);

/* Thread-local message describing the last error on this thread ("" if none). */
const char* densenet_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DENSENET_H */
