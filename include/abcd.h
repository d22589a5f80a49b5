/*
 * abcd.h -- C ABI of the ABCD active-block step on MI355X (gfx950).
 *
 * ABCD (Alpha-Composited Block Coordinate Descent) trains a radiance field one
 * spatial partition at a time: a step draws the active partition alone; its
 * image is composited between a foreground F and a background B that hold the
 * pre-accumulated renders of the frozen partitions in front of and behind it,
 * and gradients flow into the active parameters only (paper, Method section).
 * Because "over" is associative, the cached per-partition renders collapse
 * into F and B (Abstract; Method section). The renderer is 3D Gaussian
 * Splatting (Introduction), whose constants the paper does not state; they
 * are runtime parameters here (abcd_raster_params).
 *
 * One step on one camera is
 *   abcd_stage_cached     pinned host cache -> device chunk (per camera, in chunks)
 *   abcd_composite_cache  cached partition renders -> F, B (once per camera)
 *   abcd_project          parameters -> screen-space Gaussians
 *   abcd_bin_sort         -> per 16x16 tile, Gaussians sorted by (depth, index)
 *   abcd_render_fwd       -> out = F over A over B
 *   (loss gradient, e.g. abcd_loss_l1_grad)
 *   abcd_render_bwd       -> gradients of the active parameters only
 *
 * Conventions for every entry point:
 *  - Returns an abcd_status (int32). Arguments are validated on the host before
 *    any HIP call; an invalid call returns ABCD_E_INVALID and touches nothing.
 *  - Array arguments are DEVICE pointers owned by the caller unless marked
 *    "host". The library never allocates device memory: scratch space is a
 *    caller-provided workspace whose size the *_workspace_size helpers give.
 *  - All work is enqueued on `stream` and is asynchronous, except where a call
 *    is documented to synchronise.
 *  - Floating-point data is fp32 unless stated; fp16 is IEEE binary16 passed as
 *    uint16_t. Images are row-major [height][width][4] premultiplied RGBA.
 *  - Parameter arrays are contiguous structure-of-arrays:
 *      means [n][3], log_scales [n][3], quats [n][4] (w, x, y, z; any norm),
 *      opacity_logits [n], sh [n][(sh_degree+1)^2][3].
 *  - Alignment: quats, d_quats, conic_opacity and RGBA images 16 bytes,
 *    means2d 8 bytes, workspaces 256 bytes (an unaligned call is rejected).
 *  - Functions are stateless and reentrant; concurrent calls on one stream
 *    must not share a workspace.
 *  - Device arrays must be ordinary (coarse-grained) device memory, as
 *    hipMalloc and PyTorch's CUDA allocator return it. The library is built
 *    with hardware fp32 atomic adds (-munsafe-fp-atomics) for gradients,
 *    screen-space gradient sums and counters; on fine-grained, host-mapped or
 *    managed memory those atomics are not guaranteed to take effect, so the
 *    workspaces and every gradient output must not live there.
 */
#ifndef ABCD_H
#define ABCD_H

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ABCD_API __attribute__((visibility("default")))

#define ABCD_TILE 16           /* tile side in pixels */
#define ABCD_MAX_TILES 32768   /* ceil(W/16) * ceil(H/16) limit */
#define ABCD_MAX_GAUSSIANS (1LL << 30)

typedef enum {
  ABCD_OK = 0,
  ABCD_E_INVALID = 1,   /* bad argument; nothing was enqueued */
  ABCD_E_CAPACITY = 2,  /* intersection count exceeds the capacity given */
  ABCD_E_OVERFLOW = 3,  /* intersection count does not fit 32 bits */
  ABCD_E_HIP = 4        /* a HIP call failed; see abcd_last_error() */
} abcd_status;

/* Pinhole camera. x_cam = R x_world + t with OpenCV axes (x right, y down,
 * z forward); pixel (i, j) covers [i, i+1) x [j, j+1) and is sampled at its
 * centre (i + 0.5, j + 0.5). campos is the camera centre in world space (for
 * the view direction of the SH colour). Gaussians with view depth <= near_plane
 * are culled. near_plane must be positive (depth keys are the fp32 bit
 * patterns of positive depths, which sort as unsigned integers); a call with
 * near_plane <= 0 returns ABCD_E_INVALID. */
typedef struct {
  int32_t width, height;
  float fx, fy, cx, cy;
  float R[9]; /* row major */
  float t[3];
  float campos[3];
  float near_plane;
} abcd_camera;

/* Rasteriser constants of the 3D Gaussian Splatting renderer. */
typedef struct {
  float alpha_min;     /* blends with alpha below this are skipped (1/255) */
  float alpha_max;     /* alpha is clamped to this (0.99) */
  float t_min;         /* a blend that would take transmittance below this ends the pixel (1e-4) */
  float eps2d;         /* dilation added to every 2D covariance, px^2 (0.3) */
  float radius_sigmas; /* support radius in sigmas of the major axis (3) */
  float guard;         /* guard-band factor on the field of view inside the Jacobian (1.3) */
  int32_t sh_degree;   /* 0..3 */
  uint32_t flags;      /* ABCD_FLAG_* bits; others must be 0 */
} abcd_raster_params;

/* Compositing-aware stop (Limitations section: what a near-opaque foreground
 * hides need not be rendered). In abcd_render_fwd a pixel stops when the
 * weight the next blend would leave for later ones in the composited image,
 * (1 - F_alpha) T (1 - alpha), is below t_min, instead of T (1 - alpha); a
 * pixel whose F leaves it less than t_min blends nothing, and a tile whose
 * pixels all do so is skipped. Without F the rule is the plain one. The image
 * then differs from the plain rule's by at most t_min / (1 - alpha_max) per
 * channel times the largest colour plus one. abcd_render_bwd follows the
 * forward's final_T and last, so it needs no flag. */
#define ABCD_FLAG_FB_STOP 1u

/* ------------------------------------------------------------------------ */
/* Projection (3DGS EWA splatting: Introduction; Method section -- "only the
 * active partition is rendered").
 *
 * Per Gaussian i writes
 *   means2d[i][2]        pixel-space mean (u, v)
 *   conic_opacity[i][4]  (l11, l21, l22, o): the inverse 2D covariance (the
 *                        conic) [[a, b], [b, c]] as its Cholesky factor,
 *                        a = l11^2, b = l11 l21, c = l21^2 + l22^2 (computed
 *                        in fp64; the blend kernels evaluate the quadratic
 *                        form as a sum of two squares, which a badly
 *                        conditioned conic does not amplify), and opacity
 *                        o = sigmoid(logit)
 *   depth[i]             view-space z
 *   extent[i][2]         (ex, ey): half extents in pixels of the box that bins
 *                        the Gaussian: the support square (radius_sigmas times
 *                        the square root of the largest eigenvalue of the 2D
 *                        covariance) cut per axis to the extent of the ellipse
 *                        where alpha can reach alpha_min (|dx| <= sqrt(L A),
 *                        |dy| <= sqrt(L C), A and C the covariance's diagonal,
 *                        L = 1.001 tau + 0.001 and tau = 2 ((1 - e) ln 2 +
 *                        min(logit, 0)) >= 2 ln(o / alpha_min) for alpha_min =
 *                        m 2^e, m in [0.5, 1)); no pixel of a cut-off tile
 *                        could blend the Gaussian, so images are unchanged
 *   tiles_touched[i]     number of 16x16 tiles of that box
 *   rgb[i][3]            colour max(0, SH(view direction) + 0.5)
 * A culled Gaussian (behind near_plane, degenerate, non-finite, with no tile
 * on screen, or with alpha_min out of reach) gets zeros in every output. The
 * values deciding culling, the tile box and the depth key follow one fixed
 * fp32 operation order (the numerical contract of this library); extent must
 * be 8-byte aligned. n may be 0. */
ABCD_API int32_t abcd_project(const abcd_camera* cam /* host */, const abcd_raster_params* prm /* host */,
                     int64_t n, const float* means, const float* log_scales, const float* quats,
                     const float* opacity_logits, const float* sh, float* means2d,
                     float* conic_opacity, float* depth, float* extent, uint32_t* tiles_touched,
                     float* rgb, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Binning: every (tile, Gaussian) pair of the support rectangles, sorted by
 * key = tile << 32 | fp32 bits of depth, ties by Gaussian index (the unique
 * front-to-back order of each tile's list).
 *
 * Outputs: values_sorted[M] Gaussian indices; keys_sorted[M] the keys (may be
 * NULL, then not written); tile_ranges[tiles][2] = [start, end) per tile
 * (start = number of pairs of lower tiles); tile_order[tiles] (may be NULL,
 * then not written): a schedule for abcd_render_fwd, the tile indices
 * ordered by decreasing list length kept to its leading three bits (the
 * octave and its quarter), ties in tile order.
 *
 * capacity: number of elements values_sorted (and keys_sorted) can hold. If
 * the intersection count M exceeds it (or does not fit 32 bits), nothing is
 * written to values_sorted or keys_sorted, every tile range is written empty
 * (so the blend calls that follow render nothing of the active block and read
 * no list entry) and tile_order is the identity.
 * n_isect (host, may be NULL): if given, the call synchronises `stream` once,
 * stores M there and returns ABCD_E_CAPACITY when M > capacity. If NULL, the
 * call does not synchronise; M (uint64) is left at the start of the workspace,
 * where the caller can read it later (M > capacity: that call overflowed).
 * capacity must be below 2^32.
 * workspace: at least abcd_bin_sort_workspace_size(n, capacity, width, height)
 * bytes, 256-byte aligned; it grows with the capacity (8 bytes per element for
 * an intermediate list of (Gaussian, 8x8-tile block) pairs, which never holds
 * more than M elements). */
ABCD_API int32_t abcd_bin_sort_workspace_size(int64_t n, int64_t capacity, int32_t width,
                                              int32_t height, size_t* bytes);
ABCD_API int32_t abcd_bin_sort(int32_t width, int32_t height, int64_t n, const float* means2d,
                      const float* extent, const float* depth, const uint32_t* tiles_touched,
                      int64_t capacity, void* workspace, size_t ws_bytes, uint64_t* keys_sorted,
                      uint32_t* values_sorted, uint32_t* tile_ranges, uint32_t* tile_order,
                      int64_t* n_isect /* host */, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Split of long tiles between the forward and the backward (a scheduling
 * choice of this library; the paper's renderer is unchanged). The backward of
 * a tile walks its list back to front; a tile with a list of many thousand
 * entries would keep one workgroup busy after the rest of the GPU is idle.
 * With a split, whenever a tile's walk in the forward crosses a chunk
 * boundary (every `chunk` list positions, up to 63 boundaries: the 64th
 * chunk runs to the end of the list) it takes a 4 KB slot and stores each
 * pixel's transmittance and colour there, plus one slot for the end of the
 * walk; the backward then processes each (tile, chunk) as its own work item,
 * starting from those states, heaviest items first by the number of entries
 * the forward staged per chunk. Slots are taken in the forward's tile order
 * (heaviest first); a tile that finds none left is not split. The same
 * split must be given to a forward and its backward; results agree with the
 * unsplit backward up to rounding.
 * workspace: device memory of abcd_split_workspace_size(n_slots) bytes (or
 * more: the slots that fit are used), 256-byte aligned; chunk: a positive
 * multiple of 256, at most 2^24. Slots a frame needs: about (sum over tiles
 * of the longest walk in the tile) / chunk + (number of tiles split). */
typedef struct {
  void* workspace;
  size_t bytes;
  int32_t chunk;
  int32_t reserved;
} abcd_split;
ABCD_API int32_t abcd_split_workspace_size(int64_t n_slots, size_t* bytes);

/* ------------------------------------------------------------------------ */
/* Forward render and composite (Method section: F over active over B).
 *
 * Per pixel, front to back over its tile's list, starting from T = 1, C = 0:
 *   power = -(a dx^2 + c dy^2)/2 - b dx dy, (dx, dy) = pixel centre - mean;
 *   skip if power > 0; alpha = min(alpha_max, o exp(power)); skip if
 *   alpha < alpha_min; stop (without blending) if T (1 - alpha) < t_min;
 *   else C += rgb alpha T, T *= 1 - alpha.
 * The active render A = (C, 1 - T) is composited as out = F over A over B:
 *   out_rgb = F_rgb + (1 - F_a)(C + T B_rgb),
 *   out_a   = F_a + (1 - F_a)(1 - T (1 - B_a)).
 * F or B may be NULL (transparent); tile_ranges, values_sorted, means2d,
 * conic_opacity, rgb and the three outputs may not (ABCD_E_INVALID; a
 * placeholder buffer serves when the lists are empty). Also writes final_T[H][W] and last[H][W]
 * (entries of the tile's list walked up to and including the last blended
 * one), both needed by abcd_render_bwd. n_blends (may be NULL): the number of
 * blended (pixel, Gaussian) pairs of this call is ADDED to *n_blends.
 * tile_order (may be NULL): the order in which workgroups take tiles, a
 * permutation of the tiles such as abcd_bin_sort's tile_order (heaviest
 * first balances the GPU); it changes no output. NULL takes tiles in raster
 * order. split (host, may be NULL): see abcd_split. */
ABCD_API int32_t abcd_render_fwd(const abcd_camera* cam /* host */, const abcd_raster_params* prm /* host */,
                        const uint32_t* tile_ranges, const uint32_t* tile_order,
                        const uint32_t* values_sorted,
                        const float* means2d, const float* conic_opacity, const float* rgb,
                        const float* F, const float* B, float* out_rgba, float* final_T,
                        uint32_t* last, unsigned long long* n_blends, const abcd_split* split,
                        hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Cached render of a partition (Method section: the frozen partitions' renders
 * are cached per camera and refreshed after the block they belong to has been
 * trained): the forward above with F = B = transparent, written as
 * premultiplied fp16 RGBA, image_f16[H][W][4] = binary16 (round to nearest
 * even) of (C, 1 - T). Its input is that partition's projection and binning on
 * the camera; its output feeds abcd_composite_cache. tile_order as in
 * abcd_render_fwd (may be NULL). image_f16 8-byte aligned.
 * rect (device, may be NULL): int32[4] = (x0, y0, x1, y1), the bounding box
 * of the 16x16 tiles holding a pixel that blended anything, clipped to the
 * image; the image is zero outside it (x1 <= x0 when nothing blended). It is
 * the coverage box abcd_composite_cache takes. tile_ranges, values_sorted,
 * means2d, conic_opacity, rgb and image_f16 may not be NULL. */
ABCD_API int32_t abcd_render_cache(const abcd_camera* cam /* host */,
                          const abcd_raster_params* prm /* host */, const uint32_t* tile_ranges,
                          const uint32_t* tile_order, const uint32_t* values_sorted,
                          const float* means2d, const float* conic_opacity, const float* rgb,
                          uint16_t* image_f16, int32_t* rect, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Backward (Method section: gradients are back-propagated only through the
 * active parameters; F and B are constants).
 *
 * Given dL_dout[H][W][4], writes the gradient of L with respect to every
 * active parameter: d_means [n][3], d_log_scales [n][3], d_quats [n][4],
 * d_opacity_logits [n], d_sh [n][(sh_degree+1)^2][3]; d_means2d [n][2] (may be
 * NULL) receives dL/d(u, v). With accumulate != 0 the gradients are added to
 * the arrays, otherwise they overwrite them. The derivative is exact for the
 * forward above, including zero derivative of a clamped alpha and of a
 * clamped colour. Inputs are those of the forward call on the same camera.
 * workspace: at least abcd_render_bwd_workspace_size(n) bytes, 256-byte
 * aligned (screen-space gradients, 36 bytes per Gaussian with n rounded up
 * to a multiple of 1024, and the work
 * schedule of the backward, heaviest walk first, 16 bytes per tile at the
 * maximum tile count). split (host, may be NULL): the one the forward used. */
ABCD_API int32_t abcd_render_bwd_workspace_size(int64_t n, size_t* bytes);
ABCD_API int32_t abcd_render_bwd(const abcd_camera* cam /* host */, const abcd_raster_params* prm /* host */,
                        int64_t n, const float* means, const float* log_scales, const float* quats,
                        const float* opacity_logits, const float* sh, const float* means2d,
                        const float* conic_opacity, const float* rgb, const float* extent,
                        const uint32_t* tile_ranges, const uint32_t* values_sorted,
                        const float* F, const float* B, const float* final_T, const uint32_t* last,
                        const float* dL_dout, void* workspace, size_t ws_bytes, float* d_means,
                        float* d_log_scales, float* d_quats, float* d_opacity_logits, float* d_sh,
                        float* d_means2d, int32_t accumulate, const abcd_split* split,
                        hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Allocation-free backward, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): abcd_render_bwd without the workspace arguments, same outputs.
 * Its scratch (screen-space gradients and the backward's work schedule) is a
 * static device array of ABCD_NOALLOC_SCRATCH_BYTES inside the library; each
 * GPU the library runs on holds its own copy until the process ends. n may be
 * at most ABCD_NOALLOC_MAX_GAUSSIANS; a larger n returns ABCD_E_INVALID with
 * nothing enqueued. The call allocates nothing: no hipMalloc, no hipFree, no
 * allocating library routine (its first call on a device looks up that
 * device's copy of the array, with hipGetSymbolAddress, and keeps the
 * address). The calling thread's current device must be the one of `stream`.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents; each call clears what must start at zero itself (with a fill
 * kernel, no memset node). Calls that overlap on one GPU (on other streams or
 * threads) race on the array and give wrong gradients: serialise them. */
#define ABCD_NOALLOC_MAX_GAUSSIANS (1LL << 20)
#define ABCD_NOALLOC_SCRATCH_BYTES 38275072ULL /* workspace of 2^20 Gaussians */
ABCD_API int32_t abcd_render_bwd_noalloc(const abcd_camera* cam /* host */,
                                         const abcd_raster_params* prm /* host */, int64_t n,
                                         const float* means, const float* log_scales,
                                         const float* quats, const float* opacity_logits,
                                         const float* sh, const float* means2d,
                                         const float* conic_opacity, const float* rgb,
                                         const float* extent, const uint32_t* tile_ranges,
                                         const uint32_t* values_sorted, const float* F,
                                         const float* B, const float* final_T,
                                         const uint32_t* last, const float* dL_dout,
                                         float* d_means, float* d_log_scales, float* d_quats,
                                         float* d_opacity_logits, float* d_sh, float* d_means2d,
                                         int32_t accumulate, const abcd_split* split,
                                         hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Collapse of cached partition renders into F and B (Abstract; Method section:
 * the stored renders of the frozen partitions are merged, front to back in
 * their depth order, into the two layers).
 *
 * images: k premultiplied RGBA fp16 renders [k][H][W][4]. order (host): a
 * permutation of 0..k-1, front to back. F = images[order[0]] over ... over
 * images[order[n_front-1]], B = images[order[n_front]] over ... over
 * images[order[k-1]], both fp32 [H][W][4]. flags: ABCD_COMPOSITE_ACCUMULATE
 * (1) continues the fold behind the incoming F and B (F <- F over fold, B <- B
 * over fold), so chunks of cached images can stream in front to back;
 * without it they are overwritten. k = 0 writes transparent F and B (or
 * leaves them unchanged when accumulating). ABCD_COMPOSITE_BESIDE (2) runs the
 * collapse on at most two workgroups per CU, each taking many pixels, so that
 * work enqueued on other streams meanwhile (the binning of the same step)
 * finds room on the CUs; alone on the GPU it is slower. Other bits:
 * ABCD_E_INVALID.
 * rects (device, may be NULL, 16-byte aligned): int32 [k][4] = (x0, y0, x1,
 * y1) per image, the pixel box [x0, x1) x [y0, y1) outside which that image
 * is fully transparent (all four channels zero), as abcd_render_cache
 * reports it; the image is not read outside its box. A box that cuts off
 * non-zero pixels gives wrong results. NULL: every image covers the frame.
 * stop_t (0 <= stop_t < 1; Limitations section: occluded renders can be
 * ignored): 0 folds every layer; above 0 a front layer is skipped once
 * 1 - F_alpha < stop_t and a back layer once (1 - F_alpha)(1 - B_alpha) <
 * stop_t (alphas accumulated so far), which changes F over B by at most
 * 2 stop_t per channel. */
ABCD_API int32_t abcd_composite_cache(int32_t width, int32_t height, int32_t k, const uint16_t* images,
                             const int32_t* order /* host */, int32_t n_front,
                             const int32_t* rects, float stop_t, float* F, float* B,
                             int32_t flags, hipStream_t stream);
#define ABCD_COMPOSITE_ACCUMULATE 1
#define ABCD_COMPOSITE_BESIDE 2

/* ------------------------------------------------------------------------ */
/* Upload of cached renders from pinned host memory (Method section: the cache
 * of camera-partition renders is kept in system memory or on disk, and the
 * renders a camera needs go to the GPU when a block becomes active). For each
 * j < k, copies the coverage box rects[j] (as in abcd_composite_cache; NULL:
 * the whole image) of host_images[j] (fp16 RGBA [H][W][4] in pinned host
 * memory) to the same pixels of dst[j] (device, [k][H][W][4]), as one 2D
 * copy per image, asynchronously on `stream`. Pixels of dst outside the box
 * keep their old contents, which abcd_composite_cache with the same rects
 * never reads; an empty box copies nothing. host_images (k pointers) and rects
 * ([k][4] int32) are host arrays; the host images must stay unchanged until
 * the copies complete. A box outside the image is an error. */
ABCD_API int32_t abcd_stage_cached(int32_t width, int32_t height, int32_t k,
                          const uint16_t* const* host_images /* host */,
                          const int32_t* rects /* host */, uint16_t* dst, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* L1 reconstruction loss gradient (the paper evaluates a reconstruction loss
 * without naming it, Method section). img = out_rgb + (1 - out_a) bg;
 * dL/dimg = sign(img - target) / (3 H W) (sign(0) = 0); writes dL_dout[H][W][4]
 * (alpha channel -sum_c bg_c dL/dimg_c). bg (host) may be NULL (black). loss
 * (may be NULL): sum |img - target| / (3 H W) is ADDED to *loss. */
ABCD_API int32_t abcd_loss_l1_grad(int32_t width, int32_t height, const float* out_rgba,
                          const float* target_rgb, const float* bg /* host, 3 floats */,
                          float* dL_dout, float* loss, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Adam update of the active parameters after the backward (the step on the
 * optimizer side; the paper trains with gradient steps but does not name the
 * optimizer, the 3DGS line it builds on uses Adam with one learning rate per
 * parameter group). For every element of every group, in place, fp32:
 *   m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2;
 *   param -= lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * (Kingma and Ba 2015, Algorithm 1). groups (host array of n_groups <=
 * ABCD_ADAM_MAX_GROUPS): device arrays of `count` floats each; param,
 * exp_avg (m) and exp_avg_sq (v) are read and written, grad is read; a group
 * with count 0 is skipped. step >= 1 counts the updates made so far, this one
 * included; 0 <= beta1, beta2 < 1; eps >= 0. One launch. */
#define ABCD_ADAM_MAX_GROUPS 8
typedef struct abcd_adam_group {
  float* param;
  const float* grad;
  float* exp_avg;
  float* exp_avg_sq;
  int64_t count;
  float lr;
} abcd_adam_group;
ABCD_API int32_t abcd_adam_step(const abcd_adam_group* groups /* host */, int32_t n_groups,
                                float beta1, float beta2, float eps, int64_t step,
                                hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Helpers. abcd_last_error: message of the last failure on this thread.
 * abcd_timing_*: optional per-kernel HIP-event timing of every launch made by
 * this thread (off by default; enabling it adds two event records per launch
 * on the caller's stream). abcd_timing_read synchronises, and returns the
 * accumulated milliseconds and launch count of the kernel named `kernel`
 * (names: composite, project, bin_zero, depth_keys, radix_pass, l1_place,
 * l2_count, l2_scatter, bin_small_sort, bin_small_collect, bin_empty,
 * render_fwd, loss_l1, zero_fill, bwd_order, render_bwd, project_bwd, adam,
 * render_cache, cache_rect_init). */
ABCD_API const char* abcd_last_error(void);
ABCD_API const char* abcd_version(void);
ABCD_API const char* abcd_status_string(int32_t status);
ABCD_API int32_t abcd_timing_enable(int32_t enable);
ABCD_API int32_t abcd_timing_reset(void);
ABCD_API int32_t abcd_timing_read(const char* kernel, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* ABCD_H */
