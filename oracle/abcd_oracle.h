/*
 * abcd_oracle.h -- CPU oracle for the ABCD active-block step.
 *
 * TEST INFRASTRUCTURE ONLY. This library is a plain, slow, deliberately
 * unoptimised restatement of what one step of Alpha-Composited Block
 * Coordinate Descent computes (paper: Method section -- render only the active
 * partition, composite it between the pre-accumulated foreground F and
 * background B, back-propagate into the active parameters only; Abstract --
 * associativity of alpha blending lets frozen partitions be collapsed into F
 * and B). It is used by the tests, by the smoke check and by the CPU-baseline
 * leg of the benchmark. The product path never links or calls it, and it shares
 * no code, header, table or constant with the GPU library.
 *
 * The paper inherits its renderer from 3D Gaussian Splatting and states none of
 * its constants; every constant below is a runtime parameter (see the
 * numerical contract in the design notes of this repository).
 *
 * Precision: the values that decide integers (tile rectangles, sort keys, the
 * intersection count) are computed in fp32 with one fixed operation order, the
 * precision of the GPU kernels. Everything else (2D conics, opacities, colours,
 * the blend, all gradients, the "over" fold) is computed in fp64.
 */
#ifndef ABCD_ORACLE_H
#define ABCD_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_TILE 16

typedef struct {
  int32_t width, height;   /* image size in pixels */
  float fx, fy, cx, cy;    /* pinhole intrinsics; pixel (i,j) is sampled at (i+0.5, j+0.5) */
  float R[9];              /* world->camera rotation, row major (x right, y down, z forward) */
  float t[3];              /* world->camera translation: x_cam = R x_world + t */
  float campos[3];         /* camera centre in world coordinates (view direction for SH) */
  float near_plane;        /* Gaussians with view depth <= near_plane are culled */
} orc_camera;

typedef struct {
  float alpha_min;      /* blends with alpha below this are skipped */
  float alpha_max;      /* alpha is clamped to this */
  float t_min;          /* a blend that would take transmittance below this ends the pixel */
  float eps2d;          /* isotropic dilation added to every 2D covariance (px^2) */
  float radius_sigmas;  /* support radius in standard deviations of the major axis */
  float guard;          /* guard-band factor on the field of view, used inside the Jacobian only */
  int32_t sh_degree;    /* 0..3 */
  int32_t fb_stop;      /* compositing-aware stop: a blend ends the pixel when the weight
                           (1 - F_alpha) T (1 - alpha) that later blends would get in the
                           composited image falls below t_min (0: plain t_min rule) */
} orc_params;

/* ---- projection -------------------------------------------------------- */

/* fp32 chain that decides visibility, the tile rectangle and the sort key.
 * radius[i] = support radius (radius_sigmas sqrt(lambda_max)); extent[2*i..]
 * = half extents of the binning box (the support square cut per axis to the
 * ellipse where alpha can reach alpha_min); rect[4*i..] = (tx0, ty0, tx1,
 * ty1) inclusive; all outputs are zero for a culled Gaussian. */
void orc_project_bin_f32(const orc_camera* cam, const orc_params* prm, int64_t n,
                         const float* means, const float* log_scales, const float* quats,
                         const float* opacity_logits, float* means2d, float* depth,
                         float* radius, float* extent, int32_t* rect, uint32_t* tiles_touched);

/* fp64 values of the same projection (means2d, conic (a,b,c), opacity, rgb);
 * Gaussians with tiles_touched == 0 get zeros. */
void orc_project_values_f64(const orc_camera* cam, const orc_params* prm, int64_t n,
                            const float* means, const float* log_scales, const float* quats,
                            const float* opacity_logits, const float* sh,
                            const uint32_t* tiles_touched,
                            double* means2d, double* conic, double* opacity, double* rgb);

/* ---- binning ------------------------------------------------------------ */

/* total number of (Gaussian, tile) intersections */
int64_t orc_count_isect(int64_t n, const uint32_t* tiles_touched);

/* Lists every (tile, Gaussian) pair, key = tile << 32 | fp32 bits of depth,
 * sorted by (key, Gaussian index); tile_ranges[2*t..] = [start, end). The
 * pairs are grouped by tile and each tile's group sorted by (depth bits,
 * index), the same sequence as one sort of all pairs by (key, index). */
void orc_bin(int32_t width, int32_t height, int64_t n, const float* depth, const int32_t* rect,
             const uint32_t* tiles_touched, uint64_t* keys, uint32_t* values,
             uint32_t* tile_ranges);

/* ---- rasterisation ------------------------------------------------------ */

/* Front-to-back blend of the sorted tile lists, then out = F over A over B
 * (premultiplied RGBA). F, B may be NULL (transparent). knife/t_stop may be
 * NULL; knife[p] != 0 marks a pixel one of whose threshold decisions lies
 * within its margin of its threshold: rel_margin (relative) for every
 * decision when f32_kappa = 0; with f32_kappa > 0 the alpha decisions
 * (alpha_min, alpha_max) take rel_margin plus f32_kappa 2^-24 times the
 * magnitude of the terms of the quadratic form in its Cholesky form (a bound
 * on the relative error of alpha evaluated in fp32), and the stop decision
 * rel_margin plus the accumulated bound of the transmittance. The power > 0
 * test always takes rel_margin times the magnitude of its terms. With
 * prm->fb_stop the stop test is (1 - F_alpha) T_next < t_min instead of
 * T_next < t_min. */
void orc_render_fwd(const orc_camera* cam, const orc_params* prm, const uint32_t* tile_ranges,
                    const uint32_t* values, const double* means2d, const double* conic,
                    const double* opacity, const double* rgb, const double* F, const double* B,
                    double* out, double* final_T, uint32_t* last, uint64_t* n_blends,
                    double rel_margin, double f32_kappa, uint8_t* knife, double* t_stop);

/* Per-pixel backward: accumulates, per Gaussian, the 9 screen-space gradients
 * g2d[9*i..] = dL/d(u, v, a, b, c, opacity, r, g, b). g2d is overwritten. */
void orc_render_bwd_2d(const orc_camera* cam, const orc_params* prm, int64_t n,
                       const uint32_t* tile_ranges, const uint32_t* values,
                       const double* means2d, const double* conic, const double* opacity,
                       const double* rgb, const double* F, const double* B,
                       const double* dL_dout, double* g2d);

/* Per-Gaussian chain rule from screen-space gradients to the parameters. */
void orc_project_bwd(const orc_camera* cam, const orc_params* prm, int64_t n,
                     const float* means, const float* log_scales, const float* quats,
                     const float* opacity_logits, const float* sh,
                     const uint32_t* tiles_touched, const double* g2d,
                     double* d_means, double* d_log_scales, double* d_quats,
                     double* d_opacity_logits, double* d_sh);

/* ---- "over" collapse of cached renders ---------------------------------- */

/* F = fold_over(images[order[0..n_front)]), B = fold_over(images[order[n_front..k)]),
 * images are premultiplied RGBA IEEE binary16, [pool][h][w][4], every order[j]
 * indexes that pool and k is the number of layers folded. With accumulate,
 * the fold continues behind the incoming F and B. stop_t > 0 drops the layers
 * that can no longer be seen (Limitations section: occluded renders can be
 * ignored): a front layer is skipped once 1 - F_alpha < stop_t, a back layer
 * once (1 - F_alpha)(1 - B_alpha) < stop_t, with the alphas accumulated so
 * far. knife (may be NULL) marks pixels with such a decision within
 * rel_margin of stop_t. */
void orc_composite(int32_t width, int32_t height, int32_t k, const uint16_t* images,
                   const int32_t* order, int32_t n_front, double* F, double* B,
                   int32_t accumulate, double stop_t, double rel_margin, uint8_t* knife);

/* ---- helpers exposed for the pin tests --------------------------------- */

/* Adam (Kingma and Ba, "Adam: A Method for Stochastic Optimization", 2015,
 * Algorithm 1), one step t >= 1 on n elements, in place, fp64:
 *   m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2;
 *   theta = theta - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
 * The paper does not name its optimizer; the 3DGS line it builds on uses Adam
 * with a learning rate per parameter group, so the step takes one lr. */
void orc_adam(int64_t n, double* theta, const double* g, double* m, double* v, double lr,
              double b1, double b2, double eps, int64_t t);

double orc_half_to_double(uint16_t h);
/* real orthonormal SH basis Y_i(d), i = l^2 + l + m, 16 values; grad[3*i..] = dY_i/dd */
void orc_sh_basis(const double* dir, double* y, double* grad);
/* rotation matrix (row major) of the normalised quaternion (w, x, y, z) */
void orc_quat_to_rot(const double* q, double* Rm);

#ifdef __cplusplus
}
#endif
#endif
