// abcd_internal.h -- internal declarations of the gfx950 library behind abcd.h.
//
// Kernels are written for CDNA4: 64-lane wavefronts, 16x16 pixel tiles mapped
// to 256-thread workgroups (4 waves), LDS staging, wave-level ballots and
// shuffles. Nothing here is a dense contraction, so no MFMA is used.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "abcd.h"

namespace abcd {

constexpr int kTile = ABCD_TILE;
constexpr int kBlock = 256;  // threads per workgroup = pixels per tile
constexpr int kWave = 64;

inline int tiles_x(int w) { return (w + kTile - 1) / kTile; }
inline int tiles_y(int h) { return (h + kTile - 1) / kTile; }

// ---------------------------------------------------------------- errors

void set_error(const char* fmt, ...);
int32_t hip_fail(hipError_t e, const char* what);

#define ABCD_HIP(call)                                   \
  do {                                                   \
    hipError_t e_ = (call);                              \
    if (e_ != hipSuccess) return abcd::hip_fail(e_, #call); \
  } while (0)

// ---------------------------------------------------------------- timing

// Records HIP events around a launch when timing is enabled on this thread.
struct TimedLaunch {
  TimedLaunch(const char* name, hipStream_t s);
  ~TimedLaunch();
  const char* name;
  hipStream_t stream;
  void* rec;
};

#define ABCD_LAUNCH(name, kernel, grid, block, lds, stream, ...)            \
  do {                                                                      \
    abcd::TimedLaunch tl_(name, stream);                                    \
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(block), lds, stream, __VA_ARGS__); \
  } while (0)

// ------------------------------------------------- shared device helpers

// Tile rectangle of the support square [u - r, u + r] x [v - r, v + r]:
// floor of the corner divided by the tile side, clamped to the grid; part of
// the fixed fp32 operation order (scaling by 1/16 is exact). Returns false if
// the rectangle is empty.
__device__ __forceinline__ bool tile_rect(float u, float v, float r, int ntx, int nty, int& x0,
                                          int& y0, int& x1, int& y1) {
#pragma clang fp contract(off)
  float fx0 = floorf((u - r) * 0.0625f);
  float fx1 = floorf((u + r) * 0.0625f);
  float fy0 = floorf((v - r) * 0.0625f);
  float fy1 = floorf((v + r) * 0.0625f);
  const float mx = (float)(ntx - 1), my = (float)(nty - 1);
  fx0 = fx0 < 0.0f ? 0.0f : fx0;
  fy0 = fy0 < 0.0f ? 0.0f : fy0;
  fx1 = fx1 > mx ? mx : fx1;
  fy1 = fy1 > my ? my : fy1;
  if (!(fx0 <= fx1) || !(fy0 <= fy1)) return false;
  x0 = (int)fx0;
  y0 = (int)fy0;
  x1 = (int)fx1;
  y1 = (int)fy1;
  return true;
}

// Alpha of a screen-space Gaussian at pixel offset (dx, dy) = centre - mean.
// The forward and backward kernels both call this, so their skip / clamp
// decisions are bit-identical.
struct AlphaEval {
  float alpha;   // clamped alpha (valid when !skip)
  float e;       // exp(power)
  bool skip;     // power > 0 or alpha < alpha_min
  bool clamped;  // o * exp(power) > alpha_max
};

__device__ __forceinline__ AlphaEval eval_alpha(float dx, float dy, float a, float b, float c,
                                                float o, float alpha_min, float alpha_max) {
  AlphaEval r;
  const float power = -0.5f * (a * dx * dx + c * dy * dy) - b * dx * dy;
  r.e = __expf(power);
  const float raw = o * r.e;
  r.clamped = raw > alpha_max;
  r.alpha = r.clamped ? alpha_max : raw;
  r.skip = (power > 0.0f) || (r.alpha < alpha_min);
  return r;
}

// Wave-wide helpers (wave64).
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ------------------------------------------------------ kernel launchers

// project.hip
int32_t launch_project(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                       const float* means, const float* log_scales, const float* quats,
                       const float* opacity_logits, const float* sh, float* means2d,
                       float* conic_opacity, float* depth, float* radius, uint32_t* tiles_touched,
                       float* rgb, hipStream_t stream);
int32_t launch_project_bwd(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                           const float* means, const float* log_scales, const float* quats,
                           const float* opacity_logits, const float* sh, const float* radius,
                           const float* g2d, float* d_means, float* d_log_scales, float* d_quats,
                           float* d_opacity_logits, float* d_sh, float* d_means2d,
                           int accumulate, hipStream_t stream);

// binning.hip
size_t bin_sort_workspace_bytes(int64_t n, int ntiles);
int32_t launch_bin_sort(int width, int height, int64_t n, const float* means2d, const float* radius,
                        const float* depth, const uint32_t* tiles_touched, int64_t capacity,
                        void* workspace, uint64_t* keys_sorted, uint32_t* values_sorted,
                        uint32_t* tile_ranges, hipStream_t stream);

// render.hip
size_t render_bwd_workspace_bytes(int64_t n);
int32_t launch_render_fwd(const abcd_camera& cam, const abcd_raster_params& prm,
                          const uint32_t* tile_ranges, const uint32_t* values_sorted,
                          const float* means2d, const float* conic_opacity, const float* rgb,
                          const float* F, const float* B, float* out_rgba, float* final_T,
                          uint32_t* last, unsigned long long* n_blends, hipStream_t stream);
int32_t launch_render_bwd_pixels(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                                 const uint32_t* tile_ranges, const uint32_t* values_sorted,
                                 const float* means2d, const float* conic_opacity,
                                 const float* rgb, const float* F, const float* B,
                                 const float* final_T, const uint32_t* last,
                                 const float* dL_dout, float* g2d, hipStream_t stream);
int32_t launch_zero(float* p, int64_t count, hipStream_t stream);
int32_t launch_loss_l1(int width, int height, const float* out_rgba, const float* target_rgb,
                       float bg0, float bg1, float bg2, float* dL_dout, float* loss,
                       hipStream_t stream);

// composite.hip
int32_t launch_composite(int width, int height, int k, const uint16_t* images,
                         const int32_t* order, int n_front, float* F, float* B, int accumulate,
                         hipStream_t stream);

}  // namespace abcd
