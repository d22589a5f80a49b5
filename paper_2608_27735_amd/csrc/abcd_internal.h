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

#define TRY_STATUS(call)            \
  do {                              \
    const int32_t st_ = (call);     \
    if (st_ != ABCD_OK) return st_; \
  } while (0)

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

// Tile rectangle of the screen box [u - rx, u + rx] x [v - ry, v + ry]:
// floor of the corner divided by the tile side, clamped to the grid; part of
// the fixed fp32 operation order (scaling by 1/16 is exact). Returns false if
// the rectangle is empty.
__device__ __forceinline__ bool tile_rect(float u, float v, float rx, float ry, int ntx, int nty,
                                          int& x0, int& y0, int& x1, int& y1) {
#pragma clang fp contract(off)
  float fx0 = floorf((u - rx) * 0.0625f);
  float fx1 = floorf((u + rx) * 0.0625f);
  float fy0 = floorf((v - ry) * 0.0625f);
  float fy1 = floorf((v + ry) * 0.0625f);
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

// A screen-space Gaussian as the blend kernels stage it in LDS: the conic is
// pre-scaled so that p2 = qa dx^2 + qb dx dy + qc dy^2 = power * log2(e), and
// alpha = min(alpha_max, o 2^p2) is one v_exp_f32 away.
constexpr float kLog2e = 1.4426950408889634f;

// conic_opacity holds (l11, l21, l22, o): the conic [[a, b], [b, c]] as its
// Cholesky factor L = [[l11, 0], [l21, l22]], and the opacity.
struct Splat {
  float u, v;          // mean
  float qa, qb, qc;    // s l11, s l21, s l22 with s^2 = log2(e) / 2
  float o;             // opacity
};

constexpr float kHalfLog2eSqrt = 0.84932180028801904f;  // sqrt(log2(e) / 2)

__device__ __forceinline__ Splat make_splat(float2 m, float4 co) {
  Splat s;
  s.u = m.x;
  s.v = m.y;
  s.qa = kHalfLog2eSqrt * co.x;
  s.qb = kHalfLog2eSqrt * co.y;
  s.qc = kHalfLog2eSqrt * co.z;
  s.o = co.w;
  return s;
}

// The conic (a, b, c) = L L^T of a factor (l11, l21, l22): for the tile test
// (splat_rows) and the chain rule to the mean.
__device__ __forceinline__ float3 conic_of(float4 co) {
  return make_float3(co.x * co.x, co.x * co.y, co.y * co.y + co.z * co.z);
}

// Alpha of a splat at pixel offset (dx, dy) = centre - mean. The forward and
// backward kernels both call this one function, so their skip and clamp
// decisions are bit-identical.
struct AlphaEval {
  float alpha;   // clamped alpha (valid when !skip)
  float raw;     // o * exp(power), before the clamp
  float e;       // exp(power)
  bool skip;     // power > 0 or alpha < alpha_min
  bool clamped;  // o * exp(power) > alpha_max
};

__device__ __forceinline__ AlphaEval eval_alpha(float dx, float dy, float qa, float qb, float qc,
                                                float o, float alpha_min, float alpha_max) {
  AlphaEval r;
  // -log2(e) q / 2 with q = d^T L L^T d: minus a sum of two squares
  const float e1 = qa * dx + qb * dy, e2 = qc * dy;
  const float p2 = -(e1 * e1 + e2 * e2);
  r.e = __builtin_amdgcn_exp2f(p2);
  r.raw = o * r.e;
  r.clamped = r.raw > alpha_max;
  r.alpha = fminf(r.raw, alpha_max);  // raw is finite: the clamp
  // alpha_min <= alpha_max (checked on the host), so the clamped alpha is
  // below alpha_min exactly when the raw value is
  r.skip = (p2 > 0.0f) || (r.raw < alpha_min);
  return r;
}

// Wave64 sum with DPP row operations; the total is returned to every lane.
__device__ __forceinline__ float wave_sum(float x) {
  const int xi0 = __float_as_int(x);
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, xi0, 0xB1, 0xF, 0xF, false));  // quad [1,0,3,2]
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));  // [2,3,0,1]
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));  // half mirror
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));  // mirror
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xA, 0xF, false));  // bcast15
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xC, 0xF, false));  // bcast31
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

__device__ __forceinline__ unsigned int wave_sum_u32(unsigned int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// ------------------------------------------------------ split workspace

// Long tiles are split for the backward: while a tile's walk crosses every
// ch-th position of its list (up to kMaxChunks - 1 boundaries), the forward stores each pixel's transmittance
// and colour there (and, for a tile that crossed one, at the end of its walk),
// and the backward processes each (tile, chunk) as a work item of its own.
// Slots are taken as the walks cross boundaries, so memory follows the walks,
// not the list lengths; a tile that finds no free slot is not split. Layout
// of the caller's workspace:
//   hdr[16]                  [0] checkpoint slots taken
//   slot_of[MAX][kMaxChunks] per tile: [0] end-of-walk slot, [b] boundary b
//   work[MAX]                per tile: the most entries the forward staged
//                            (kept by the tile test) within one chunk of its
//                            walk, the whole walk if it is not split; bit 31
//                            (kSplitTile) set when the tile has an end-of-walk
//                            slot (the schedule then needs no read of slot_of)
//   walk[MAX]                per tile: the largest per-pixel walk length
//   items[MAX + slots]       backward work items (tile, chunk), 8 bytes each
//   ckpt[slots][256]         (T, C_r, C_g, C_b) per pixel, 256-byte aligned
constexpr uint32_t kNoSlot = 0xFFFFFFFFu;
constexpr uint32_t kMaxChunks = 64;
constexpr uint32_t kSplitTile = 1u << 31;

struct SplitLayout {
  uint32_t* hdr;
  uint32_t* slot_of;
  uint32_t* work;
  uint32_t* walk;
  uint2* items;
  float4* ckpt;
  uint32_t nslots;
  int ch;  // list positions per chunk (the last chunk takes the rest); 0: no split
};

// Chunk j of a split tile holds list positions [j ch, (j + 1) ch) of its
// list; the last one (j = kMaxChunks - 1) runs to the end. The boundaries are
// fixed multiples of ch whatever the list length: a long list whose walks stop
// early (a dense front) still splits into chunks of ch.
__host__ __device__ inline uint32_t chunk_hi(uint32_t j, uint32_t ch) {
  return j + 1 < kMaxChunks ? (j + 1) * ch : 0xFFFFFFFFu;
}

inline size_t split_fixed_bytes(uint32_t nslots) {
  const size_t head = 64 + 4 * (size_t)ABCD_MAX_TILES * (kMaxChunks + 2) +
                      8 * ((size_t)ABCD_MAX_TILES + nslots);
  return (head + 255) & ~size_t(255);
}
inline size_t split_bytes(uint32_t nslots) {
  return split_fixed_bytes(nslots) + (size_t)nslots * 256 * sizeof(float4);
}
// Slots that fit `bytes` (0 if not even one does).
inline uint32_t split_slots(size_t bytes) {
  if (bytes < split_bytes(1)) return 0;
  uint64_t ns = (bytes - split_fixed_bytes(0)) / (256 * sizeof(float4) + 8);
  if (ns > 0x7FFF0000ull) ns = 0x7FFF0000ull;
  while (ns > 0 && split_bytes((uint32_t)ns) > bytes) --ns;
  return (uint32_t)ns;
}
inline SplitLayout split_layout(void* ws, size_t bytes, int ch) {
  SplitLayout s{};
  if (!ws || ch <= 0) return s;
  s.nslots = split_slots(bytes);
  if (s.nslots == 0) return s;
  char* b = reinterpret_cast<char*>(ws);
  s.hdr = reinterpret_cast<uint32_t*>(b);
  s.slot_of = reinterpret_cast<uint32_t*>(b + 64);
  s.work = reinterpret_cast<uint32_t*>(b + 64 + 4 * (size_t)ABCD_MAX_TILES * kMaxChunks);
  s.walk = reinterpret_cast<uint32_t*>(b + 64 + 4 * (size_t)ABCD_MAX_TILES * (kMaxChunks + 1));
  s.items = reinterpret_cast<uint2*>(b + 64 + 4 * (size_t)ABCD_MAX_TILES * (kMaxChunks + 2));
  s.ckpt = reinterpret_cast<float4*>(b + split_fixed_bytes(s.nslots));
  s.ch = ch;
  return s;
}

// ------------------------------------------------------ kernel launchers

// project.hip
int32_t launch_project(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                       const float* means, const float* log_scales, const float* quats,
                       const float* opacity_logits, const float* sh, float* means2d,
                       float* conic_opacity, float* depth, float* extent, uint32_t* tiles_touched,
                       float* rgb, hipStream_t stream);
int32_t launch_project_bwd(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                           const float* means, const float* log_scales, const float* quats,
                           const float* opacity_logits, const float* sh, const float* extent,
                           const float* g2d, float* d_means, float* d_log_scales, float* d_quats,
                           float* d_opacity_logits, float* d_sh, float* d_means2d,
                           int accumulate, hipStream_t stream);

// binning.hip
size_t bin_sort_workspace_bytes(int64_t n, int64_t capacity, int width, int height);
int32_t launch_bin_sort(int width, int height, int64_t n, const float* means2d, const float* extent,
                        const float* depth, const uint32_t* tiles_touched, int64_t capacity,
                        void* workspace, uint64_t* keys_sorted, uint32_t* values_sorted,
                        uint32_t* tile_ranges, uint32_t* tile_order, hipStream_t stream);

// render_fwd.hip, render_bwd.hip, loss.hip
// The backward's workspace: the screen-space gradients g2d, field-major
// (field q of Gaussian i at q * g2d_stride(n) + i, fp32), then per tile the
// work estimate, the order and the work items (when not split), then the
// queue counters. Field-major, the nine atomic adds of one Gaussian fall on
// nine cache lines instead of one or two (adds to one line are serialised in
// L2); the stride is a multiple of 1024 floats.
constexpr int64_t g2d_stride(int64_t n) { return (n + 1023) & ~int64_t(1023); }
constexpr size_t bwd_g2d_bytes(int64_t n) { return (size_t)9 * sizeof(float) * (size_t)g2d_stride(n); }
constexpr size_t bwd_workspace_bytes(int64_t n) {
  return bwd_g2d_bytes(n) + 2 * sizeof(uint32_t) * ABCD_MAX_TILES + 8 * (size_t)ABCD_MAX_TILES +
         sizeof(uint32_t) * 64 * 8;
}
size_t render_bwd_workspace_bytes(int64_t n);
int32_t launch_render_fwd(const abcd_camera& cam, const abcd_raster_params& prm,
                          const uint32_t* tile_ranges, const uint32_t* values_sorted,
                          const float* means2d, const float* conic_opacity, const float* rgb,
                          const float* F, const float* B, float* out_rgba, float* final_T,
                          uint32_t* last, unsigned long long* n_blends, const uint32_t* tile_order,
                          const SplitLayout& split, hipStream_t stream);
int32_t launch_render_cache(const abcd_camera& cam, const abcd_raster_params& prm,
                            const uint32_t* tile_ranges, const uint32_t* tile_order,
                            const uint32_t* values_sorted, const float* means2d,
                            const float* conic_opacity, const float* rgb, uint16_t* image_f16,
                            int32_t* rect, hipStream_t stream);
int32_t launch_render_bwd_pixels(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                                 const uint32_t* tile_ranges, const uint32_t* values_sorted,
                                 const float* means2d, const float* conic_opacity,
                                 const float* rgb, const float* F, const float* B,
                                 const float* final_T, const uint32_t* last,
                                 const float* dL_dout, float* g2d, const SplitLayout& split,
                                 hipStream_t stream);
// (launch_render_bwd_pixels clears g2d, 9 g2d_stride(n) floats, itself)
int32_t launch_zero(float* p, int64_t count, hipStream_t stream);
int32_t launch_loss_l1(int width, int height, const float* out_rgba, const float* target_rgb,
                       float bg0, float bg1, float bg2, float* dL_dout, float* loss,
                       hipStream_t stream);

// schedule.hip: the backward's schedule (work items heaviest first) and the
// per-tile maximum of the forward's walk lengths as a work estimate.
// The backward's work queue: queue[0] = number of items, then kQueues
// counters kQueueStride words apart (one cache line each): item i is served
// by queue i mod kQueues, whose counter is queue[kQueueStride q + 1].
constexpr int kQueues = 8;
constexpr int kQueueStride = 64;
// The same launch clears zero[0, zero_count) (16-byte aligned, a multiple of
// 4 floats) with workgroups of its own, beside the one that schedules.
int32_t launch_bwd_schedule(int ntiles, const uint32_t* key, const uint32_t* walk,
                            uint32_t* order, const SplitLayout& split, void* items, uint32_t cap,
                            uint32_t* queue, float* zero, int64_t zero_count,
                            hipStream_t stream);
int32_t launch_tile_walk(int width, int height, const uint32_t* last, uint32_t* work,
                         hipStream_t stream);

// adam.hip
int32_t launch_adam(const abcd_adam_group* groups, int ngroups, float beta1, float beta2, float eps,
                    int64_t t, hipStream_t stream);

// staging.hip
int32_t stage_cached(int width, int height, int k, const uint16_t* const* host_images,
                     const int32_t* rects, uint16_t* dst, hipStream_t stream);

// composite.hip
// beside: at most two workgroups per CU (room for other streams' work)
int32_t launch_composite(int width, int height, int k, const uint16_t* images,
                         const int32_t* order, int n_front, const int32_t* rects, float stop_t,
                         float* F, float* B, int accumulate, bool beside, hipStream_t stream);

}  // namespace abcd
