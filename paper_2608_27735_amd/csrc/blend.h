// blend.h -- pieces shared by the forward and backward tile blend kernels:
// the launch constants, the tile schedule lookup, list-entry loads, the
// tile's pixel-centre box and the block-wide compaction of staged entries.
//
// One 256-thread workgroup (4 wave64) per 16x16 tile, one thread per pixel.
// Gaussians of the tile's depth-sorted list are staged through LDS in batches
// of 256; an entry is kept only if its alpha >= alpha_min ellipse reaches the
// tile's pixel-centre box.
#pragma once

#include "abcd_internal.h"

namespace abcd {
namespace {


struct BlendConsts {
  int width, height, ntx, ntiles, per_xcd;
  float alpha_min, alpha_max, t_min;
};

// Tile of this workgroup: the given schedule (heaviest tiles first), or, with
// none, raster order with each of the 8 XCDs (which take workgroups round
// robin) given a contiguous band of tiles, so that neighbouring tiles (which
// share Gaussians) share an L2.
__device__ __forceinline__ int tile_of_block(const BlendConsts& k, const uint32_t* order) {
  const int b = blockIdx.x;
  if (order) return (int)order[b];
  return (b & 7) * k.per_xcd + (b >> 3);
}

// One list entry as loaded from global memory by one thread.
struct Rec {
  float2 m;
  float4 co;
  float r, g, b;
  uint32_t gid;
  bool valid;
};

// The gathers of one entry, for a Gaussian index read earlier. The loads are
// unconditional (an invalid entry reads a valid index, see the callers):
// loads under a divergent branch would make the compiler wait for them at the
// branch's end instead of where the values are first used, which serialised
// the staging of every batch.
__device__ __forceinline__ Rec gather_rec(uint32_t gid, bool valid,
                                          const float2* __restrict__ means2d,
                                          const float4* __restrict__ conic_opacity,
                                          const float* __restrict__ rgb) {
  Rec r;
  r.valid = valid;
  r.gid = gid;
  r.m = means2d[gid];
  r.co = conic_opacity[gid];
  r.r = rgb[3 * gid];
  r.g = rgb[3 * gid + 1];
  r.b = rgb[3 * gid + 2];
  return r;
}

// Pixel-centre box of a tile, clipped to the image.
struct TileBox {
  float x0, x1, y0, y1;
};

__device__ __forceinline__ TileBox tile_box(const BlendConsts& k, int tile) {
  const int tx = tile % k.ntx, ty = tile / k.ntx;
  TileBox b;
  b.x0 = (float)(tx * kTile) + 0.5f;
  b.y0 = (float)(ty * kTile) + 0.5f;
  b.x1 = (float)(min(tx * kTile + kTile, k.width) - 1) + 0.5f;
  b.y1 = (float)(min(ty * kTile + kTile, k.height) - 1) + 0.5f;
  return b;
}

// Block-wide stream compaction of this thread's entry into slot `*pos`;
// returns the number kept. s_wcnt holds 4 wave counts.
__device__ __forceinline__ int compact(bool keep, int* s_wcnt, int& pos) {
  const int w = threadIdx.x >> 6;
  const uint64_t bal = __ballot(keep);
  if ((threadIdx.x & 63) == 0) s_wcnt[w] = __popcll(bal);
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int c = s_wcnt[k];
    off += k < w ? c : 0;
    tot += c;
  }
  pos = off + __popcll(bal & ((1ull << (threadIdx.x & 63)) - 1ull));
  return __builtin_amdgcn_readfirstlane(tot);  // uniform: loops over it branch on scalars
}

// Tile test and rows mask of an entry in one: bit w set when some pixel
// centre of rows 4w .. 4w + 3 of the tile (clipped to the image) can see the
// Gaussian with alpha >= alpha_min, i.e. d^T Q d <= tau = 2 ln(o / alpha_min);
// 0: the entry is dropped. With the tile's column range fixed, the minimum of
// the convex quadratic over dx is a convex function of dy whose minimiser y*
// is 0 when the mean's column lies in the range, else -b dx_e / c on the
// nearer edge dx_e; the minimum over a band is at y* clamped to the band, with
// dx = -b dy / a clamped to the columns. The margin keeps every entry whose
// per-pixel decision could go either way in fp32 (no pixel that blends is
// ever dropped, so the outputs do not depend on this test).
__device__ __forceinline__ uint32_t splat_rows(float u, float v, float a, float b, float c, float o,
                                               float alpha_min, const TileBox& box) {
  if (!(o >= alpha_min)) return 0u;
  const float tau = 2.0f * (__logf(o) - __logf(alpha_min));
  const float lim = tau * 1.001f + 1e-3f;
  const float ia = a > 0.0f ? 1.0f / a : 0.0f, ic = c > 0.0f ? 1.0f / c : 0.0f;
  const float dx0 = box.x0 - u, dx1 = box.x1 - u;
  const float dxe = dx0 > 0.0f ? dx0 : (dx1 < 0.0f ? dx1 : 0.0f);
  const float ys = -b * dxe * ic;
  uint32_t rows = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float yb0 = box.y0 + 4.0f * (float)w, yb1 = fminf(box.y1, yb0 + 3.0f);
    const float dy = fminf(fmaxf(ys, yb0 - v), yb1 - v);
    const float dx = fminf(fmaxf(-b * dy * ia, dx0), dx1);
    const float q = a * dx * dx + 2.0f * b * dx * dy + c * dy * dy;
    if (yb0 <= yb1 && q <= lim) rows |= 1u << w;
  }
  return rows;
}

// The same test for single pixel rows: bit w set when pixel row row0 + w of
// the tile (clipped to the image) can see the Gaussian. With the row fixed,
// the minimum over the columns is at dx = -b dy / a clamped to the columns.
__device__ __forceinline__ uint32_t splat_rows_single(float u, float v, float a, float b, float c,
                                                      float o, float alpha_min, const TileBox& box,
                                                      int row0) {
  if (!(o >= alpha_min)) return 0u;
  const float tau = 2.0f * (__logf(o) - __logf(alpha_min));
  const float lim = tau * 1.001f + 1e-3f;
  const float ia = a > 0.0f ? 1.0f / a : 0.0f;
  const float dx0 = box.x0 - u, dx1 = box.x1 - u;
  uint32_t rows = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float yb = box.y0 + (float)(row0 + w);
    const float dy = yb - v;
    const float dx = fminf(fmaxf(-b * dy * ia, dx0), dx1);
    const float q = a * dx * dx + 2.0f * b * dx * dy + c * dy * dy;
    if (yb <= box.y1 && q <= lim) rows |= 1u << w;
  }
  return rows;
}

// Block-wide compaction of the staged entries (as compact() does) and, for
// each wave w, the list of the staged slots whose rows mask has bit w, in
// list order, into s_idx[w]. s_cnt holds 5 x 4 wave counts. Returns the
// number kept; wcnt is the length of the calling wave's list (both uniform).
__device__ __forceinline__ int compact_rows(bool keep, uint32_t rows, int (*s_cnt)[4],
                                            uint8_t (*s_idx)[256], int& pos, int& wcnt) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const uint64_t below = (1ull << l) - 1ull;
  const uint64_t bal = __ballot(keep);
  uint64_t rb[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) rb[r] = __ballot((rows >> r) & 1u);
  if (l == 0) {
    s_cnt[0][w] = __popcll(bal);
#pragma unroll
    for (int r = 0; r < 4; ++r) s_cnt[1 + r][w] = __popcll(rb[r]);
  }
  __syncthreads();
  int off = 0, tot = 0, mine = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int c = s_cnt[0][v];
    off += v < w ? c : 0;
    tot += c;
    mine += s_cnt[1 + w][v];
  }
  pos = off + __popcll(bal & below);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if ((rows >> r) & 1u) {
      int o = 0;
#pragma unroll
      for (int v = 0; v < 4; ++v) o += v < w ? s_cnt[1 + r][v] : 0;
      s_idx[r][o + __popcll(rb[r] & below)] = (uint8_t)pos;
    }
  }
  wcnt = __builtin_amdgcn_readfirstlane(mine);
  return __builtin_amdgcn_readfirstlane(tot);
}

// Frames of at most this many tiles (without a split) take the forward and
// backward kernels that give each tile four workgroups, one pixel row per
// wave and four list entries per step of a wave.
constexpr int kRowsTiles = 256;

// Lane-bit-4 and lane-bit-5 exchanges. v_permlane16_swap of (x, x) leaves
// rows (0, 0, 2, 2) of x in its first result and rows (1, 1, 3, 3) in its
// second; v_permlane32_swap of (x, x) leaves halves (low, low) and (high,
// high). Either way the two results combined give the pair's total with the
// same operands in the same order on both partners, and a lane with the
// exchanged bit set finds its partner's value in the first result.
struct Swapped {
  float first, second;
};
__device__ __forceinline__ Swapped swap_bit4(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_int(x), __float_as_int(x), false, false);
  return Swapped{__int_as_float(p[0]), __int_as_float(p[1])};
}
__device__ __forceinline__ Swapped swap_bit5(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_int(x), __float_as_int(x), false, false);
  return Swapped{__int_as_float(p[0]), __int_as_float(p[1])};
}

constexpr int kGroup = 8;
constexpr int kBwdGroup = 4;  // the backward's group (register budget: 5 waves per SIMD)

BlendConsts consts(const abcd_camera& cam, const abcd_raster_params& prm) {
  BlendConsts k;
  k.width = cam.width;
  k.height = cam.height;
  k.ntx = tiles_x(cam.width);
  k.ntiles = k.ntx * tiles_y(cam.height);
  k.per_xcd = (k.ntiles + 7) / 8;
  k.alpha_min = prm.alpha_min;
  k.alpha_max = prm.alpha_max;
  k.t_min = prm.t_min;
  return k;
}

}  // namespace
}  // namespace abcd
