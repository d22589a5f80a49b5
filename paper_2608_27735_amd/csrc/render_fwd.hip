// render_fwd.hip -- forward tile rasterisation of the active partition,
// composited between F and B (paper, Method section), and the cached-render
// variant (F = B = transparent, fp16 store) used to refresh a partition's
// cached images.
//
// The forward blends each pixel's list front to back and stops a pixel once
// the next blend would take its transmittance below t_min; the workgroup
// stops when all its pixels have stopped.
//
// Each wave (four pixel rows of the tile) walks only the staged entries whose
// alpha >= alpha_min ellipse reaches its rows: the others cannot blend at any
// of its pixels, so the result is the same, and in tiles of many small
// Gaussians a wave's walk is a fraction of the tile's list.
#include <type_traits>

#include "blend.h"

namespace abcd {
namespace {

// kHalf: the cached-render variant: F = B = transparent, the image is written
// as fp16 RGBA to out16 (round to nearest even), no final T or walk lengths.
// Register budget: four waves per SIMD (at most 128 VGPRs).
template <bool kHalf>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void render_fwd_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    float4* __restrict__ out, float* __restrict__ final_T, uint32_t* __restrict__ last,
    unsigned long long* __restrict__ n_blends, const uint32_t* __restrict__ order,
    uint2* __restrict__ out16, int* __restrict__ rect, int fb_stop, SplitLayout sp) {
  __shared__ float4 s_ga[256];  // u, v, qa, qb
  __shared__ float4 s_gb[256];  // qc, o, r, g
  __shared__ float4 s_bl[256];  // b (16-byte stride: one address serves all three reads)
  __shared__ int s_pos[256];    // position in the tile's list
  __shared__ __align__(8) uint8_t s_idx[4][256];  // per wave: staged slots reaching its rows
  __shared__ int s_wcnt[5][4];
  __shared__ unsigned long long s_nb;
  __shared__ uint32_t s_base;
  __shared__ uint32_t s_walk;  // largest walk of the tile (split only)
  const int tile = tile_of_block(k, order);
  if ((unsigned)tile >= (unsigned)k.ntiles) return;
  const int tid = threadIdx.x;
  const int px = (tile % k.ntx) * kTile + (tid & 15);
  const int py = (tile / k.ntx) * kTile + (tid >> 4);
  const bool inside = px < k.width && py < k.height;
  const TileBox box = tile_box(k, tile);
  const uint32_t start = tile_ranges[2 * tile], end = tile_ranges[2 * tile + 1];
  const float fx = (float)px + 0.5f, fy = (float)py + 0.5f;
  float T = 1.0f, cr = 0.0f, cg = 0.0f, cb = 0.0f;
  uint32_t lastk = 0, nb = 0;
  bool done = !inside;
  // Stop threshold on the next transmittance. The compositing-aware rule
  // (1 - F_a) T_next < t_min is applied as T_next < t_min / (1 - F_a); a pixel
  // whose F leaves it less than t_min of weight blends nothing.
  float thr = k.t_min;
  if (!kHalf && fb_stop && F && inside) {
    const float vis = 1.0f - F[(int64_t)py * k.width + px].w;
    thr = vis > 0.0f ? k.t_min / vis : __builtin_huge_valf();
    done = vis < k.t_min;
  }
  // alpha below which the lane blends nothing: alpha_min, infinite once the
  // pixel has stopped
  float amin_l = done ? __builtin_huge_valf() : k.alpha_min;
  if (tid == 0) {
    s_nb = 0;
    s_walk = 0;
  }
  // Checkpoints for the split backward (uniform state): a slot per boundary
  // the walk crosses, taken when it crosses
  const uint32_t len = end - start;
  const uint32_t cht = (!kHalf && sp.ckpt) ? (uint32_t)sp.ch : 0u;
  const uint32_t chd = cht != 0u ? cht : 1u;  // divisor (only used when splitting)
  bool split_ok = cht != 0u && len > cht;
  bool crossed = false;
  // entries staged in the current chunk and the most in any chunk so far: the
  // backward's cost estimate for ordering its work items
  uint32_t staged = 0, staged_max = 0;
  // Loads run two batches ahead of use: the list values of batch b + 2 and
  // the gathers of batch b + 1 are in flight while batch b blends. Positions
  // past the list read its last entry (valid == false), so every load is
  // unconditional and in bounds.
  const uint32_t lastpos = end > start ? end - 1 : start;
  Rec rec{};
  uint32_t gid_next = 0;
  if (end > start) {  // uniform
    const uint32_t gid0 = values[min(start + tid, lastpos)];
    gid_next = values[min(start + 256 + tid, lastpos)];
    rec = gather_rec(gid0, start + tid < end, means2d, conic_opacity, rgb);
  }
  for (uint32_t b0 = start; b0 < end; b0 += 256) {
    if (__syncthreads_count(done) == 256) break;
    if (split_ok && b0 > start && (b0 - start) % chd == 0 && (b0 - start) / chd < kMaxChunks) {
      // state after the positions before b0; no pixel walks past a boundary
      // the loop did not reach
      if (tid == 0) {
        const uint32_t got = atomicAdd(&sp.hdr[0], 1u);
        s_base = got < sp.nslots ? got : kNoSlot;
        sp.slot_of[(size_t)tile * kMaxChunks + (b0 - start) / chd] = s_base;
      }
      __syncthreads();
      const uint32_t slot = s_base;
      if (slot == kNoSlot) {
        split_ok = false;  // out of slots: the backward takes this tile whole
      } else {
        sp.ckpt[(size_t)slot * 256 + tid] = make_float4(T, cr, cg, cb);
        crossed = true;
        staged_max = max(staged_max, staged);
        staged = 0;
      }
    }
    const float3 cn = conic_of(rec.co);
    // each wave walks only the staged entries whose ellipse reaches its four
    // pixel rows: the others contribute nothing to any of its pixels
    const uint32_t rows =
        rec.valid ? splat_rows(rec.m.x, rec.m.y, cn.x, cn.y, cn.z, rec.co.w, k.alpha_min, box) : 0u;
    const bool keep = rows != 0u;
    int pos, wcnt;
    const int cnt = compact_rows(keep, rows, s_wcnt, s_idx, pos, wcnt);
    staged += (uint32_t)cnt;
    if (keep) {
      const Splat sp = make_splat(rec.m, rec.co);
      s_ga[pos] = make_float4(sp.u, sp.v, sp.qa, sp.qb);
      s_gb[pos] = make_float4(sp.qc, sp.o, rec.r, rec.g);
      s_bl[pos].x = rec.b;
      s_pos[pos] = (int)(b0 - start) + tid;
    }
    __syncthreads();
    // gathers of the next batch and list values of the one after overlap the
    // blend of this one
    const uint32_t nxt = b0 + 256 + tid;
    const uint32_t gid_after = values[min(b0 + 512 + tid, lastpos)];
    rec = gather_rec(gid_next, nxt < end, means2d, conic_opacity, rgb);
    gid_next = gid_after;
    if (__ballot(!done)) {
      // The wave walks its own list of staged slots, kGroup entries at a
      // time; all LDS reads of a group are issued before the first is used,
      // so the LDS latency is paid once per group.
      static_assert(kGroup % 4 == 0, "slot indices are read four at a time");
      const uint32_t* my_idx = reinterpret_cast<const uint32_t*>(s_idx[tid >> 6]);
      int jl = -1;  // position in the wave's list of the last entry the lane blended
      // One group; kTail: the list ends inside it, and positions past the end
      // read the group's first entry and blend nothing (every value read is
      // finite). Returns true when no pixel of the wave is left.
      auto group = [&](const int j0, auto tail) -> bool {
        constexpr bool kTail = decltype(tail)::value;
        uint32_t iw[kGroup / 4];
#pragma unroll
        for (int h = 0; h < kGroup / 4; ++h) iw[h] = __builtin_amdgcn_readfirstlane(my_idx[j0 / 4 + h]);
        float4 ga[kGroup], gb[kGroup];
        float bl[kGroup];
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
          int j = (int)((iw[i >> 2] >> (8 * (i & 3))) & 255u);
          if (kTail && j0 + i >= wcnt) j = (int)(iw[0] & 255u);
          ga[i] = s_ga[j];
          gb[i] = s_gb[j];
          bl[i] = s_bl[j].x;
        }
        // keep the group's reads ahead of the arithmetic (the compiler would
        // otherwise sink each read to its use)
#pragma unroll
        for (int i = 0; i < kGroup; ++i)
          asm volatile("" ::"v"(ga[i].x), "v"(ga[i].y), "v"(ga[i].z), "v"(ga[i].w), "v"(gb[i].x),
                       "v"(gb[i].y), "v"(gb[i].z), "v"(gb[i].w), "v"(bl[i]));
        // alpha of each entry at this pixel, 0 where the lane does not blend
        // it: below alpha_min (eval_alpha's skip: its power is minus a sum of
        // squares, never positive), or the pixel has stopped (amin_l = inf)
        float a[kGroup];
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
          const AlphaEval ae = eval_alpha(fx - ga[i].x, fy - ga[i].y, ga[i].z, ga[i].w, gb[i].x,
                                          gb[i].y, k.alpha_min, k.alpha_max);
          a[i] = ae.alpha < amin_l ? 0.0f : ae.alpha;
          if (kTail && j0 + i >= wcnt) a[i] = 0.0f;
        }
        // The chain Tc of every hit blended, T (1 - alpha) with one rounding
        // (exactly T where alpha = 0), holds the values of the entry-by-entry
        // walk up to its first stop. T never increases and only hits change
        // it, so an entry blends exactly when its next value is still at or
        // above the threshold (ok): the first hit below stops the pixel and
        // every later value is below too. No branch depends on the stop.
        float Tc = T;
        int jg = -1;  // the lane's last blended entry of the group
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
          const float Tn = fmaf(-Tc, a[i], Tc);
          const bool ok = Tn >= thr;
          // a zero weight adds exactly zero (colours are finite and >= 0)
          const float wgt = ok ? a[i] * Tc : 0.0f;
          cr = fmaf(gb[i].z, wgt, cr);
          cg = fmaf(gb[i].w, wgt, cg);
          cb = fmaf(bl[i], wgt, cb);
          const bool blend = ok && a[i] != 0.0f;
          jg = blend ? i : jg;
          nb += blend ? 1u : 0u;
          T = ok ? Tn : T;
          Tc = Tn;
        }
        jl = jg >= 0 ? j0 + jg : jl;
        done = done || Tc < thr;
        amin_l = done ? __builtin_huge_valf() : amin_l;
        return !__ballot(!done);
      };
      int j0 = 0;
      bool over = false;
      for (; j0 + kGroup <= wcnt && !over; j0 += kGroup) over = group(j0, std::false_type{});
      if (!over && j0 < wcnt) group(j0, std::true_type{});
      if (jl >= 0) lastk = (uint32_t)s_pos[s_idx[tid >> 6][jl]] + 1;
    }
    // s_wcnt is rewritten only after the next barrier
  }
  if (cht != 0u) {
    // the tile's largest walk, for the backward's schedule
    uint32_t wmax = lastk;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) wmax = max(wmax, (uint32_t)__shfl_xor((int)wmax, off, 64));
    if ((tid & 63) == 0 && wmax) atomicMax(&s_walk, wmax);
    __syncthreads();  // every thread has read s_base; s_walk is complete
    if (tid == 0) {
      sp.walk[tile] = s_walk;
      uint32_t fin = kNoSlot;
      if (split_ok && crossed) {
        const uint32_t got = atomicAdd(&sp.hdr[0], 1u);
        if (got < sp.nslots) fin = got;
      }
      s_base = fin;
      sp.slot_of[(size_t)tile * kMaxChunks] = fin;
      sp.work[tile] = min(max(staged_max, staged), kSplitTile - 1u) | (fin != kNoSlot ? kSplitTile : 0u);
    }
    __syncthreads();
    const uint32_t slot = s_base;
    if (slot != kNoSlot) sp.ckpt[(size_t)slot * 256 + tid] = make_float4(T, cr, cg, cb);
  }
  if (kHalf && rect) {
    // coverage of the cached image: tiles holding any pixel that blended
    if (__syncthreads_or(inside && T < 1.0f) && tid == 0) {
      const int tx = tile % k.ntx, ty = tile / k.ntx;
      atomicMin(&rect[0], tx * kTile);
      atomicMin(&rect[1], ty * kTile);
      atomicMax(&rect[2], min(tx * kTile + kTile, k.width));
      atomicMax(&rect[3], min(ty * kTile + kTile, k.height));
    }
  }
  if (inside) {
    const int64_t p = (int64_t)py * k.width + px;
    if (kHalf) {
      const _Float16 h[4] = {(_Float16)cr, (_Float16)cg, (_Float16)cb, (_Float16)(1.0f - T)};
      out16[p] = __builtin_bit_cast(uint2, h);
    } else {
      const float4 f = F ? F[p] : make_float4(0, 0, 0, 0);
      const float4 bb = B ? B[p] : make_float4(0, 0, 0, 0);
      const float s = 1.0f - f.w;
      out[p] = make_float4(f.x + s * (cr + T * bb.x), f.y + s * (cg + T * bb.y),
                           f.z + s * (cb + T * bb.z), f.w + s * (1.0f - T * (1.0f - bb.w)));
      final_T[p] = T;
      last[p] = lastk;
    }
  }
  if (n_blends) {
    const unsigned long long wsum = wave_sum_u32(nb);
    __syncthreads();
    if ((tid & 63) == 0) atomicAdd(&s_nb, wsum);
    __syncthreads();
    if (tid == 0 && s_nb) atomicAdd(n_blends, s_nb);
  }
}

// Small frames (at most kRowsTiles tiles, no split): four workgroups per
// tile (rows 4q .. 4q + 3 for quarter q), one pixel row per wave and four
// list entries per step of a wave, as in the backward for small frames. Lane
// l holds column l & 15 of the wave's row and entry l >> 4 of the step (entry
// 0 the frontmost). Per step, the transmittance before and after each entry
// is the running chain T times an exclusive and an inclusive prefix product of
// 1 - alpha over the step's entries (scans over lane bits 4 and 5). The
// inclusive products never increase along the step (each is a rounded product
// of the one before and a factor at most 1), so an entry blends exactly when
// its product is still at or above the threshold, and the first entry that
// fails stops the pixel. Each lane sums the colour, blend count and walk end
// of its own entries; the four rows are combined once, at the end (the
// pixel's transmittance is the smallest of the rows' last blended values).
template <bool kHalf>
__global__ __launch_bounds__(256) void render_fwd_rows_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    float4* __restrict__ out, float* __restrict__ final_T, uint32_t* __restrict__ last,
    unsigned long long* __restrict__ n_blends, uint2* __restrict__ out16, int* __restrict__ rect,
    int fb_stop) {
  __shared__ float4 s_ga[256];  // u, v, qa, qb
  __shared__ float4 s_gb[256];  // qc, o, r, g
  __shared__ float s_bl[256];   // b
  __shared__ int s_pos[256];    // position in the tile's list
  __shared__ __align__(4) uint8_t s_idx[4][256];  // per wave: staged slots reaching its row
  __shared__ int s_wcnt[5][4];
  __shared__ unsigned long long s_nb;
  const int tile = (int)(blockIdx.x >> 2), quarter = (int)(blockIdx.x & 3);
  const int tid = threadIdx.x, lane = tid & 63, col = lane & 15, e = lane >> 4;
  const int px = (tile % k.ntx) * kTile + col;
  const int py = (tile / k.ntx) * kTile + 4 * quarter + (tid >> 6);
  const bool inside = px < k.width && py < k.height;
  const TileBox box = tile_box(k, tile);
  const uint32_t start = tile_ranges[2 * tile], end = tile_ranges[2 * tile + 1];
  const float fx = (float)px + 0.5f, fy = (float)py + 0.5f;
  bool done = !inside;
  float thr = k.t_min;  // stop threshold on the next transmittance (see render_fwd_kernel)
  if (!kHalf && fb_stop && F && inside) {
    const float vis = 1.0f - F[(int64_t)py * k.width + px].w;
    thr = vis > 0.0f ? k.t_min / vis : __builtin_huge_valf();
    done = vis < k.t_min;
  }
  float amin_l = done ? __builtin_huge_valf() : k.alpha_min;
  float T = 1.0f;      // the pixel's chain through the steps so far (same in its four lanes)
  float Tlast = 1.0f;  // the chain after this lane's last entry that passed the threshold
  float cr = 0.0f, cg = 0.0f, cb = 0.0f;
  uint32_t lastk = 0, nb = 0;
  const bool odd = lane & 16, high = lane & 32;
  if (tid == 0) s_nb = 0;
  const uint32_t lastpos = end > start ? end - 1 : start;
  Rec rec{};
  uint32_t gid_next = 0;
  if (end > start) {  // uniform
    const uint32_t gid0 = values[min(start + tid, lastpos)];
    gid_next = values[min(start + 256 + tid, lastpos)];
    rec = gather_rec(gid0, start + tid < end, means2d, conic_opacity, rgb);
  }
  for (uint32_t b0 = start; b0 < end; b0 += 256) {
    if (__syncthreads_count(done) == 256) break;
    const float3 cn = conic_of(rec.co);
    const uint32_t rows = rec.valid ? splat_rows_single(rec.m.x, rec.m.y, cn.x, cn.y, cn.z,
                                                        rec.co.w, k.alpha_min, box, 4 * quarter)
                                    : 0u;
    const bool keep = rows != 0u;
    int pos, wcnt;
    compact_rows(keep, rows, s_wcnt, s_idx, pos, wcnt);
    if (keep) {
      const Splat sp = make_splat(rec.m, rec.co);
      s_ga[pos] = make_float4(sp.u, sp.v, sp.qa, sp.qb);
      s_gb[pos] = make_float4(sp.qc, sp.o, rec.r, rec.g);
      s_bl[pos] = rec.b;
      s_pos[pos] = (int)(b0 - start) + tid;
    }
    __syncthreads();
    const uint32_t nxt = b0 + 256 + tid;
    const uint32_t gid_after = values[min(b0 + 512 + tid, lastpos)];
    rec = gather_rec(gid_next, nxt < end, means2d, conic_opacity, rgb);
    gid_next = gid_after;
    if (__ballot(!done)) {
      // lanes past the end of the wave's list read the step's first entry
      // (every value read is finite) and blend nothing
      const uint8_t* my_idx = s_idx[tid >> 6];
      int jl = -1;  // position in the wave's list of the lane's last blended entry
      for (int j0 = 0; j0 < wcnt; j0 += 4) {
        const int jw = j0 + e;
        const int j = my_idx[jw < wcnt ? jw : j0];
        const float4 ga = s_ga[j], gb = s_gb[j];
        const float bl = s_bl[j];
        const AlphaEval ae = eval_alpha(fx - ga.x, fy - ga.y, ga.z, ga.w, gb.x, gb.y, k.alpha_min,
                                        k.alpha_max);
        // 0 where the lane blends nothing: past the list, below alpha_min
        // (eval_alpha's power is never positive), or the pixel has stopped
        const float a = (jw < wcnt && !(ae.alpha < amin_l)) ? ae.alpha : 0.0f;
        const float om = 1.0f - a;
        const Swapped p1 = swap_bit4(om);
        const float t1 = p1.first * p1.second;
        const Swapped p2 = swap_bit5(t1);
        const float in1 = odd ? t1 : om, ex1 = odd ? p1.first : 1.0f;
        const float Tn = T * (high ? in1 * p2.first : in1);  // after the entry
        const float Tc = T * (high ? ex1 * p2.first : ex1);  // before it
        const bool ok = Tn >= thr;
        // a zero weight adds exactly zero (colours are finite and >= 0)
        const float wgt = ok ? a * Tc : 0.0f;
        cr = fmaf(gb.z, wgt, cr);
        cg = fmaf(gb.w, wgt, cg);
        cb = fmaf(bl, wgt, cb);
        const bool blend = ok && a != 0.0f;
        jl = blend ? jw : jl;
        nb += blend ? 1u : 0u;
        Tlast = ok ? Tn : Tlast;
        T *= p2.first * p2.second;  // through the step's four entries
        done = done || T < thr;
        amin_l = done ? __builtin_huge_valf() : amin_l;
        if (!__ballot(!done)) break;  // wave-uniform
      }
      if (jl >= 0) lastk = (uint32_t)s_pos[my_idx[jl]] + 1;
    }
    // s_wcnt is rewritten only after the next barrier
  }
  // combine the pixel's four lanes
  {
    const Swapped r1 = swap_bit4(cr), g1 = swap_bit4(cg), c1 = swap_bit4(cb), t1 = swap_bit4(Tlast);
    const Swapped r2 = swap_bit5(r1.first + r1.second), g2 = swap_bit5(g1.first + g1.second),
                  c2 = swap_bit5(c1.first + c1.second), t2 = swap_bit5(fminf(t1.first, t1.second));
    cr = r2.first + r2.second;
    cg = g2.first + g2.second;
    cb = c2.first + c2.second;
    T = fminf(t2.first, t2.second);
    const Swapped k1 = swap_bit4(__uint_as_float(lastk));
    const uint32_t l1 = max(__float_as_uint(k1.first), __float_as_uint(k1.second));
    const Swapped k2 = swap_bit5(__uint_as_float(l1));
    lastk = max(__float_as_uint(k2.first), __float_as_uint(k2.second));
  }
  if (kHalf && rect) {
    // coverage of the cached image: tiles holding any pixel that blended
    if (__syncthreads_or(inside && T < 1.0f) && tid == 0) {
      const int tx = tile % k.ntx, ty = tile / k.ntx;
      atomicMin(&rect[0], tx * kTile);
      atomicMin(&rect[1], ty * kTile);
      atomicMax(&rect[2], min(tx * kTile + kTile, k.width));
      atomicMax(&rect[3], min(ty * kTile + kTile, k.height));
    }
  }
  if (inside && e == 0) {
    const int64_t p = (int64_t)py * k.width + px;
    if (kHalf) {
      const _Float16 h[4] = {(_Float16)cr, (_Float16)cg, (_Float16)cb, (_Float16)(1.0f - T)};
      out16[p] = __builtin_bit_cast(uint2, h);
    } else {
      const float4 f = F ? F[p] : make_float4(0, 0, 0, 0);
      const float4 bb = B ? B[p] : make_float4(0, 0, 0, 0);
      const float s = 1.0f - f.w;
      out[p] = make_float4(f.x + s * (cr + T * bb.x), f.y + s * (cg + T * bb.y),
                           f.z + s * (cb + T * bb.z), f.w + s * (1.0f - T * (1.0f - bb.w)));
      final_T[p] = T;
      last[p] = lastk;
    }
  }
  if (n_blends) {
    const unsigned long long wsum = wave_sum_u32(nb);
    __syncthreads();
    if (lane == 0) atomicAdd(&s_nb, wsum);
    __syncthreads();
    if (tid == 0 && s_nb) atomicAdd(n_blends, s_nb);
  }
}

__global__ void rect_init_kernel(int* __restrict__ rect, int width, int height) {
  if (threadIdx.x == 0) {
    rect[0] = width;
    rect[1] = height;
    rect[2] = 0;
    rect[3] = 0;
  }
}

}  // namespace

int32_t launch_render_fwd(const abcd_camera& cam, const abcd_raster_params& prm,
                          const uint32_t* tile_ranges, const uint32_t* values_sorted,
                          const float* means2d, const float* conic_opacity, const float* rgb,
                          const float* F, const float* B, float* out_rgba, float* final_T,
                          uint32_t* last, unsigned long long* n_blends, const uint32_t* tile_order,
                          const SplitLayout& split, hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  const int grid = tile_order ? k.ntiles : 8 * k.per_xcd;
  if (!split.ckpt && k.ntiles <= kRowsTiles) {
    ABCD_LAUNCH("render_fwd", render_fwd_rows_kernel<false>, 4 * k.ntiles, kBlock, 0, stream, k,
                tile_ranges, values_sorted, reinterpret_cast<const float2*>(means2d),
                reinterpret_cast<const float4*>(conic_opacity), rgb,
                reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B),
                reinterpret_cast<float4*>(out_rgba), final_T, last, n_blends, nullptr, nullptr,
                (int)(prm.flags & ABCD_FLAG_FB_STOP));
    ABCD_HIP(hipGetLastError());
    return ABCD_OK;
  }
  if (split.ckpt) TRY_STATUS(launch_zero(reinterpret_cast<float*>(split.hdr), 16, stream));
  ABCD_LAUNCH("render_fwd", render_fwd_kernel<false>, grid, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb,
              reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B),
              reinterpret_cast<float4*>(out_rgba), final_T, last, n_blends, tile_order, nullptr,
              nullptr, (int)(prm.flags & ABCD_FLAG_FB_STOP), split);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_render_cache(const abcd_camera& cam, const abcd_raster_params& prm,
                            const uint32_t* tile_ranges, const uint32_t* tile_order,
                            const uint32_t* values_sorted, const float* means2d,
                            const float* conic_opacity, const float* rgb, uint16_t* image_f16,
                            int32_t* rect, hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  const int grid = tile_order ? k.ntiles : 8 * k.per_xcd;
  if (rect) {
    ABCD_LAUNCH("cache_rect_init", rect_init_kernel, 1, 64, 0, stream, rect, k.width, k.height);
    ABCD_HIP(hipGetLastError());
  }
  if (k.ntiles <= kRowsTiles) {
    ABCD_LAUNCH("render_cache", render_fwd_rows_kernel<true>, 4 * k.ntiles, kBlock, 0, stream, k,
                tile_ranges, values_sorted, reinterpret_cast<const float2*>(means2d),
                reinterpret_cast<const float4*>(conic_opacity), rgb, nullptr, nullptr, nullptr,
                nullptr, nullptr, nullptr, reinterpret_cast<uint2*>(image_f16), rect, 0);
    ABCD_HIP(hipGetLastError());
    return ABCD_OK;
  }
  ABCD_LAUNCH("render_cache", render_fwd_kernel<true>, grid, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb, nullptr, nullptr, nullptr,
              nullptr, nullptr, nullptr, tile_order, reinterpret_cast<uint2*>(image_f16), rect, 0,
              SplitLayout{});
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd
