// render.hip -- tile rasterisation of the active partition, composited between
// F and B (paper, Method section), and its backward pass.
//
// One 256-thread workgroup (4 wave64) per 16x16 tile, one thread per pixel.
// Gaussians of the tile's depth-sorted list are staged through LDS in batches
// of 256. The forward blends front to back and stops a pixel once the next
// blend would take its transmittance below t_min; the workgroup stops when all
// its pixels have stopped. The backward walks each pixel's list back to front
// from its last blended entry, reduces each Gaussian's 9 screen-space
// gradients across the wave with cross-lane adds, combines the 4 waves in LDS
// and issues one global fp32 atomic per Gaussian and field per tile.
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

__device__ __forceinline__ Rec load_rec(const uint32_t* __restrict__ values, uint32_t idx,
                                        bool valid, const float2* __restrict__ means2d,
                                        const float4* __restrict__ conic_opacity,
                                        const float* __restrict__ rgb) {
  Rec r;
  r.valid = valid;
  r.gid = 0;
  if (valid) {
    r.gid = values[idx];
    r.m = means2d[r.gid];
    r.co = conic_opacity[r.gid];
    r.r = rgb[3 * r.gid];
    r.g = rgb[3 * r.gid + 1];
    r.b = rgb[3 * r.gid + 2];
  }
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
  return tot;
}

constexpr int kGroup = 8;
constexpr int kBwdGroup = 8;  // the backward's group

// kHalf: the cached-render variant: F = B = transparent, the image is written
// as fp16 RGBA to out16 (round to nearest even), no final T or walk lengths.
template <bool kHalf>
__global__ __launch_bounds__(256) void render_fwd_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    float4* __restrict__ out, float* __restrict__ final_T, uint32_t* __restrict__ last,
    unsigned long long* __restrict__ n_blends, const uint32_t* __restrict__ order,
    uint2* __restrict__ out16) {
  __shared__ float4 s_ga[256];  // u, v, qa, qb
  __shared__ float4 s_gb[256];  // qc, o, r, g
  __shared__ float s_bl[256];   // b
  __shared__ int s_pos[256];    // position in the tile's list
  __shared__ int s_wcnt[4];
  __shared__ unsigned long long s_nb;
  const int tile = tile_of_block(k, order);
  if (tile >= k.ntiles) return;
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
  if (tid == 0) s_nb = 0;
  Rec rec = load_rec(values, start + tid, start + tid < end, means2d, conic_opacity, rgb);
  for (uint32_t b0 = start; b0 < end; b0 += 256) {
    if (__syncthreads_count(done) == 256) break;
    const bool keep = rec.valid && splat_touches_box(rec.m.x, rec.m.y, rec.co.x, rec.co.y, rec.co.z,
                                                     rec.co.w, k.alpha_min, box.x0, box.x1,
                                                     box.y0, box.y1);
    int pos;
    const int cnt = compact(keep, s_wcnt, pos);
    if (keep) {
      const Splat sp = make_splat(rec.m, rec.co);
      s_ga[pos] = make_float4(sp.u, sp.v, sp.qa, sp.qb);
      s_gb[pos] = make_float4(sp.qc, sp.o, rec.r, rec.g);
      s_bl[pos] = rec.b;
      s_pos[pos] = (int)(b0 - start) + tid;
    }
    __syncthreads();
    // gathers of the next batch overlap the blend of this one
    const uint32_t nxt = b0 + 256 + tid;
    rec = load_rec(values, nxt, nxt < end, means2d, conic_opacity, rgb);
    if (__ballot(!done)) {
      // Lanes step through the entries together without divergent branches:
      // a lane that skips an entry, or has stopped, blends with weight 0.
      // Entries are read from LDS kGroup at a time, all reads issued before
      // the first is used, so the LDS latency is paid once per group.
      int jl = -1;  // last entry of this batch the lane blended
      for (int j0 = 0; j0 < cnt; j0 += kGroup) {
        float4 ga[kGroup], gb[kGroup];
        float bl[kGroup];
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
          const int j = min(j0 + i, 255);
          ga[i] = s_ga[j];
          gb[i] = s_gb[j];
          bl[i] = s_bl[j];
        }
#pragma unroll
        for (int i = 0; i < kGroup; ++i) {
          if (j0 + i >= cnt) break;  // wave-uniform
          const AlphaEval ae = eval_alpha(fx - ga[i].x, fy - ga[i].y, ga[i].z, ga[i].w, gb[i].x,
                                          gb[i].y, k.alpha_min, k.alpha_max);
          const float Tn = T * (1.0f - ae.alpha);
          const bool hit = !done && !ae.skip;
          const bool stop = hit && Tn < k.t_min;
          const bool blend = hit && !stop;
          done = done || stop;
          const float wgt = blend ? ae.alpha * T : 0.0f;
          cr += gb[i].z * wgt;
          cg += gb[i].w * wgt;
          cb += bl[i] * wgt;
          T = blend ? Tn : T;
          jl = blend ? j0 + i : jl;
          nb += blend ? 1u : 0u;
        }
        if (!__ballot(!done)) break;  // wave-uniform
      }
      if (jl >= 0) lastk = (uint32_t)s_pos[jl] + 1;
    }
    // s_wcnt is rewritten only after the next barrier
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


// DPP lane move inside the wave (all rows and banks enabled).
template <int kCtrl>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xF, 0xF, false));
}

// Wave64 sum of nine values at once, by recursive halving: at each of the
// first three exchanges a lane keeps half of its values and receives the
// partner's partial sums of that half (quad xor 1, quad xor 2, row rotate 4),
// the fourth pairs the survivor with the ninth value (row rotate 8), and two
// cross-row swaps (v_permlane16_swap, v_permlane32_swap) finish. A rotation
// by 4 (by 8) within a 16-lane row pairs lanes that differ in bit 2 (bit 3)
// and agree in the lower bits, so partners hold partial sums of the same
// values over disjoint lane sets. About 30 instructions, all VALU, instead of
// 9 separate six-step reductions. On return, lane l < 16 holds the wave
// total of value sum9_slot(l); every row holds the same totals.
__device__ __forceinline__ float wave_sum9(const float (&g)[9], int lane) {
  const bool b0 = lane & 1, b1 = lane & 2, b2 = lane & 4, b3 = lane & 8;
  float a[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float keep = b0 ? g[q + 4] : g[q];
    const float send = b0 ? g[q] : g[q + 4];
    a[q] = keep + dpp_mov<0xB1>(send);
  }
  float v8 = g[8] + dpp_mov<0xB1>(g[8]);
  float b[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const float keep = b1 ? a[q + 2] : a[q];
    const float send = b1 ? a[q] : a[q + 2];
    b[q] = keep + dpp_mov<0x4E>(send);
  }
  v8 += dpp_mov<0x4E>(v8);
  const float c = (b2 ? b[1] : b[0]) + dpp_mov<0x124>(b2 ? b[0] : b[1]);
  v8 += dpp_mov<0x124>(v8);
  float d = (b3 ? v8 : c) + dpp_mov<0x128>(b3 ? c : v8);
  // across rows: v_permlane16_swap / v_permlane32_swap exchange rows 0 <-> 1,
  // 2 <-> 3 (halves 0 <-> 1); of the two registers each lane gets back, one
  // is its own value and the other its partner's, so their sum is the pair sum
  {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_int(d), __float_as_int(d), false,
                                                    false);
    d = __int_as_float(p[0]) + __int_as_float(p[1]);
  }
  {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_int(d), __float_as_int(d), false,
                                                    false);
    d = __int_as_float(p[0]) + __int_as_float(p[1]);
  }
  return d;
}

// Which of the nine values lane l (< 16) holds after wave_sum9.
__device__ __forceinline__ int sum9_slot(int l) {
  return l < 8 ? 4 * (l & 1) + 2 * ((l >> 1) & 1) + ((l >> 2) & 1) : 8;
}

__global__ __launch_bounds__(256) void render_bwd_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    const float* __restrict__ final_T, const uint32_t* __restrict__ last,
    const float4* __restrict__ dL_dout, float* __restrict__ g2d, const uint32_t* __restrict__ order) {
  __shared__ float4 s_ga[256];  // u, v, qa, qb
  __shared__ float4 s_gb[256];  // qc, o, r, g
  __shared__ float4 s_gc[256];  // a, b, c (conic), colour b
  __shared__ int s_pos[256];
  __shared__ uint32_t s_g[256];
  __shared__ float s_acc[9 * 256];  // entry-major: [entry][9]
  __shared__ int s_wcnt[4];
  __shared__ uint32_t s_max;
  const int tile = tile_of_block(k, order);
  if (tile >= k.ntiles) return;
  const int tid = threadIdx.x;
  const int px = (tile % k.ntx) * kTile + (tid & 15);
  const int py = (tile / k.ntx) * kTile + (tid >> 4);
  const bool inside = px < k.width && py < k.height;
  const TileBox box = tile_box(k, tile);
  const uint32_t start = tile_ranges[2 * tile];
  const float fx = (float)px + 0.5f, fy = (float)py + 0.5f;
  float T = 1.0f, gcr = 0, gcg = 0, gcb = 0, gT = 0;
  uint32_t lastp = 0;
  if (tid == 0) s_max = 0;
  __syncthreads();
  if (inside) {
    const int64_t p = (int64_t)py * k.width + px;
    T = final_T[p];
    lastp = last[p];
    const float4 G = dL_dout[p];
    const float4 f = F ? F[p] : make_float4(0, 0, 0, 0);
    const float4 bb = B ? B[p] : make_float4(0, 0, 0, 0);
    const float s = 1.0f - f.w;
    gcr = s * G.x;
    gcg = s * G.y;
    gcb = s * G.z;
    gT = s * (G.x * bb.x + G.y * bb.y + G.z * bb.z - G.w * (1.0f - bb.w));
    if (lastp) atomicMax(&s_max, lastp);
  }
  const float Tfin = T;
  // RG = sum over channels of gc_ch R_ch, where R is the colour accumulated
  // behind the current entry (normalised by its transmittance): the
  // alpha-derivative needs R only through this sum.
  float RG = 0.0f;
  __syncthreads();
  const uint32_t nent = s_max;
  const int lane = tid & 63, slot = sum9_slot(lane & 15);
  uint32_t wml = lastp;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) wml = max(wml, (uint32_t)__shfl_xor((int)wml, off, 64));
  // entry j of a batch is list position bend - 1 - j (back to front)
  uint32_t bend = start + nent;
  Rec rec = load_rec(values, bend - 1 - tid, tid < (int)nent, means2d, conic_opacity, rgb);
  while (bend > start) {
    const uint32_t bbeg = bend - min(256u, bend - start);
    __syncthreads();
    const bool keep = rec.valid && splat_touches_box(rec.m.x, rec.m.y, rec.co.x, rec.co.y, rec.co.z,
                                                     rec.co.w, k.alpha_min, box.x0, box.x1,
                                                     box.y0, box.y1);
    int pos;
    const int cnt = compact(keep, s_wcnt, pos);
    if (keep) {
      const Splat sp = make_splat(rec.m, rec.co);
      s_ga[pos] = make_float4(sp.u, sp.v, sp.qa, sp.qb);
      s_gb[pos] = make_float4(sp.qc, sp.o, rec.r, rec.g);
      s_gc[pos] = make_float4(rec.co.x, rec.co.y, rec.co.z, rec.b);
      s_pos[pos] = (int)(bend - 1 - tid - start);
      s_g[pos] = rec.gid;
#pragma unroll
      for (int q = 0; q < 9; ++q) s_acc[9 * pos + q] = 0.0f;
    }
    __syncthreads();
    {
      const uint32_t nxt_end = bbeg;
      const bool v = (uint32_t)tid < nxt_end - start;
      rec = load_rec(values, nxt_end - 1 - tid, v, means2d, conic_opacity, rgb);
    }
    // Entries are read from LDS kGroup at a time, all reads issued before the
    // first is used, so the LDS latency is paid once per group.
    for (int j0 = 0; j0 < cnt; j0 += kBwdGroup) {
    float4 gav[kBwdGroup], gbv[kBwdGroup], gcv[kBwdGroup];
    uint32_t kkv[kBwdGroup];
#pragma unroll
    for (int i = 0; i < kBwdGroup; ++i) {
      const int j = min(j0 + i, 255);
      gav[i] = s_ga[j];
      gbv[i] = s_gb[j];
      gcv[i] = s_gc[j];
      kkv[i] = (uint32_t)s_pos[j];
    }
#pragma unroll
    for (int i = 0; i < kBwdGroup; ++i) {
      const int j = j0 + i;
      if (j >= cnt) break;  // wave-uniform
      const uint32_t kk = kkv[i];
      const float4 ga = gav[i], gb = gbv[i], gc = gcv[i];
      if (kk >= wml) continue;  // wave-uniform: no pixel of this wave reaches entry kk
      const float dx = fx - ga.x, dy = fy - ga.y;
      const AlphaEval ae = eval_alpha(dx, dy, ga.z, ga.w, gb.x, gb.y, k.alpha_min, k.alpha_max);
      const bool contrib = kk < lastp && !ae.skip;
      if (!__ballot(contrib)) continue;  // wave-uniform
      // Branch-free per lane: a lane that does not blend this entry takes
      // alpha = 0, which leaves T and R unchanged, and a zero mask on the
      // alpha-derivative terms.
      const float a = contrib ? ae.alpha : 0.0f;
      const float om = 1.0f - a;
      const float iom = __builtin_amdgcn_rcpf(om);  // om >= 1 - alpha_max > 0
      const float Tk = T * iom;
      const float wgt = a * Tk;
      float gr[9];
      gr[6] = wgt * gcr;
      gr[7] = wgt * gcg;
      gr[8] = wgt * gcb;
      const float CG = gb.z * gcr + gb.w * gcg + gc.w * gcb;
      const float dLda = Tk * (CG - RG) - (Tfin * iom) * gT;
      RG = a * CG + om * RG;
      T = Tk;
      const float dm = (contrib && !ae.clamped) ? dLda : 0.0f;
      const float gp = a * dm;
      // first and second moments of gp over the pixels; the conic and the
      // constant factors are applied once per entry at the flush
      const float q = gp * dx, r = gp * dy;
      gr[0] = q;
      gr[1] = r;
      gr[2] = q * dx;
      gr[3] = q * dy;
      gr[4] = r * dy;
      gr[5] = ae.e * dm;
      const float v = wave_sum9(gr, lane);
      if (lane < 9) atomicAdd(&s_acc[9 * j + slot], v);
    }
    }
    __syncthreads();
    if (tid < cnt) {
      // moments -> dL/d(u, v, a, b, c): with q = dL/dpower * (dx, dy),
      // d power / d(u, v) = (a dx + b dy, b dx + c dy), d power / d(a, b, c)
      // = (-dx^2 / 2, -dx dy, -dy^2 / 2)
      const float4 co = s_gc[tid];
      float g[9];
#pragma unroll
      for (int q = 0; q < 9; ++q) g[q] = s_acc[9 * tid + q];
      const float mx = g[0], my = g[1];
      g[0] = co.x * mx + co.y * my;
      g[1] = co.y * mx + co.z * my;
      g[2] = -0.5f * g[2];
      g[3] = -g[3];
      g[4] = -0.5f * g[4];
      float* dst = g2d + 9 * (int64_t)s_g[tid];
#pragma unroll
      for (int q = 0; q < 9; ++q)
        if (g[q] != 0.0f) atomicAdd(dst + q, g[q]);
    }
    bend = bbeg;
  }
}

__global__ void zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

// Grid-stride over pixels; one global atomic per workgroup for the loss.
__global__ __launch_bounds__(256) void loss_l1_kernel(int64_t npix, const float4* __restrict__ out,
                                                      const float* __restrict__ target, float bg0,
                                                      float bg1, float bg2, float scale,
                                                      float4* __restrict__ dL_dout,
                                                      float* __restrict__ loss) {
  __shared__ float s_loss;
  if (threadIdx.x == 0) s_loss = 0.0f;
  __syncthreads();
  float l = 0.0f;
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < npix;
       p += (int64_t)gridDim.x * blockDim.x) {
    const float4 o = out[p];
    const float ia = 1.0f - o.w;
    const float d0 = o.x + ia * bg0 - target[3 * p];
    const float d1 = o.y + ia * bg1 - target[3 * p + 1];
    const float d2 = o.z + ia * bg2 - target[3 * p + 2];
    const float s0 = (d0 > 0.0f) - (d0 < 0.0f), s1 = (d1 > 0.0f) - (d1 < 0.0f),
                s2 = (d2 > 0.0f) - (d2 < 0.0f);
    const float g0 = s0 * scale, g1 = s1 * scale, g2 = s2 * scale;
    dL_dout[p] = make_float4(g0, g1, g2, -(bg0 * g0 + bg1 * g1 + bg2 * g2));
    l += (fabsf(d0) + fabsf(d1) + fabsf(d2)) * scale;
  }
  if (loss) {
    l = wave_sum(l);
    if ((threadIdx.x & 63) == 0) atomicAdd(&s_loss, l);
    __syncthreads();
    if (threadIdx.x == 0) atomicAdd(loss, s_loss);
  }
}

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

static size_t g2d_bytes(int64_t n) {
  return ((size_t)9 * sizeof(float) * (size_t)n + 255) & ~size_t(255);
}

// g2d[n][9], then the backward's tile work and tile order.
size_t render_bwd_workspace_bytes(int64_t n) {
  return g2d_bytes(n) + 2 * sizeof(uint32_t) * ABCD_MAX_TILES;
}

int32_t launch_render_fwd(const abcd_camera& cam, const abcd_raster_params& prm,
                          const uint32_t* tile_ranges, const uint32_t* values_sorted,
                          const float* means2d, const float* conic_opacity, const float* rgb,
                          const float* F, const float* B, float* out_rgba, float* final_T,
                          uint32_t* last, unsigned long long* n_blends, const uint32_t* tile_order,
                          hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  const int grid = tile_order ? k.ntiles : 8 * k.per_xcd;
  ABCD_LAUNCH("render_fwd", render_fwd_kernel<false>, grid, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb,
              reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B),
              reinterpret_cast<float4*>(out_rgba), final_T, last, n_blends, tile_order, nullptr);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_render_cache(const abcd_camera& cam, const abcd_raster_params& prm,
                            const uint32_t* tile_ranges, const uint32_t* tile_order,
                            const uint32_t* values_sorted, const float* means2d,
                            const float* conic_opacity, const float* rgb, uint16_t* image_f16,
                            hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  const int grid = tile_order ? k.ntiles : 8 * k.per_xcd;
  ABCD_LAUNCH("render_cache", render_fwd_kernel<true>, grid, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb, nullptr, nullptr, nullptr,
              nullptr, nullptr, nullptr, tile_order, reinterpret_cast<uint2*>(image_f16));
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_render_bwd_pixels(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                                 const uint32_t* tile_ranges, const uint32_t* values_sorted,
                                 const float* means2d, const float* conic_opacity,
                                 const float* rgb, const float* F, const float* B,
                                 const float* final_T, const uint32_t* last,
                                 const float* dL_dout, float* g2d, hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  uint32_t* work = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(g2d) + g2d_bytes(n));
  uint32_t* order = work + ABCD_MAX_TILES;
  TRY_STATUS(launch_tile_walk(k.width, k.height, last, work, stream));
  TRY_STATUS(launch_tile_order(k.ntiles, work, order, nullptr, "bwd_order", stream));
  ABCD_LAUNCH("render_bwd", render_bwd_kernel, k.ntiles, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb,
              reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B), final_T,
              last, reinterpret_cast<const float4*>(dL_dout), g2d, order);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_zero(float* p, int64_t count, hipStream_t stream) {
  if (count == 0) return ABCD_OK;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
  ABCD_LAUNCH("zero_fill", zero_kernel, blocks, 256, 0, stream, p, count);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_loss_l1(int width, int height, const float* out_rgba, const float* target_rgb,
                       float bg0, float bg1, float bg2, float* dL_dout, float* loss,
                       hipStream_t stream) {
  const int64_t npix = (int64_t)width * height;
  const float scale = 1.0f / (3.0f * (float)npix);
  const int64_t blocks = std::min<int64_t>((npix + 255) / 256, 1024);
  ABCD_LAUNCH("loss_l1", loss_l1_kernel, blocks, 256, 0, stream, npix,
              reinterpret_cast<const float4*>(out_rgba), target_rgb, bg0, bg1, bg2, scale,
              reinterpret_cast<float4*>(dL_dout), loss);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd
