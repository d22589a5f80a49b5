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

// Workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous
// band of tiles so neighbouring tiles (which share Gaussians) share an L2.
__device__ __forceinline__ int tile_of_block(const BlendConsts& k) {
  const int b = blockIdx.x;
  return (b & 7) * k.per_xcd + (b >> 3);
}

__global__ __launch_bounds__(256) void render_fwd_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    float4* __restrict__ out, float* __restrict__ final_T, uint32_t* __restrict__ last,
    unsigned long long* __restrict__ n_blends) {
  __shared__ float2 s_xy[256];
  __shared__ float4 s_co[256];
  __shared__ float4 s_rgb[256];
  __shared__ unsigned long long s_nb;
  const int tile = tile_of_block(k);
  if (tile >= k.ntiles) return;
  const int tid = threadIdx.x;
  const int px = (tile % k.ntx) * kTile + (tid & 15);
  const int py = (tile / k.ntx) * kTile + (tid >> 4);
  const bool inside = px < k.width && py < k.height;
  const uint32_t start = tile_ranges[2 * tile], end = tile_ranges[2 * tile + 1];
  const float fx = (float)px + 0.5f, fy = (float)py + 0.5f;
  float T = 1.0f, cr = 0.0f, cg = 0.0f, cb = 0.0f;
  uint32_t lastk = 0, nb = 0;
  bool done = !inside;
  if (tid == 0) s_nb = 0;
  for (uint32_t b0 = start; b0 < end; b0 += 256) {
    if (__syncthreads_count(done) == 256) break;
    const uint32_t idx = b0 + tid;
    if (idx < end) {
      const uint32_t g = values[idx];
      s_xy[tid] = means2d[g];
      s_co[tid] = conic_opacity[g];
      s_rgb[tid] = make_float4(rgb[3 * g], rgb[3 * g + 1], rgb[3 * g + 2], 0.0f);
    }
    __syncthreads();
    const int cnt = (int)min(256u, end - b0);
    if (!done) {
      for (int j = 0; j < cnt; ++j) {
        const float2 m = s_xy[j];
        const float4 co = s_co[j];
        const AlphaEval ae = eval_alpha(fx - m.x, fy - m.y, co.x, co.y, co.z, co.w, k.alpha_min,
                                        k.alpha_max);
        if (ae.skip) continue;
        const float Tn = T * (1.0f - ae.alpha);
        if (Tn < k.t_min) {
          done = true;
          break;
        }
        const float4 c = s_rgb[j];
        const float wgt = ae.alpha * T;
        cr += c.x * wgt;
        cg += c.y * wgt;
        cb += c.z * wgt;
        T = Tn;
        lastk = b0 - start + j + 1;
        ++nb;
      }
    }
  }
  if (inside) {
    const int64_t p = (int64_t)py * k.width + px;
    const float4 f = F ? F[p] : make_float4(0, 0, 0, 0);
    const float4 bb = B ? B[p] : make_float4(0, 0, 0, 0);
    const float s = 1.0f - f.w;
    out[p] = make_float4(f.x + s * (cr + T * bb.x), f.y + s * (cg + T * bb.y),
                         f.z + s * (cb + T * bb.z), f.w + s * (1.0f - T * (1.0f - bb.w)));
    final_T[p] = T;
    last[p] = lastk;
  }
  if (n_blends) {
    unsigned int x = nb;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    const unsigned long long wsum = x;
    __syncthreads();
    if ((tid & 63) == 0) atomicAdd(&s_nb, wsum);
    __syncthreads();
    if (tid == 0 && s_nb) atomicAdd(n_blends, s_nb);
  }
}

__global__ __launch_bounds__(256) void render_bwd_kernel(
    BlendConsts k, const uint32_t* __restrict__ tile_ranges, const uint32_t* __restrict__ values,
    const float2* __restrict__ means2d, const float4* __restrict__ conic_opacity,
    const float* __restrict__ rgb, const float4* __restrict__ F, const float4* __restrict__ B,
    const float* __restrict__ final_T, const uint32_t* __restrict__ last,
    const float4* __restrict__ dL_dout, float* __restrict__ g2d) {
  __shared__ float2 s_xy[256];
  __shared__ float4 s_co[256];
  __shared__ float4 s_rgb[256];
  __shared__ uint32_t s_g[256];
  __shared__ float s_acc[9][256];
  __shared__ uint32_t s_max;
  const int tile = tile_of_block(k);
  if (tile >= k.ntiles) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int px = (tile % k.ntx) * kTile + (tid & 15);
  const int py = (tile / k.ntx) * kTile + (tid >> 4);
  const bool inside = px < k.width && py < k.height;
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
    atomicMax(&s_max, lastp);
  }
  const float Tfin = T;
  float Rr = 0.0f, Rg = 0.0f, Rb = 0.0f;
  __syncthreads();
  const uint32_t nent = s_max;
  for (uint32_t bend = start + nent; bend > start;) {
    const uint32_t bbeg = bend - min(256u, bend - start);
    const int cnt = (int)(bend - bbeg);
    __syncthreads();
    if (tid < cnt) {
      const uint32_t g = values[bend - 1 - tid];
      s_g[tid] = g;
      s_xy[tid] = means2d[g];
      s_co[tid] = conic_opacity[g];
      s_rgb[tid] = make_float4(rgb[3 * g], rgb[3 * g + 1], rgb[3 * g + 2], 0.0f);
#pragma unroll
      for (int q = 0; q < 9; ++q) s_acc[q][tid] = 0.0f;
    }
    __syncthreads();
    for (int j = 0; j < cnt; ++j) {
      const uint32_t kk = bend - 1 - j - start;  // position in the tile's list
      float gr[9];
      bool contrib = false;
      if (kk < lastp) {
        const float2 m = s_xy[j];
        const float4 co = s_co[j];
        const float dx = fx - m.x, dy = fy - m.y;
        const AlphaEval ae = eval_alpha(dx, dy, co.x, co.y, co.z, co.w, k.alpha_min, k.alpha_max);
        if (!ae.skip) {
          contrib = true;
          const float4 c = s_rgb[j];
          const float om = 1.0f - ae.alpha;
          const float Tk = T / om;
          const float wgt = ae.alpha * Tk;
          gr[6] = wgt * gcr;
          gr[7] = wgt * gcg;
          gr[8] = wgt * gcb;
          const float dLda = Tk * ((c.x - Rr) * gcr + (c.y - Rg) * gcg + (c.z - Rb) * gcb) -
                             (Tfin / om) * gT;
          Rr = ae.alpha * c.x + om * Rr;
          Rg = ae.alpha * c.y + om * Rg;
          Rb = ae.alpha * c.z + om * Rb;
          T = Tk;
          if (ae.clamped) {
            gr[0] = gr[1] = gr[2] = gr[3] = gr[4] = gr[5] = 0.0f;
          } else {
            const float gp = ae.alpha * dLda;
            gr[5] = ae.e * dLda;
            gr[0] = gp * (co.x * dx + co.y * dy);
            gr[1] = gp * (co.y * dx + co.z * dy);
            gr[2] = -0.5f * gp * dx * dx;
            gr[3] = -gp * dx * dy;
            gr[4] = -0.5f * gp * dy * dy;
          }
        }
      }
      if (__ballot(contrib)) {
        if (!contrib) {
#pragma unroll
          for (int q = 0; q < 9; ++q) gr[q] = 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 9; ++q) {
          const float v = wave_sum(gr[q]);
          if (lane == 0) atomicAdd(&s_acc[q][j], v);
        }
      }
    }
    __syncthreads();
    if (tid < cnt) {
      float* dst = g2d + 9 * (int64_t)s_g[tid];
#pragma unroll
      for (int q = 0; q < 9; ++q) {
        const float v = s_acc[q][tid];
        if (v != 0.0f) atomicAdd(dst + q, v);
      }
    }
    bend = bbeg;
  }
}

__global__ void zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

__global__ __launch_bounds__(256) void loss_l1_kernel(int64_t npix, const float4* __restrict__ out,
                                                      const float* __restrict__ target, float bg0,
                                                      float bg1, float bg2, float scale,
                                                      float4* __restrict__ dL_dout,
                                                      float* __restrict__ loss) {
  __shared__ float s_loss;
  if (threadIdx.x == 0) s_loss = 0.0f;
  __syncthreads();
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  float l = 0.0f;
  if (p < npix) {
    const float4 o = out[p];
    const float ia = 1.0f - o.w;
    const float d0 = o.x + ia * bg0 - target[3 * p];
    const float d1 = o.y + ia * bg1 - target[3 * p + 1];
    const float d2 = o.z + ia * bg2 - target[3 * p + 2];
    const float s0 = (d0 > 0.0f) - (d0 < 0.0f), s1 = (d1 > 0.0f) - (d1 < 0.0f),
                s2 = (d2 > 0.0f) - (d2 < 0.0f);
    const float g0 = s0 * scale, g1 = s1 * scale, g2 = s2 * scale;
    dL_dout[p] = make_float4(g0, g1, g2, -(bg0 * g0 + bg1 * g1 + bg2 * g2));
    l = (fabsf(d0) + fabsf(d1) + fabsf(d2)) * scale;
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

size_t render_bwd_workspace_bytes(int64_t n) {
  return ((size_t)9 * sizeof(float) * (size_t)n + 255) & ~size_t(255);
}

int32_t launch_render_fwd(const abcd_camera& cam, const abcd_raster_params& prm,
                          const uint32_t* tile_ranges, const uint32_t* values_sorted,
                          const float* means2d, const float* conic_opacity, const float* rgb,
                          const float* F, const float* B, float* out_rgba, float* final_T,
                          uint32_t* last, unsigned long long* n_blends, hipStream_t stream) {
  const BlendConsts k = consts(cam, prm);
  ABCD_LAUNCH("render_fwd", render_fwd_kernel, 8 * k.per_xcd, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb,
              reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B),
              reinterpret_cast<float4*>(out_rgba), final_T, last, n_blends);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_render_bwd_pixels(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                                 const uint32_t* tile_ranges, const uint32_t* values_sorted,
                                 const float* means2d, const float* conic_opacity,
                                 const float* rgb, const float* F, const float* B,
                                 const float* final_T, const uint32_t* last,
                                 const float* dL_dout, float* g2d, hipStream_t stream) {
  (void)n;
  const BlendConsts k = consts(cam, prm);
  ABCD_LAUNCH("render_bwd", render_bwd_kernel, 8 * k.per_xcd, kBlock, 0, stream, k, tile_ranges,
              values_sorted, reinterpret_cast<const float2*>(means2d),
              reinterpret_cast<const float4*>(conic_opacity), rgb,
              reinterpret_cast<const float4*>(F), reinterpret_cast<const float4*>(B), final_T,
              last, reinterpret_cast<const float4*>(dL_dout), g2d);
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
  ABCD_LAUNCH("loss_l1", loss_l1_kernel, (npix + 255) / 256, 256, 0, stream, npix,
              reinterpret_cast<const float4*>(out_rgba), target_rgb, bg0, bg1, bg2, scale,
              reinterpret_cast<float4*>(dL_dout), loss);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd
