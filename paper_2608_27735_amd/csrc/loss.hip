// loss.hip -- the L1 reconstruction loss and its image gradient, and a fill
// kernel that clears device buffers (used instead of memsets, which HIP graph
// capture handles poorly).
#include "abcd_internal.h"

namespace abcd {
namespace {

// Clears `count` floats: the floats before p's first 16-byte boundary and
// after the last whole float4 one by one, the rest as float4 stores.
__global__ void zero_kernel(float* __restrict__ p, int64_t count, int64_t head) {
  const int64_t n4 = (count - head) / 4;
  const int64_t tail = head + 4 * n4;
  float4* __restrict__ q = reinterpret_cast<float4*>(p + head);
  const int64_t first = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = first; i < n4; i += stride) q[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (first < head) p[first] = 0.0f;
  if (tail + first < count) p[tail + first] = 0.0f;
}

// Each thread takes kLossUnroll pixels a grid apart, all loads issued before
// the first is used (a launch normally covers the image in one pass, a larger
// image is strided over); one global atomic per workgroup for the loss. Atomic
// adds to one address are serialised, so the workgroups are few and large.
constexpr int kLossUnroll = 8;
constexpr int kLossThreads = 512;

__global__ __launch_bounds__(kLossThreads) void loss_l1_kernel(int64_t npix, const float4* __restrict__ out,
                                                      const float* __restrict__ target, float bg0,
                                                      float bg1, float bg2, float scale,
                                                      float4* __restrict__ dL_dout,
                                                      float* __restrict__ loss) {
  __shared__ float s_loss;
  if (threadIdx.x == 0) s_loss = 0.0f;
  __syncthreads();
  float l = 0.0f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t p0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p0 < npix;
       p0 += kLossUnroll * stride) {
    float4 o[kLossUnroll];
    float t0[kLossUnroll], t1[kLossUnroll], t2[kLossUnroll];
#pragma unroll
    for (int u = 0; u < kLossUnroll; ++u) {
      const int64_t p = min(p0 + u * stride, npix - 1);  // past the end: a valid pixel, unused
      o[u] = out[p];
      t0[u] = target[3 * p];
      t1[u] = target[3 * p + 1];
      t2[u] = target[3 * p + 2];
    }
#pragma unroll
    for (int u = 0; u < kLossUnroll; ++u) {
      const int64_t p = p0 + u * stride;
      if (p >= npix) break;
      const float ia = 1.0f - o[u].w;
      const float d0 = o[u].x + ia * bg0 - t0[u];
      const float d1 = o[u].y + ia * bg1 - t1[u];
      const float d2 = o[u].z + ia * bg2 - t2[u];
      const float s0 = (d0 > 0.0f) - (d0 < 0.0f), s1 = (d1 > 0.0f) - (d1 < 0.0f),
                  s2 = (d2 > 0.0f) - (d2 < 0.0f);
      const float g0 = s0 * scale, g1 = s1 * scale, g2 = s2 * scale;
      dL_dout[p] = make_float4(g0, g1, g2, -(bg0 * g0 + bg1 * g1 + bg2 * g2));
      l += (fabsf(d0) + fabsf(d1) + fabsf(d2)) * scale;
    }
  }
  if (loss) {
    l = wave_sum(l);
    if ((threadIdx.x & 63) == 0) atomicAdd(&s_loss, l);
    __syncthreads();
    if (threadIdx.x == 0) atomicAdd(loss, s_loss);
  }
}

}  // namespace

int32_t launch_zero(float* p, int64_t count, hipStream_t stream) {
  if (count == 0) return ABCD_OK;
  // p is float aligned: 0-3 floats up to its first 16-byte boundary
  const int64_t head =
      std::min<int64_t>(count, (int64_t)((16 - (reinterpret_cast<uintptr_t>(p) & 15)) & 15) / 4);
  const int64_t blocks = std::min<int64_t>((count / 4 + 255) / 256 + 1, 4096);
  ABCD_LAUNCH("zero_fill", zero_kernel, blocks, 256, 0, stream, p, count, head);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_loss_l1(int width, int height, const float* out_rgba, const float* target_rgb,
                       float bg0, float bg1, float bg2, float* dL_dout, float* loss,
                       hipStream_t stream) {
  const int64_t npix = (int64_t)width * height;
  const float scale = 1.0f / (3.0f * (float)npix);
  constexpr int64_t per_block = (int64_t)kLossThreads * kLossUnroll;
  const int64_t blocks = std::min<int64_t>((npix + per_block - 1) / per_block, 1024);
  ABCD_LAUNCH("loss_l1", loss_l1_kernel, blocks, kLossThreads, 0, stream, npix,
              reinterpret_cast<const float4*>(out_rgba), target_rgb, bg0, bg1, bg2, scale,
              reinterpret_cast<float4*>(dL_dout), loss);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd
