// loss.hip -- the L1 reconstruction loss and its image gradient, and a fill
// kernel that clears device buffers (used instead of memsets, which HIP graph
// capture handles poorly).
#include "abcd_internal.h"

namespace abcd {
namespace {

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

}  // namespace

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
