// adam.hip -- Adam update of the active parameters after a step's backward.
//
// The paper trains the active block with gradient steps and does not name the
// optimizer; the 3DGS line it builds on uses Adam (Kingma and Ba 2015,
// Algorithm 1) with one learning rate per parameter group. One launch updates
// every group in place: a pure HBM stream (parameter, gradient and both
// moments read, parameter and moments written: 28 bytes per element).
// Workgroups are dealt to the groups in proportion to their sizes; a thread
// takes 16 consecutive elements as four 16-byte loads when the group's arrays
// allow it, else element by element.
#include <math.h>

#include "abcd_internal.h"

namespace abcd {
namespace {

constexpr int kMaxGroups = ABCD_ADAM_MAX_GROUPS;
constexpr int kPerThread = 16;
constexpr int64_t kPerBlock = (int64_t)kBlock * kPerThread;

struct AdamArgs {
  float* theta[kMaxGroups];
  const float* g[kMaxGroups];
  float* m[kMaxGroups];
  float* v[kMaxGroups];
  int64_t count[kMaxGroups];
  float step[kMaxGroups];          // lr / (1 - beta1^t)
  int64_t block0[kMaxGroups + 1];  // first workgroup of each group
  int vec[kMaxGroups];             // 16-byte aligned arrays, count % 4 == 0
  int ngroups;
};

__device__ __forceinline__ void adam_one(float& th, float g, float& m, float& v, float b1,
                                         float b2, float ic2, float eps, float step) {
  m = b1 * m + (1.0f - b1) * g;
  v = b2 * v + (1.0f - b2) * (g * g);
  th = th - step * m / (sqrtf(v * ic2) + eps);
}

__global__ __launch_bounds__(kBlock) void adam_kernel(AdamArgs a, float b1, float b2, float ic2,
                                                      float eps) {
  int gi = 0;
  while (gi + 1 < a.ngroups && (int64_t)blockIdx.x >= a.block0[gi + 1]) ++gi;
  const int64_t e0 = ((int64_t)blockIdx.x - a.block0[gi]) * kPerBlock +
                     (int64_t)threadIdx.x * kPerThread;
  const int64_t n = a.count[gi];
  if (e0 >= n) return;
  float* th = a.theta[gi] + e0;
  const float* g = a.g[gi] + e0;
  float* m = a.m[gi] + e0;
  float* v = a.v[gi] + e0;
  const float step = a.step[gi];
  if (a.vec[gi] && e0 + kPerThread <= n) {
    float4 T[4], G[4], M[4], V[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      T[q] = reinterpret_cast<const float4*>(th)[q];
      G[q] = reinterpret_cast<const float4*>(g)[q];
      M[q] = reinterpret_cast<const float4*>(m)[q];
      V[q] = reinterpret_cast<const float4*>(v)[q];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      adam_one(T[q].x, G[q].x, M[q].x, V[q].x, b1, b2, ic2, eps, step);
      adam_one(T[q].y, G[q].y, M[q].y, V[q].y, b1, b2, ic2, eps, step);
      adam_one(T[q].z, G[q].z, M[q].z, V[q].z, b1, b2, ic2, eps, step);
      adam_one(T[q].w, G[q].w, M[q].w, V[q].w, b1, b2, ic2, eps, step);
      reinterpret_cast<float4*>(th)[q] = T[q];
      reinterpret_cast<float4*>(m)[q] = M[q];
      reinterpret_cast<float4*>(v)[q] = V[q];
    }
    return;
  }
  const int cnt = (int)min<int64_t>(kPerThread, n - e0);
  for (int i = 0; i < cnt; ++i) {
    float t = th[i], mm = m[i], vv = v[i];
    adam_one(t, g[i], mm, vv, b1, b2, ic2, eps, step);
    th[i] = t;
    m[i] = mm;
    v[i] = vv;
  }
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

int32_t launch_adam(const abcd_adam_group* groups, int ngroups, float beta1, float beta2, float eps,
                    int64_t t, hipStream_t stream) {
  AdamArgs a{};
  const double c1 = 1.0 - pow((double)beta1, (double)t);
  const double c2 = 1.0 - pow((double)beta2, (double)t);
  int64_t blocks = 0;
  int used = 0;
  for (int i = 0; i < ngroups; ++i) {
    const abcd_adam_group& gr = groups[i];
    if (gr.count == 0) continue;
    a.theta[used] = gr.param;
    a.g[used] = gr.grad;
    a.m[used] = gr.exp_avg;
    a.v[used] = gr.exp_avg_sq;
    a.count[used] = gr.count;
    a.step[used] = (float)((double)gr.lr / c1);
    a.vec[used] = aligned16(gr.param) && aligned16(gr.grad) && aligned16(gr.exp_avg) &&
                  aligned16(gr.exp_avg_sq) && gr.count % 4 == 0;
    a.block0[used] = blocks;
    blocks += (gr.count + kPerBlock - 1) / kPerBlock;
    ++used;
  }
  a.block0[used] = blocks;
  a.ngroups = used;
  if (blocks == 0) return ABCD_OK;
  ABCD_LAUNCH("adam", adam_kernel, blocks, kBlock, 0, stream, a, beta1, beta2,
              (float)(1.0 / c2), eps);
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd
